"""Benchmark of the UFP4 hot path on one MI355X.

One step = the whole hot path of one linear layer's training step under the UFP4 recipe: six fused
RHT + quantize calls (X, W rowwise along K; dY rowwise along N with SR; W^T along N; dY^T along M with SR;
X^T along M) and the three block-scaled 4-bit GEMMs fwd_y, bwd_dx, bwd_dw. Inputs are resident in HBM before
the timed region; every output buffer is allocated before it, so the timed loop only launches kernels.

Prints one JSON line. `value` is the step's GEMM work (3 x 2MNK) divided by the step time, in TFLOP/s;
`breakdown` has every kernel's average duration and its own GB/s (quantizers, 2.75 algorithmic bytes per
element) or TFLOP/s (GEMMs); `roofline` is for the GEMM kernel, the dominant one; `cpu_baseline` times the CPU
oracle on a bounded sample of the same layer.

Usage: python bench.py [--gpus 1] [--steps 20] [--warmup W] [--workload dense|tiny|moe7.9b|moe124b|square|quant1g|quant1g-t|copy1g]

Without --warmup the untimed warmup runs whole steps until at least WARMUP_SECONDS have passed: the GPU's clock
takes tens of milliseconds of load to settle, and a few milliseconds of warmup would time the ramp.
"""

from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2606_20381_amd import ufp4 as U  # noqa: E402
from paper_2606_20381_amd import workloads as WL  # noqa: E402

HBM_PEAK_GBPS = 8000.0
INT8_PEAK_TOPS = 5000.0  # dense int8 / fp8 MFMA, MI355X
FP4_PEAK_TFLOPS = 10100.0  # dense fp4 MFMA (the E2M1 baseline's block products)
# Bound of an exact per-16-block fp32-scale GEMM: one VALU FMA per output and block, i.e. 2MNK / (MNK/16) = 32
# ops per FMA, at 256 CUs x 4 SIMDs x 16 fp32 FMA lanes per clock x 2.4 GHz = 39.3 T FMA/s (non-packed).
ATTAINABLE_TOPS = 32 * 256 * 4 * 16 * 2.4e9 / 1e12
GEMM_KERNEL = {
    "ufp4": "gemm_f32_kernel (fp8 MFMA 32x32x16 per K-block + bf16 MFMA 32x32x8 scale outer product + fp32 FMA)",
    "e2m1": "gemm_f32_kernel (FP4 f8f6f4 MFMA per K-block + bf16 MFMA 32x32x8 scale outer product + fp32 FMA)",
}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
WARMUP_SECONDS = 0.5
QUANT_BYTES_PER_ELEM = 2.75  # 2 B bf16 in, 0.5 B codes + 0.25 B scale out
METRIC = "RHT+quantize GB/s and 4-bit fwd_y/bwd_dx/bwd_dw TFLOP/s (% of roofline)"


class Timeline:
    """HIP events around every launch of the timed region, on the stream the kernels run on."""

    def __init__(self):
        self.events = {}

    def run(self, label, fn, record):
        if not record:
            return fn()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        r = fn()
        e.record()
        self.events.setdefault(label, []).append((s, e))
        return r

    def mean_us(self, label):
        v = [s.elapsed_time(e) * 1e3 for s, e in self.events[label]]
        return float(np.mean(v))


# ---------------------------------------------------------------------------------------------------
# step builders: each returns (step(record) -> None, kernel table)
# kernel table: label -> ("quant", elements) or ("gemm", flops)
# ---------------------------------------------------------------------------------------------------

# Per recipe: the quantizer and, for fwd_y / bwd_dx / bwd_dw, whether the RHT is applied to that GEMM's
# operands (Table 1: UFP4 rotates all three; the E2M1 baseline only bwd_dw's).
RECIPES = {
    "ufp4": (U.UNIFORM, (True, True, True), "ufp4: uniform -7..7, RHT16 on all GEMMs, SR on dY"),
    "e2m1": (U.E2M1, (False, False, True), "e2m1 baseline: E2M1 grid, RHT16 on bwd_dw only, SR on dY"),
}


def _quantizers(recipe: str):
    fmt, (r_y, r_dx, r_dw), _ = RECIPES[recipe]
    fn = U.rht_quantize if fmt == U.UNIFORM else U.e2m1_quantize
    return fmt, fn, r_y, r_dx, r_dw


def dense_step(wl, tl: Timeline, recipe: str = "ufp4"):
    m, s = wl.sign_mask, wl.seed
    fmt, Q, r_y, r_dx, r_dw = _quantizers(recipe)
    x, w, dy = (t.cuda() for t in (wl.x, wl.w, wl.dy))
    M, K = x.shape
    N = w.shape[0]
    q = {
        "x": U.empty_qtensor(M, K, fmt), "w": U.empty_qtensor(N, K, fmt), "dy": U.empty_qtensor(M, N, fmt),
        "wt": U.empty_qtensor(K, N, fmt), "dyt": U.empty_qtensor(N, M, fmt), "xt": U.empty_qtensor(K, M, fmt),
    }
    y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    dx = torch.empty(M, K, dtype=torch.bfloat16, device="cuda")
    dw = torch.empty(N, K, dtype=torch.float32, device="cuda")

    def step(rec):
        tl.run("quant_x", lambda: Q(x, rht=r_y, sign_mask=m, out=q["x"]), rec)
        tl.run("quant_w", lambda: Q(w, rht=r_y, sign_mask=m, out=q["w"]), rec)
        tl.run("quant_dy_sr", lambda: Q(dy, rht=r_dx, sign_mask=m, rounding=U.SR, seed=s, stream_id=0,
                                        out=q["dy"]), rec)
        tl.run("quant_wt", lambda: Q(w, transpose=True, rht=r_dx, sign_mask=m, out=q["wt"]), rec)
        tl.run("quant_dyt_sr", lambda: Q(dy, transpose=True, rht=r_dw, sign_mask=m, rounding=U.SR, seed=s,
                                         stream_id=1, out=q["dyt"]), rec)
        tl.run("quant_xt", lambda: Q(x, transpose=True, rht=r_dw, sign_mask=m, out=q["xt"]), rec)
        tl.run("gemm_fwd_y", lambda: U.gemm_fwd_y(q["x"], q["w"], out=y), rec)
        tl.run("gemm_bwd_dx", lambda: U.gemm_bwd_dx(q["dy"], q["wt"], out=dx), rec)
        tl.run("gemm_bwd_dw", lambda: U.gemm_bwd_dw(q["dyt"], q["xt"], out=dw), rec)

    kern = {
        "quant_x": ("quant", M * K), "quant_w": ("quant", N * K), "quant_dy_sr": ("quant", M * N),
        "quant_wt": ("quant", N * K), "quant_dyt_sr": ("quant", M * N), "quant_xt": ("quant", M * K),
        "gemm_fwd_y": ("gemm", 2 * M * N * K), "gemm_bwd_dx": ("gemm", 2 * M * N * K),
        "gemm_bwd_dw": ("gemm", 2 * M * N * K),
    }
    return step, kern


def moe_step(wl, tl: Timeline, recipe: str = "ufp4"):
    m, s = wl.sign_mask, wl.seed
    fmt, Q, r_y, r_dx, r_dw = _quantizers(recipe)
    E, N, K = wl.w.shape
    x, dy = wl.x.cuda(), wl.dy.cuda()
    w2 = wl.w.reshape(E * N, K).cuda()
    M = x.shape[0]
    off, poff, red = U.group_offsets(wl.counts)
    eoff, epoff, ered = U.group_offsets([N] * E)
    q = {
        "x": U.empty_qtensor(M, K, fmt), "w": U.empty_qtensor(E * N, K, fmt), "dy": U.empty_qtensor(M, N, fmt),
        "wt": U.empty_qtensor(K, E * N, fmt), "dyt": U.empty_qtensor(N, red, fmt), "xt": U.empty_qtensor(K, red, fmt),
    }
    y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    dx = torch.empty(M, K, dtype=torch.bfloat16, device="cuda")
    dw = torch.empty(E, N, K, dtype=torch.float32, device="cuda")

    def step(rec):
        tl.run("quant_x", lambda: Q(x, rht=r_y, sign_mask=m, out=q["x"]), rec)
        tl.run("quant_w", lambda: Q(w2, rht=r_y, sign_mask=m, out=q["w"]), rec)
        tl.run("quant_dy_sr", lambda: Q(dy, rht=r_dx, sign_mask=m, rounding=U.SR, seed=s, stream_id=0,
                                        out=q["dy"]), rec)
        tl.run("quant_wt", lambda: U.quantize_grouped_t(w2, eoff, epoff, ered, fmt=fmt, rht=r_dx, sign_mask=m,
                                                        out=q["wt"]), rec)
        tl.run("quant_dyt_sr", lambda: U.quantize_grouped_t(dy, off, poff, red, fmt=fmt, rht=r_dw, sign_mask=m,
                                                            rounding=U.SR, seed=s, stream_id=1, out=q["dyt"]), rec)
        tl.run("quant_xt", lambda: U.quantize_grouped_t(x, off, poff, red, fmt=fmt, rht=r_dw, sign_mask=m,
                                                        out=q["xt"]), rec)
        tl.run("gemm_fwd_y", lambda: U.gemm_fwd_y_grouped(q["x"], q["w"], off, N, out=y), rec)
        tl.run("gemm_bwd_dx", lambda: U.gemm_bwd_dx_grouped(q["dy"], q["wt"], off, out=dx), rec)
        tl.run("gemm_bwd_dw", lambda: U.gemm_bwd_dw_grouped(q["dyt"], q["xt"], poff, out=dw), rec)

    flops = 2 * M * N * K
    kern = {
        "quant_x": ("quant", M * K), "quant_w": ("quant", E * N * K), "quant_dy_sr": ("quant", M * N),
        "quant_wt": ("quant", E * N * K), "quant_dyt_sr": ("quant", M * N), "quant_xt": ("quant", M * K),
        "gemm_fwd_y": ("gemm", flops), "gemm_bwd_dx": ("gemm", flops), "gemm_bwd_dw": ("gemm", flops),
    }
    return step, kern


def copy1g_step(tl: Timeline):
    """Plain device copy of the 1 GiB quantizer tensor: the calibration kernel for HBM byte counters."""
    t = WL.quantizer_tensor().cuda()
    dst = torch.empty_like(t)

    def step(rec):
        tl.run("copy", lambda: dst.copy_(t), rec)

    return step, {"copy": ("copy", t.numel() * t.element_size())}


def quant1g_step(tl: Timeline, transpose: bool):
    """The quantizer alone on a 1 GiB bf16 tensor, rowwise (reduction along its 16384 columns) or transposed
    (operand X^T, reduction along its 32768 rows)."""
    t = WL.quantizer_tensor().cuda()
    R, C = t.shape
    q = U.empty_qtensor(C, R) if transpose else U.empty_qtensor(R, C)
    label = "quant_cols_rtne" if transpose else "quant_rows_rtne"

    def step(rec):
        tl.run(label, lambda: U.rht_quantize(t, transpose=transpose, sign_mask=0x6A09, out=q), rec)

    return step, {label: ("quant", R * C)}


# ---------------------------------------------------------------------------------------------------
# measured HBM traffic (rocprofv3 FETCH_SIZE / WRITE_SIZE runs, scaled by a 1 GiB copy), valid only for the
# kernel source it was measured on
# ---------------------------------------------------------------------------------------------------

TRAFFIC_SOURCES = {"gemm": "ufp4_gemm.hip", "quant": "ufp4_quant.hip"}


def _source_digest(name: str) -> str:
    import hashlib

    path = os.path.join(ROOT, "paper_2606_20381_amd", "csrc", name)
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(kind: str, workload: str):
    """HBM bytes per launch of the dominant kernel from profiles/traffic.json, or None when there is no
    entry for this workload or the kernel source changed since the counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            table = json.load(f)
    except (OSError, ValueError):
        return None
    entry = table.get(kind, {}).get(workload)
    if not entry or entry.get("source_sha256") != _source_digest(TRAFFIC_SOURCES[kind]):
        return None
    return entry["bytes_per_launch"]


# ---------------------------------------------------------------------------------------------------
# CPU oracle baseline: the same layer step on a bounded sample of tokens
# ---------------------------------------------------------------------------------------------------

def cpu_baseline(wl, tokens: int = 512, recipe: str = "ufp4"):
    from oracle import ufp4_oracle as O
    from threadpoolctl import threadpool_info

    x = WL.bf16_bits(wl.x[:tokens].contiguous())
    dy = WL.bf16_bits(wl.dy[:tokens].contiguous())
    w = WL.bf16_bits(wl.w)
    M, K = x.shape
    N = w.shape[0]
    t0 = time.perf_counter()
    O.layer_gemms(x, w, dy, recipe, sign_mask=wl.sign_mask, seed=wl.seed)
    dt = time.perf_counter() - t0
    flops = 3 * 2 * M * N * K
    blas = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    return {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": int(blas),
        "kind": "oracle",
        "sample": (f"whole UFP4 layer step (6 quantizations + 3 fp64 GEMMs) on {tokens} of {wl.x.shape[0]} "
                   f"tokens, full {N}x{K} weight; {dt:.1f} s; elementwise numpy on 1 thread, fp64 matmul on "
                   f"{blas} BLAS threads; host {platform.processor() or platform.machine()}, "
                   f"os.cpu_count()={os.cpu_count()}"),
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=None, help="untimed steps (default: steps for WARMUP_SECONDS)")
    ap.add_argument("--workload", default="dense",
                    choices=["dense", "tiny", "moe7.9b", "moe124b", "square", "quant1g", "quant1g-t", "copy1g"])
    ap.add_argument("--recipe", default="ufp4", choices=sorted(RECIPES),
                    help="ufp4 (the method) or e2m1 (the comparison baseline of Table 1)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); the multi-GPU layout "
              f"is described in DESIGN.md but not run", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    U.lib()

    tl = Timeline()
    wl = None
    if args.workload in ("quant1g", "quant1g-t"):
        transpose = args.workload == "quant1g-t"
        step, kern = quant1g_step(tl, transpose)
        wname = (f"standalone quantizer: 32768x16384 bf16 (1 GiB), {'transposed' if transpose else 'rowwise'} "
                 f"RTNE with RHT")
    elif args.workload == "copy1g":
        step, kern = copy1g_step(tl)
        wname = "calibration: device copy of a 1 GiB bf16 tensor (read 1 GiB + write 1 GiB)"
    else:
        wl = WL.CONFIGS[args.workload]()
        step, kern = (moe_step if wl.grouped else dense_step)(wl, tl, args.recipe)
        wname = wl.name
    torch.cuda.synchronize()

    if args.warmup is None:
        # whole untimed steps until the clock has settled
        warm, tw = 0, time.perf_counter()
        while warm < 3 or time.perf_counter() - tw < WARMUP_SECONDS:
            step(False)
            torch.cuda.synchronize()
            warm += 1
        args.warmup = warm
    else:
        for _ in range(args.warmup):
            step(False)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for _ in range(args.steps):
        step(True)
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = start.elapsed_time(end) / args.steps

    breakdown = {}
    gemm_flops = 0
    quant_bytes = 0.0
    for label, (kind, work) in kern.items():
        us = tl.mean_us(label)
        if kind == "copy":
            gbps = 2 * work / (us * 1e-6) / 1e9
            breakdown[label] = {"us": round(us, 2), "GB/s": round(gbps, 1), "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4)}
            quant_bytes += 2 * work
        elif kind == "quant":
            gbps = work * QUANT_BYTES_PER_ELEM / (us * 1e-6) / 1e9
            breakdown[label] = {"us": round(us, 2), "GB/s": round(gbps, 1), "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4)}
            quant_bytes += work * QUANT_BYTES_PER_ELEM
        else:
            tf = work / (us * 1e-6) / 1e12
            breakdown[label] = {"us": round(us, 2), "TFLOP/s": round(tf, 1), "frac_int8": round(tf / INT8_PEAK_TOPS, 4)}
            gemm_flops += work

    gemm_labels = [k for k, (kind, _) in kern.items() if kind == "gemm"]
    quant_labels = [k for k, (kind, _) in kern.items() if kind in ("quant", "copy")]
    if gemm_labels:
        value = gemm_flops / (ms_per_step * 1e-3) / 1e12
        unit = "TFLOP/s"
        per_launch = np.mean([kern[k][1] for k in gemm_labels])
        avg_us = np.mean([tl.mean_us(k) for k in gemm_labels])
        ach = per_launch / (avg_us * 1e-6) / 1e12
        peak = INT8_PEAK_TOPS if args.recipe == "ufp4" else FP4_PEAK_TFLOPS
        roof = {"bound": "mfma", "kernel": GEMM_KERNEL[args.recipe],
                "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(ach / peak, 4), "traffic": measured_traffic("gemm", wname + "/" + args.recipe),
                "attainable": {"peak": round(ATTAINABLE_TOPS, 1), "frac": round(ach / ATTAINABLE_TOPS, 4),
                               "why": "one fp32 VALU FMA per output and 16-block"}}
    else:
        value = quant_bytes / (ms_per_step * 1e-3) / 1e9
        unit = "GB/s"
        label = quant_labels[0]
        us = tl.mean_us(label)
        per_launch = kern[label][1] * (QUANT_BYTES_PER_ELEM if kern[label][0] == "quant" else 2)
        ach = per_launch / (us * 1e-6) / 1e9
        kname = {"quant_rows_rtne": "quant_rows_kernel", "quant_cols_rtne": "quant_cols_kernel"}.get(label, "copy")
        roof = {"bound": "hbm", "kernel": kname, "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS,
                "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBPS, 4),
                "traffic": measured_traffic("quant", wname) if kname != "copy" else None}
    if quant_labels and gemm_labels:
        qus = sum(tl.mean_us(k) for k in quant_labels)
        breakdown["quant_all"] = {"us": round(qus, 2), "GB/s": round(quant_bytes / (qus * 1e-6) / 1e9, 1)}

    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if gemm_labels else "f64+f32",
        "data": "synthetic (seeded, shapes and distributions of the workload; no real tensors)",
        "config": {"workload": wname, "recipe": RECIPES[args.recipe][2],
                   "outputs": "Y bf16, dX bf16, dW fp32" if gemm_labels else "codes + fp32 scales",
                   "wall_s": round(wall, 3)},
        "roofline": roof,
        "breakdown": breakdown,
    }
    if wl is not None and not args.no_cpu_baseline and not wl.grouped:
        out["cpu_baseline"] = cpu_baseline(wl, recipe=args.recipe)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
