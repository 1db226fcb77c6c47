"""Benchmark of the UFP4 hot path on one MI355X.

One step = the whole hot path of one linear layer's training step under the UFP4 recipe: the six fused
RHT + quantized operands (X, W rowwise along K; dY rowwise along N with SR; W^T along N; dY^T along M with SR;
X^T along M) and the three block-scaled 4-bit GEMMs fwd_y, bwd_dx, bwd_dw. By default X and W each go through
the two-operand quantizer (one read, both operands) and dY through the two single-output kernels (faster for
SR); --quant separate uses six single-output calls. Inputs are resident in HBM before the timed region; every
output buffer is allocated before it, so the timed loop only launches kernels.

The default workload is the square 16384^3 layer, the largest that the paper's configurations put on one GPU.

Prints one JSON line. `value` is the step's GEMM work (3 x 2MNK) divided by the step time, in TFLOP/s;
`breakdown` has every kernel's average duration and its own GB/s (algorithmic bytes: 2.75 per element for a
single-output quantizer, 3.5 for the two-operand one) or TFLOP/s (GEMMs); `roofline` is for the GEMM kernel,
the dominant one; `cpu_baseline` times the CPU oracle on a bounded sample of the same layer (a block of tokens
and of W's rows). For a layer workload under the ufp4 recipe the line also carries, untimed by `value`:
`e2m1_step`, the same step under the E2M1 baseline recipe of Table 1 on the same inputs, and
`quantizer_1gib`, every quantizer kernel on a 1 GiB bf16 tensor (Sec. 5 Q5).

Usage: python bench.py [--gpus 1] [--steps 20] [--warmup W] [--quant dual|separate]
                       [--workload square|dense|tiny|moe7.9b|moe124b|quant1g|quant1g-t|quant1g-dual|copy1g|
                                   quality-dense|quality-moe124b] [--no-compare] [--no-cpu-baseline]

The quant1g workloads time one quantizer on a 1 GiB bf16 tensor; they also time the same kernel without the
RHT (plain block quantization) and report the ratio, the quantity the paper gives for its own fused kernel.
The quality workloads print the Sec. 3.2 diagnostics of every GEMM operand of the layer (four grids, without
and with the RHT), computed on the GPU at full size by the statistics kernel, and that kernel's throughput.

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

from paper_2606_20381_amd import recipe as R  # noqa: E402
from paper_2606_20381_amd import ufp4 as U  # noqa: E402
from paper_2606_20381_amd import workloads as WL  # noqa: E402

HBM_PEAK_GBPS = 8000.0
INT8_PEAK_TOPS = 5000.0  # dense int8 / fp8 MFMA, MI355X
FP4_PEAK_TFLOPS = 10100.0  # dense fp4 / fp6 MFMA (the power-of-two-scale GEMM's FP6 operands)
# Bound of the per-16-block fp32-scale GEMM kernel: per 32x32 output tile and 16-block two MFMAs of 32 cycles each
# (block product, scale outer product) keep the matrix core busy 64 cycles (the counter SQ_VALU_MFMA_BUSY_CYCLES
# reads exactly that) for 32*32*16*2 ops, i.e. 512 ops per cycle per SIMD, at 256 CUs x 4 SIMDs x 2.4 GHz. The 16
# fp32 FMAs per tile-block (acc += D_b * (sA sB)_b) run on the VALU beside the MFMAs; the bound assumes they hide.
ATTAINABLE_TOPS = 32 * 32 * 16 * 2 / 64 * 256 * 4 * 2.4e9 / 1e12
GEMM_KERNEL = {
    "mxufp4": "gemm_mx_kernel (scaled f8f6f4 MFMA 32x32x64, FP6 E2M3 operands, E8M0 scales applied in the matrix core)",
    "ufp4": "gemm_f32_kernel (fp8 MFMA 32x32x16 per K-block + bf16 MFMA 32x32x8 scale outer product + fp32 FMA)",
    "e2m1": "gemm_f32_kernel (fp8 MFMA 32x32x16 per K-block on the E2M1 levels as e4m3 + bf16 MFMA 32x32x8 scale "
            "outer product + fp32 FMA)",
}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
WARMUP_SECONDS = 0.5
QUANT_BYTES_PER_ELEM = 2.75  # 2 B bf16 in, 0.5 B codes + 0.25 B scale out
DUAL_BYTES_PER_ELEM = 3.5  # two-operand quantizer: 2 B in, 2 x 0.75 B out
BYTES_PER_ELEM = {"quant": QUANT_BYTES_PER_ELEM, "quant2": DUAL_BYTES_PER_ELEM, "copy": 2.0,
                  "quantmx": 2.0 + 0.75 + 1.0 / 32,  # power-of-two scales: 0.75 B FP6 codes + 1/32 B E8M0 out
                  "quant2mx": 2.0 + 2 * (0.75 + 1.0 / 32)}
METRIC = "RHT+quantize GB/s and 4-bit fwd_y/bwd_dx/bwd_dw TFLOP/s (% of roofline)"


def gemm_family(recipe: str) -> str:
    """Which GEMM kernel a recipe runs: mxufp4 (FP6 scaled MFMA), ufp4 or e2m1 (fp8 MFMA per block)."""
    if recipe == "mxufp4":
        return "mxufp4"
    return "ufp4" if R.RECIPES[recipe].fmt == U.UNIFORM else "e2m1"


# The arithmetic each GEMM family computes in: 4-bit codes times per-block scales, fp32 accumulation.
ARITH = {
    "ufp4": "int4xf32",   # integer codes -7..7 (as exact fp8 e4m3 values on the fp8 MFMA), fp32 1x16 scales
    "e2m1": "fp4xf32",    # E2M1 codes (as exact fp8 e4m3 values on the fp8 MFMA), fp32 1x16 scales
    "mxufp4": "int4xe8m0",  # integer codes -7..7 (as FP6 E2M3 values), power-of-two 1x32 scales in the MFMA
}


def gemm_peak(recipe: str) -> float:
    """Dense MFMA peak of the GEMM's operand type: fp8 (= int8) for both per-16 grids, fp6 (the fp4 rate) for the
    power-of-two-scale GEMM."""
    return FP4_PEAK_TFLOPS if gemm_family(recipe) == "mxufp4" else INT8_PEAK_TOPS


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

# Recipes (paper_2606_20381_amd.recipe: Table 1, the Table 2 ablations, Sec. 5 Q4 and the Appendix search
# space) and the power-of-two-scale variant.
RECIPE_NOTES = {name: f"{name}: {r.note}" for name, r in R.RECIPES.items()}
RECIPE_NOTES["mxufp4"] = ("mxufp4: uniform -7..7 with power-of-two 1x32 (E8M0) scales, FP6 E2M3 codes, RHT16 on all "
                          "GEMMs, SR on dY")


def _quantizers(recipe: str):
    r = R.RECIPES[recipe]
    fn = U.rht_quantize if r.fmt == U.UNIFORM else U.e2m1_quantize
    return r.fmt, fn, r.rht[0], r.rht[1], r.rht[2]


def dense_step_mx(wl, tl: Timeline, dual: bool = True):
    """The layer step with power-of-two 1x32 scales: six quantizations (RHT16 everywhere, SR on dY; X and W
    through the two-operand quantizer unless `dual` is off) and the three passes on the scaled FP6 matrix-core
    instruction."""
    m, s = wl.sign_mask, wl.seed
    x, w, dy = (t.cuda() for t in (wl.x, wl.w, wl.dy))
    M, K = x.shape
    N = w.shape[0]
    E = U.empty_qtensor_mx
    q = {"x": E(M, K), "w": E(N, K), "dy": E(M, N), "wt": E(K, N), "dyt": E(N, M), "xt": E(K, M)}
    y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    dx = torch.empty(M, K, dtype=torch.bfloat16, device="cuda")
    dw = torch.empty(N, K, dtype=torch.float32, device="cuda")
    Q = U.mx_quantize
    src = {"x": x, "w": w}

    def step(rec):
        for a in ("x", "w"):
            if dual:
                tl.run(f"quant_{a}_{a}t", lambda a=a: U.mx_quantize_dual(
                    src[a], sign_mask_rows=m, sign_mask_cols=m, out_rows=q[a], out_cols=q[a + "t"]), rec)
            else:
                tl.run(f"quant_{a}", lambda a=a: Q(src[a], sign_mask=m, out=q[a]), rec)
                tl.run(f"quant_{a}t", lambda a=a: Q(src[a], transpose=True, sign_mask=m, out=q[a + "t"]), rec)
        tl.run("quant_dy_sr", lambda: Q(dy, sign_mask=m, rounding=U.SR, seed=s, stream_id=0, out=q["dy"]), rec)
        tl.run("quant_dyt_sr", lambda: Q(dy, transpose=True, sign_mask=m, rounding=U.SR, seed=s, stream_id=1,
                                         out=q["dyt"]), rec)
        tl.run("gemm_fwd_y", lambda: U.mx_gemm_fwd_y(q["x"], q["w"], out=y), rec)
        tl.run("gemm_bwd_dx", lambda: U.mx_gemm_bwd_dx(q["dy"], q["wt"], out=dx), rec)
        tl.run("gemm_bwd_dw", lambda: U.mx_gemm_bwd_dw(q["dyt"], q["xt"], out=dw), rec)

    elems = {"x": M * K, "w": N * K}
    kern = {}
    for a in ("x", "w"):
        if dual:
            kern[f"quant_{a}_{a}t"] = ("quant2mx", elems[a])
        else:
            kern.update({f"quant_{a}": ("quantmx", elems[a]), f"quant_{a}t": ("quantmx", elems[a])})
    kern.update({
        "quant_dy_sr": ("quantmx", M * N), "quant_dyt_sr": ("quantmx", M * N),
        "gemm_fwd_y": ("gemm", 2 * M * N * K), "gemm_bwd_dx": ("gemm", 2 * M * N * K),
        "gemm_bwd_dw": ("gemm", 2 * M * N * K),
    })
    return step, kern


def dense_step(wl, tl: Timeline, recipe: str = "ufp4", dual: bool = True):
    """The layer step under a recipe of paper_2606_20381_amd.recipe: six quantizations (X and W through the
    two-operand quantizer where the recipe allows it) and the three GEMMs."""
    if recipe == "mxufp4":
        return dense_step_mx(wl, tl, dual)
    m, s = wl.sign_mask, wl.seed
    r = R.RECIPES[recipe]
    x, w, dy = (t.cuda() for t in (wl.x, wl.w, wl.dy))
    M, K = x.shape
    N = w.shape[0]
    ls = R.LayerStep(M, N, K, r, dual=dual)
    q, src = ls.q, {"x": x, "w": w, "dy": dy}
    pairs = [(a, b) for a, b in (("x", "xt"), ("w", "wt")) if dual and R.dual_ok(r, a, b)]
    singles = [op for op in R.OPERANDS if not any(op in p for p in pairs)]

    def label(op):
        return "quant_" + op + ("_sr" if r.rounding(op) == U.SR else "")

    def step(rec):
        for a, b in pairs:
            tl.run(f"quant_{a}_{b}", lambda a=a, b=b: U.quantize_dual(
                src[a], fmt=r.fmt, rht_rows=r.rotated(a), rht_cols=r.rotated(b), sign_mask_rows=m, sign_mask_cols=m,
                rounding=r.rounding(a), seed=s, stream_rows=R.LAYOUT[a][3], stream_cols=R.LAYOUT[b][3],
                out_rows=q[a], out_cols=q[b]), rec)
        for op in singles:
            tl.run(label(op), lambda op=op: R.quantize_operand(src[R.LAYOUT[op][0]], op, r, m, s, out=q[op]), rec)
        tl.run("gemm_fwd_y", lambda: U.gemm_fwd_y(q["x"], q["w"], out=ls.y), rec)
        tl.run("gemm_bwd_dx", lambda: U.gemm_bwd_dx(q["dy"], q["wt"], out=ls.dx), rec)
        tl.run("gemm_bwd_dw", lambda: U.gemm_bwd_dw(q["dyt"], q["xt"], out=ls.dw), rec)

    elems = {"x": M * K, "w": N * K, "dy": M * N, "wt": N * K, "dyt": M * N, "xt": M * K}
    kern = {f"quant_{a}_{b}": ("quant2", elems[a]) for a, b in pairs}
    kern.update({label(op): ("quant", elems[op]) for op in singles})
    kern.update({"gemm_fwd_y": ("gemm", 2 * M * N * K), "gemm_bwd_dx": ("gemm", 2 * M * N * K),
                 "gemm_bwd_dw": ("gemm", 2 * M * N * K)})
    return step, kern


def moe_step(wl, tl: Timeline, recipe: str = "ufp4", dual: bool = True):
    if recipe == "mxufp4":
        return moe_step_mx(wl, tl, dual)
    m, s = wl.sign_mask, wl.seed
    fmt, Q, r_y, r_dx, r_dw = _quantizers(recipe)
    E, N, K = wl.w.shape
    x, dy = wl.x.cuda(), wl.dy.cuda()
    w2 = wl.w.reshape(E * N, K).cuda()
    M = x.shape[0]
    off, red = U.group_offsets(wl.counts)
    eoff, ered = U.group_offsets([N] * E)
    q = {
        "x": U.empty_qtensor(M, K, fmt), "w": U.empty_qtensor(E * N, K, fmt), "dy": U.empty_qtensor(M, N, fmt),
        "wt": U.empty_qtensor(K, E * N, fmt), "dyt": U.empty_qtensor(N, red, fmt), "xt": U.empty_qtensor(K, red, fmt),
    }
    y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    dx = torch.empty(M, K, dtype=torch.bfloat16, device="cuda")
    dw = torch.empty(E, N, K, dtype=torch.float32, device="cuda")

    def step(rec):
        tl.run("quant_x", lambda: Q(x, rht=r_y, sign_mask=m, out=q["x"]), rec)
        if dual:  # W^T's expert groups are N rows each (N % 16 == 0): no padding, the plain transposed operand
            tl.run("quant_w_wt", lambda: U.quantize_dual(w2, fmt=fmt, rht_rows=r_y, rht_cols=r_dx, sign_mask_rows=m,
                                                         sign_mask_cols=m, out_rows=q["w"], out_cols=q["wt"]), rec)
        else:
            tl.run("quant_w", lambda: Q(w2, rht=r_y, sign_mask=m, out=q["w"]), rec)
            tl.run("quant_wt", lambda: U.quantize_grouped_t(w2, eoff, ered, fmt=fmt, rht=r_dx, sign_mask=m,
                                                            out=q["wt"]), rec)
        tl.run("quant_dy_sr", lambda: Q(dy, rht=r_dx, sign_mask=m, rounding=U.SR, seed=s, stream_id=0,
                                        out=q["dy"]), rec)
        tl.run("quant_dyt_sr", lambda: U.quantize_grouped_t(dy, off, red, fmt=fmt, rht=r_dw, sign_mask=m,
                                                            rounding=U.SR, seed=s, stream_id=1, out=q["dyt"]), rec)
        tl.run("quant_xt", lambda: U.quantize_grouped_t(x, off, red, fmt=fmt, rht=r_dw, sign_mask=m,
                                                        out=q["xt"]), rec)
        tl.run("gemm_fwd_y", lambda: U.gemm_fwd_y_grouped(q["x"], q["w"], off, out=y), rec)
        tl.run("gemm_bwd_dx", lambda: U.gemm_bwd_dx_grouped(q["dy"], q["wt"], off, out=dx), rec)
        tl.run("gemm_bwd_dw", lambda: U.gemm_bwd_dw_grouped(q["dyt"], q["xt"], off, out=dw), rec)

    flops = 2 * M * N * K
    kern = {"quant_x": ("quant", M * K)}
    if dual:
        kern["quant_w_wt"] = ("quant2", E * N * K)
    else:
        kern.update({"quant_w": ("quant", E * N * K), "quant_wt": ("quant", E * N * K)})
    kern.update({
        "quant_dy_sr": ("quant", M * N), "quant_dyt_sr": ("quant", M * N), "quant_xt": ("quant", M * K),
        "gemm_fwd_y": ("gemm", flops), "gemm_bwd_dx": ("gemm", flops), "gemm_bwd_dw": ("gemm", flops),
    })
    return step, kern


def moe_step_mx(wl, tl: Timeline, dual: bool = True):
    """The expert layer step with power-of-two 1x32 scales: X and dY in the grouped-rows form (each expert's rows
    from a panel boundary) for the ragged-M passes, X^T and dY^T with each expert's tokens padded to 32 for
    bwd_dw, W and W^T plain (from the two-operand quantizer unless `dual` is off: W^T's expert groups are N
    rows each, N % 32 == 0, so the plain transposed operand is the grouped one); RHT16 everywhere, SR on dY."""
    m, s = wl.sign_mask, wl.seed
    E, N, K = wl.w.shape
    x, dy = wl.x.cuda(), wl.dy.cuda()
    w2 = wl.w.reshape(E * N, K).cuda()
    M = x.shape[0]
    off, prow = U.group_offsets(wl.counts, block=128)
    _, red32 = U.group_offsets(wl.counts, block=32)
    Q = U.empty_qtensor_mx
    q = {"x": Q(prow, K), "w": Q(E * N, K), "dy": Q(prow, N), "wt": Q(K, E * N), "dyt": Q(N, red32),
         "xt": Q(K, red32)}
    y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    dx = torch.empty(M, K, dtype=torch.bfloat16, device="cuda")
    dw = torch.empty(E, N, K, dtype=torch.float32, device="cuda")
    G = U.mx_quantize_grouped

    def step(rec):
        tl.run("quant_x", lambda: G(x, off, prow, transpose=False, sign_mask=m, out=q["x"]), rec)
        if dual:
            tl.run("quant_w_wt", lambda: U.mx_quantize_dual(w2, sign_mask_rows=m, sign_mask_cols=m, out_rows=q["w"],
                                                            out_cols=q["wt"]), rec)
        else:
            tl.run("quant_w", lambda: U.mx_quantize(w2, sign_mask=m, out=q["w"]), rec)
            tl.run("quant_wt", lambda: U.mx_quantize(w2, transpose=True, sign_mask=m, out=q["wt"]), rec)
        tl.run("quant_dy_sr", lambda: G(dy, off, prow, transpose=False, sign_mask=m, rounding=U.SR, seed=s,
                                        stream_id=0, out=q["dy"]), rec)
        tl.run("quant_dyt_sr", lambda: G(dy, off, red32, transpose=True, sign_mask=m, rounding=U.SR, seed=s,
                                         stream_id=1, out=q["dyt"]), rec)
        tl.run("quant_xt", lambda: G(x, off, red32, transpose=True, sign_mask=m, out=q["xt"]), rec)
        tl.run("gemm_fwd_y", lambda: U.mx_gemm_fwd_y_grouped(q["x"], q["w"], off, M, out=y), rec)
        tl.run("gemm_bwd_dx", lambda: U.mx_gemm_bwd_dx_grouped(q["dy"], q["wt"], off, M, out=dx), rec)
        tl.run("gemm_bwd_dw", lambda: U.mx_gemm_bwd_dw_grouped(q["dyt"], q["xt"], off, out=dw), rec)

    flops = 2 * M * N * K
    kern = {"quant_x": ("quantmx", M * K)}
    if dual:
        kern["quant_w_wt"] = ("quant2mx", E * N * K)
    else:
        kern.update({"quant_w": ("quantmx", E * N * K), "quant_wt": ("quantmx", E * N * K)})
    kern.update({
        "quant_dy_sr": ("quantmx", M * N), "quant_dyt_sr": ("quantmx", M * N), "quant_xt": ("quantmx", M * K),
        "gemm_fwd_y": ("gemm", flops), "gemm_bwd_dx": ("gemm", flops), "gemm_bwd_dw": ("gemm", flops),
    })
    return step, kern


def copy1g_step(tl: Timeline):
    """Plain device copy of the 1 GiB quantizer tensor: the calibration kernel for HBM byte counters."""
    t = WL.quantizer_tensor().cuda()
    dst = torch.empty_like(t)

    def step(rec):
        tl.run("copy", lambda: dst.copy_(t), rec)

    return step, {"copy": ("copy", t.numel() * t.element_size())}


def quant1g_step(tl: Timeline, mode: str, sr: bool = False):
    """One quantizer on a 1 GiB bf16 tensor: rowwise (reduction along its 16384 columns), transposed (operand
    X^T, reduction along its 32768 rows) or both operands in one pass, rounding RTNE or SR. Returns (step, kernel
    table, plain step, unfused step): the plain step runs the same kernel without the RHT."""
    t = WL.quantizer_tensor().cuda()
    R, C = t.shape
    rnd, rname = (U.SR, "sr") if sr else (U.RTNE, "rtne")
    if mode == "dual":
        qr, qc = U.empty_qtensor(R, C), U.empty_qtensor(C, R)

        def run(rht):
            return U.quantize_dual(t, rht_rows=rht, rht_cols=rht, sign_mask_rows=0x6A09, sign_mask_cols=0x6A09,
                                   rounding=rnd, seed=7, stream_rows=0, stream_cols=1, out_rows=qr, out_cols=qc)

        label, kind = "quant_dual_" + rname, "quant2"
    else:
        transpose = mode == "cols"
        q = U.empty_qtensor(C, R) if transpose else U.empty_qtensor(R, C)

        def run(rht):
            return U.rht_quantize(t, transpose=transpose, rht=rht, sign_mask=0x6A09, rounding=rnd, seed=7,
                                  stream_id=int(transpose), out=q)

        label, kind = ("quant_cols_" if transpose else "quant_rows_") + rname, "quant"

    def step(rec):
        tl.run(label, lambda: run(True), rec)

    def plain(rec):
        tl.run(label + "_plain", lambda: run(False), rec)

    unfused = None
    if mode == "rows" and not sr:
        # the unfused form: standalone RHT into an fp32 tensor, then the fp32-input quantizer (same codes)
        y = torch.empty((R, C), dtype=torch.float32, device="cuda")
        qu = U.empty_qtensor(R, C)

        def unfused(rec):
            tl.run(label + "_unfused_rht", lambda: U.rht(t, sign_mask=0x6A09, out=y), rec)
            tl.run(label + "_unfused_quant", lambda: U.quantize_f32(y, out=qu), rec)

    return step, {label: (kind, R * C)}, plain, unfused


# ---------------------------------------------------------------------------------------------------
# extras of a layer run: the E2M1 baseline step on the same inputs, every quantizer on a 1 GiB tensor
# ---------------------------------------------------------------------------------------------------

def time_steps(step, steps: int, warmup: int, warm_seconds: float = 0.0) -> float:
    """`warmup` untimed calls (more until `warm_seconds` have passed), then `steps` calls between two events on
    the current stream: ms per call."""
    n, t0 = 0, time.perf_counter()
    while n < warmup or time.perf_counter() - t0 < warm_seconds:
        step(False)
        n += 1
        if n % 16 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(steps):
        step(True)
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / steps


def e2m1_comparison(wl, steps: int, warmup: int, dual: bool) -> dict:
    """The same layer step under the E2M1 recipe of Table 1 (RHT on bwd_dw only, SR on dY), same inputs."""
    tl = Timeline()
    step, kern = (moe_step if wl.grouped else dense_step)(wl, tl, "e2m1", dual)
    ms = time_steps(step, steps, warmup)
    gemms, flops, qus = {}, 0, 0.0
    for label, (kind, work) in kern.items():
        us = tl.mean_us(label)
        if kind == "gemm":
            tf = work / (us * 1e-6) / 1e12
            gemms[label] = {"us": round(us, 2), "TFLOP/s": round(tf, 1), "frac_peak": round(tf / gemm_peak("e2m1"), 4)}
            flops += work
        else:
            qus += us
    return {"recipe": RECIPE_NOTES["e2m1"], "kernel": GEMM_KERNEL["e2m1"], "ms_per_step": round(ms, 4),
            "TFLOP/s": round(flops / (ms * 1e-3) / 1e12, 3), "gemms": gemms, "quant_all_us": round(qus, 2)}


def quantizer_1gib(steps: int, warmup: int) -> dict:
    """Each quantizer kernel on the 1 GiB bf16 tensor [32768, 16384] (Sec. 5 Q5's measurement): RHT16, both
    roundings, rowwise, transposed and both operands in one pass, the E2M1 grid, and the power-of-two-scale
    quantizers (rowwise, transposed, both in one pass)."""
    t = WL.quantizer_tensor().cuda()
    rows, cols = t.shape
    qr, qc = U.empty_qtensor(rows, cols), U.empty_qtensor(cols, rows)
    er = U.empty_qtensor(rows, cols, U.E2M1)
    mr, mc = U.empty_qtensor_mx(rows, cols), U.empty_qtensor_mx(cols, rows)
    m = 0x6A09
    cases = {
        "rows_rtne": (lambda: U.rht_quantize(t, sign_mask=m, out=qr), "quant"),
        "cols_rtne": (lambda: U.rht_quantize(t, transpose=True, sign_mask=m, out=qc), "quant"),
        "rows_sr": (lambda: U.rht_quantize(t, sign_mask=m, rounding=U.SR, seed=7, out=qr), "quant"),
        "cols_sr": (lambda: U.rht_quantize(t, transpose=True, sign_mask=m, rounding=U.SR, seed=7, stream_id=1,
                                           out=qc), "quant"),
        "dual_rtne": (lambda: U.quantize_dual(t, sign_mask_rows=m, sign_mask_cols=m, out_rows=qr, out_cols=qc),
                      "quant2"),
        "rows_e2m1_rtne": (lambda: U.e2m1_quantize(t, rht=True, sign_mask=m, out=er), "quant"),
        "mx_rows_rtne": (lambda: U.mx_quantize(t, sign_mask=m, out=mr), "quantmx"),
        "mx_cols_rtne": (lambda: U.mx_quantize(t, transpose=True, sign_mask=m, out=mc), "quantmx"),
        "mx_dual_rtne": (lambda: U.mx_quantize_dual(t, sign_mask_rows=m, sign_mask_cols=m, out_rows=mr,
                                                    out_cols=mc), "quant2mx"),
    }
    out = {}
    for label, (fn, kind) in cases.items():
        us = time_steps(lambda rec, fn=fn: fn(), steps, warmup, WARMUP_SECONDS) * 1e3
        gbps = rows * cols * BYTES_PER_ELEM[kind] / (us * 1e-6) / 1e9
        out[label] = {"us": round(us, 2), "GB/s": round(gbps, 1), "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4)}
    del t, qr, qc, er, mr, mc
    return out


# ---------------------------------------------------------------------------------------------------
# quality diagnostics (Sec. 3.2) on the layer's tensors at full size, from ufp4_quant_stats
# ---------------------------------------------------------------------------------------------------

QUALITY_GRIDS = [("uniform", U.UNIFORM, 0.0), ("e2m1", U.E2M1, 0.0), ("e2m1 max_fpx=4", U.E2M1, 4.0),
                 ("e2m1 max_fpx=2", U.E2M1, 2.0)]


def quality_report(wl, steps: int):
    """NMSE / SQNR / alpha / B_eff of every GEMM operand of the layer, per grid, without and with the RHT,
    Delta SQNR (Sec. 3.2), and the coherent attenuation eta = alpha_A alpha_B of each GEMM; plus the
    statistics kernel's own throughput on the first operand."""
    x, dy = wl.x.cuda(), wl.dy.cuda()
    w = wl.w.reshape(-1, wl.w.shape[-1]).cuda()  # experts stacked along N (multiples of 16)
    # operand: (tensor, transpose, rounding, SR stream), as in the layer step
    ops = {"X (fwd_y)": (x, False, U.RTNE, 0), "W (fwd_y)": (w, False, U.RTNE, 0),
           "dY (bwd_dx)": (dy, False, U.SR, 0), "W^T (bwd_dx)": (w, True, U.RTNE, 0),
           "dY^T (bwd_dw)": (dy, True, U.SR, 1), "X^T (bwd_dw)": (x, True, U.RTNE, 0)}
    table = {}
    for gname, fmt, mf in QUALITY_GRIDS:
        rows, stats = {}, {}
        for oname, (t, tr, rnd, st) in ops.items():
            r, recs = {}, {}
            for rht in (False, True):
                q = U.quant_stats(t, fmt, max_fpx=mf, transpose=tr, rht=rht, sign_mask=wl.sign_mask, rounding=rnd,
                                  seed=wl.seed, stream_id=st)
                recs[rht] = q
                r["rht" if rht else "raw"] = {"nmse": q.nmse, "sqnr_db": round(q.sqnr_db, 3),
                                              "alpha": round(q.alpha, 6), "beff": round(q.beff, 4)}
            r["delta_sqnr_db"] = round(U.delta_sqnr_db(recs[False], recs[True]), 3)
            rows[oname], stats[oname] = r, recs
        eta = {}
        for gemm, (a, b) in {"fwd_y": ("X (fwd_y)", "W (fwd_y)"), "bwd_dx": ("dY (bwd_dx)", "W^T (bwd_dx)"),
                             "bwd_dw": ("dY^T (bwd_dw)", "X^T (bwd_dw)")}.items():
            eta[gemm] = {("rht" if k else "raw"): round(U.gemm_attenuation(stats[a][k], stats[b][k]), 6)
                         for k in (False, True)}
        table[gname] = {"operands": rows, "eta": eta}
    # timing of the statistics kernel (uniform grid, RHT, X rowwise)
    rec = torch.empty(U.STATS_BYTES // 8, dtype=torch.float64, device="cuda")
    lib = U.lib()

    def launch():
        return lib.ufp4_quant_stats(U.UNIFORM, 0.0, x.data_ptr(), x.shape[0], x.shape[1], x.stride(0), 0, 1,
                                    wl.sign_mask, U.RTNE, 0, 0, rec.data_ptr(), U._stream())

    for _ in range(3):
        launch()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(steps):
        launch()
    e.record()
    torch.cuda.synchronize()
    us = s.elapsed_time(e) * 1e3 / steps
    gbps = x.numel() * 2 / (us * 1e-6) / 1e9
    return table, {"us": round(us, 2), "GB/s": round(gbps, 1), "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4),
                   "work": f"quant_stats_kernel + record clear on X {tuple(x.shape)} (reads 2 B per element)"}


# ---------------------------------------------------------------------------------------------------
# measured HBM traffic (rocprofv3 FETCH_SIZE / WRITE_SIZE runs, scaled by a 1 GiB copy), valid only for the
# kernel source it was measured on
# ---------------------------------------------------------------------------------------------------

TRAFFIC_SOURCES = {"gemm": "ufp4_gemm.hip", "gemm_mx": "ufp4_gemm_mx.hip", "quant": "ufp4_quant.hip"}


def _source_digest(name: str) -> str:
    """sha256 of a kernel source with its comments and blank space removed: a figure measured on a kernel stays
    valid across edits of its comments, and becomes stale with any change of the code."""
    import hashlib
    import re

    path = os.path.join(ROOT, "paper_2606_20381_amd", "csrc", name)
    with open(path, encoding="utf-8") as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)  # block comments
    text = re.sub(r"//[^\n]*", " ", text)                # line comments (the sources have no '//' in strings)
    code = " ".join(text.split())
    return hashlib.sha256(code.encode()).hexdigest()


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

def cpu_baseline(wl, tokens: int = 1280, wrows: int = 1280, recipe: str = "ufp4"):
    """The oracle's layer step (six quantizations, three fp64 GEMMs) on the first `tokens` rows of X and dY and
    the first `wrows` rows of W (dY's matching columns): the same arithmetic per element as the full layer, on
    a sample that fits a few seconds of host time. The rate is per sampled work."""
    from oracle import ufp4_oracle as O
    from threadpoolctl import threadpool_info

    M_full, K = wl.x.shape
    N_full = wl.w.shape[0]
    m, n = min(tokens, M_full), min(wrows, N_full)
    x = WL.bf16_bits(wl.x[:m].contiguous())
    dy = WL.bf16_bits(wl.dy[:m, :n].contiguous())
    w = WL.bf16_bits(wl.w[:n].contiguous())
    times = {}
    t0 = time.perf_counter()
    O.layer_gemms(x, w, dy, recipe, sign_mask=wl.sign_mask, seed=wl.seed, times=times)
    dt = time.perf_counter() - t0
    flops = 3 * 2 * m * n * K
    quant_elems = 2 * (m * K + n * K + m * n)  # the six operands
    blas = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    per_op = {k: round(v, 3) for k, v in times.items()}
    return {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": int(blas),
        "kind": "oracle",
        "per_op_s": per_op,
        "quantize_GB/s": round(quant_elems * QUANT_BYTES_PER_ELEM / times["quantize"] / 1e9, 3),
        "gemm_TFLOP/s": round(float(2 * m * n * K / np.mean([times[k] for k in ("fwd_y", "bwd_dx", "bwd_dw")])) / 1e12, 4),
        "sample": (f"whole {recipe} layer step (6 quantizations + 3 fp64 GEMMs) on {m} of {M_full} tokens and {n} "
                   f"of {N_full} output features (X [{m}, {K}], W [{n}, {K}], dY [{m}, {n}]); {dt:.1f} s; "
                   f"elementwise numpy on 1 thread, fp64 matmul on {blas} BLAS threads; host "
                   f"{platform.processor() or platform.machine()}, os.cpu_count()={os.cpu_count()}"),
    }


def progress(msg: str) -> None:
    """A line on stderr per finished stage (the JSON result is the only stdout line)."""
    print(f"bench.py: {msg}", file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=None, help="untimed steps (default: steps for WARMUP_SECONDS)")
    ap.add_argument("--workload", default="square",
                    choices=["square", "dense", "tiny", "moe7.9b", "moe124b", "quant1g", "quant1g-t", "quant1g-dual",
                             "copy1g", "quality-dense", "quality-moe124b"])
    ap.add_argument("--recipe", default="ufp4", choices=sorted(RECIPE_NOTES),
                    help="ufp4 (the method) or e2m1 (the comparison baseline of Table 1)")
    ap.add_argument("--quant", default="dual", choices=["dual", "separate"],
                    help="dual: X and W quantized to both operands in one pass (dY, SR, uses the single-output "
                         "kernels, measured faster); separate: six single-output quantizations")
    ap.add_argument("--rounding", default="rtne", choices=["rtne", "sr"],
                    help="rounding of the quant1g workloads (the layer step rounds dY stochastically, the rest RTNE)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-compare", action="store_true",
                    help="skip the E2M1 step and the 1 GiB quantizer runs that a ufp4 layer run carries")
    ap.add_argument("--graph", action="store_true",
                    help="also capture the layer step once in a HIP graph and time its replays (reported beside "
                         "`value`, which stays the eagerly launched step)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the hot path runs on one GPU only (asked for --gpus {args.gpus}); sharding it over "
              f"several GPUs is a design note, not an implemented mode", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    U.lib()

    if args.workload.startswith("quality"):
        wl = WL.CONFIGS["dense" if args.workload == "quality-dense" else "moe124b"]()
        table, kern_time = quality_report(wl, args.steps)
        print(json.dumps({
            "metric": "quantization quality of the layer's GEMM operands (Sec. 3.2): NMSE, SQNR, alpha, B_eff, "
                      "Delta SQNR; eta = alpha_A alpha_B per GEMM",
            "value": kern_time["GB/s"], "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
            "higher_is_better": True, "vs_baseline": None, "dtype": "f64+f32",
            "data": "synthetic (seeded, shapes and distributions of the workload; no real tensors)",
            "config": {"workload": wl.name, "note": "transposed operands of grouped tensors are taken along the "
                       "concatenated token axis, without the per-expert padding of the grouped quantizer"},
            "stats_kernel": kern_time, "quality": table}), flush=True)
        return

    tl = Timeline()
    wl = None
    plain = unfused = None
    if args.workload in ("quant1g", "quant1g-t", "quant1g-dual"):
        mode = {"quant1g": "rows", "quant1g-t": "cols", "quant1g-dual": "dual"}[args.workload]
        step, kern, plain, unfused = quant1g_step(tl, mode, args.rounding == "sr")
        what = {"rows": "rowwise", "cols": "transposed", "dual": "rowwise + transposed in one pass"}[mode]
        wname = f"standalone quantizer: 32768x16384 bf16 (1 GiB), {what} {args.rounding.upper()} with RHT"
    elif args.workload == "copy1g":
        step, kern = copy1g_step(tl)
        wname = "calibration: device copy of a 1 GiB bf16 tensor (read 1 GiB + write 1 GiB)"
    else:
        wl = WL.CONFIGS[args.workload]()
        if wl.grouped and args.recipe not in ("ufp4", "e2m1", "mxufp4"):
            print("bench.py: grouped (MoE) layers run the ufp4, e2m1 and mxufp4 recipes only", file=sys.stderr)
            sys.exit(2)
        step, kern = (moe_step if wl.grouped else dense_step)(wl, tl, args.recipe, args.quant == "dual")
        wname = wl.name
    torch.cuda.synchronize()
    progress(f"inputs of '{wname}' resident; warming up")

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
    context = None
    if plain is not None:
        # the same kernel without the RHT, timed after the measured steps (not part of `value`)
        for _ in range(args.warmup):
            plain(False)
        for _ in range(args.steps):
            plain(True)
        torch.cuda.synchronize()
        (label,) = kern
        fused_us, plain_us = tl.mean_us(label), tl.mean_us(label + "_plain")
        context = {"plain_quant_us": round(plain_us, 2), "fused_us": round(fused_us, 2),
                   "fused_over_plain": round(fused_us / plain_us, 3),
                   "paper": "fused / plain quantization latency ~1.06x (SM90), ~1.07x (SM100); Sec. 5 Q5"}
        if unfused is not None:
            for _ in range(args.warmup):
                unfused(False)
            for _ in range(args.steps):
                unfused(True)
            torch.cuda.synchronize()
            r_us, q_us = tl.mean_us(label + "_unfused_rht"), tl.mean_us(label + "_unfused_quant")
            context.update({
                "unfused_rht_us": round(r_us, 2), "unfused_quant_us": round(q_us, 2),
                "unfused_over_fused": round((r_us + q_us) / fused_us, 3),
                "unfused_form": "standalone RHT writing fp32 y (2 B in, 4 B out per element), then the fp32-input "
                                "quantizer (4 B in, 0.75 B out); same codes as the fused kernel",
                "paper_unfused": "unfused / fused latency 1.62x (SM90), 1.41x (SM100); Sec. 5 Q5"})

    progress(f"timed {args.steps} steps: {ms_per_step:.3f} ms per step")

    extras = {}
    if wl is not None and args.recipe == "ufp4" and not args.no_compare:
        extras["e2m1_step"] = e2m1_comparison(wl, args.steps, args.warmup, args.quant == "dual")
        extras["e2m1_step"]["ufp4_over_e2m1_speed"] = round(extras["e2m1_step"]["ms_per_step"] / ms_per_step, 3)
        progress("E2M1 step timed")
        extras["quantizer_1gib"] = quantizer_1gib(args.steps, 5)
        progress("1 GiB quantizers timed")

    graph_ctx = None
    if args.graph and wl is not None:
        # the library only launches kernels (no allocation, memset or synchronization), so the whole step can be
        # captured; replays skip the per-launch host overhead
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step(False)
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step(False)
        for _ in range(max(3, args.warmup)):
            graph.replay()
        torch.cuda.synchronize()
        gs, ge = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        gs.record()
        for _ in range(args.steps):
            graph.replay()
        ge.record()
        torch.cuda.synchronize()
        g_ms = gs.elapsed_time(ge) / args.steps
        graph_ctx = {"ms_per_step": round(g_ms, 4), "eager_ms_per_step": round(ms_per_step, 4),
                     "eager_over_graph": round(ms_per_step / g_ms, 3)}

    breakdown = {}
    gemm_flops = 0
    quant_bytes = 0.0
    for label, (kind, work) in kern.items():
        us = tl.mean_us(label)
        if kind == "copy":
            gbps = 2 * work / (us * 1e-6) / 1e9
            breakdown[label] = {"us": round(us, 2), "GB/s": round(gbps, 1), "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4)}
            quant_bytes += 2 * work
        elif kind in ("quant", "quant2", "quantmx", "quant2mx"):
            gbps = work * BYTES_PER_ELEM[kind] / (us * 1e-6) / 1e9
            breakdown[label] = {"us": round(us, 2), "GB/s": round(gbps, 1), "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4)}
            quant_bytes += work * BYTES_PER_ELEM[kind]
        else:
            tf = work / (us * 1e-6) / 1e12
            breakdown[label] = {"us": round(us, 2), "TFLOP/s": round(tf, 1),
                                "frac_peak": round(tf / gemm_peak(args.recipe), 4)}
            gemm_flops += work

    gemm_labels = [k for k, (kind, _) in kern.items() if kind == "gemm"]
    quant_kinds = ("quant", "quant2", "quantmx", "quant2mx", "copy")
    quant_labels = [k for k, (kind, _) in kern.items() if kind in quant_kinds]
    if gemm_labels:
        value = gemm_flops / (ms_per_step * 1e-3) / 1e12
        unit = "TFLOP/s"
        per_launch = np.mean([kern[k][1] for k in gemm_labels])
        avg_us = np.mean([tl.mean_us(k) for k in gemm_labels])
        ach = per_launch / (avg_us * 1e-6) / 1e12
        peak = gemm_peak(args.recipe)
        roof = {"bound": "mfma", "kernel": GEMM_KERNEL[gemm_family(args.recipe)],
                "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(ach / peak, 4),
                "traffic": measured_traffic("gemm_mx" if args.recipe == "mxufp4" else "gemm", wname + "/" + args.recipe)}
        if args.recipe != "mxufp4":  # per-16 fp32 scales: a scale outer product per tile and block
            roof["attainable"] = {"peak": round(ATTAINABLE_TOPS, 1), "frac": round(ach / ATTAINABLE_TOPS, 4),
                                  "why": "two 32-cycle MFMAs per 32x32 tile and 16-block (block product and "
                                         "scale outer product); the 16 fp32 FMAs per tile-block hidden beside them"}
    else:
        value = quant_bytes / (ms_per_step * 1e-3) / 1e9
        unit = "GB/s"
        label = quant_labels[0]
        us = tl.mean_us(label)
        per_launch = kern[label][1] * BYTES_PER_ELEM[kern[label][0]]
        ach = per_launch / (us * 1e-6) / 1e9
        kname = {"quant_rows_rtne": "quant_rows_kernel", "quant_cols_rtne": "quant_cols_kernel",
                 "quant_rows_sr": "quant_rows_kernel", "quant_cols_sr": "quant_cols_kernel",
                 "quant_dual_sr": "quant_dual_kernel",
                 "quant_dual_rtne": "quant_dual_kernel"}.get(label, "copy")
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
        "dtype": ARITH[gemm_family(args.recipe)] if gemm_labels else "bf16->int4xf32",
        "data": "synthetic (seeded, shapes and distributions of the workload; no real tensors)",
        "config": {"workload": wname, "recipe": RECIPE_NOTES[args.recipe],
                   "outputs": "Y bf16, dX bf16, dW fp32" if gemm_labels else "codes + fp32 scales",
                   "wall_s": round(wall, 3)},
        "roofline": roof,
        "breakdown": breakdown,
    }
    if wl is not None:
        # the step re-reads the same inputs every time: tensors that fit the 256 MB last-level cache (MALL) may
        # be served from it, so the per-kernel quantizer rates of a layer step are cache-warm figures
        out["breakdown_note"] = ("per-kernel means inside the timed steps; the inputs are reused across steps, so "
                                 "tensors under the 256 MB MALL may be read warm")
    if context is not None:
        out["rht_cost"] = context
    if graph_ctx is not None:
        out["graph_replay"] = graph_ctx
    out.update(extras)
    if wl is not None:
        out["config"]["quant"] = args.quant
    if wl is not None and not args.no_cpu_baseline and not wl.grouped:
        progress("timing the CPU oracle on a sample of the layer")
        out["cpu_baseline"] = cpu_baseline(wl, recipe=args.recipe)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
