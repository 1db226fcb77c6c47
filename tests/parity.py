"""Parity helpers: run one operand or GEMM through the oracle (on sampled rows when the tensor is large)
and through the HIP library, and compare. The oracle never sees a value produced by the HIP path."""

from __future__ import annotations

import numpy as np
import torch

from oracle import ufp4_oracle as O
from paper_2606_20381_amd import ufp4 as U
from paper_2606_20381_amd.workloads import bf16_bits

# name -> (layout, rounding, SR stream) for the six operands of one layer step (Sec. 2.2 last sentence;
# Table 1: SR on dY only). "t" marks a transposed operand.
OPERANDS = {
    "x": ("rows", O.RTNE, 0),
    "w": ("rows", O.RTNE, 0),
    "dy": ("rows", O.SR, 0),
    "wt": ("cols", O.RTNE, 0),
    "dyt": ("cols", O.SR, 1),
    "xt": ("cols", O.RTNE, 0),
}
SOURCE = {"x": "x", "w": "w", "dy": "dy", "wt": "w", "dyt": "dy", "xt": "x"}


def oracle_operand(t_bits: np.ndarray, layout: str, fmt: int, rounding: int, rht: bool, mask: int, seed: int,
                   stream: int, rows=None):
    """Oracle quantization of operand rows `rows` (None = all). Rowwise: A = T; transposed: A = T^T."""
    if layout == "rows":
        ids = np.arange(t_bits.shape[0]) if rows is None else np.asarray(rows)
        a = O.bf16_bits_to_f32(t_bits[ids])
    else:
        ids = np.arange(t_bits.shape[1]) if rows is None else np.asarray(rows)
        a = np.ascontiguousarray(O.bf16_bits_to_f32(t_bits[:, ids]).T)
    idx, sc = O.quantize_rows(a, fmt, rounding, rht, mask, seed, stream, row_ids=ids)
    return idx, sc


def oracle_operand_grouped(t_bits: np.ndarray, counts, fmt, rounding, rht, mask, seed, stream, rows=None):
    """Oracle grouped-transposed operand (rows = columns of T), restricted to operand rows `rows`."""
    ids = np.arange(t_bits.shape[1]) if rows is None else np.asarray(rows)
    a, poff = O.operand_colwise_grouped(np.ascontiguousarray(t_bits[:, ids]), counts)
    idx, sc = O.quantize_rows(a, fmt, rounding, rht, mask, seed, stream, row_ids=ids)
    return idx, sc, poff


def gpu_operand(t_dev: torch.Tensor, layout: str, fmt: int, rounding: int, rht: bool, mask: int, seed: int,
                stream: int) -> U.QTensor:
    fn = U.rht_quantize if fmt == O.UNIFORM else U.e2m1_quantize
    return fn(t_dev, transpose=(layout == "cols"), rht=rht, sign_mask=mask, rounding=rounding, seed=seed,
              stream_id=stream)


def gpu_rows(q: U.QTensor, rows=None):
    """(packed codes, scales) of the GPU operand as row-major host arrays, restricted to `rows`."""
    codes, scales = q.codes_rows(), q.scales_rows()
    if rows is not None:
        idx = torch.as_tensor(np.asarray(rows), dtype=torch.int64, device=codes.device)
        codes, scales = codes[idx], scales[idx]
    return codes.cpu().numpy(), scales.cpu().numpy()


def assert_codes_equal(gpu_codes, gpu_scales, idx, sc, fmt, what=""):
    want_codes = O.pack_codes(idx, fmt)
    if not np.array_equal(gpu_codes, want_codes):
        bad = np.argwhere(gpu_codes != want_codes)
        r, c = bad[0]
        raise AssertionError(f"{what}: {len(bad)} code bytes differ; first at row {r} byte {c}: "
                             f"gpu {gpu_codes[r, c]:#04x} oracle {want_codes[r, c]:#04x}")
    gs = np.ascontiguousarray(gpu_scales).view(np.uint32)
    ws = np.ascontiguousarray(sc.astype(np.float32)).view(np.uint32)
    if not np.array_equal(gs, ws):
        bad = np.argwhere(gs != ws)
        r, c = bad[0]
        raise AssertionError(f"{what}: {len(bad)} scales differ; first at row {r} block {c}: "
                             f"gpu {gpu_scales[r, c]!r} oracle {sc[r, c]!r}")


def rel_fro(got: np.ndarray, want: np.ndarray) -> float:
    want = np.asarray(want, dtype=np.float64)
    num = np.linalg.norm(np.asarray(got, dtype=np.float64) - want)
    den = np.linalg.norm(want)
    return float(num / den) if den > 0 else float(num)


def to_numpy(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()


def layer_bits(wl):
    return {k: bf16_bits(getattr(wl, k)) for k in ("x", "w", "dy")}


def sample(n: int, k: int, rng: np.random.Generator) -> np.ndarray:
    """k sorted distinct indices in [0, n), always including the first and the last."""
    if n <= k:
        return np.arange(n)
    s = rng.choice(np.arange(1, n - 1), size=k - 2, replace=False)
    return np.sort(np.concatenate([[0, n - 1], s]))
