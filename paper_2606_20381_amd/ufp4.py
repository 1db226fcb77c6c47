"""Python binding of libufp4 (ctypes). Argument marshalling only: every step runs in the HIP library.

Tensors are torch tensors on the GPU; torch supplies device memory and the current stream. The library
must be built (``python -m paper_2606_20381_amd.build``); without it every call raises.
"""

from __future__ import annotations

import ctypes
import math
import os
import struct
from dataclasses import dataclass

import torch

UNIFORM = 0
E2M1 = 1
RTNE = 0
SR = 1
OUT_F32 = 0
OUT_BF16 = 1

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libufp4.so")
_lib = None

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32 = ctypes.c_int32
_INT = ctypes.c_int
_U32 = ctypes.c_uint32
_U64 = ctypes.c_uint64

_QUANT_ARGS = [_P, _I64, _I64, _I64, _INT, _INT, _U32, _INT, _U64, _U32, _P, _I64, _P, _I64, _P]
_GEMM_ARGS = [_P, _I64, _P, _I64, _P, _I64, _P, _I64, _I64, _I64, _I64, _INT, _P, _I64, _INT, _P]
_GEMM_MX_ARGS = [_P, _I64, _P, _I64, _P, _I64, _P, _I64, _I64, _I64, _I64, _P, _I64, _INT, _P]
SIGNATURES = {
    "ufp4_status_string": ([_INT], ctypes.c_char_p),
    "ufp4_version": ([], ctypes.c_char_p),
    "ufp4_rht_quantize": (_QUANT_ARGS, _INT),
    "ufp4_e2m1_quantize": (_QUANT_ARGS, _INT),
    "ufp4_quantize_grouped_t": ([_INT, _P, _I64, _I64, _I64, _P, _P, _I32, _I64, _INT, _U32, _INT, _U64, _U32, _P,
                                 _I64, _P, _I64, _P], _INT),
    "ufp4_quantize_dual": ([_INT, _P, _I64, _I64, _I64, _INT, _U32, _U32, _INT, _U32, _U32, _INT, _U64, _P, _I64, _P,
                            _I64, _P, _I64, _P, _I64, _P], _INT),
    "ufp4_e2m1_quantize_range": ([_P, _I64, _I64, _I64, _INT, _INT, _U32, _INT, _U64, _U32, ctypes.c_float, _P, _I64,
                                  _P, _I64, _P], _INT),
    "ufp4_quant_stats": ([_INT, ctypes.c_float, _P, _I64, _I64, _I64, _INT, _INT, _U32, _INT, _U64, _U32, _P, _P], _INT),
    "ufp4_quantize_rht_block": ([_INT, _P, _I64, _I64, _I64, _INT, _INT, _P, _INT, _U64, _U32, _P, _I64, _P, _I64, _P],
                                _INT),
    "ufp4_rht": ([_P, _I64, _I64, _I64, _U32, _P, _I64, _P], _INT),
    "ufp4_quantize_f32": ([_INT, _P, _I64, _I64, _I64, _INT, _U64, _U32, _P, _I64, _P, _I64, _P], _INT),
    "ufp4_mx_quantize": (_QUANT_ARGS, _INT),
    "ufp4_mx_gemm_fwd_y": (_GEMM_MX_ARGS, _INT),
    "ufp4_mx_gemm_bwd_dx": (_GEMM_MX_ARGS, _INT),
    "ufp4_mx_gemm_bwd_dw": (_GEMM_MX_ARGS, _INT),
    "ufp4_gemm_fwd_y": (_GEMM_ARGS, _INT),
    "ufp4_gemm_bwd_dx": (_GEMM_ARGS, _INT),
    "ufp4_gemm_bwd_dw": (_GEMM_ARGS, _INT),
    "ufp4_gemm_fwd_y_grouped": ([_P, _I64, _P, _I64, _P, _I64, _P, _I64, _P, _I32, _I64, _I64, _I64, _INT, _P, _I64,
                                 _INT, _P], _INT),
    "ufp4_gemm_bwd_dx_grouped": ([_P, _I64, _P, _I64, _P, _I64, _P, _I64, _P, _I32, _I64, _I64, _I64, _INT, _P, _I64,
                                  _INT, _P], _INT),
    "ufp4_gemm_bwd_dw_grouped": ([_P, _I64, _P, _I64, _P, _I64, _P, _I64, _P, _I32, _I64, _I64, _I64, _INT, _P, _I64,
                                  _INT, _P], _INT),
}


def library_path() -> str:
    return _LIB_PATH


def lib() -> ctypes.CDLL:
    """Load libufp4.so (once) and declare the C signatures. Raises if the library is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is not built; run `python -m paper_2606_20381_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        for name, (args, res) in SIGNATURES.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


class UFP4Error(RuntimeError):
    def __init__(self, status: int, call: str):
        msg = lib().ufp4_status_string(status).decode()
        super().__init__(f"{call}: {msg} (status {status})")
        self.status = status


def _check(status: int, call: str) -> None:
    if status != 0:
        raise UFP4Error(status, call)


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


PANEL_ROWS = 128  # rows per panel of a quantized operand


@dataclass
class QTensor:
    """A quantized operand [rows, red] in the library's panel layout.

    Rows are grouped in panels of 128; within a panel, block b (16 reduction positions) of all 128 rows is
    contiguous: 128 x 8 bytes of codes at b * 1024 and 128 fp32 scales at b * 128. Rows past ``rows`` in the
    last panel hold zeros. ``codes_rows()`` / ``scales_rows()`` give the plain row-major views.
    """

    codes: torch.Tensor  # uint8 [panels, >= 1024 * red/16]
    scales: torch.Tensor  # float32 [panels, >= 128 * red/16]
    fmt: int
    rows: int
    red: int

    @property
    def code_panel_ld(self) -> int:
        return self.codes.stride(0)

    @property
    def scale_panel_ld(self) -> int:
        return self.scales.stride(0)

    @property
    def panels(self) -> int:
        return self.codes.shape[0]

    def codes_rows(self) -> torch.Tensor:
        """Codes as uint8 [rows, red/2], row-major (a copy)."""
        nkb = self.red // 16
        v = self.codes[:, : nkb * 1024].reshape(self.panels, nkb, PANEL_ROWS, 8).permute(0, 2, 1, 3)
        return v.reshape(self.panels * PANEL_ROWS, nkb * 8)[: self.rows]

    def scales_rows(self) -> torch.Tensor:
        """Scales as float32 [rows, red/16], row-major (a copy)."""
        nkb = self.red // 16
        v = self.scales[:, : nkb * PANEL_ROWS].reshape(self.panels, nkb, PANEL_ROWS).permute(0, 2, 1)
        return v.reshape(self.panels * PANEL_ROWS, nkb)[: self.rows]


def empty_qtensor(rows: int, red: int, fmt: int = UNIFORM, device="cuda") -> QTensor:
    panels = max(1, -(-rows // PANEL_ROWS))
    nkb = red // 16
    codes = torch.empty((panels, max(16, nkb * 1024)), dtype=torch.uint8, device=device)
    scales = torch.empty((panels, max(4, nkb * PANEL_ROWS)), dtype=torch.float32, device=device)
    return QTensor(codes, scales, fmt, rows, red)


def _quantize_call(name, fmt, x, transpose, rht, sign_mask, rounding, seed, stream_id, out):
    if x.dtype != torch.bfloat16 or not x.is_cuda or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D row-major bf16 CUDA tensor")
    rows, cols = x.shape
    qrows, red = (cols, rows) if transpose else (rows, cols)
    q = out if out is not None else empty_qtensor(qrows, red, fmt, x.device)
    st = getattr(lib(), name)(x.data_ptr(), rows, cols, x.stride(0), int(transpose), int(rht), sign_mask, rounding,
                              seed & 0xFFFFFFFFFFFFFFFF, stream_id, q.codes.data_ptr(), q.code_panel_ld,
                              q.scales.data_ptr(), q.scale_panel_ld, _stream())
    _check(st, name)
    return q


def rht_quantize(x: torch.Tensor, *, transpose: bool = False, rht: bool = True, sign_mask: int = 0,
                 rounding: int = RTNE, seed: int = 0, stream_id: int = 0, out: QTensor | None = None) -> QTensor:
    """Fused RHT + uniform-grid quantization (ufp4_rht_quantize)."""
    return _quantize_call("ufp4_rht_quantize", UNIFORM, x, transpose, rht, sign_mask, rounding, seed, stream_id, out)


def e2m1_quantize(x: torch.Tensor, *, transpose: bool = False, rht: bool = False, sign_mask: int = 0,
                  rounding: int = RTNE, seed: int = 0, stream_id: int = 0, out: QTensor | None = None) -> QTensor:
    """Fused (optional) RHT + E2M1 quantization (ufp4_e2m1_quantize), the comparison baseline."""
    return _quantize_call("ufp4_e2m1_quantize", E2M1, x, transpose, rht, sign_mask, rounding, seed, stream_id, out)


def e2m1_quantize_range(x: torch.Tensor, max_fpx: float, *, transpose: bool = False, rht: bool = False,
                        sign_mask: int = 0, rounding: int = RTNE, seed: int = 0, stream_id: int = 0,
                        out: QTensor | None = None) -> QTensor:
    """E2M1 quantization on the grid cut at max_fpx in {2, 4, 6} (ufp4_e2m1_quantize_range)."""
    if x.dtype != torch.bfloat16 or not x.is_cuda or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D row-major bf16 CUDA tensor")
    rows, cols = x.shape
    qrows, red = (cols, rows) if transpose else (rows, cols)
    q = out if out is not None else empty_qtensor(qrows, red, E2M1, x.device)
    st = lib().ufp4_e2m1_quantize_range(x.data_ptr(), rows, cols, x.stride(0), int(transpose), int(rht), sign_mask,
                                        rounding, seed & 0xFFFFFFFFFFFFFFFF, stream_id, float(max_fpx),
                                        q.codes.data_ptr(), q.code_panel_ld, q.scales.data_ptr(), q.scale_panel_ld,
                                        _stream())
    _check(st, "ufp4_e2m1_quantize_range")
    return q


def quantize_rht_block(x: torch.Tensor, fmt: int = UNIFORM, *, rht_block: int = 16, sign_mask: int = 0,
                       transpose: bool = False, rounding: int = RTNE, seed: int = 0, stream_id: int = 0,
                       out: QTensor | None = None) -> QTensor:
    """RHT over n-blocks (n = rht_block, sign_mask an n-bit integer), then 1x16 quantization
    (ufp4_quantize_rht_block)."""
    if x.dtype != torch.bfloat16 or not x.is_cuda or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D row-major bf16 CUDA tensor")
    rows, cols = x.shape
    qrows, red = (cols, rows) if transpose else (rows, cols)
    q = out if out is not None else empty_qtensor(qrows, red, fmt, x.device)
    words = (ctypes.c_uint16 * 8)(*[(sign_mask >> (16 * k)) & 0xFFFF for k in range(8)])
    st = lib().ufp4_quantize_rht_block(fmt, x.data_ptr(), rows, cols, x.stride(0), int(transpose), rht_block,
                                       ctypes.cast(words, ctypes.c_void_p), rounding, seed & 0xFFFFFFFFFFFFFFFF,
                                       stream_id, q.codes.data_ptr(), q.code_panel_ld, q.scales.data_ptr(),
                                       q.scale_panel_ld, _stream())
    _check(st, "ufp4_quantize_rht_block")
    return q


def rht(x: torch.Tensor, *, sign_mask: int = 0, out: torch.Tensor | None = None) -> torch.Tensor:
    """Standalone block-16 RHT along the rows of x (ufp4_rht): fp32 [rows, cols]."""
    if x.dtype != torch.bfloat16 or not x.is_cuda or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D row-major bf16 CUDA tensor")
    y = out if out is not None else torch.empty(x.shape, dtype=torch.float32, device=x.device)
    if y.dtype != torch.float32 or y.shape != x.shape or y.stride(1) != 1:
        raise ValueError("out must be a row-major fp32 tensor of x's shape")
    st = lib().ufp4_rht(x.data_ptr(), x.shape[0], x.shape[1], x.stride(0), sign_mask, y.data_ptr(), y.stride(0),
                        _stream())
    _check(st, "ufp4_rht")
    return y


def quantize_f32(x: torch.Tensor, fmt: int = UNIFORM, *, rounding: int = RTNE, seed: int = 0, stream_id: int = 0,
                 out: QTensor | None = None) -> QTensor:
    """Rowwise quantization of an fp32 tensor, no transform (ufp4_quantize_f32)."""
    if x.dtype != torch.float32 or not x.is_cuda or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D row-major fp32 CUDA tensor")
    rows, cols = x.shape
    q = out if out is not None else empty_qtensor(rows, cols, fmt, x.device)
    st = lib().ufp4_quantize_f32(fmt, x.data_ptr(), rows, cols, x.stride(0), rounding, seed & 0xFFFFFFFFFFFFFFFF,
                                 stream_id, q.codes.data_ptr(), q.code_panel_ld, q.scales.data_ptr(),
                                 q.scale_panel_ld, _stream())
    _check(st, "ufp4_quantize_f32")
    return q


# number of levels (magnitude buckets, zero included) of each grid: B_eff's K
def grid_levels(fmt: int, max_fpx: float = 0.0) -> int:
    if fmt == UNIFORM or max_fpx in (0.0, 6.0):
        return 8
    return {2.0: 5, 4.0: 7}[float(max_fpx)]


@dataclass
class QuantStats:
    """Record of ufp4_quant_stats: fp64 sums over the elements and the magnitude-code histogram."""

    err2: float
    ref2: float
    cross: float
    hist: list
    fmt: int
    max_fpx: float

    @property
    def nmse(self) -> float:
        return self.err2 / self.ref2 if self.ref2 > 0 else float("nan")

    @property
    def sqnr_db(self) -> float:
        return -10.0 * math.log10(self.nmse) if self.err2 > 0 else float("inf")

    @property
    def alpha(self) -> float:
        return self.cross / self.ref2 if self.ref2 > 0 else float("nan")

    @property
    def beff(self) -> float:
        k = grid_levels(self.fmt, self.max_fpx)
        n = sum(self.hist[:k])
        ent = -sum((h / n) * math.log(h / n + 1e-12) for h in self.hist[:k]) if n else 0.0
        return math.exp(ent) / k


STATS_BYTES = 88  # 3 doubles + 8 uint64


def quant_stats(x: torch.Tensor, fmt: int = UNIFORM, *, max_fpx: float = 0.0, transpose: bool = False,
                rht: bool = True, sign_mask: int = 0, rounding: int = RTNE, seed: int = 0, stream_id: int = 0,
                out: torch.Tensor | None = None) -> QuantStats:
    """Quality statistics of one quantization of x (ufp4_quant_stats); synchronizes to read the record."""
    if x.dtype != torch.bfloat16 or not x.is_cuda or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D row-major bf16 CUDA tensor")
    rows, cols = x.shape
    rec = out if out is not None else torch.empty(STATS_BYTES // 8, dtype=torch.float64, device=x.device)
    st = lib().ufp4_quant_stats(fmt, float(max_fpx), x.data_ptr(), rows, cols, x.stride(0), int(transpose), int(rht),
                                sign_mask, rounding, seed & 0xFFFFFFFFFFFFFFFF, stream_id, rec.data_ptr(), _stream())
    _check(st, "ufp4_quant_stats")
    raw = rec.cpu().numpy().tobytes()
    vals = struct.unpack("<3d8Q", raw[:STATS_BYTES])
    return QuantStats(vals[0], vals[1], vals[2], list(vals[3:]), fmt, float(max_fpx))


def delta_sqnr_db(raw: QuantStats, rotated: QuantStats) -> float:
    """10 log10(NMSE_I / NMSE_H16) (Sec. 3.2): positive when the rotation lowers the quantization error."""
    return 10.0 * math.log10(raw.nmse / rotated.nmse)


def quantize_dual(x: torch.Tensor, *, fmt: int = UNIFORM, rht_rows: bool = True, rht_cols: bool = True,
                  sign_mask_rows: int = 0, sign_mask_cols: int = 0, rounding: int = RTNE, seed: int = 0,
                  stream_rows: int = 0, stream_cols: int = 0, out_rows: QTensor | None = None,
                  out_cols: QTensor | None = None) -> tuple[QTensor, QTensor]:
    """Both operands of x [rows, cols] from one read (ufp4_quantize_dual): (Q_r [rows, cols] along cols,
    Q_c [cols, rows] along rows)."""
    if x.dtype != torch.bfloat16 or not x.is_cuda or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D row-major bf16 CUDA tensor")
    rows, cols = x.shape
    qr = out_rows if out_rows is not None else empty_qtensor(rows, cols, fmt, x.device)
    qc = out_cols if out_cols is not None else empty_qtensor(cols, rows, fmt, x.device)
    st = lib().ufp4_quantize_dual(fmt, x.data_ptr(), rows, cols, x.stride(0), int(rht_rows), sign_mask_rows,
                                  stream_rows, int(rht_cols), sign_mask_cols, stream_cols, rounding,
                                  seed & 0xFFFFFFFFFFFFFFFF, qr.codes.data_ptr(), qr.code_panel_ld,
                                  qr.scales.data_ptr(), qr.scale_panel_ld, qc.codes.data_ptr(), qc.code_panel_ld,
                                  qc.scales.data_ptr(), qc.scale_panel_ld, _stream())
    _check(st, "ufp4_quantize_dual")
    return qr, qc


@dataclass
class QTensorMX:
    """An operand quantized with power-of-two 1x32 scales, [rows, red] in panels of 128 rows: 32-block b of the
    panel's rows is contiguous, 3072 bytes of FP6 E2M3 codes at b * 3072 (three planes of 128 x 8 bytes: row
    i's 24-byte string is plane 0, 1, 2 at i * 8) and 128 E8M0 bytes at b * 128."""

    codes: torch.Tensor  # uint8 [panels, >= 3072 * red/32]
    scales: torch.Tensor  # uint8 [panels, >= 128 * red/32]
    rows: int
    red: int

    @property
    def code_panel_ld(self) -> int:
        return self.codes.stride(0)

    @property
    def scale_panel_ld(self) -> int:
        return self.scales.stride(0)

    @property
    def panels(self) -> int:
        return self.codes.shape[0]

    def codes_rows(self) -> torch.Tensor:
        """Codes as uint8 [rows, red * 3/4] (24 bytes per 32-block), row-major (a copy)."""
        nkb = self.red // 32
        v = self.codes[:, : nkb * 3072].reshape(self.panels, nkb, 3, PANEL_ROWS, 8).permute(0, 3, 1, 2, 4)
        return v.reshape(self.panels * PANEL_ROWS, nkb * 24)[: self.rows]

    def scales_rows(self) -> torch.Tensor:
        """E8M0 scale bytes as uint8 [rows, red/32], row-major (a copy)."""
        nkb = self.red // 32
        v = self.scales[:, : nkb * PANEL_ROWS].reshape(self.panels, nkb, PANEL_ROWS).permute(0, 2, 1)
        return v.reshape(self.panels * PANEL_ROWS, nkb)[: self.rows]


def empty_qtensor_mx(rows: int, red: int, device="cuda") -> QTensorMX:
    panels = max(1, -(-rows // PANEL_ROWS))
    nkb = red // 32
    codes = torch.empty((panels, max(16, nkb * 3072)), dtype=torch.uint8, device=device)
    scales = torch.empty((panels, max(16, nkb * PANEL_ROWS)), dtype=torch.uint8, device=device)
    return QTensorMX(codes, scales, rows, red)


def mx_quantize(x: torch.Tensor, *, transpose: bool = False, rht: bool = True, sign_mask: int = 0,
                rounding: int = RTNE, seed: int = 0, stream_id: int = 0, out: QTensorMX | None = None) -> QTensorMX:
    """Fused RHT + uniform-grid quantization with power-of-two 1x32 scales (ufp4_mx_quantize)."""
    if x.dtype != torch.bfloat16 or not x.is_cuda or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D row-major bf16 CUDA tensor")
    rows, cols = x.shape
    qrows, red = (cols, rows) if transpose else (rows, cols)
    q = out if out is not None else empty_qtensor_mx(qrows, red, x.device)
    st = lib().ufp4_mx_quantize(x.data_ptr(), rows, cols, x.stride(0), int(transpose), int(rht), sign_mask, rounding,
                                seed & 0xFFFFFFFFFFFFFFFF, stream_id, q.codes.data_ptr(), q.code_panel_ld,
                                q.scales.data_ptr(), q.scale_panel_ld, _stream())
    _check(st, "ufp4_mx_quantize")
    return q


def _gemm_mx_call(name, a: QTensorMX, b: QTensorMX, M, N, K, c: torch.Tensor):
    if c.dim() != 2 or c.stride(1) != 1:
        raise ValueError("output must be a 2-D row-major tensor")
    st = getattr(lib(), name)(a.codes.data_ptr(), a.code_panel_ld, a.scales.data_ptr(), a.scale_panel_ld,
                              b.codes.data_ptr(), b.code_panel_ld, b.scales.data_ptr(), b.scale_panel_ld, M, N, K,
                              c.data_ptr(), c.stride(0), _odt(c), _stream())
    _check(st, name)
    return c


def mx_gemm_fwd_y(xq: QTensorMX, wq: QTensorMX, out_dtype=torch.float32, out=None) -> torch.Tensor:
    """Y [M, N] = Q(X H') Q(W H')^T with power-of-two scales (ufp4_mx_gemm_fwd_y)."""
    M, K, N = xq.rows, xq.red, wq.rows
    return _gemm_mx_call("ufp4_mx_gemm_fwd_y", xq, wq, M, N, K, _out(M, N, out_dtype, xq.codes.device, out))


def mx_gemm_bwd_dx(dyq: QTensorMX, wtq: QTensorMX, out_dtype=torch.float32, out=None) -> torch.Tensor:
    """dX [M, K] = Q(dY H') Q(W^T H')^T (ufp4_mx_gemm_bwd_dx)."""
    M, N, K = dyq.rows, dyq.red, wtq.rows
    return _gemm_mx_call("ufp4_mx_gemm_bwd_dx", dyq, wtq, M, N, K, _out(M, K, out_dtype, dyq.codes.device, out))


def mx_gemm_bwd_dw(dytq: QTensorMX, xtq: QTensorMX, out_dtype=torch.float32, out=None) -> torch.Tensor:
    """dW [N, K] = Q(dY^T H') Q(X^T H')^T (ufp4_mx_gemm_bwd_dw)."""
    N, M, K = dytq.rows, dytq.red, xtq.rows
    return _gemm_mx_call("ufp4_mx_gemm_bwd_dw", dytq, xtq, M, N, K, _out(N, K, out_dtype, dytq.codes.device, out))


def group_offsets(counts, device="cuda"):
    """(token offsets, padded offsets, padded total) for per-group row counts; offsets as int64 device
    tensors of length G + 1."""
    off = [0]
    poff = [0]
    for c in counts:
        off.append(off[-1] + int(c))
        poff.append(poff[-1] + -(-int(c) // 16) * 16)
    return (torch.tensor(off, dtype=torch.int64, device=device), torch.tensor(poff, dtype=torch.int64, device=device),
            poff[-1])


def quantize_grouped_t(x: torch.Tensor, offsets: torch.Tensor, padded_offsets: torch.Tensor, red_total: int, *,
                       fmt: int = UNIFORM, rht: bool = True, sign_mask: int = 0, rounding: int = RTNE, seed: int = 0,
                       stream_id: int = 0, out: QTensor | None = None) -> QTensor:
    """Grouped transposed quantization (ufp4_quantize_grouped_t): Q [cols, red_total]."""
    if x.dtype != torch.bfloat16 or not x.is_cuda or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D row-major bf16 CUDA tensor")
    rows, cols = x.shape
    G = offsets.numel() - 1
    q = out if out is not None else empty_qtensor(cols, red_total, fmt, x.device)
    st = lib().ufp4_quantize_grouped_t(fmt, x.data_ptr(), rows, cols, x.stride(0), offsets.data_ptr(),
                                       padded_offsets.data_ptr(), G, red_total, int(rht), sign_mask, rounding,
                                       seed & 0xFFFFFFFFFFFFFFFF, stream_id, q.codes.data_ptr(), q.code_panel_ld,
                                       q.scales.data_ptr(), q.scale_panel_ld, _stream())
    _check(st, "ufp4_quantize_grouped_t")
    return q


def _out(rows, cols, out_dtype, device, out):
    if out is not None:
        return out
    return torch.empty((rows, cols), dtype=out_dtype, device=device)


def _odt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return OUT_F32
    if t.dtype == torch.bfloat16:
        return OUT_BF16
    raise ValueError("output must be float32 or bfloat16")


def _gemm(name, a: QTensor, b: QTensor, M, N, K, c: torch.Tensor):
    if a.fmt != b.fmt:
        raise ValueError("operands quantized to different grids")
    st = getattr(lib(), name)(a.codes.data_ptr(), a.code_panel_ld, a.scales.data_ptr(), a.scale_panel_ld, b.codes.data_ptr(),
                              b.code_panel_ld, b.scales.data_ptr(), b.scale_panel_ld, M, N, K, a.fmt, c.data_ptr(), c.stride(0),
                              _odt(c), _stream())
    _check(st, name)
    return c


def gemm_fwd_y(xq: QTensor, wq: QTensor, out_dtype=torch.float32, out=None) -> torch.Tensor:
    """Y [M, N] = Q(X H') Q(W H')^T (ufp4_gemm_fwd_y)."""
    M, K, N = xq.rows, xq.red, wq.rows
    return _gemm("ufp4_gemm_fwd_y", xq, wq, M, N, K, _out(M, N, out_dtype, xq.codes.device, out))


def gemm_bwd_dx(dyq: QTensor, wtq: QTensor, out_dtype=torch.float32, out=None) -> torch.Tensor:
    """dX [M, K] = Q(dY H') Q(W^T H')^T (ufp4_gemm_bwd_dx)."""
    M, N, K = dyq.rows, dyq.red, wtq.rows
    return _gemm("ufp4_gemm_bwd_dx", dyq, wtq, M, N, K, _out(M, K, out_dtype, dyq.codes.device, out))


def gemm_bwd_dw(dytq: QTensor, xtq: QTensor, out_dtype=torch.float32, out=None) -> torch.Tensor:
    """dW [N, K] = Q(dY^T H') Q(X^T H')^T (ufp4_gemm_bwd_dw)."""
    N, M, K = dytq.rows, dytq.red, xtq.rows
    return _gemm("ufp4_gemm_bwd_dw", dytq, xtq, M, N, K, _out(N, K, out_dtype, dytq.codes.device, out))


def gemm_fwd_y_grouped(xq: QTensor, wq: QTensor, offsets: torch.Tensor, n_per_group: int, out_dtype=torch.float32,
                       out=None) -> torch.Tensor:
    """Y_g = Qx[group g rows] Qw[g*N:(g+1)*N]^T, Y [M_total, N] (ufp4_gemm_fwd_y_grouped)."""
    G = offsets.numel() - 1
    M, K, N = xq.rows, xq.red, n_per_group
    c = _out(M, N, out_dtype, xq.codes.device, out)
    st = lib().ufp4_gemm_fwd_y_grouped(xq.codes.data_ptr(), xq.code_panel_ld, xq.scales.data_ptr(), xq.scale_panel_ld,
                                       wq.codes.data_ptr(), wq.code_panel_ld, wq.scales.data_ptr(), wq.scale_panel_ld,
                                       offsets.data_ptr(), G, M, N, K, xq.fmt, c.data_ptr(), c.stride(0), _odt(c),
                                       _stream())
    _check(st, "ufp4_gemm_fwd_y_grouped")
    return c


def gemm_bwd_dx_grouped(dyq: QTensor, wtq: QTensor, offsets: torch.Tensor, out_dtype=torch.float32,
                        out=None) -> torch.Tensor:
    """dX_g = Qdy[group g rows] Qwt[:, g*N:(g+1)*N]^T, dX [M_total, K] (ufp4_gemm_bwd_dx_grouped)."""
    G = offsets.numel() - 1
    M, N, K = dyq.rows, dyq.red, wtq.rows
    c = _out(M, K, out_dtype, dyq.codes.device, out)
    st = lib().ufp4_gemm_bwd_dx_grouped(dyq.codes.data_ptr(), dyq.code_panel_ld, dyq.scales.data_ptr(), dyq.scale_panel_ld,
                                        wtq.codes.data_ptr(), wtq.code_panel_ld, wtq.scales.data_ptr(), wtq.scale_panel_ld,
                                        offsets.data_ptr(), G, M, N, K, dyq.fmt, c.data_ptr(), c.stride(0), _odt(c),
                                        _stream())
    _check(st, "ufp4_gemm_bwd_dx_grouped")
    return c


def gemm_bwd_dw_grouped(dytq: QTensor, xtq: QTensor, padded_offsets: torch.Tensor, out_dtype=torch.float32,
                        out=None) -> torch.Tensor:
    """dW_g = Qdyt[:, pad_g:pad_{g+1}] Qxt[:, pad_g:pad_{g+1}]^T, dW [G, N, K] (ufp4_gemm_bwd_dw_grouped)."""
    G = padded_offsets.numel() - 1
    N, K = dytq.rows, xtq.rows
    c = out if out is not None else torch.empty((G, N, K), dtype=out_dtype, device=dytq.codes.device)
    st = lib().ufp4_gemm_bwd_dw_grouped(dytq.codes.data_ptr(), dytq.code_panel_ld, dytq.scales.data_ptr(), dytq.scale_panel_ld,
                                        xtq.codes.data_ptr(), xtq.code_panel_ld, xtq.scales.data_ptr(), xtq.scale_panel_ld,
                                        padded_offsets.data_ptr(), G, dytq.red, N, K, dytq.fmt, c.data_ptr(), c.stride(-2),
                                        _odt(c), _stream())
    _check(st, "ufp4_gemm_bwd_dw_grouped")
    return c
