"""Python binding of libufp4 (ctypes). Argument marshalling only: every step runs in the HIP library, and the
layout, padding and metric arithmetic is the library's too (ufp4_qtensor_bytes, ufp4_grouped_reduction,
ufp4_quant_metrics and friends).

Tensors are torch tensors on the GPU; torch supplies device memory and the current stream. The library
must be built (``python -m paper_2606_20381_amd.build``); without it every call raises.
"""

from __future__ import annotations

import ctypes
import os
import struct

import torch

UNIFORM = 0
E2M1 = 1
UNIFORM_MX32 = 2  # uniform grid with power-of-two 1x32 scales
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
_F = ctypes.c_float
_D = ctypes.c_double


class QDesc(ctypes.Structure):
    """ufp4_qtensor: storage set by the caller, contents written by the quantizer (include/ufp4.h)."""

    _fields_ = [("codes", _P), ("scales", _P), ("code_panel_ld", _I64), ("scale_panel_ld", _I64), ("panels", _I64),
                ("rows", _I64), ("red", _I64), ("format", _I32), ("rht_block", _I32),
                ("sign_words", ctypes.c_uint16 * 8), ("max_fpx", _F), ("rounding", _I32), ("layout", _I32),
                ("reserved", _I32)]


assert ctypes.sizeof(QDesc) == 96
# ufp4_qtensor.layout
LAYOUT_PLAIN, LAYOUT_GROUPED_ROWS, LAYOUT_GROUPED_RED = 0, 1, 2


class Metrics(ctypes.Structure):
    """ufp4_quant_metrics_t."""

    _fields_ = [("nmse", _D), ("sqnr_db", _D), ("alpha", _D), ("entropy", _D), ("beff", _D)]


_Q = ctypes.POINTER(QDesc)
_M = ctypes.POINTER(Metrics)
_QUANT_ARGS = [_P, _I64, _I64, _I64, _INT, _INT, _U32, _INT, _U64, _U32, _Q, _P]
_GEMM_ARGS = [_Q, _Q, _P, _I64, _INT, _P]
_GEMM_G_ARGS = [_Q, _Q, _P, _I32, _P, _I64, _INT, _P]
SIGNATURES = {
    "ufp4_status_string": ([_INT], ctypes.c_char_p),
    "ufp4_version": ([], ctypes.c_char_p),
    "ufp4_qtensor_bytes": ([_INT, _I64, _I64, _P, _P, _P, _P, _P], _INT),
    "ufp4_grouped_reduction": ([_P, _I32, _I32, _P, _P], _INT),
    "ufp4_rht_quantize": (_QUANT_ARGS, _INT),
    "ufp4_e2m1_quantize": (_QUANT_ARGS, _INT),
    "ufp4_e2m1_quantize_range": ([_P, _I64, _I64, _I64, _INT, _INT, _U32, _INT, _U64, _U32, _F, _Q, _P], _INT),
    "ufp4_quantize_rht_block": ([_INT, _P, _I64, _I64, _I64, _INT, _INT, _P, _INT, _U64, _U32, _Q, _P], _INT),
    "ufp4_quant_stats": ([_INT, _F, _P, _I64, _I64, _I64, _INT, _INT, _U32, _INT, _U64, _U32, _P, _P], _INT),
    "ufp4_quant_metrics": ([_P, _INT, _F, _M], _INT),
    "ufp4_rotation_gain": ([_M, _M, _P], _INT),
    "ufp4_gemm_attenuation": ([_M, _M, _P], _INT),
    "ufp4_rht": ([_P, _I64, _I64, _I64, _U32, _P, _I64, _P], _INT),
    "ufp4_quantize_f32": ([_INT, _P, _I64, _I64, _I64, _INT, _U32, _INT, _U64, _U32, _Q, _P], _INT),
    "ufp4_quantize_grouped_t": ([_INT, _P, _I64, _I64, _I64, _P, _I32, _I64, _INT, _U32, _INT, _U64, _U32, _Q, _P],
                                _INT),
    "ufp4_quantize_dual": ([_INT, _P, _I64, _I64, _I64, _INT, _U32, _U32, _INT, _U32, _U32, _INT, _U64, _Q, _Q, _P],
                           _INT),
    "ufp4_mx_quantize": (_QUANT_ARGS, _INT),
    "ufp4_mx_quantize_dual": ([_P, _I64, _I64, _I64, _INT, _U32, _U32, _INT, _U32, _U32, _INT, _U64, _Q, _Q, _P],
                              _INT),
    "ufp4_mx_gemm_fwd_y": (_GEMM_ARGS, _INT),
    "ufp4_mx_gemm_bwd_dx": (_GEMM_ARGS, _INT),
    "ufp4_mx_gemm_bwd_dw": (_GEMM_ARGS, _INT),
    "ufp4_mx_quantize_grouped": ([_P, _I64, _I64, _I64, _INT, _P, _I32, _I64, _INT, _U32, _INT, _U64, _U32, _Q, _P],
                                 _INT),
    "ufp4_mx_gemm_fwd_y_grouped": ([_Q, _Q, _P, _I32, _I64, _P, _I64, _INT, _P], _INT),
    "ufp4_mx_gemm_bwd_dx_grouped": ([_Q, _Q, _P, _I32, _I64, _P, _I64, _INT, _P], _INT),
    "ufp4_mx_gemm_bwd_dw_grouped": (_GEMM_G_ARGS, _INT),
    "ufp4_gemm_fwd_y": (_GEMM_ARGS, _INT),
    "ufp4_gemm_bwd_dx": (_GEMM_ARGS, _INT),
    "ufp4_gemm_bwd_dw": (_GEMM_ARGS, _INT),
    "ufp4_gemm_fwd_y_grouped": (_GEMM_G_ARGS, _INT),
    "ufp4_gemm_bwd_dx_grouped": (_GEMM_G_ARGS, _INT),
    "ufp4_gemm_bwd_dw_grouped": (_GEMM_G_ARGS, _INT),
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


def _bf16_2d(x: torch.Tensor) -> None:
    if x.dtype != torch.bfloat16 or not x.is_cuda or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D row-major bf16 CUDA tensor")


PANEL_ROWS = 128  # rows per panel of a quantized operand


class QTensor:
    """A quantized operand [rows, red] in the library's panel layout: the two device buffers and the ufp4_qtensor
    descriptor (`desc`) that points at them. The quantizers fill the descriptor's contents (rows, reduction length,
    grid, RHT block and signs); the GEMMs read it.

    Rows are grouped in panels of 128; within a panel, block b (16 reduction positions) of all 128 rows is
    contiguous: 128 x 8 bytes of codes at b * 1024 and 128 fp32 scales at b * 128 (power-of-two scales: 32-blocks
    of 3 x 1024 code bytes and 128 E8M0 bytes). ``codes_rows()`` / ``scales_rows()`` give plain row-major copies.
    """

    def __init__(self, codes: torch.Tensor, scales: torch.Tensor, desc: QDesc):
        self.codes, self.scales, self.desc = codes, scales, desc

    fmt = property(lambda self: self.desc.format)
    rows = property(lambda self: self.desc.rows)
    red = property(lambda self: self.desc.red)
    rht_block = property(lambda self: self.desc.rht_block)
    code_panel_ld = property(lambda self: self.desc.code_panel_ld)
    scale_panel_ld = property(lambda self: self.desc.scale_panel_ld)
    panels = property(lambda self: self.desc.panels)
    layout = property(lambda self: self.desc.layout)

    @property
    def sign_mask(self) -> int:
        """The RHT signs as one integer (bit j: eps_j = -1), 0 without RHT."""
        return sum(int(w) << (16 * k) for k, w in enumerate(self.desc.sign_words))

    def ref(self):
        return ctypes.byref(self.desc)

    def codes_rows(self) -> torch.Tensor:
        """Codes as uint8 [rows, red/2] (power-of-two scales: [rows, red * 3/4]), row-major (a copy)."""
        if self.fmt == UNIFORM_MX32:
            nkb = self.red // 32
            v = self.codes[:, : nkb * 3072].reshape(self.panels, nkb, 3, PANEL_ROWS, 8).permute(0, 3, 1, 2, 4)
            return v.reshape(self.panels * PANEL_ROWS, nkb * 24)[: self.rows]
        nkb = self.red // 16
        v = self.codes[:, : nkb * 1024].reshape(self.panels, nkb, PANEL_ROWS, 8).permute(0, 2, 1, 3)
        return v.reshape(self.panels * PANEL_ROWS, nkb * 8)[: self.rows]

    def scales_rows(self) -> torch.Tensor:
        """Scales as [rows, red/16] fp32 (power-of-two scales: [rows, red/32] E8M0 bytes), row-major (a copy)."""
        nkb = self.red // (32 if self.fmt == UNIFORM_MX32 else 16)
        v = self.scales[:, : nkb * PANEL_ROWS].reshape(self.panels, nkb, PANEL_ROWS).permute(0, 2, 1)
        return v.reshape(self.panels * PANEL_ROWS, nkb)[: self.rows]


def empty_qtensor(rows: int, red: int, fmt: int = UNIFORM, device="cuda") -> QTensor:
    """Buffers for a [rows, red] operand of `fmt`, sized by the library (ufp4_qtensor_bytes)."""
    p, cld, sld = _I64(), _I64(), _I64()
    _check(lib().ufp4_qtensor_bytes(fmt, rows, red, ctypes.byref(p), ctypes.byref(cld), ctypes.byref(sld), None, None),
           "ufp4_qtensor_bytes")
    codes = torch.empty((p.value, cld.value), dtype=torch.uint8, device=device)
    sdt = torch.uint8 if fmt == UNIFORM_MX32 else torch.float32
    scales = torch.empty((p.value, sld.value), dtype=sdt, device=device)
    desc = QDesc(codes=codes.data_ptr(), scales=scales.data_ptr(), code_panel_ld=cld.value, scale_panel_ld=sld.value,
                 panels=p.value, rows=rows, red=red, format=fmt)
    return QTensor(codes, scales, desc)


def empty_qtensor_mx(rows: int, red: int, device="cuda") -> QTensor:
    return empty_qtensor(rows, red, UNIFORM_MX32, device)


def _quantize_call(name, fmt, x, transpose, rht, sign_mask, rounding, seed, stream_id, out):
    _bf16_2d(x)
    rows, cols = x.shape
    qrows, red = (cols, rows) if transpose else (rows, cols)
    q = out if out is not None else empty_qtensor(qrows, red, fmt, x.device)
    st = getattr(lib(), name)(x.data_ptr(), rows, cols, x.stride(0), int(transpose), int(rht), sign_mask, rounding,
                              seed & 0xFFFFFFFFFFFFFFFF, stream_id, q.ref(), _stream())
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
    _bf16_2d(x)
    rows, cols = x.shape
    qrows, red = (cols, rows) if transpose else (rows, cols)
    q = out if out is not None else empty_qtensor(qrows, red, E2M1, x.device)
    st = lib().ufp4_e2m1_quantize_range(x.data_ptr(), rows, cols, x.stride(0), int(transpose), int(rht), sign_mask,
                                        rounding, seed & 0xFFFFFFFFFFFFFFFF, stream_id, float(max_fpx), q.ref(),
                                        _stream())
    _check(st, "ufp4_e2m1_quantize_range")
    return q


def quantize_rht_block(x: torch.Tensor, fmt: int = UNIFORM, *, rht_block: int = 16, sign_mask: int = 0,
                       transpose: bool = False, rounding: int = RTNE, seed: int = 0, stream_id: int = 0,
                       out: QTensor | None = None) -> QTensor:
    """RHT over n-blocks (n = rht_block, sign_mask an n-bit integer), then 1x16 quantization
    (ufp4_quantize_rht_block)."""
    _bf16_2d(x)
    rows, cols = x.shape
    qrows, red = (cols, rows) if transpose else (rows, cols)
    q = out if out is not None else empty_qtensor(qrows, red, fmt, x.device)
    words = (ctypes.c_uint16 * 8)(*[(sign_mask >> (16 * k)) & 0xFFFF for k in range(8)])
    st = lib().ufp4_quantize_rht_block(fmt, x.data_ptr(), rows, cols, x.stride(0), int(transpose), rht_block,
                                       ctypes.cast(words, ctypes.c_void_p), rounding, seed & 0xFFFFFFFFFFFFFFFF,
                                       stream_id, q.ref(), _stream())
    _check(st, "ufp4_quantize_rht_block")
    return q


def rht(x: torch.Tensor, *, sign_mask: int = 0, out: torch.Tensor | None = None) -> torch.Tensor:
    """Standalone block-16 RHT along the rows of x (ufp4_rht): fp32 [rows, cols]."""
    _bf16_2d(x)
    y = out if out is not None else torch.empty(x.shape, dtype=torch.float32, device=x.device)
    if y.dtype != torch.float32 or y.shape != x.shape or y.stride(1) != 1 or y.device != x.device:
        raise ValueError("out must be a row-major fp32 tensor of x's shape on x's device")
    st = lib().ufp4_rht(x.data_ptr(), x.shape[0], x.shape[1], x.stride(0), sign_mask, y.data_ptr(), y.stride(0),
                        _stream())
    _check(st, "ufp4_rht")
    return y


def quantize_f32(x: torch.Tensor, fmt: int = UNIFORM, *, rht: bool = False, sign_mask: int = 0, rounding: int = RTNE,
                 seed: int = 0, stream_id: int = 0, out: QTensor | None = None) -> QTensor:
    """Rowwise quantization of an fp32 tensor, no transform (ufp4_quantize_f32). rht / sign_mask record the
    block-16 RHT the input already carries (the output of ufp4_rht), for the GEMMs' operand check."""
    if x.dtype != torch.float32 or not x.is_cuda or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D row-major fp32 CUDA tensor")
    rows, cols = x.shape
    q = out if out is not None else empty_qtensor(rows, cols, fmt, x.device)
    st = lib().ufp4_quantize_f32(fmt, x.data_ptr(), rows, cols, x.stride(0), int(rht), sign_mask, rounding,
                                 seed & 0xFFFFFFFFFFFFFFFF, stream_id, q.ref(), _stream())
    _check(st, "ufp4_quantize_f32")
    return q


# ---------------------------------------------------------------------------------------------------
# quality diagnostics (Sec. 3.2)
# ---------------------------------------------------------------------------------------------------

STATS_BYTES = 88  # ufp4_quant_stats_t: 3 doubles + 8 uint64


class QuantStats:
    """Record of ufp4_quant_stats (fp64 sums and the magnitude-code histogram) and its Sec. 3.2 metrics, computed by
    the library (ufp4_quant_metrics)."""

    def __init__(self, raw: bytes, fmt: int, max_fpx: float):
        self.raw = raw
        vals = struct.unpack("<3d8Q", raw)
        self.err2, self.ref2, self.cross = vals[:3]
        self.hist = list(vals[3:])
        self.fmt, self.max_fpx = fmt, float(max_fpx)
        self.metrics = Metrics()
        buf = ctypes.create_string_buffer(raw, STATS_BYTES)
        _check(lib().ufp4_quant_metrics(buf, fmt, self.max_fpx, ctypes.byref(self.metrics)), "ufp4_quant_metrics")

    nmse = property(lambda self: self.metrics.nmse)
    sqnr_db = property(lambda self: self.metrics.sqnr_db)
    alpha = property(lambda self: self.metrics.alpha)
    entropy = property(lambda self: self.metrics.entropy)
    beff = property(lambda self: self.metrics.beff)


def quant_stats(x: torch.Tensor, fmt: int = UNIFORM, *, max_fpx: float = 0.0, transpose: bool = False,
                rht: bool = True, sign_mask: int = 0, rounding: int = RTNE, seed: int = 0, stream_id: int = 0,
                out: torch.Tensor | None = None) -> QuantStats:
    """Quality statistics of one quantization of x (ufp4_quant_stats); synchronizes to read the record."""
    _bf16_2d(x)
    rows, cols = x.shape
    rec = out if out is not None else torch.empty(STATS_BYTES // 8, dtype=torch.float64, device=x.device)
    if rec.numel() * rec.element_size() < STATS_BYTES or not rec.is_cuda or not rec.is_contiguous():
        raise ValueError("out must be a contiguous CUDA buffer of at least 88 bytes")
    st = lib().ufp4_quant_stats(fmt, float(max_fpx), x.data_ptr(), rows, cols, x.stride(0), int(transpose), int(rht),
                                sign_mask, rounding, seed & 0xFFFFFFFFFFFFFFFF, stream_id, rec.data_ptr(), _stream())
    _check(st, "ufp4_quant_stats")
    return QuantStats(rec.cpu().numpy().tobytes()[:STATS_BYTES], fmt, max_fpx)


def delta_sqnr_db(raw: QuantStats, rotated: QuantStats) -> float:
    """Delta SQNR of the rotation (ufp4_rotation_gain, Sec. 3.2): positive when it lowers the error."""
    out = _D()
    _check(lib().ufp4_rotation_gain(ctypes.byref(raw.metrics), ctypes.byref(rotated.metrics), ctypes.byref(out)),
           "ufp4_rotation_gain")
    return out.value


def gemm_attenuation(a: QuantStats, b: QuantStats) -> float:
    """eta = alpha_A alpha_B of a GEMM's two operands (ufp4_gemm_attenuation, Sec. 3.2)."""
    out = _D()
    _check(lib().ufp4_gemm_attenuation(ctypes.byref(a.metrics), ctypes.byref(b.metrics), ctypes.byref(out)),
           "ufp4_gemm_attenuation")
    return out.value


def quantize_dual(x: torch.Tensor, *, fmt: int = UNIFORM, rht_rows: bool = True, rht_cols: bool = True,
                  sign_mask_rows: int = 0, sign_mask_cols: int = 0, rounding: int = RTNE, seed: int = 0,
                  stream_rows: int = 0, stream_cols: int = 0, out_rows: QTensor | None = None,
                  out_cols: QTensor | None = None) -> tuple[QTensor, QTensor]:
    """Both operands of x [rows, cols] from one read (ufp4_quantize_dual): (Q_r [rows, cols] along cols,
    Q_c [cols, rows] along rows)."""
    _bf16_2d(x)
    rows, cols = x.shape
    qr = out_rows if out_rows is not None else empty_qtensor(rows, cols, fmt, x.device)
    qc = out_cols if out_cols is not None else empty_qtensor(cols, rows, fmt, x.device)
    st = lib().ufp4_quantize_dual(fmt, x.data_ptr(), rows, cols, x.stride(0), int(rht_rows), sign_mask_rows,
                                  stream_rows, int(rht_cols), sign_mask_cols, stream_cols, rounding,
                                  seed & 0xFFFFFFFFFFFFFFFF, qr.ref(), qc.ref(), _stream())
    _check(st, "ufp4_quantize_dual")
    return qr, qc


def mx_quantize(x: torch.Tensor, *, transpose: bool = False, rht: bool = True, sign_mask: int = 0,
                rounding: int = RTNE, seed: int = 0, stream_id: int = 0, out: QTensor | None = None) -> QTensor:
    """Fused RHT + uniform-grid quantization with power-of-two 1x32 scales (ufp4_mx_quantize)."""
    return _quantize_call("ufp4_mx_quantize", UNIFORM_MX32, x, transpose, rht, sign_mask, rounding, seed, stream_id,
                          out)


def mx_quantize_dual(x: torch.Tensor, *, rht_rows: bool = True, rht_cols: bool = True, sign_mask_rows: int = 0,
                     sign_mask_cols: int = 0, rounding: int = RTNE, seed: int = 0, stream_rows: int = 0,
                     stream_cols: int = 0, out_rows: QTensor | None = None,
                     out_cols: QTensor | None = None) -> tuple[QTensor, QTensor]:
    """Both power-of-two-scale operands of x [rows, cols] from one read (ufp4_mx_quantize_dual): (Q_r [rows, cols]
    along cols, Q_c [cols, rows] along rows)."""
    _bf16_2d(x)
    rows, cols = x.shape
    qr = out_rows if out_rows is not None else empty_qtensor_mx(rows, cols, x.device)
    qc = out_cols if out_cols is not None else empty_qtensor_mx(cols, rows, x.device)
    st = lib().ufp4_mx_quantize_dual(x.data_ptr(), rows, cols, x.stride(0), int(rht_rows), sign_mask_rows,
                                     stream_rows, int(rht_cols), sign_mask_cols, stream_cols, rounding,
                                     seed & 0xFFFFFFFFFFFFFFFF, qr.ref(), qc.ref(), _stream())
    _check(st, "ufp4_mx_quantize_dual")
    return qr, qc


# ---------------------------------------------------------------------------------------------------
# grouped (MoE) operands
# ---------------------------------------------------------------------------------------------------

def group_offsets(counts, device="cuda", block: int = 16):
    """(token offsets as an int64 tensor [G + 1] on `device`, the padded length of the grouped axis from
    ufp4_grouped_reduction: `block` 16 for the grouped transposed operands, 32 for their power-of-two-scale form,
    128 for the grouped rows of the power-of-two-scale ragged-M passes)."""
    off = [0]
    for c in counts:
        off.append(off[-1] + int(c))
    arr = (ctypes.c_int64 * len(off))(*off)
    red = _I64()
    _check(lib().ufp4_grouped_reduction(ctypes.cast(arr, ctypes.c_void_p), len(off) - 1, block, None,
                                        ctypes.byref(red)), "ufp4_grouped_reduction")
    return torch.tensor(off, dtype=torch.int64, device=device), red.value


def padded_offsets(offsets_host, block: int = 16) -> list:
    """The padded offsets of a grouped axis (ufp4_grouped_reduction), from host token offsets."""
    off = [int(v) for v in offsets_host]
    arr = (ctypes.c_int64 * len(off))(*off)
    pad = (ctypes.c_int64 * len(off))()
    _check(lib().ufp4_grouped_reduction(ctypes.cast(arr, ctypes.c_void_p), len(off) - 1, block,
                                        ctypes.cast(pad, ctypes.c_void_p), None), "ufp4_grouped_reduction")
    return list(pad)


def _offsets(offsets: torch.Tensor) -> int:
    if offsets.dtype != torch.int64 or not offsets.is_cuda or not offsets.is_contiguous() or offsets.dim() != 1:
        raise ValueError("offsets must be a contiguous int64 CUDA tensor [G + 1]")
    return offsets.numel() - 1


def quantize_grouped_t(x: torch.Tensor, offsets: torch.Tensor, red_total: int, *, fmt: int = UNIFORM,
                       rht: bool = True, sign_mask: int = 0, rounding: int = RTNE, seed: int = 0, stream_id: int = 0,
                       out: QTensor | None = None) -> QTensor:
    """Grouped transposed quantization (ufp4_quantize_grouped_t): Q [cols, red_total]."""
    _bf16_2d(x)
    rows, cols = x.shape
    G = _offsets(offsets)
    q = out if out is not None else empty_qtensor(cols, red_total, fmt, x.device)
    st = lib().ufp4_quantize_grouped_t(fmt, x.data_ptr(), rows, cols, x.stride(0), offsets.data_ptr(), G, red_total,
                                       int(rht), sign_mask, rounding, seed & 0xFFFFFFFFFFFFFFFF, stream_id, q.ref(),
                                       _stream())
    _check(st, "ufp4_quantize_grouped_t")
    return q


# ---------------------------------------------------------------------------------------------------
# GEMMs
# ---------------------------------------------------------------------------------------------------

def _out(shape, out_dtype, device, out):
    if out is None:
        return torch.empty(shape, dtype=out_dtype, device=device)
    if tuple(out.shape) != tuple(shape) or out.stride(-1) != 1 or out.device != torch.device(device):
        raise ValueError(f"out must be a row-major tensor of shape {tuple(shape)} on {device}")
    if out.dim() == 3 and out.shape[0] > 1 and out.stride(0) != out.shape[1] * out.stride(1):
        raise ValueError("out [G, N, K] must hold its groups N rows apart")
    _odt(out)
    return out


def _odt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return OUT_F32
    if t.dtype == torch.bfloat16:
        return OUT_BF16
    raise ValueError("output must be float32 or bfloat16")


def _gemm(name, a: QTensor, b: QTensor, c: torch.Tensor):
    st = getattr(lib(), name)(a.ref(), b.ref(), c.data_ptr(), c.stride(-2), _odt(c), _stream())
    _check(st, name)
    return c


def gemm_fwd_y(xq: QTensor, wq: QTensor, out_dtype=torch.float32, out=None) -> torch.Tensor:
    """Y [M, N] = Q(X H') Q(W H')^T (ufp4_gemm_fwd_y)."""
    return _gemm("ufp4_gemm_fwd_y", xq, wq, _out((xq.rows, wq.rows), out_dtype, xq.codes.device, out))


def gemm_bwd_dx(dyq: QTensor, wtq: QTensor, out_dtype=torch.float32, out=None) -> torch.Tensor:
    """dX [M, K] = Q(dY H') Q(W^T H')^T (ufp4_gemm_bwd_dx)."""
    return _gemm("ufp4_gemm_bwd_dx", dyq, wtq, _out((dyq.rows, wtq.rows), out_dtype, dyq.codes.device, out))


def gemm_bwd_dw(dytq: QTensor, xtq: QTensor, out_dtype=torch.float32, out=None) -> torch.Tensor:
    """dW [N, K] = Q(dY^T H') Q(X^T H')^T (ufp4_gemm_bwd_dw)."""
    return _gemm("ufp4_gemm_bwd_dw", dytq, xtq, _out((dytq.rows, xtq.rows), out_dtype, dytq.codes.device, out))


def mx_gemm_fwd_y(xq: QTensor, wq: QTensor, out_dtype=torch.float32, out=None) -> torch.Tensor:
    """Y [M, N] = Q(X H') Q(W H')^T with power-of-two scales (ufp4_mx_gemm_fwd_y)."""
    return _gemm("ufp4_mx_gemm_fwd_y", xq, wq, _out((xq.rows, wq.rows), out_dtype, xq.codes.device, out))


def mx_gemm_bwd_dx(dyq: QTensor, wtq: QTensor, out_dtype=torch.float32, out=None) -> torch.Tensor:
    """dX [M, K] = Q(dY H') Q(W^T H')^T (ufp4_mx_gemm_bwd_dx)."""
    return _gemm("ufp4_mx_gemm_bwd_dx", dyq, wtq, _out((dyq.rows, wtq.rows), out_dtype, dyq.codes.device, out))


def mx_gemm_bwd_dw(dytq: QTensor, xtq: QTensor, out_dtype=torch.float32, out=None) -> torch.Tensor:
    """dW [N, K] = Q(dY^T H') Q(X^T H')^T (ufp4_mx_gemm_bwd_dw)."""
    return _gemm("ufp4_mx_gemm_bwd_dw", dytq, xtq, _out((dytq.rows, xtq.rows), out_dtype, dytq.codes.device, out))


def _gemm_grouped(name, a: QTensor, b: QTensor, offsets: torch.Tensor, c: torch.Tensor):
    st = getattr(lib(), name)(a.ref(), b.ref(), offsets.data_ptr(), _offsets(offsets), c.data_ptr(), c.stride(-2),
                              _odt(c), _stream())
    _check(st, name)
    return c


def gemm_fwd_y_grouped(xq: QTensor, wq: QTensor, offsets: torch.Tensor, out_dtype=torch.float32,
                       out=None) -> torch.Tensor:
    """Y_g = Qx[group g rows] Qw[g*N:(g+1)*N]^T, Y [M_total, N] (ufp4_gemm_fwd_y_grouped); N = Qw rows / G."""
    n = wq.rows // _offsets(offsets)
    return _gemm_grouped("ufp4_gemm_fwd_y_grouped", xq, wq, offsets,
                         _out((xq.rows, n), out_dtype, xq.codes.device, out))


def gemm_bwd_dx_grouped(dyq: QTensor, wtq: QTensor, offsets: torch.Tensor, out_dtype=torch.float32,
                        out=None) -> torch.Tensor:
    """dX_g = Qdy[group g rows] Qwt[:, g*N:(g+1)*N]^T, dX [M_total, K] (ufp4_gemm_bwd_dx_grouped)."""
    return _gemm_grouped("ufp4_gemm_bwd_dx_grouped", dyq, wtq, offsets,
                         _out((dyq.rows, wtq.rows), out_dtype, dyq.codes.device, out))


def gemm_bwd_dw_grouped(dytq: QTensor, xtq: QTensor, offsets: torch.Tensor, out_dtype=torch.float32,
                        out=None) -> torch.Tensor:
    """dW_g = Qdyt[:, pad_g:pad_{g+1}] Qxt[:, pad_g:pad_{g+1}]^T, dW [G, N, K] (ufp4_gemm_bwd_dw_grouped); the
    token offsets are those the grouped operands were quantized with."""
    G = _offsets(offsets)
    return _gemm_grouped("ufp4_gemm_bwd_dw_grouped", dytq, xtq, offsets,
                         _out((G, dytq.rows, xtq.rows), out_dtype, dytq.codes.device, out))


# ---------------------------------------------------------------------------------------------------
# grouped (MoE) operands and GEMMs with power-of-two 1x32 scales
# ---------------------------------------------------------------------------------------------------

def mx_quantize_grouped(x: torch.Tensor, offsets: torch.Tensor, padded_total: int, *, transpose: bool, rht: bool = True,
                        sign_mask: int = 0, rounding: int = RTNE, seed: int = 0, stream_id: int = 0,
                        out: QTensor | None = None) -> QTensor:
    """ufp4_mx_quantize_grouped: transpose False gives the grouped-rows operand [padded_total, cols] (each group of
    X's rows from a panel boundary; padded_total from group_offsets(..., block=128)), True the grouped-reduction
    operand [cols, padded_total] (each group's tokens padded to 32; block=32)."""
    _bf16_2d(x)
    rows, cols = x.shape
    G = _offsets(offsets)
    qrows, red = (cols, padded_total) if transpose else (padded_total, cols)
    q = out if out is not None else empty_qtensor(qrows, red, UNIFORM_MX32, x.device)
    st = lib().ufp4_mx_quantize_grouped(x.data_ptr(), rows, cols, x.stride(0), int(transpose), offsets.data_ptr(), G,
                                        padded_total, int(rht), sign_mask, rounding, seed & 0xFFFFFFFFFFFFFFFF,
                                        stream_id, q.ref(), _stream())
    _check(st, "ufp4_mx_quantize_grouped")
    return q


def _mx_gemm_ragged_m(name, a: QTensor, b: QTensor, offsets: torch.Tensor, m_total: int, c: torch.Tensor):
    st = getattr(lib(), name)(a.ref(), b.ref(), offsets.data_ptr(), _offsets(offsets), m_total, c.data_ptr(),
                              c.stride(-2), _odt(c), _stream())
    _check(st, name)
    return c


def mx_gemm_fwd_y_grouped(xq: QTensor, wq: QTensor, offsets: torch.Tensor, m_total: int, out_dtype=torch.float32,
                          out=None) -> torch.Tensor:
    """Y [m_total, N] per group from the grouped-rows X and W [G*N, K] (ufp4_mx_gemm_fwd_y_grouped)."""
    n = wq.rows // _offsets(offsets)
    return _mx_gemm_ragged_m("ufp4_mx_gemm_fwd_y_grouped", xq, wq, offsets, m_total,
                             _out((m_total, n), out_dtype, xq.codes.device, out))


def mx_gemm_bwd_dx_grouped(dyq: QTensor, wtq: QTensor, offsets: torch.Tensor, m_total: int, out_dtype=torch.float32,
                           out=None) -> torch.Tensor:
    """dX [m_total, K] per group from the grouped-rows dY and W^T [K, G*N] (ufp4_mx_gemm_bwd_dx_grouped)."""
    return _mx_gemm_ragged_m("ufp4_mx_gemm_bwd_dx_grouped", dyq, wtq, offsets, m_total,
                             _out((m_total, wtq.rows), out_dtype, dyq.codes.device, out))


def mx_gemm_bwd_dw_grouped(dytq: QTensor, xtq: QTensor, offsets: torch.Tensor, out_dtype=torch.float32,
                           out=None) -> torch.Tensor:
    """dW [G, N, K] from the grouped-reduction dY^T and X^T (ufp4_mx_gemm_bwd_dw_grouped)."""
    G = _offsets(offsets)
    return _gemm_grouped("ufp4_mx_gemm_bwd_dw_grouped", dytq, xtq, offsets,
                         _out((G, dytq.rows, xtq.rows), out_dtype, dytq.codes.device, out))
