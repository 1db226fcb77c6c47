"""CPU checks of the C ABI library: it loads, exports every function include/ufp4.h declares, computes its host-side
arithmetic (layout sizes, grouped padding, Sec. 3.2 metrics), and rejects bad arguments -- including GEMM operands
quantized differently -- on the host before any GPU call. Every call below either is host-only or fails validation,
so nothing is launched."""

import ctypes
import math
import os
import re
import struct

import pytest

from paper_2606_20381_amd import ufp4 as U

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ufp4.h")

OK, INVALID, SHAPE, ALIGN, MISMATCH, UNSUPPORTED = 0, 1, 2, 3, 4, 5


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ufp4_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(U.library_path()):
        pytest.skip("libufp4.so not built")
    return U.lib()


def test_header_declares_the_boundary():
    names = _declared()
    for required in ("ufp4_rht_quantize", "ufp4_e2m1_quantize", "ufp4_gemm_fwd_y", "ufp4_gemm_bwd_dx",
                     "ufp4_gemm_bwd_dw", "ufp4_qtensor_bytes", "ufp4_grouped_reduction", "ufp4_quant_metrics"):
        assert required in names
    assert "UFP4_ERR_MISMATCH = 4" in open(HEADER).read()


def test_every_declared_symbol_is_exported(lib):
    raw = ctypes.CDLL(U.library_path())
    for name in _declared():
        assert hasattr(raw, name), name
        assert name in U.SIGNATURES, f"binding lacks a signature for {name}"


def test_status_strings(lib):
    assert lib.ufp4_status_string(0) == b"ok"
    assert lib.ufp4_status_string(3).startswith(b"misaligned")
    assert lib.ufp4_status_string(4).startswith(b"operands quantized differently")
    assert lib.ufp4_version() == b"0.3.0"


FAKE = 1 << 20  # a 1 MiB-aligned non-null address that is never dereferenced: every call below fails validation


def _desc(rows=16, red=32, fmt=U.UNIFORM, rht_block=16, mask=0, codes=FAKE, scales=FAKE, cld=None, sld=None,
          panels=1, layout=0):
    """A descriptor as a quantizer would leave it (storage at FAKE, minimal strides unless given)."""
    mx = fmt == U.UNIFORM_MX32
    nkb = red // (32 if mx else 16)
    d = U.QDesc(codes=codes, scales=scales, code_panel_ld=cld if cld is not None else max(16, nkb * (3072 if mx else 1024)),
                scale_panel_ld=sld if sld is not None else max(16 if mx else 4, nkb * 128), panels=panels, rows=rows,
                red=red, format=fmt, rht_block=rht_block, layout=layout)
    for k in range(8):
        d.sign_words[k] = (mask >> (16 * k)) & 0xFFFF if k < rht_block // 16 else 0
    return d


R = ctypes.byref


# ------------------------------------------------------------------------------------------------
# host-side arithmetic
# ------------------------------------------------------------------------------------------------

def test_qtensor_bytes(lib):
    p, c, s = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    cb, sb = ctypes.c_size_t(), ctypes.c_size_t()
    assert lib.ufp4_qtensor_bytes(0, 200, 48, R(p), R(c), R(s), R(cb), R(sb)) == OK
    # 200 rows -> 2 panels; 3 blocks of 16: 3 x 128 x 8 code bytes and 3 x 128 fp32 scales per panel
    assert (p.value, c.value, s.value, cb.value, sb.value) == (2, 3072, 384, 6144, 3072)
    assert lib.ufp4_qtensor_bytes(2, 129, 64, R(p), R(c), R(s), R(cb), R(sb)) == OK  # power-of-two scales
    assert (p.value, c.value, s.value, cb.value, sb.value) == (2, 2 * 3072, 256, 12288, 512)
    assert lib.ufp4_qtensor_bytes(0, 0, 0, R(p), R(c), R(s), None, None) == OK  # empty: one minimal panel
    assert (p.value, c.value, s.value) == (1, 16, 4)
    assert lib.ufp4_qtensor_bytes(0, 16, 24, None, None, None, None, None) == SHAPE
    assert lib.ufp4_qtensor_bytes(2, 16, 48, None, None, None, None, None) == SHAPE
    assert lib.ufp4_qtensor_bytes(3, 16, 32, None, None, None, None, None) == INVALID
    assert lib.ufp4_qtensor_bytes(0, -1, 32, None, None, None, None, None) == INVALID


def _grouped(lib, offsets, block=16):
    arr = (ctypes.c_int64 * len(offsets))(*offsets)
    pad = (ctypes.c_int64 * len(offsets))()
    red = ctypes.c_int64()
    st = lib.ufp4_grouped_reduction(ctypes.cast(arr, ctypes.c_void_p), len(offsets) - 1, block,
                                    ctypes.cast(pad, ctypes.c_void_p), R(red))
    return st, list(pad), red.value


def test_grouped_reduction(lib):
    # counts 0, 1, 16, 17, 33: each rounded up to a multiple of 16 (Sec. 2.2 needs whole RHT blocks per group)
    st, pad, red = _grouped(lib, [0, 0, 1, 17, 34, 67])
    assert st == OK and pad == [0, 0, 16, 32, 64, 112] and red == 112
    # power-of-two scales: whole 32-blocks along the reduction, whole 128-row panels for grouped rows
    assert _grouped(lib, [0, 0, 1, 17, 34, 67], 32)[1:] == ([0, 0, 32, 64, 96, 160], 160)
    assert _grouped(lib, [0, 0, 1, 129, 300], 128)[1:] == ([0, 0, 128, 256, 512], 512)
    assert _grouped(lib, [0, 5, 3])[0] == INVALID      # decreasing offsets
    assert _grouped(lib, [2, 5])[0] == INVALID         # first offset not 0
    assert _grouped(lib, [0, 5], 24)[0] == INVALID     # padding block
    assert lib.ufp4_grouped_reduction(None, 1, 16, None, None) == INVALID


def _metrics(lib, err2, ref2, cross, hist, fmt=0, max_fpx=0.0):
    rec = ctypes.create_string_buffer(struct.pack("<3d8Q", err2, ref2, cross, *hist), 88)
    m = U.Metrics()
    assert lib.ufp4_quant_metrics(rec, fmt, max_fpx, R(m)) == OK
    return m


def test_quant_metrics_closed_forms(lib):
    m = _metrics(lib, 1.0, 100.0, 99.0, [10, 10, 10, 10, 10, 10, 10, 10])
    assert m.nmse == 0.01 and m.sqnr_db == pytest.approx(20.0) and m.alpha == 0.99
    assert m.beff == pytest.approx(1.0, abs=1e-9)  # all 8 buckets equally used
    m = _metrics(lib, 0.0, 4.0, 4.0, [5, 0, 0, 0, 0, 0, 0, 3])
    assert m.sqnr_db == math.inf and m.alpha == 1.0
    p = [5 / 8, 3 / 8]
    assert m.entropy == pytest.approx(-sum(q * math.log(q + 1e-12) for q in p))
    assert m.beff == pytest.approx(math.exp(m.entropy) / 8)
    # E2M1 cut at 2 has K = 5 levels (0, .5, 1, 1.5, 2): the sixth bucket and up are not counted
    m = _metrics(lib, 1.0, 2.0, 1.0, [1, 1, 1, 1, 1, 7, 7, 7], fmt=1, max_fpx=2.0)
    assert m.beff == pytest.approx(1.0, abs=1e-9)
    m = _metrics(lib, 0.0, 0.0, 0.0, [0] * 8)  # an all-zero operand
    assert math.isnan(m.nmse) and math.isnan(m.alpha)
    raw, rot = _metrics(lib, 2.0, 100.0, 99.0, [1] * 8), _metrics(lib, 1.0, 100.0, 98.0, [1] * 8)
    out = ctypes.c_double()
    assert lib.ufp4_rotation_gain(R(raw), R(rot), R(out)) == OK
    assert out.value == pytest.approx(10 * math.log10(2.0))
    assert lib.ufp4_gemm_attenuation(R(raw), R(rot), R(out)) == OK
    assert out.value == pytest.approx(0.99 * 0.98)
    rec = ctypes.create_string_buffer(88)
    assert lib.ufp4_quant_metrics(rec, 0, 4.0, R(U.Metrics())) == INVALID  # max_fpx on the uniform grid
    assert lib.ufp4_quant_metrics(None, 0, 0.0, R(U.Metrics())) == INVALID


# ------------------------------------------------------------------------------------------------
# quantizer validation
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("args,dkw,status", [
    # (x, rows, cols, ld, transpose, rht, mask, rounding, seed, stream_id), descriptor storage
    ((None, 16, 16, 16, 0, 1, 0, 0, 0, 0), {}, INVALID),            # null input
    ((FAKE, 16, 24, 24, 0, 1, 0, 0, 0, 0), {}, SHAPE),              # cols % 16
    ((FAKE, 24, 16, 16, 1, 1, 0, 0, 0, 0), {}, SHAPE),              # transposed: rows % 16
    ((FAKE, 16, 32, 30, 0, 1, 0, 0, 0, 0), {}, SHAPE),              # ld < cols
    ((FAKE, 16, 32, 36, 0, 1, 0, 0, 0, 0), {}, SHAPE),              # ld % 8
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0), dict(cld=1024), SHAPE),  # code panel stride < 1024 nkb
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0), dict(sld=128), SHAPE),   # scale panel stride < 128 nkb
    ((FAKE, 200, 32, 32, 0, 1, 0, 0, 0, 0), dict(panels=1), SHAPE),  # 200 rows need 2 panels
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0), dict(cld=2048 + 8), ALIGN),  # code panel stride % 16
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0), dict(sld=256 + 2), ALIGN),   # scale panel stride % 4
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0), dict(codes=FAKE + 8), ALIGN),  # codes alignment
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0), dict(scales=FAKE + 4), ALIGN),  # scales alignment
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0), dict(codes=None), INVALID),  # no code buffer
    ((FAKE + 2, 16, 32, 32, 0, 1, 0, 0, 0, 0), {}, ALIGN),          # input alignment
    ((FAKE, 16, 32, 32, 0, 1, 0, 2, 0, 0), {}, INVALID),            # rounding enum
    ((FAKE, 16, 32, 32, 2, 1, 0, 0, 0, 0), {}, INVALID),            # transpose flag
    ((FAKE, 16, 32, 32, 0, 1, 0x10000, 0, 0, 0), {}, INVALID),      # sign mask > 16 bits
    ((FAKE, -1, 32, 32, 0, 1, 0, 0, 0, 0), {}, INVALID),            # negative size
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0), dict(cld=1 << 30), UNSUPPORTED),  # code panel stride > 2^29
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0), dict(sld=1 << 28), UNSUPPORTED),  # scale panel stride > 2^27
])
def test_quantize_validation(lib, args, dkw, status):
    for fn in (lib.ufp4_rht_quantize, lib.ufp4_e2m1_quantize):
        d = _desc(rows=0, red=0, **dkw)
        d.code_panel_ld = dkw.get("cld", 2048)
        d.scale_panel_ld = dkw.get("sld", 256)
        assert fn(*args, R(d), None) == status
    assert lib.ufp4_rht_quantize(FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, None, None) == INVALID  # no descriptor


def test_empty_tensors_need_no_storage(lib):
    """A tensor with no element is never accessed: a NULL pointer and any leading dimension are accepted (as
    torch hands them over for empty tensors), the call returns OK without launching, and the descriptor
    records the empty operand. Non-empty tensors still need both."""
    for fn in (lib.ufp4_rht_quantize, lib.ufp4_e2m1_quantize, lib.ufp4_mx_quantize):
        mx = dict(fmt=U.UNIFORM_MX32) if fn is lib.ufp4_mx_quantize else {}
        for rows, cols, ld, transpose in [(0, 64, 64, 0), (70, 0, 1, 0), (0, 0, 1, 1), (0, 64, 64, 1)]:
            d = _desc(rows=7, red=128, **mx)  # storage for any of the shapes
            assert fn(None, rows, cols, ld, transpose, 1, 0, 0, 0, 0, R(d), None) == OK
            assert (d.rows, d.red) == ((cols, rows) if transpose else (rows, cols))
        assert fn(None, 16, 32 if mx else 16, 32, 0, 1, 0, 0, 0, 0, R(_desc(**mx)), None) == INVALID
        assert fn(FAKE, 16, 32, 36, 0, 1, 0, 0, 0, 0, R(_desc(**mx)), None) == SHAPE  # ld % 8 still checked
    assert _dual(lib, rows=0, x=None, ld=1) == OK
    assert lib.ufp4_rht(None, 0, 32, 32, 0, None, 1, None) == OK
    assert lib.ufp4_quantize_f32(0, None, 0, 32, 1, 1, 0, 0, 0, 0, R(_desc()), None) == OK
    # a GEMM whose output has no element: NULL output, OK, no launch
    assert lib.ufp4_gemm_fwd_y(R(_desc(rows=0)), R(_desc(rows=40)), None, 40, 0, None) == OK
    assert lib.ufp4_gemm_fwd_y(R(_desc(rows=16)), R(_desc(rows=0)), None, 0, 1, None) == OK
    mx = dict(fmt=U.UNIFORM_MX32)
    assert lib.ufp4_mx_gemm_fwd_y(R(_desc(rows=0, **mx)), R(_desc(rows=40, **mx)), None, 40, 0, None) == OK
    assert lib.ufp4_gemm_fwd_y(R(_desc(rows=16)), R(_desc(rows=40)), None, 40, 0, None) == INVALID  # not empty


def _dual(lib, rows=32, cols=48, ld=48, fmt=0, rht_r=1, mask_r=0, rht_c=1, mask_c=0, rnd=0, x=FAKE, dr=None, dc=None):
    dr = dr or _desc(cld=3 * 1024, sld=3 * 128)
    dc = dc or _desc(cld=2 * 1024, sld=2 * 128)
    return lib.ufp4_quantize_dual(fmt, x, rows, cols, ld, rht_r, mask_r, 0, rht_c, mask_c, 1, rnd, 0, R(dr), R(dc),
                                  None)


@pytest.mark.parametrize("kw,status", [
    (dict(x=None), INVALID),                                # null input
    (dict(dc=_desc(codes=None)), INVALID),                  # null transposed codes
    (dict(fmt=2), INVALID),                                 # format enum
    (dict(rnd=2), INVALID),                                 # rounding enum
    (dict(rht_c=3), INVALID),                               # rht flag
    (dict(mask_r=0x10000), INVALID),                        # sign mask > 16 bits
    (dict(rows=-16), INVALID),                              # negative size
    (dict(rows=24), SHAPE),                                 # rows % 16 (the transposed output's reduction)
    (dict(cols=40, ld=40), SHAPE),                          # cols % 16 (the rowwise output's reduction)
    (dict(ld=40), SHAPE),                                   # ld < cols
    (dict(ld=52), SHAPE),                                   # ld % 8
    (dict(dr=_desc(cld=2 * 1024, sld=3 * 128)), SHAPE),     # rowwise code panel stride < 1024 cols/16
    (dict(dc=_desc(cld=2 * 1024, sld=128)), SHAPE),         # transposed scale panel stride < 128 rows/16
    (dict(dc=_desc(cld=2 * 1024 + 8, sld=256)), ALIGN),     # panel stride % 16
    (dict(x=FAKE + 2), ALIGN),                              # input alignment
    (dict(dr=_desc(scales=FAKE + 4, cld=3 * 1024, sld=3 * 128)), ALIGN),  # scales alignment
    (dict(dc=_desc(cld=1 << 30, sld=256)), UNSUPPORTED),    # panel stride > 2^29
])
def test_dual_validation(lib, kw, status):
    assert _dual(lib, **kw) == status


def test_grouped_quantizer_validation(lib):
    d = _desc(cld=2 * 1024, sld=2 * 128)
    q = lib.ufp4_quantize_grouped_t
    # (format, x, rows, cols, ld, offsets, G, red_total, rht, mask, rounding, seed, stream, out)
    assert q(0, FAKE, 32, 16, 16, None, 2, 32, 1, 0, 0, 0, 0, R(d), None) == INVALID      # null offsets
    assert q(0, FAKE, 32, 16, 16, FAKE, 5000, 32, 1, 0, 0, 0, 0, R(d), None) == UNSUPPORTED  # too many groups
    assert q(0, FAKE, 64, 16, 16, FAKE, 2, 32, 1, 0, 0, 0, 0, R(d), None) == SHAPE         # red_total < rows
    assert q(0, FAKE, 32, 16, 16, FAKE, 2, 48, 1, 0, 0, 0, 0, R(d), None) == SHAPE         # 3 blocks, room for 2


def test_mx_quantizer_validation(lib):
    C32, S32 = 3072, 128  # panel strides for one 32-block
    q = lib.ufp4_mx_quantize

    def d(cld=2 * C32, sld=2 * S32, **kw):
        return R(_desc(fmt=U.UNIFORM_MX32, cld=cld, sld=sld, **kw))

    assert q(FAKE, 16, 48, 48, 0, 1, 0, 0, 0, 0, d(), None) == SHAPE             # cols % 32
    assert q(FAKE, 48, 16, 16, 1, 1, 0, 0, 0, 0, d(), None) == SHAPE             # transposed: rows % 32
    assert q(FAKE, 16, 64, 64, 0, 1, 0, 0, 0, 0, d(cld=C32), None) == SHAPE      # code stride < 3072 nkb
    assert q(FAKE, 16, 64, 64, 0, 1, 0, 0, 0, 0, d(sld=S32), None) == SHAPE      # scale stride < 128 nkb
    assert q(FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, d(sld=S32 + 4), None) == ALIGN  # scale stride % 16
    assert q(FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, d(scales=FAKE + 8), None) == ALIGN  # scales alignment
    assert q(None, 16, 32, 32, 0, 1, 0, 0, 0, 0, d(), None) == INVALID           # null input
    assert q(FAKE, 16, 32, 32, 0, 1, 0, 2, 0, 0, d(), None) == INVALID           # rounding enum
    assert q(FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, d(cld=1 << 30), None) == UNSUPPORTED  # stride > 2^29


def test_mx_dual_validation(lib):
    C32, S32 = 3072, 128
    q = lib.ufp4_mx_quantize_dual

    def d(rows=64, red=64, **kw):
        return _desc(rows=rows, red=red, fmt=U.UNIFORM_MX32, **kw)

    dr, dc = d(), d()

    def call(x=FAKE, rows=64, cols=64, ld=64, rht_r=1, rht_c=1, mr=0, mc=0, rnd=0, out_r=None, out_c=None):
        return q(x, rows, cols, ld, rht_r, mr, 0, rht_c, mc, 1, rnd, 0, R(out_r or dr), R(out_c or dc), None)

    assert call(rows=48, out_c=d(red=48, cld=2 * C32, sld=2 * S32)) == SHAPE  # rows % 32 (Q_c's reduction)
    assert call(cols=48, ld=48) == SHAPE                                     # cols % 32 (Q_r's reduction)
    assert call(ld=56) == SHAPE                                              # ld < cols
    assert call(cols=32, ld=36) == SHAPE                                     # ld % 8
    assert call(x=FAKE + 2) == ALIGN
    assert call(x=None) == INVALID
    assert call(rnd=2) == INVALID
    assert call(rht_c=2) == INVALID
    assert call(mr=0x10000) == INVALID
    assert call(rows=-32) == INVALID
    assert call(out_r=d(cld=C32)) == SHAPE                                   # code stride < 3072 nkb
    assert call(out_c=d(cld=2 * C32 + 8)) == ALIGN                           # code stride % 16
    assert q(FAKE, 64, 64, 64, 1, 0, 0, 1, 0, 1, 0, 0, R(dr), R(dr), None) == INVALID  # one descriptor for both


def test_quant_stats_validation(lib):
    """ufp4_quant_stats(format, max_fpx, x, rows, cols, ld, transpose, rht, mask, rounding, seed, stream, rec)"""
    ok = (0, 0.0, FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE)
    cases = [
        ((0, 4.0) + ok[2:], INVALID),            # max_fpx on the uniform grid
        ((1, 3.0) + ok[2:], INVALID),            # max_fpx not in {2, 4, 6}
        ((2,) + ok[1:], INVALID),                # format enum
        (ok[:2] + (None,) + ok[3:], INVALID),    # null input
        (ok[:12] + (None,), INVALID),            # null record
        (ok[:12] + (FAKE + 4,), ALIGN),          # record alignment
        (ok[:4] + (24, 24) + ok[6:], SHAPE),     # cols % 16
        (ok[:5] + (30,) + ok[6:], SHAPE),        # ld < cols
        (ok[:6] + (2,) + ok[7:], INVALID),       # transpose flag
        (ok[:9] + (2,) + ok[10:], INVALID),      # rounding enum
    ]
    for args, status in cases:
        assert lib.ufp4_quant_stats(*args, None) == status, args


def test_e2m1_range_validation(lib):
    args = (FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0)
    for mf in (0.0, 1.0, 3.0, 7.0):
        assert lib.ufp4_e2m1_quantize_range(*args, mf, R(_desc(fmt=1)), None) == INVALID
    assert lib.ufp4_e2m1_quantize_range(FAKE, 16, 24, 24, 0, 1, 0, 0, 0, 0, 4.0, R(_desc(fmt=1)), None) == SHAPE


def test_unfused_validation(lib):
    # ufp4_rht(x, rows, cols, ld, mask, y, ldy, stream)
    assert lib.ufp4_rht(None, 16, 32, 32, 0, FAKE, 32, None) == INVALID
    assert lib.ufp4_rht(FAKE, 16, 32, 32, 0x10000, FAKE, 32, None) == INVALID
    assert lib.ufp4_rht(FAKE, 16, 24, 24, 0, FAKE, 24, None) == SHAPE      # cols % 16
    assert lib.ufp4_rht(FAKE, 16, 32, 36, 0, FAKE, 32, None) == SHAPE      # ld % 8
    assert lib.ufp4_rht(FAKE, 16, 32, 32, 0, FAKE, 30, None) == SHAPE      # ldy < cols
    assert lib.ufp4_rht(FAKE, 16, 32, 32, 0, FAKE, 34, None) == SHAPE      # ldy % 4
    assert lib.ufp4_rht(FAKE, 16, 32, 32, 0, FAKE + 4, 32, None) == ALIGN  # y alignment
    # ufp4_quantize_f32(format, x, rows, cols, ld, rht, mask, rounding, seed, stream, out, stream)
    f = lib.ufp4_quantize_f32
    assert f(2, FAKE, 16, 32, 32, 0, 0, 0, 0, 0, R(_desc()), None) == INVALID     # format
    assert f(0, FAKE, 16, 32, 32, 0, 0, 2, 0, 0, R(_desc()), None) == INVALID     # rounding
    assert f(0, FAKE, 16, 32, 32, 2, 0, 0, 0, 0, R(_desc()), None) == INVALID     # rht flag
    assert f(0, FAKE, 16, 24, 24, 0, 0, 0, 0, 0, R(_desc()), None) == SHAPE       # cols % 16
    assert f(0, FAKE, 16, 32, 34, 0, 0, 0, 0, 0, R(_desc()), None) == SHAPE       # ld % 4
    assert f(0, FAKE + 8, 16, 32, 32, 0, 0, 0, 0, 0, R(_desc()), None) == ALIGN   # input alignment
    assert f(0, FAKE, 16, 32, 32, 0, 0, 0, 0, 0, R(_desc(cld=1024)), None) == SHAPE  # code panel stride


def test_rht_block_validation(lib):
    words = (ctypes.c_uint16 * 8)()
    w = ctypes.cast(words, ctypes.c_void_p)
    base = (0, FAKE, 16, 128, 128, 0)
    d = R(_desc(red=128))
    assert lib.ufp4_quantize_rht_block(*base, 48, w, 0, 0, 0, d, None) == INVALID          # block size
    assert lib.ufp4_quantize_rht_block(*base, 32, None, 0, 0, 0, d, None) == INVALID       # no sign words
    assert lib.ufp4_quantize_rht_block(2, *base[1:], 32, w, 0, 0, 0, d, None) == INVALID   # format
    assert lib.ufp4_quantize_rht_block(0, FAKE, 16, 96, 96, 0, 64, w, 0, 0, 0, R(_desc(red=96)), None) == SHAPE  # 96 % 64


# ------------------------------------------------------------------------------------------------
# GEMM validation: operands and output
# ------------------------------------------------------------------------------------------------

GEMMS = ("ufp4_gemm_fwd_y", "ufp4_gemm_bwd_dx", "ufp4_gemm_bwd_dw")


@pytest.mark.parametrize("name", GEMMS)
@pytest.mark.parametrize("a,b,status", [
    (dict(), dict(fmt=U.E2M1), MISMATCH),                      # grids differ
    (dict(rht_block=16), dict(rht_block=0), MISMATCH),         # one operand rotated, the other not
    (dict(mask=0x1234), dict(mask=0x1235), MISMATCH),          # different signs: different H'
    (dict(rht_block=32, mask=0x1), dict(rht_block=32, mask=0x10001), MISMATCH),  # second word of the signs
    (dict(rht_block=16, mask=0x1), dict(rht_block=32, mask=0x1), MISMATCH),      # different RHT blocks
    (dict(red=32), dict(red=48, cld=3072, sld=384), MISMATCH),  # reduction lengths differ
    (dict(fmt=U.UNIFORM_MX32), dict(fmt=U.UNIFORM_MX32), MISMATCH),  # power-of-two scales: the mx calls
    (dict(fmt=7), dict(fmt=7), INVALID),                       # unknown format
    (dict(rht_block=24), dict(rht_block=24), INVALID),         # unknown RHT block
    (dict(codes=None), dict(), INVALID),                       # no codes
    (dict(rows=200), dict(), SHAPE),                           # 200 rows in one panel
    (dict(cld=1024), dict(), SHAPE),                           # code stride < 1024 nkb
    (dict(), dict(scales=FAKE + 4), ALIGN),                    # scales alignment
    (dict(), dict(cld=1 << 30), UNSUPPORTED),                  # panel stride > 2^29
])
def test_gemm_operand_checks(lib, name, a, b, status):
    assert getattr(lib, name)(R(_desc(**a)), R(_desc(**b)), FAKE, 16, 0, None) == status


@pytest.mark.parametrize("name", GEMMS)
def test_gemm_signs_ignored_without_rht(lib, name):
    """With no RHT the sign words carry nothing: operands that differ only there pass the operand checks (the
    output check after them fails here, so nothing is launched)."""
    a, b = _desc(rht_block=0), _desc(rht_block=0)
    a.sign_words[0], b.sign_words[0] = 1, 2
    assert getattr(lib, name)(R(a), R(b), FAKE, 8, 0, None) == SHAPE


@pytest.mark.parametrize("name", GEMMS)
def test_gemm_output_checks(lib, name):
    f = getattr(lib, name)
    assert f(R(_desc()), R(_desc()), None, 16, 0, None) == INVALID        # no output
    assert f(R(_desc()), R(_desc()), FAKE, 8, 0, None) == SHAPE           # ldc < N
    assert f(R(_desc()), R(_desc()), FAKE + 1, 16, 0, None) == ALIGN      # output alignment
    assert f(R(_desc()), R(_desc()), FAKE, 16, 5, None) == INVALID        # out dtype enum
    assert f(None, R(_desc()), FAKE, 16, 0, None) == INVALID              # no operand


def test_mx_gemm_operand_checks(lib):
    mx = dict(fmt=U.UNIFORM_MX32)
    g = lib.ufp4_mx_gemm_fwd_y
    assert g(R(_desc()), R(_desc()), FAKE, 16, 0, None) == MISMATCH                     # 1x16 operands
    assert g(R(_desc(**mx)), R(_desc(red=64, **mx)), FAKE, 16, 0, None) == MISMATCH     # reductions differ
    assert g(R(_desc(mask=3, **mx)), R(_desc(mask=5, **mx)), FAKE, 16, 0, None) == MISMATCH
    assert g(R(_desc(**mx)), R(_desc(**mx)), FAKE, 8, 0, None) == SHAPE                 # ldc < N
    assert g(R(_desc(**mx)), R(_desc(**mx)), FAKE, 16, 4, None) == INVALID              # out dtype
    assert g(R(_desc(red=48, **mx)), R(_desc(red=48, **mx)), FAKE, 16, 0, None) == SHAPE  # K % 32
    for name in ("ufp4_mx_gemm_bwd_dx", "ufp4_mx_gemm_bwd_dw"):
        assert getattr(lib, name)(R(_desc()), R(_desc(**mx)), FAKE, 16, 0, None) == MISMATCH


def test_grouped_gemm_checks(lib):
    fy, fx, fw = lib.ufp4_gemm_fwd_y_grouped, lib.ufp4_gemm_bwd_dx_grouped, lib.ufp4_gemm_bwd_dw_grouped
    # (a, b, offsets, G, c, ldc, out, stream)
    for f in (fy, fx, fw):
        assert f(R(_desc()), R(_desc()), None, 2, FAKE, 16, 0, None) == INVALID          # null offsets
        assert f(R(_desc()), R(_desc()), FAKE, 0, FAKE, 16, 0, None) == INVALID          # no groups
        assert f(R(_desc()), R(_desc(fmt=1)), FAKE, 2, FAKE, 16, 0, None) == MISMATCH    # grids differ
        assert f(R(_desc(mask=1)), R(_desc(mask=2)), FAKE, 2, FAKE, 16, 0, None) == MISMATCH
    assert fy(R(_desc()), R(_desc(rows=15)), FAKE, 2, FAKE, 16, 0, None) == SHAPE        # 15 rows of W in 2 groups
    assert fy(R(_desc()), R(_desc(red=48, cld=3072, sld=384)), FAKE, 2, FAKE, 16, 0, None) == MISMATCH  # K differs
    # bwd_dx: W^T's reduction must be G times dY's
    assert fx(R(_desc(red=32)), R(_desc(red=48, cld=3072, sld=384)), FAKE, 2, FAKE, 16, 0, None) == MISMATCH
    g = dict(layout=2)  # grouped-transposed operands, as bwd_dw takes them
    assert fw(R(_desc(**g)), R(_desc(red=48, cld=3072, sld=384, **g)), FAKE, 2, FAKE, 16, 0, None) == MISMATCH
    assert fw(R(_desc()), R(_desc()), FAKE, 70000, FAKE, 16, 0, None) == UNSUPPORTED     # groups > 65535
    # operand forms: bwd_dw pads each group's tokens to 16, so plain operands are refused; fwd_y and dY take plain
    assert fw(R(_desc()), R(_desc()), FAKE, 2, FAKE, 16, 0, None) == MISMATCH
    assert fw(R(_desc(**g)), R(_desc()), FAKE, 2, FAKE, 16, 0, None) == MISMATCH
    assert fy(R(_desc(**g)), R(_desc()), FAKE, 2, FAKE, 16, 0, None) == MISMATCH
    assert fy(R(_desc()), R(_desc(**g)), FAKE, 2, FAKE, 16, 0, None) == MISMATCH
    assert fx(R(_desc(red=16, **g)), R(_desc()), FAKE, 2, FAKE, 16, 0, None) == MISMATCH


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(U, "_lib", None)
    monkeypatch.setattr(U, "_LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        U.lib()


def test_binding_descriptor_layout_matches_the_header():
    """The ctypes mirror of ufp4_qtensor: field order and offsets as the header declares them (88 bytes)."""
    src = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    body = re.search(r"typedef struct \{(.*?)\} ufp4_qtensor;", src, re.S).group(1)
    names = re.findall(r"\b(\w+)(?:\[\d+\])?;", body)
    assert names == [f[0] for f in U.QDesc._fields_]
    assert ctypes.sizeof(U.QDesc) == 96 and U.QDesc.sign_words.offset == 64 and U.QDesc.layout.offset == 88


def test_mx_grouped_quantizer_validation(lib):
    q = lib.ufp4_mx_quantize_grouped
    mx = dict(fmt=U.UNIFORM_MX32)
    # (x, rows, cols, ld, transpose, offsets, G, padded_total, rht, mask, rounding, seed, stream, out, stream)
    rows_out = _desc(rows=256, red=64, cld=2 * 3072, sld=2 * 128, panels=2, **mx)
    assert q(FAKE, 200, 64, 64, 0, None, 2, 256, 1, 0, 0, 0, 0, R(rows_out), None) == INVALID   # no offsets
    assert q(FAKE, 200, 64, 64, 0, FAKE, 0, 256, 1, 0, 0, 0, 0, R(rows_out), None) == INVALID   # no groups
    assert q(FAKE, 200, 64, 64, 0, FAKE, 2000, 256, 1, 0, 0, 0, 0, R(rows_out), None) == UNSUPPORTED
    assert q(FAKE, 200, 64, 64, 0, FAKE, 2, 200, 1, 0, 0, 0, 0, R(rows_out), None) == SHAPE  # not whole panels
    assert q(FAKE, 200, 64, 64, 0, FAKE, 2, 384, 1, 0, 0, 0, 0, R(rows_out), None) == SHAPE  # 3 panels, room for 2
    assert q(FAKE, 200, 48, 48, 0, FAKE, 2, 256, 1, 0, 0, 0, 0, R(rows_out), None) == SHAPE  # cols % 32
    assert q(FAKE, 200, 64, 64, 2, FAKE, 2, 256, 1, 0, 0, 0, 0, R(rows_out), None) == INVALID   # transpose flag
    assert q(FAKE + 8, 200, 64, 64, 0, FAKE, 2, 256, 1, 0, 0, 0, 0, R(rows_out), None) == ALIGN
    red_out = _desc(rows=64, red=256, cld=8 * 3072, sld=8 * 128, **mx)
    assert q(FAKE, 300, 64, 64, 1, FAKE, 2, 256, 1, 0, 0, 0, 0, R(red_out), None) == SHAPE   # padded < rows
    assert q(FAKE, 200, 64, 64, 1, FAKE, 2, 240, 1, 0, 0, 0, 0, R(red_out), None) == SHAPE   # 240 % 32
    assert q(FAKE, 200, 64, 64, 1, FAKE, 2, 288, 1, 0, 0, 0, 0, R(red_out), None) == SHAPE   # 9 blocks, room for 8


def test_mx_grouped_gemm_checks(lib):
    mx = dict(fmt=U.UNIFORM_MX32)
    gr = dict(layout=U.LAYOUT_GROUPED_ROWS, **mx)
    gk = dict(layout=U.LAYOUT_GROUPED_RED, **mx)
    fy, fx, fw = lib.ufp4_mx_gemm_fwd_y_grouped, lib.ufp4_mx_gemm_bwd_dx_grouped, lib.ufp4_mx_gemm_bwd_dw_grouped
    w = _desc(rows=256, red=32, panels=2, **mx)  # two groups of 128 weight rows
    # (a, b, offsets, G, m_total, c, ldc, out, stream)
    assert fy(R(_desc(**gr)), R(w), None, 2, 16, FAKE, 128, 0, None) == INVALID        # no offsets
    assert fy(R(_desc(**gr)), R(w), FAKE, 2, -1, FAKE, 128, 0, None) == INVALID        # negative rows
    assert fy(R(_desc(**mx)), R(w), FAKE, 2, 16, FAKE, 128, 0, None) == MISMATCH       # X not in grouped rows
    assert fy(R(_desc(**gr)), R(_desc(rows=256, red=32, panels=2, **gr)), FAKE, 2, 16, FAKE, 128, 0, None) == MISMATCH
    assert fy(R(_desc(**gr)), R(_desc(rows=256, red=32, panels=2)), FAKE, 2, 16, FAKE, 128, 0, None) == MISMATCH  # 1x16
    assert fy(R(_desc(red=64, cld=2 * 3072, sld=256, **gr)), R(w), FAKE, 2, 16, FAKE, 128, 0, None) == MISMATCH
    assert fy(R(_desc(**gr)), R(_desc(rows=96, red=32, **mx)), FAKE, 2, 16, FAKE, 48, 0, None) == UNSUPPORTED  # N=48
    assert fy(R(_desc(**gr)), R(_desc(rows=255, red=32, panels=2, **mx)), FAKE, 2, 16, FAKE, 128, 0, None) == SHAPE
    assert fy(R(_desc(**gr)), R(w), FAKE, 2, 16, FAKE, 64, 0, None) == SHAPE            # ldc < N
    assert fy(R(_desc(mask=1, **gr)), R(_desc(rows=256, red=32, panels=2, mask=2, **mx)), FAKE, 2, 16, FAKE, 128, 0,
              None) == MISMATCH                                                          # other signs
    wt = _desc(rows=64, red=64, cld=2 * 3072, sld=256, **mx)  # W^T [K, G*N] with N = 32, G = 2
    assert fx(R(_desc(**mx)), R(wt), FAKE, 2, 16, FAKE, 64, 0, None) == MISMATCH         # dY not in grouped rows
    assert fx(R(_desc(**gr)), R(_desc(rows=64, red=96, cld=3 * 3072, sld=384, **mx)), FAKE, 2, 16, FAKE, 64, 0,
              None) == MISMATCH                                                          # W^T red != G * N
    assert fx(R(_desc(**gr)), R(wt), FAKE, 2, 16, FAKE, 32, 0, None) == SHAPE             # ldc < K
    # bwd_dw: both operands grouped along the reduction
    assert fw(R(_desc(**gk)), R(_desc(**mx)), FAKE, 2, FAKE, 16, 0, None) == MISMATCH
    assert fw(R(_desc(**gk)), R(_desc(red=64, cld=2 * 3072, sld=256, **gk)), FAKE, 2, FAKE, 16, 0, None) == MISMATCH
    assert fw(R(_desc(**gk)), R(_desc(**gk)), FAKE, 70000, FAKE, 16, 0, None) == UNSUPPORTED
    assert fw(R(_desc(**gk)), R(_desc(**gk)), FAKE, 2, FAKE, 8, 0, None) == SHAPE          # ldc < K
