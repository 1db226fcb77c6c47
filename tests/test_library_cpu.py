"""CPU checks of the C ABI library: it loads, exports every function include/ufp4.h declares, and rejects
bad arguments on the host before any GPU call (no compute runs here)."""

import ctypes
import os
import re

import pytest

from paper_2606_20381_amd import ufp4 as U

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ufp4.h")


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
                     "ufp4_gemm_bwd_dw"):
        assert required in names


def test_every_declared_symbol_is_exported(lib):
    raw = ctypes.CDLL(U.library_path())
    for name in _declared():
        assert hasattr(raw, name), name
        assert name in U.SIGNATURES, f"binding lacks a signature for {name}"


def test_status_strings(lib):
    assert lib.ufp4_status_string(0) == b"ok"
    assert lib.ufp4_status_string(3).startswith(b"misaligned")
    assert lib.ufp4_version() == b"0.1.0"


FAKE = 1 << 20  # a 1 MiB-aligned non-null address that is never dereferenced: every call below fails validation


# panel strides for one and two 16-blocks of reduction
C1, S1, C2, S2 = 1024, 128, 2048, 256


@pytest.mark.parametrize("args,status", [
    # (x, rows, cols, ld, transpose, rht, mask, rounding, seed, stream_id, codes, code_panel_ld, scales,
    #  scale_panel_ld)
    ((None, 16, 16, 16, 0, 1, 0, 0, 0, 0, FAKE, C1, FAKE, S1), 1),          # null input
    ((FAKE, 16, 24, 24, 0, 1, 0, 0, 0, 0, FAKE, C2, FAKE, S2), 2),          # cols % 16
    ((FAKE, 24, 16, 16, 1, 1, 0, 0, 0, 0, FAKE, C2, FAKE, S2), 2),          # transposed: rows % 16
    ((FAKE, 16, 32, 30, 0, 1, 0, 0, 0, 0, FAKE, C2, FAKE, S2), 2),          # ld < cols
    ((FAKE, 16, 32, 36, 0, 1, 0, 0, 0, 0, FAKE, C2, FAKE, S2), 2),          # ld % 8
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE, C1, FAKE, S2), 2),          # code panel stride < 1024 nkb
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE, C2, FAKE, S1), 2),          # scale panel stride < 128 nkb
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE, C2 + 8, FAKE, S2), 3),      # code panel stride % 16
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE, C2, FAKE, S2 + 2), 3),      # scale panel stride % 4
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE + 8, C2, FAKE, S2), 3),      # codes alignment
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE, C2, FAKE + 4, S2), 3),      # scales alignment
    ((FAKE + 2, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE, C2, FAKE, S2), 3),      # input alignment
    ((FAKE, 16, 32, 32, 0, 1, 0, 2, 0, 0, FAKE, C2, FAKE, S2), 1),          # rounding enum
    ((FAKE, 16, 32, 32, 2, 1, 0, 0, 0, 0, FAKE, C2, FAKE, S2), 1),          # transpose flag
    ((FAKE, 16, 32, 32, 0, 1, 0x10000, 0, 0, 0, FAKE, C2, FAKE, S2), 1),    # sign mask > 16 bits
    ((FAKE, -1, 32, 32, 0, 1, 0, 0, 0, 0, FAKE, C2, FAKE, S2), 1),          # negative size
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE, 1 << 30, FAKE, S2), 5),     # code panel stride > 2^29
    ((FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE, C2, FAKE, 1 << 28), 5),     # scale panel stride > 2^27
])
def test_quantize_validation(lib, args, status):
    for fn in (lib.ufp4_rht_quantize, lib.ufp4_e2m1_quantize):
        assert fn(*args, None) == status


@pytest.mark.parametrize("args,status", [
    # (a, a_panel_ld, as, as_panel_ld, b, b_panel_ld, bs, bs_panel_ld, M, N, K, fmt, c, ldc, out)
    ((None, C1, FAKE, S1, FAKE, C1, FAKE, S1, 16, 16, 16, 0, FAKE, 16, 0), 1),
    ((FAKE, C2, FAKE, S2, FAKE, C2, FAKE, S2, 16, 16, 24, 0, FAKE, 16, 0), 2),      # K % 16
    ((FAKE, C1, FAKE, S2, FAKE, C2, FAKE, S2, 16, 16, 32, 0, FAKE, 16, 0), 2),      # A panel stride < 1024 K/16
    ((FAKE, C2, FAKE, S2, FAKE, C2, FAKE, S1, 16, 16, 32, 0, FAKE, 16, 0), 2),      # B scale stride < 128 K/16
    ((FAKE, C2, FAKE, S2, FAKE, C2, FAKE, S2, 16, 16, 32, 0, FAKE, 8, 0), 2),       # ldc < N
    ((FAKE, C1 + 8, FAKE, S1, FAKE, C1, FAKE, S1, 16, 16, 16, 0, FAKE, 16, 0), 3),  # A panel stride % 16
    ((FAKE, C1, FAKE, S1, FAKE + 4, C1, FAKE, S1, 16, 16, 16, 0, FAKE, 16, 0), 3),  # B codes alignment
    ((FAKE, C2, FAKE, S2, FAKE, C2, FAKE, S2, 16, 16, 32, 3, FAKE, 16, 0), 1),      # format enum
    ((FAKE, C2, FAKE, S2, FAKE, C2, FAKE, S2, 16, 16, 32, 0, FAKE, 16, 5), 1),      # out dtype enum
    ((FAKE, C2, FAKE, S2, FAKE, C2, FAKE, S2, 16, 16, 32, 0, FAKE + 1, 16, 0), 3),  # output alignment
    ((FAKE, C2, FAKE, S2, FAKE, 1 << 30, FAKE, S2, 16, 16, 32, 0, FAKE, 16, 0), 5), # B panel stride > 2^29
])
def test_gemm_validation(lib, args, status):
    # the dense entry points map (M, N, K) onto (rows_a, rows_b, reduction) differently; pick the layout each
    # expects so the same failure shows up
    assert lib.ufp4_gemm_fwd_y(*args, None) == status


def test_gemm_validation_per_pass_layout(lib):
    # bwd_dx: dY [M, N] . Wt [K, N]^T -> dX [M, K]; the reduction is N
    assert lib.ufp4_gemm_bwd_dx(FAKE, C2, FAKE, S2, FAKE, C2, FAKE, S2, 16, 24, 16, 0, FAKE, 16, 0, None) == 2
    # bwd_dw: dYt [N, M] . Xt [K, M]^T -> dW [N, K]; the reduction is M
    assert lib.ufp4_gemm_bwd_dw(FAKE, C2, FAKE, S2, FAKE, C2, FAKE, S2, 24, 16, 16, 0, FAKE, 16, 0, None) == 2


def _dual_args(rows=32, cols=48, ld=48, fmt=0, rht_r=1, mask_r=0, rht_c=1, mask_c=0, rnd=0, x=FAKE, cr=FAKE,
               cr_ld=3 * 1024, sr=FAKE, sr_ld=3 * 128, cc=FAKE, cc_ld=2 * 1024, sc=FAKE, sc_ld=2 * 128):
    # (fmt, x, rows, cols, ld, rht_r, mask_r, stream_r, rht_c, mask_c, stream_c, rounding, seed,
    #  codes_r, code_panel_ld_r, scales_r, scale_panel_ld_r, codes_c, ..., stream)
    return (fmt, x, rows, cols, ld, rht_r, mask_r, 0, rht_c, mask_c, 1, rnd, 0, cr, cr_ld, sr, sr_ld, cc, cc_ld, sc,
            sc_ld, None)


@pytest.mark.parametrize("kw,status", [
    (dict(x=None), 1),                          # null input
    (dict(cc=None), 1),                         # null transposed codes
    (dict(fmt=2), 1),                           # format enum
    (dict(rnd=2), 1),                           # rounding enum
    (dict(rht_c=3), 1),                         # rht flag
    (dict(mask_r=0x10000), 1),                  # sign mask > 16 bits
    (dict(rows=-16), 1),                        # negative size
    (dict(rows=24), 2),                         # rows % 16 (the transposed output's reduction)
    (dict(cols=40, ld=40), 2),                  # cols % 16 (the rowwise output's reduction)
    (dict(ld=40), 2),                           # ld < cols
    (dict(ld=52), 2),                           # ld % 8
    (dict(cr_ld=2 * 1024), 2),                  # rowwise code panel stride < 1024 cols/16
    (dict(sc_ld=128), 2),                       # transposed scale panel stride < 128 rows/16
    (dict(cc_ld=2 * 1024 + 8), 3),              # panel stride % 16
    (dict(x=FAKE + 2), 3),                      # input alignment
    (dict(sr=FAKE + 4), 3),                     # scales alignment
    (dict(cc_ld=1 << 30), 5),                   # panel stride > 2^29
])
def test_dual_validation(lib, kw, status):
    assert lib.ufp4_quantize_dual(*_dual_args(**kw)) == status


def test_grouped_validation(lib):
    # null offsets
    assert lib.ufp4_quantize_grouped_t(0, FAKE, 32, 16, 16, None, FAKE, 2, 32, 1, 0, 0, 0, 0, FAKE, 16, FAKE, 2,
                                       None) == 1
    # too many groups for one launch
    assert lib.ufp4_quantize_grouped_t(0, FAKE, 32, 16, 16, FAKE, FAKE, 5000, 32, 1, 0, 0, 0, 0, FAKE, 16, FAKE, 2,
                                       None) == 5
    # padded total smaller than the rows
    assert lib.ufp4_quantize_grouped_t(0, FAKE, 64, 16, 16, FAKE, FAKE, 2, 32, 1, 0, 0, 0, 0, FAKE, 16, FAKE, 2,
                                       None) == 2
    assert lib.ufp4_gemm_fwd_y_grouped(FAKE, 8, FAKE, 1, FAKE, 8, FAKE, 1, None, 2, 16, 16, 16, 0, FAKE, 16, 0,
                                       None) == 1
    assert lib.ufp4_gemm_bwd_dx_grouped(FAKE, 8, FAKE, 1, FAKE, 8, FAKE, 1, FAKE, 0, 16, 16, 16, 0, FAKE, 16, 0,
                                        None) == 1
    assert lib.ufp4_gemm_bwd_dw_grouped(FAKE, 8, FAKE, 1, FAKE, 8, FAKE, 1, FAKE, 2, 32, 16, 16, 3, FAKE, 16, 0,
                                        None) == 1
    # red_total wider than the operands' panels
    assert lib.ufp4_gemm_bwd_dw_grouped(FAKE, C1, FAKE, S1, FAKE, C1, FAKE, S1, FAKE, 2, 32, 16, 16, 0, FAKE, 16,
                                        0, None) == 2


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(U, "_lib", None)
    monkeypatch.setattr(U, "_LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        U.lib()


def test_mx_validation(lib):
    # (x, rows, cols, ld, transpose, rht, mask, rounding, seed, stream, codes, code_pld, scales, scale_pld)
    C32, S32 = 3072, 128  # panel strides for one 32-block
    q = lib.ufp4_mx_quantize
    assert q(FAKE, 16, 48, 48, 0, 1, 0, 0, 0, 0, FAKE, 2 * C32, FAKE, 2 * S32, None) == 2   # cols % 32
    assert q(FAKE, 48, 16, 16, 1, 1, 0, 0, 0, 0, FAKE, 2 * C32, FAKE, 2 * S32, None) == 2   # transposed: rows % 32
    assert q(FAKE, 16, 64, 64, 0, 1, 0, 0, 0, 0, FAKE, C32, FAKE, 2 * S32, None) == 2       # code stride < 3072 nkb
    assert q(FAKE, 16, 64, 64, 0, 1, 0, 0, 0, 0, FAKE, 2 * C32, FAKE, S32, None) == 2       # scale stride < 128 nkb
    assert q(FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE, C32, FAKE, S32 + 4, None) == 3       # scale stride % 16
    assert q(FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE, C32, FAKE + 8, S32, None) == 3       # scales alignment
    assert q(None, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE, C32, FAKE, S32, None) == 1           # null input
    assert q(FAKE, 16, 32, 32, 0, 1, 0, 2, 0, 0, FAKE, C32, FAKE, S32, None) == 1           # rounding enum
    assert q(FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE, 1 << 30, FAKE, S32, None) == 5       # stride > 2^29
    g = lib.ufp4_mx_gemm_fwd_y
    # (a, a_pld, as, as_pld, b, b_pld, bs, bs_pld, M, N, K, c, ldc, out)
    assert g(FAKE, C32, FAKE, S32, FAKE, C32, FAKE, S32, 16, 16, 48, FAKE, 16, 0, None) == 2  # K % 32
    assert g(FAKE, C32, FAKE, S32, FAKE, C32, FAKE, S32, 16, 16, 64, FAKE, 16, 0, None) == 2  # strides < 2 blocks
    assert g(FAKE, C32, FAKE, S32, FAKE, C32, FAKE, S32, 16, 16, 32, FAKE, 8, 0, None) == 2   # ldc < N
    assert g(FAKE, C32, FAKE, S32, FAKE, C32, FAKE, S32, 16, 16, 32, FAKE, 16, 4, None) == 1  # out dtype
    assert g(None, C32, FAKE, S32, FAKE, C32, FAKE, S32, 16, 16, 32, FAKE, 16, 0, None) == 1  # null operand
    assert g(FAKE, C32, FAKE, S32, FAKE, C32, FAKE, S32, 16, 16, 32, FAKE + 2, 16, 0, None) == 3  # out alignment
    assert lib.ufp4_mx_gemm_bwd_dx(FAKE, C32, FAKE, S32, FAKE, C32, FAKE, S32, 16, 48, 16, FAKE, 16, 0,
                                   None) == 2  # reduction N % 32
    assert lib.ufp4_mx_gemm_bwd_dw(FAKE, C32, FAKE, S32, FAKE, C32, FAKE, S32, 48, 16, 16, FAKE, 16, 0,
                                   None) == 2  # reduction M % 32


def test_quant_stats_validation(lib):
    """ufp4_quant_stats(format, max_fpx, x, rows, cols, ld, transpose, rht, mask, rounding, seed, stream, rec)"""
    ok = (0, 0.0, FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0, FAKE)
    cases = [
        ((0, 4.0) + ok[2:], 1),                  # max_fpx on the uniform grid
        ((1, 3.0) + ok[2:], 1),                  # max_fpx not in {2, 4, 6}
        ((2,) + ok[1:], 1),                      # format enum
        (ok[:2] + (None,) + ok[3:], 1),          # null input
        (ok[:12] + (None,), 1),                  # null record
        (ok[:12] + (FAKE + 4,), 3),              # record alignment
        (ok[:4] + (24, 24) + ok[6:], 2),         # cols % 16
        (ok[:5] + (30,) + ok[6:], 2),            # ld < cols
        (ok[:6] + (2,) + ok[7:], 1),             # transpose flag
        (ok[:9] + (2,) + ok[10:], 1),            # rounding enum
    ]
    for args, status in cases:
        assert lib.ufp4_quant_stats(*args, None) == status, args


def test_e2m1_range_validation(lib):
    args = (FAKE, 16, 32, 32, 0, 1, 0, 0, 0, 0)
    for mf in (0.0, 1.0, 3.0, 7.0):
        assert lib.ufp4_e2m1_quantize_range(*args, mf, FAKE, 2 * 1024, FAKE, 2 * 128, None) == 1
    assert lib.ufp4_e2m1_quantize_range(FAKE, 16, 24, 24, 0, 1, 0, 0, 0, 0, 4.0, FAKE, 2048, FAKE, 256, None) == 2


def test_unfused_validation(lib):
    # ufp4_rht(x, rows, cols, ld, mask, y, ldy, stream)
    assert lib.ufp4_rht(None, 16, 32, 32, 0, FAKE, 32, None) == 1
    assert lib.ufp4_rht(FAKE, 16, 32, 32, 0x10000, FAKE, 32, None) == 1
    assert lib.ufp4_rht(FAKE, 16, 24, 24, 0, FAKE, 24, None) == 2      # cols % 16
    assert lib.ufp4_rht(FAKE, 16, 32, 36, 0, FAKE, 32, None) == 2      # ld % 8
    assert lib.ufp4_rht(FAKE, 16, 32, 32, 0, FAKE, 30, None) == 2      # ldy < cols
    assert lib.ufp4_rht(FAKE, 16, 32, 32, 0, FAKE, 34, None) == 2      # ldy % 4
    assert lib.ufp4_rht(FAKE, 16, 32, 32, 0, FAKE + 4, 32, None) == 3  # y alignment
    # ufp4_quantize_f32(format, x, rows, cols, ld, rounding, seed, stream, codes, cld, scales, sld, stream)
    assert lib.ufp4_quantize_f32(2, FAKE, 16, 32, 32, 0, 0, 0, FAKE, C2, FAKE, S2, None) == 1
    assert lib.ufp4_quantize_f32(0, FAKE, 16, 32, 32, 2, 0, 0, FAKE, C2, FAKE, S2, None) == 1
    assert lib.ufp4_quantize_f32(0, FAKE, 16, 24, 24, 0, 0, 0, FAKE, C2, FAKE, S2, None) == 2
    assert lib.ufp4_quantize_f32(0, FAKE, 16, 32, 34, 0, 0, 0, FAKE, C2, FAKE, S2, None) == 2   # ld % 4
    assert lib.ufp4_quantize_f32(0, FAKE + 8, 16, 32, 32, 0, 0, 0, FAKE, C2, FAKE, S2, None) == 3
    assert lib.ufp4_quantize_f32(0, FAKE, 16, 32, 32, 0, 0, 0, FAKE, C1, FAKE, S2, None) == 2   # code panel stride


def test_rht_block_validation(lib):
    words = (ctypes.c_uint16 * 8)()
    w = ctypes.cast(words, ctypes.c_void_p)
    base = (0, FAKE, 16, 128, 128, 0)
    tail = (0, 0, 0, FAKE, 8 * 1024, FAKE, 8 * 128, None)
    assert lib.ufp4_quantize_rht_block(*base, 48, w, *tail) == 1         # block size
    assert lib.ufp4_quantize_rht_block(*base, 32, None, *tail) == 1      # no sign words
    assert lib.ufp4_quantize_rht_block(2, *base[1:], 32, w, *tail) == 1  # format
    assert lib.ufp4_quantize_rht_block(0, FAKE, 16, 96, 96, 0, 64, w, 0, 0, 0, FAKE, 6 * 1024, FAKE, 6 * 128,
                                       None) == 2                        # 96 % 64
