"""GPU parity of the two-operand quantizer (ufp4_quantize_dual): both outputs bit-exact against the oracle's
two quantizations of the same tensor, through the C ABI (ctypes binding)."""

import numpy as np
import pytest
import torch

from oracle import ufp4_oracle as O
from paper_2606_20381_amd import ufp4 as U
from paper_2606_20381_amd import workloads as WL
from tests import parity as P

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    U.lib()


def _poisoned(rows, red, fmt):
    """An output operand filled with 0xFF bytes, so padding the kernel fails to write shows up."""
    q = U.empty_qtensor(rows, red, fmt)
    q.codes.fill_(0xFF)
    q.scales.view(torch.int32).fill_(-1)
    return q


def _check_dual(t_cpu, fmt, rounding, rht_r, rht_c, mask_r, mask_c, seed, st_r, st_c, rows_r=None, rows_c=None,
                what=""):
    bits = WL.bf16_bits(t_cpu)
    R, C = bits.shape
    qr, qc = _poisoned(R, C, fmt), _poisoned(C, R, fmt)
    U.quantize_dual(t_cpu.cuda(), fmt=fmt, rht_rows=rht_r, rht_cols=rht_c, sign_mask_rows=mask_r,
                    sign_mask_cols=mask_c, rounding=rounding, seed=seed, stream_rows=st_r, stream_cols=st_c,
                    out_rows=qr, out_cols=qc)
    torch.cuda.synchronize()
    for q, layout, rht, mask, st, rows in ((qr, "rows", rht_r, mask_r, st_r, rows_r),
                                           (qc, "cols", rht_c, mask_c, st_c, rows_c)):
        gc, gs = P.gpu_rows(q, rows)
        idx, sc = P.oracle_operand(bits, layout, fmt, rounding, rht, mask, seed, st, rows)
        P.assert_codes_equal(gc, gs, idx, sc, fmt, f"{what} dual {layout} fmt={fmt} rnd={rounding} rht={rht}")
        # padding rows of the last panel: zero codes and zero scales
        nkb = q.red // 16
        tail = q.panels * U.PANEL_ROWS - q.rows
        if tail:
            last_c = q.codes[-1, : nkb * 1024].reshape(nkb, U.PANEL_ROWS, 8)[:, U.PANEL_ROWS - tail:]
            last_s = q.scales[-1, : nkb * U.PANEL_ROWS].reshape(nkb, U.PANEL_ROWS)[:, U.PANEL_ROWS - tail:]
            assert int(last_c.count_nonzero()) == 0, f"{what} {layout}: padding codes not zero"
            assert int(last_s.count_nonzero()) == 0, f"{what} {layout}: padding scales not zero"
    return qr, qc


RHT_PAIRS = [(True, True), (False, True), (True, False), (False, False)]


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
@pytest.mark.parametrize("rht_r,rht_c", RHT_PAIRS)
def test_dual_tiny_layer_tensors(fmt, rounding, rht_r, rht_c):
    wl = WL.tiny()
    for name in ("x", "w", "dy"):
        t = getattr(wl, name)
        print(f"tiny {name} {tuple(t.shape)} fmt={fmt} rnd={rounding} rht={rht_r},{rht_c}", flush=True)
        _check_dual(t, fmt, rounding, rht_r, rht_c, wl.sign_mask, wl.sign_mask ^ 0x5A5A, wl.seed, 0, 1, what=name)


@pytest.mark.parametrize("shape", [(16, 16), (48, 80), (272, 208), (144, 400), (400, 144), (16, 2048),
                                   (2064, 16), (128, 64), (256, 192)])
def test_dual_ragged_shapes(shape):
    """Several 64-column tiles and 512-row workgroup spans, ragged tails on both axes, padding on both
    outputs' last panels."""
    g = torch.Generator().manual_seed(shape[0] * 1000 + shape[1])
    t = torch.randn(*shape, generator=g).bfloat16()
    print(f"ragged {shape}", flush=True)
    _check_dual(t, O.UNIFORM, O.RTNE, True, True, 0x1357, 0x2468, 9, 0, 0, what=str(shape))
    _check_dual(t, O.UNIFORM, O.SR, True, True, 0x1357, 0x1357, 9, 0, 1, what=str(shape))
    _check_dual(t, O.E2M1, O.SR, False, True, 0x1357, 0x1357, 9, 0, 1, what=str(shape))


def test_dual_edge_blocks():
    """Zero blocks, a lone outlier, ties of both grids and extreme magnitudes, arranged in 16-row groups so that
    the column blocks stay inside the exact-RHT domain too."""
    rng = np.random.default_rng(0)
    g0 = np.zeros((16, 64))
    g0[3, 17] = 3.0e4
    g0[3, 32:48] = np.linspace(-1e-6, 1e-6, 16)
    g1 = rng.standard_normal((16, 64)) * 1e-30
    g2 = rng.standard_normal((16, 64)) * 1e30
    tie_u = np.array([7.0, -7.0] + [k + 0.5 for k in range(-7, 7)] + list(range(-7, 8)) + [0.0] * 33)
    e = [6.0, 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, -0.25, -0.75, -1.25, -1.75, -2.5, -3.5, -5.0, -6.0]
    tie_e = np.array(e * 4)
    signs = np.where(rng.random((16, 1)) < 0.5, -1.0, 1.0)
    g3 = signs * tie_u[None, :]
    g4 = signs[::-1] * tie_e[None, :]
    t = torch.tensor(np.concatenate([g0, g1, g2, g3, g4]).astype(np.float32)).bfloat16()  # 80 x 64
    for fmt in (O.UNIFORM, O.E2M1):
        for rounding in (O.RTNE, O.SR):
            _check_dual(t, fmt, rounding, True, True, 0xA5A5, 0x0F0F, 3, 0, 1, what="edge")
            _check_dual(t, fmt, rounding, False, False, 0, 0, 3, 2, 3, what="edge")


def test_dual_strided_input():
    g = torch.Generator().manual_seed(17)
    big = torch.randn(96, 264, generator=g).bfloat16()
    t = big[:, 8:200]  # ld 264, 192 columns
    bits_t = t.contiguous()
    qr, qc = U.quantize_dual(big.cuda()[:, 8:200], rht_rows=True, rht_cols=True, sign_mask_rows=0x0F0F,
                             sign_mask_cols=0x0F0F, rounding=O.SR, seed=5, stream_rows=0, stream_cols=1)
    torch.cuda.synchronize()
    bits = WL.bf16_bits(bits_t)
    for q, layout, st in ((qr, "rows", 0), (qc, "cols", 1)):
        gc, gs = P.gpu_rows(q)
        idx, sc = P.oracle_operand(bits, layout, O.UNIFORM, O.SR, True, 0x0F0F, 5, st)
        P.assert_codes_equal(gc, gs, idx, sc, O.UNIFORM, f"strided {layout}")


def _equal_to_separate_calls(dev, fmt, rounding, rht_r, rht_c, mask_r, mask_c, seed, st_r, st_c):
    qr, qc = U.quantize_dual(dev, fmt=fmt, rht_rows=rht_r, rht_cols=rht_c, sign_mask_rows=mask_r,
                             sign_mask_cols=mask_c, rounding=rounding, seed=seed, stream_rows=st_r,
                             stream_cols=st_c)
    fn = U.rht_quantize if fmt == O.UNIFORM else U.e2m1_quantize
    sr = fn(dev, transpose=False, rht=rht_r, sign_mask=mask_r, rounding=rounding, seed=seed, stream_id=st_r)
    sc = fn(dev, transpose=True, rht=rht_c, sign_mask=mask_c, rounding=rounding, seed=seed, stream_id=st_c)
    torch.cuda.synchronize()
    for a, b, what in ((qr, sr, "rows"), (qc, sc, "cols")):
        assert torch.equal(a.codes, b.codes), f"dual {what} codes differ from the single-output kernel"
        assert torch.equal(a.scales.view(torch.int32), b.scales.view(torch.int32)), f"dual {what} scales differ"
    return qr, qc


def test_dual_dense_ffn_sampled():
    """Dense-1.5B FFN tensors at full size: sampled operand rows against the oracle, and every byte against
    the single-output kernels (which are themselves oracle-checked)."""
    wl = WL.dense_ffn()
    rng = np.random.default_rng(3)
    plan = (("x", O.RTNE, 0, 0), ("w", O.RTNE, 0, 0), ("dy", O.SR, 0, 1))
    for name, rounding, st_r, st_c in plan:
        t = getattr(wl, name)
        bits = WL.bf16_bits(t)
        dev = t.cuda()
        print(f"dense {name} {tuple(t.shape)}", flush=True)
        for fmt, rht_r, rht_c in ((O.UNIFORM, True, True), (O.E2M1, False, True)):
            qr, qc = _equal_to_separate_calls(dev, fmt, rounding, rht_r, rht_c, wl.sign_mask, wl.sign_mask,
                                              wl.seed, st_r, st_c)
            for q, layout, rht, st in ((qr, "rows", rht_r, st_r), (qc, "cols", rht_c, st_c)):
                rows = P.sample(q.rows, 24, rng)
                gc, gs = P.gpu_rows(q, rows)
                idx, sc = P.oracle_operand(bits, layout, fmt, rounding, rht, wl.sign_mask, wl.seed, st, rows)
                P.assert_codes_equal(gc, gs, idx, sc, fmt, f"dense {name} {layout} fmt={fmt}")
            del qr, qc


def test_dual_1gib_tensor_sampled():
    t = WL.quantizer_tensor()
    bits = WL.bf16_bits(t)
    dev = t.cuda()
    rng = np.random.default_rng(2)
    qr, qc = U.quantize_dual(dev, rht_rows=True, rht_cols=True, sign_mask_rows=0x6A09, sign_mask_cols=0x6A09,
                             rounding=O.RTNE, seed=5)
    torch.cuda.synchronize()
    for q, layout in ((qr, "rows"), (qc, "cols")):
        rows = P.sample(q.rows, 16, rng)
        gc, gs = P.gpu_rows(q, rows)
        idx, sc = P.oracle_operand(bits, layout, O.UNIFORM, O.RTNE, True, 0x6A09, 5, 0, rows)
        P.assert_codes_equal(gc, gs, idx, sc, O.UNIFORM, f"1GiB dual {layout}")


def test_dual_empty_and_invalid_calls():
    lib = U.lib()
    x = torch.zeros(32, 48, dtype=torch.bfloat16, device="cuda")
    qr, qc = U.empty_qtensor(32, 48), U.empty_qtensor(48, 32)
    qr.codes.fill_(0xAB)
    args = lambda rows, cols, ld, rnd=0: (0, x.data_ptr(), rows, cols, ld, 1, 0, 0, 1, 0, 1, rnd, 0, qr.ref(),
                                          qc.ref(), None)
    assert lib.ufp4_quantize_dual(*args(0, 48, 48)) == 0  # empty: nothing written
    assert lib.ufp4_quantize_dual(*args(32, 0, 48)) == 0
    torch.cuda.synchronize()
    assert int((qr.codes != 0xAB).sum()) == 0
    assert lib.ufp4_quantize_dual(*args(24, 48, 48)) == 2  # rows % 16
    assert lib.ufp4_quantize_dual(*args(32, 40, 48)) == 2  # cols % 16
    assert lib.ufp4_quantize_dual(*args(32, 48, 48, rnd=3)) == 1
    assert lib.ufp4_quantize_dual(0, x.data_ptr(), 32, 48, 48, 1, 0, 0, 1, 0, 1, 0, 0, qr.ref(), qr.ref(),
                                  None) == 1  # one descriptor for both outputs


def test_dual_transposed_equals_equal_group_transpose():
    """For per-expert weights W [E*N, K] with N % 16 == 0 the grouped-transposed operand (groups of N rows, no
    padding) is the plain transposed one, so the two-operand quantizer's Q_c can stand in for it."""
    E, N, K = 6, 176, 256
    g = torch.Generator().manual_seed(23)
    w = (torch.randn(E * N, K, generator=g) * 0.02).bfloat16().cuda()
    eoff, ered = U.group_offsets([N] * E)
    for fmt in (O.UNIFORM, O.E2M1):
        _, qc = U.quantize_dual(w, fmt=fmt, rht_rows=True, rht_cols=True, sign_mask_rows=0x3C3C,
                                sign_mask_cols=0x3C3C)
        qg = U.quantize_grouped_t(w, eoff, ered, fmt=fmt, rht=True, sign_mask=0x3C3C)
        torch.cuda.synchronize()
        assert torch.equal(qc.codes, qg.codes)
        assert torch.equal(qc.scales.view(torch.int32), qg.scales.view(torch.int32))
