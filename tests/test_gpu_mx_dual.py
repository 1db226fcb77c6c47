"""GPU parity of the two-operand power-of-two-scale quantizer (ufp4_mx_quantize_dual): both outputs bit-exact
against the oracle's two quantizations of the same tensor (rowwise along the columns, and of the transpose along
the rows), padding rows zero, through the C ABI (ctypes binding)."""

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


def _oracle(bits, layout, rounding, rht, mask, seed, stream, rows=None):
    """Oracle operand rows `rows`: rows of T (layout "rows") or of T^T (layout "cols")."""
    if layout == "rows":
        ids = np.arange(bits.shape[0]) if rows is None else np.asarray(rows)
        a = O.bf16_bits_to_f32(bits[ids])
    else:
        ids = np.arange(bits.shape[1]) if rows is None else np.asarray(rows)
        a = np.ascontiguousarray(O.bf16_bits_to_f32(bits[:, ids]).T)
    return O.quantize_rows_mx(a, rounding, rht, mask, seed, stream, row_ids=ids)


def _assert_equal(q, idx, e8, rows, what):
    gc, gs = q.codes_rows(), q.scales_rows()
    if rows is not None:
        sel = torch.as_tensor(np.asarray(rows), dtype=torch.int64, device=gc.device)
        gc, gs = gc[sel], gs[sel]
    gc, gs = gc.cpu().numpy(), gs.cpu().numpy()
    want = O.pack_fp6(idx)
    if not np.array_equal(gc, want):
        r, c = np.argwhere(gc != want)[0]
        raise AssertionError(f"{what}: code bytes differ; first at row {r} byte {c}: gpu {gc[r, c]:#04x} "
                             f"oracle {want[r, c]:#04x}")
    if not np.array_equal(gs, e8):
        r, c = np.argwhere(gs != e8)[0]
        raise AssertionError(f"{what}: scale bytes differ; first at row {r} block {c}: gpu {gs[r, c]} "
                             f"oracle {e8[r, c]}")


def _poisoned(rows, red):
    q = U.empty_qtensor_mx(rows, red)
    q.codes.fill_(0xFF)
    q.scales.fill_(0xFF)
    return q


def _padding_zero(q, what):
    tail = q.panels * U.PANEL_ROWS - q.rows
    if tail:
        nkb = q.red // 32
        lc = q.codes[-1, : nkb * 3072].reshape(nkb, 3, U.PANEL_ROWS, 8)[:, :, U.PANEL_ROWS - tail:]
        ls = q.scales[-1, : nkb * U.PANEL_ROWS].reshape(nkb, U.PANEL_ROWS)[:, U.PANEL_ROWS - tail:]
        assert int(lc.count_nonzero()) == 0 and int(ls.count_nonzero()) == 0, f"{what}: padding not zero"


def _check_dual(t_cpu, rounding, rht_r, rht_c, mask_r, mask_c, seed, st_r, st_c, dev=None, what=""):
    bits = WL.bf16_bits(t_cpu.contiguous())
    R, C = bits.shape
    qr, qc = _poisoned(R, C), _poisoned(C, R)
    U.mx_quantize_dual(t_cpu.cuda() if dev is None else dev, rht_rows=rht_r, rht_cols=rht_c, sign_mask_rows=mask_r,
                       sign_mask_cols=mask_c, rounding=rounding, seed=seed, stream_rows=st_r, stream_cols=st_c,
                       out_rows=qr, out_cols=qc)
    torch.cuda.synchronize()
    for q, layout, rht, mask, st in ((qr, "rows", rht_r, mask_r, st_r), (qc, "cols", rht_c, mask_c, st_c)):
        tag = f"{what} mx dual {layout} rnd={rounding} rht={rht}"
        idx, e8 = _oracle(bits, layout, rounding, rht, mask, seed, st)
        _assert_equal(q, idx, e8, None, tag)
        _padding_zero(q, tag)
    return qr, qc


RHT_PAIRS = [(True, True), (False, True), (True, False), (False, False)]


@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
@pytest.mark.parametrize("rht_r,rht_c", RHT_PAIRS)
def test_mx_dual_tiny_layer_tensors(rounding, rht_r, rht_c):
    wl = WL.tiny()
    for name in ("x", "w", "dy"):
        t = getattr(wl, name)
        print(f"mx dual tiny {name} {tuple(t.shape)} rnd={rounding} rht={rht_r},{rht_c}", flush=True)
        _check_dual(t, rounding, rht_r, rht_c, wl.sign_mask, wl.sign_mask ^ 0x5A5A, wl.seed, 0, 1, what=name)


@pytest.mark.parametrize("shape", [(32, 32), (64, 288), (160, 544), (288, 96), (96, 256), (416, 800), (32, 2080),
                                   (2080, 32), (256, 512)])
def test_mx_dual_ragged_shapes(shape):
    """32 x 256 workgroup tiles: several tiles on both axes, a partial last column tile, padding rows on both
    outputs' last panels (row tiles past the input write only zeros)."""
    g = torch.Generator().manual_seed(shape[0] * 1000 + shape[1])
    t = torch.randn(*shape, generator=g).bfloat16()
    print(f"mx dual ragged {shape}", flush=True)
    _check_dual(t, O.RTNE, True, True, 0x1357, 0x2468, 9, 0, 0, what=str(shape))
    _check_dual(t, O.SR, True, False, 0x1357, 0x1357, 9, 0, 1, what=str(shape))


def test_mx_dual_edge_blocks():
    """Zero blocks, a lone outlier, exact top levels, ties and extreme magnitudes in 32-row groups, so the column
    blocks see them too."""
    rng = np.random.default_rng(0)
    g0 = np.zeros((32, 64))
    g0[3, 17] = 3.0e4
    g0[3, 32:48] = np.linspace(-1e-6, 1e-6, 16)
    g1 = rng.standard_normal((32, 64)) * 1e-30
    g2 = rng.standard_normal((32, 64)) * 1e30
    ties = np.array([7.0, -7.0] + [k + 0.5 for k in range(-7, 7)] + list(range(-7, 8)) + [0.0] * 33)
    signs = np.where(rng.random((32, 1)) < 0.5, -1.0, 1.0)
    g3 = signs * ties[None, :]
    t = torch.tensor(np.concatenate([g0, g1, g2, g3]).astype(np.float32)).bfloat16()  # 128 x 64
    for rounding in (O.RTNE, O.SR):
        _check_dual(t, rounding, True, True, 0xA5A5, 0x0F0F, 3, 0, 1, what="edge")
        _check_dual(t, rounding, False, False, 0, 0, 3, 2, 3, what="edge")


def test_mx_dual_strided_input():
    g = torch.Generator().manual_seed(17)
    big = torch.randn(96, 328, generator=g).bfloat16()
    t = big[:, 8:296]  # ld 328, 288 columns
    _check_dual(t, O.SR, True, True, 0x0F0F, 0x0F0F, 5, 0, 1, dev=big.cuda()[:, 8:296], what="strided")


def _equal_to_separate_calls(dev, rounding, rht_r, rht_c, mask_r, mask_c, seed, st_r, st_c):
    qr, qc = U.mx_quantize_dual(dev, rht_rows=rht_r, rht_cols=rht_c, sign_mask_rows=mask_r, sign_mask_cols=mask_c,
                                rounding=rounding, seed=seed, stream_rows=st_r, stream_cols=st_c)
    sr = U.mx_quantize(dev, transpose=False, rht=rht_r, sign_mask=mask_r, rounding=rounding, seed=seed,
                       stream_id=st_r)
    sc = U.mx_quantize(dev, transpose=True, rht=rht_c, sign_mask=mask_c, rounding=rounding, seed=seed,
                       stream_id=st_c)
    torch.cuda.synchronize()
    for a, b, what in ((qr, sr, "rows"), (qc, sc, "cols")):
        assert torch.equal(a.codes, b.codes), f"mx dual {what} codes differ from the single-output kernel"
        assert torch.equal(a.scales, b.scales), f"mx dual {what} scales differ from the single-output kernel"
    return qr, qc


def test_mx_dual_dense_ffn_sampled():
    """Dense-1.5B FFN tensors at full size: sampled operand rows against the oracle, and every byte against the
    single-output kernels (which are themselves oracle-checked)."""
    wl = WL.dense_ffn()
    rng = np.random.default_rng(3)
    plan = (("x", O.RTNE, 0, 0), ("w", O.RTNE, 0, 0), ("dy", O.SR, 0, 1))
    for name, rounding, st_r, st_c in plan:
        t = getattr(wl, name)
        bits = WL.bf16_bits(t)
        print(f"mx dual dense {name} {tuple(t.shape)}", flush=True)
        qr, qc = _equal_to_separate_calls(t.cuda(), rounding, True, True, wl.sign_mask, wl.sign_mask, wl.seed,
                                          st_r, st_c)
        for q, layout, st in ((qr, "rows", st_r), (qc, "cols", st_c)):
            rows = P.sample(q.rows, 24, rng)
            idx, e8 = _oracle(bits, layout, rounding, True, wl.sign_mask, wl.seed, st, rows)
            _assert_equal(q, idx, e8, rows, f"dense {name} {layout}")
        del qr, qc


def test_mx_dual_1gib_tensor_sampled():
    """The 1 GiB quantizer tensor (32768 x 16384): every byte against the single-output kernels, sampled rows of
    both outputs against the oracle."""
    t = WL.quantizer_tensor()
    bits = WL.bf16_bits(t)
    rng = np.random.default_rng(8)
    print(f"mx dual 1GiB {tuple(t.shape)}", flush=True)
    qr, qc = _equal_to_separate_calls(t.cuda(), O.SR, True, True, 0x6A09, 0x6A09, 5, 0, 1)
    for q, layout, st in ((qr, "rows", 0), (qc, "cols", 1)):
        rows = P.sample(q.rows, 8, rng)
        idx, e8 = _oracle(bits, layout, O.SR, True, 0x6A09, 5, st, rows)
        _assert_equal(q, idx, e8, rows, f"1GiB {layout}")


def test_mx_dual_empty_and_invalid_calls():
    lib = U.lib()
    x = torch.zeros(64, 96, dtype=torch.bfloat16, device="cuda")
    qr, qc = U.empty_qtensor_mx(64, 96), U.empty_qtensor_mx(96, 64)
    qr.codes.fill_(0xAB)

    def call(rows, cols, ld, rnd=0, out_cols=None):
        return lib.ufp4_mx_quantize_dual(x.data_ptr(), rows, cols, ld, 1, 0, 0, 1, 0, 1, rnd, 0, qr.ref(),
                                         (out_cols or qc).ref(), None)

    assert call(0, 96, 96) == 0  # empty: nothing written
    assert call(64, 0, 96) == 0
    torch.cuda.synchronize()
    assert int((qr.codes != 0xAB).sum()) == 0
    assert call(48, 96, 96) == 2  # rows % 32
    assert call(64, 80, 96) == 2  # cols % 32
    assert call(64, 96, 96, rnd=3) == 1
    assert call(64, 96, 96, out_cols=qr) == 1  # one descriptor for both outputs
