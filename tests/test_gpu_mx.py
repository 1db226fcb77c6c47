"""GPU parity of the power-of-two-scale variant (1x32 E8M0 scales, FP6 E2M3 codes): quantized codes and scale
bytes bit-exact against the oracle, GEMMs within relative Frobenius error 1e-5 (fp32 output) and 4e-3 (bf16)
of the oracle's fp64 product of its own dequantized operands. Called through the C ABI (ctypes binding)."""

import numpy as np
import pytest
import torch

from oracle import ufp4_oracle as O
from paper_2606_20381_amd import ufp4 as U
from paper_2606_20381_amd import workloads as WL
from tests import parity as P

pytestmark = pytest.mark.gpu

TOL = {torch.float32: 1e-5, torch.bfloat16: 4e-3}
PASSES = {
    "fwd_y": ("x", "w", U.mx_gemm_fwd_y),
    "bwd_dx": ("dy", "wt", U.mx_gemm_bwd_dx),
    "bwd_dw": ("dyt", "xt", U.mx_gemm_bwd_dw),
}


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    U.lib()


def _oracle_mx(bits, layout, rounding, rht, mask, seed, stream, rows=None):
    if layout == "rows":
        ids = np.arange(bits.shape[0]) if rows is None else np.asarray(rows)
        a = O.bf16_bits_to_f32(bits[ids])
    else:
        ids = np.arange(bits.shape[1]) if rows is None else np.asarray(rows)
        a = np.ascontiguousarray(O.bf16_bits_to_f32(bits[:, ids]).T)
    return O.quantize_rows_mx(a, rounding, rht, mask, seed, stream, row_ids=ids)


def _gpu_mx(t_dev, layout, rounding, rht, mask, seed, stream, out=None):
    return U.mx_quantize(t_dev, transpose=(layout == "cols"), rht=rht, sign_mask=mask, rounding=rounding, seed=seed,
                         stream_id=stream, out=out)


def _assert_mx_equal(q, idx, e8, rows=None, what=""):
    gc, gs = q.codes_rows(), q.scales_rows()
    if rows is not None:
        sel = torch.as_tensor(np.asarray(rows), dtype=torch.int64, device=gc.device)
        gc, gs = gc[sel], gs[sel]
    gc, gs = gc.cpu().numpy(), gs.cpu().numpy()
    want = O.pack_fp6(idx)
    if not np.array_equal(gc, want):
        bad = np.argwhere(gc != want)
        r, c = bad[0]
        raise AssertionError(f"{what}: {len(bad)} code bytes differ; first at row {r} byte {c}: "
                             f"gpu {gc[r, c]:#04x} oracle {want[r, c]:#04x}")
    if not np.array_equal(gs, e8):
        bad = np.argwhere(gs != e8)
        r, c = bad[0]
        raise AssertionError(f"{what}: {len(bad)} scale bytes differ; first at row {r} block {c}: "
                             f"gpu {gs[r, c]} oracle {e8[r, c]}")


def _check(t_cpu, layout, rounding, rht, mask, seed, stream, what=""):
    bits = WL.bf16_bits(t_cpu)
    R, C = bits.shape
    qrows, red = (C, R) if layout == "cols" else (R, C)
    q = U.empty_qtensor_mx(qrows, red)
    q.codes.fill_(0xFF)
    q.scales.fill_(0xFF)
    _gpu_mx(t_cpu.cuda(), layout, rounding, rht, mask, seed, stream, out=q)
    torch.cuda.synchronize()
    idx, e8 = _oracle_mx(bits, layout, rounding, rht, mask, seed, stream)
    _assert_mx_equal(q, idx, e8, what=f"{what} {layout} rnd={rounding} rht={rht}")
    tail = q.panels * U.PANEL_ROWS - q.rows  # padding rows of the last panel are zero
    if tail:
        nkb = red // 32
        lc = q.codes[-1, : nkb * 3072].reshape(nkb, 3, U.PANEL_ROWS, 8)[:, :, U.PANEL_ROWS - tail:]
        ls = q.scales[-1, : nkb * U.PANEL_ROWS].reshape(nkb, U.PANEL_ROWS)[:, U.PANEL_ROWS - tail:]
        assert int(lc.count_nonzero()) == 0 and int(ls.count_nonzero()) == 0, f"{what}: padding not zero"


@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
@pytest.mark.parametrize("rht", [True, False])
def test_mx_quantize_tiny_layer(rounding, rht):
    wl = WL.tiny()
    for name in ("x", "w", "dy"):
        t = getattr(wl, name)
        print(f"mx tiny {name} rnd={rounding} rht={rht}", flush=True)
        _check(t, "rows", rounding, rht, wl.sign_mask, wl.seed, 0, name)
        _check(t, "cols", rounding, rht, wl.sign_mask, wl.seed, 1, name)


@pytest.mark.parametrize("shape", [(37, 96), (32, 32), (130, 64), (64, 200), (96, 136), (288, 64), (32, 8),
                                   (320, 1024)])
def test_mx_quantize_ragged(shape):
    g = torch.Generator().manual_seed(shape[0] * 1000 + shape[1])
    t = torch.randn(*shape, generator=g).bfloat16()
    print(f"mx ragged {shape}", flush=True)
    if shape[1] % 32 == 0:
        _check(t, "rows", O.RTNE, True, 0x1357, 9, 0, str(shape))
        _check(t, "rows", O.SR, True, 0x1357, 9, 0, str(shape))
    if shape[0] % 32 == 0:
        _check(t, "cols", O.RTNE, True, 0x2468, 9, 0, str(shape))
        _check(t, "cols", O.SR, False, 0x2468, 9, 1, str(shape))


def test_mx_quantize_edge_blocks():
    """Zero blocks, a lone outlier, exact top levels, ties, extreme magnitudes; 32-row groups keep the column
    blocks inside the exact-RHT domain too."""
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
        for rht in (False, True):
            _check(t, "rows", rounding, rht, 0xA5A5, 3, 0, "edge")
            _check(t, "cols", rounding, rht, 0x0F0F, 3, 1, "edge")


def _layer(wl_or_tensors, mask, seed):
    x, w, dy = wl_or_tensors
    dev = {"x": x.cuda(), "w": w.cuda(), "dy": dy.cuda()}
    q = {}
    for name, (layout, rnd, st) in P.OPERANDS.items():
        q[name] = _gpu_mx(dev[P.SOURCE[name]], layout, rnd, True, mask, seed, st)
    return q


def _oracle_pass(bits, pas, mask, seed, rows=None, cols=None):
    a, b, _ = PASSES[pas]
    la, ra, sa = P.OPERANDS[a]
    lb, rb, sb = P.OPERANDS[b]
    ia, ea = _oracle_mx(bits[P.SOURCE[a]], la, ra, True, mask, seed, sa, rows)
    ib, eb = _oracle_mx(bits[P.SOURCE[b]], lb, rb, True, mask, seed, sb, cols)
    return O.gemm_nt_mx(ia, ea, ib, eb)


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_mx_gemm_tiny_layer(out_dtype):
    wl = WL.tiny()
    bits = P.layer_bits(wl)
    q = _layer((wl.x, wl.w, wl.dy), wl.sign_mask, wl.seed)
    for pas, (a, b, fn) in PASSES.items():
        print(f"mx tiny {pas} {out_dtype}", flush=True)
        got = P.to_numpy(fn(q[a], q[b], out_dtype=out_dtype))
        want = _oracle_pass(bits, pas, wl.sign_mask, wl.seed)
        assert got.shape == want.shape
        err = P.rel_fro(got, want)
        assert err <= TOL[out_dtype], (pas, err)


@pytest.mark.parametrize("mnk", [(200, 72, 96), (32, 32, 32), (1, 300, 416), (257, 129, 2080), (128, 128, 128),
                                 (130, 260, 160)])
def test_mx_gemm_ragged_shapes(mnk):
    """128 x 128 tiles and 128-deep stages: partial tiles on both axes, partial last stage, single blocks."""
    m, n, k = mnk
    g = torch.Generator().manual_seed(m * 7 + n * 13 + k)
    a = torch.randn(m, k, generator=g).bfloat16()
    b = (torch.randn(n, k, generator=g) * 0.02).bfloat16()
    print(f"mx ragged gemm {mnk}", flush=True)
    qa = U.mx_quantize(a.cuda(), rht=True, sign_mask=0x3C3C)
    qb = U.mx_quantize(b.cuda(), rht=True, sign_mask=0x3C3C)
    ia, ea = O.quantize_rows_mx(O.bf16_bits_to_f32(WL.bf16_bits(a)), O.RTNE, True, 0x3C3C)
    ib, eb = O.quantize_rows_mx(O.bf16_bits_to_f32(WL.bf16_bits(b)), O.RTNE, True, 0x3C3C)
    want = O.gemm_nt_mx(ia, ea, ib, eb)
    for out_dtype in (torch.float32, torch.bfloat16):
        got = P.to_numpy(U.mx_gemm_fwd_y(qa, qb, out_dtype=out_dtype))
        assert P.rel_fro(got, want) <= TOL[out_dtype], (mnk, out_dtype)


def test_mx_gemm_output_leading_dimension():
    g = torch.Generator().manual_seed(5)
    a = torch.randn(64, 96, generator=g).bfloat16()
    b = torch.randn(48, 96, generator=g).bfloat16()
    qa, qb = U.mx_quantize(a.cuda()), U.mx_quantize(b.cuda())
    big = torch.full((64, 80), 7.0, device="cuda")
    U.mx_gemm_fwd_y(qa, qb, out=big[:, 8:56])
    torch.cuda.synchronize()
    ia, ea = O.quantize_rows_mx(O.bf16_bits_to_f32(WL.bf16_bits(a)), O.RTNE, True)
    ib, eb = O.quantize_rows_mx(O.bf16_bits_to_f32(WL.bf16_bits(b)), O.RTNE, True)
    want = O.gemm_nt_mx(ia, ea, ib, eb)
    got = big.cpu().numpy()
    assert P.rel_fro(got[:, 8:56], want) <= 1e-5
    assert np.all(got[:, :8] == 7.0) and np.all(got[:, 56:] == 7.0)


def test_mx_dense_ffn_sampled():
    """Dense-1.5B FFN layer at full size: sampled operand rows bit-exact, and sampled rows x columns of each
    pass against the oracle."""
    wl = WL.dense_ffn()
    bits = P.layer_bits(wl)
    rng = np.random.default_rng(4)
    q = _layer((wl.x, wl.w, wl.dy), wl.sign_mask, wl.seed)
    for name, (layout, rnd, st) in P.OPERANDS.items():
        rows = P.sample(q[name].rows, 16, rng)
        idx, e8 = _oracle_mx(bits[P.SOURCE[name]], layout, rnd, True, wl.sign_mask, wl.seed, st, rows)
        _assert_mx_equal(q[name], idx, e8, rows, f"dense {name}")
    for pas, (a, b, fn) in PASSES.items():
        print(f"mx dense {pas}", flush=True)
        c = fn(q[a], q[b], out_dtype=torch.float32)
        rows = P.sample(c.shape[0], 12, rng)
        cols = P.sample(c.shape[1], 64, rng)
        got = c[torch.as_tensor(rows, device="cuda")][:, torch.as_tensor(cols, device="cuda")].cpu().numpy()
        want = _oracle_pass(bits, pas, wl.sign_mask, wl.seed, rows, cols)
        assert P.rel_fro(got, want) <= 1e-5, pas


def test_mx_square_sampled():
    """The 16384^3 layer at full size with the output types of the timed layer step (Y and dX bf16, dW fp32):
    sampled operand rows bit-exact, sampled rows x columns of each pass against the oracle."""
    wl = WL.square()
    bits = P.layer_bits(wl)
    rng = np.random.default_rng(6)
    q = _layer((wl.x, wl.w, wl.dy), wl.sign_mask, wl.seed)
    for name, (layout, rnd, st) in P.OPERANDS.items():
        rows = P.sample(q[name].rows, 8, rng)
        idx, e8 = _oracle_mx(bits[P.SOURCE[name]], layout, rnd, True, wl.sign_mask, wl.seed, st, rows)
        _assert_mx_equal(q[name], idx, e8, rows, f"square {name}")
    out = {"fwd_y": torch.bfloat16, "bwd_dx": torch.bfloat16, "bwd_dw": torch.float32}
    for pas, (a, b, fn) in PASSES.items():
        print(f"mx square {pas}", flush=True)
        c = fn(q[a], q[b], out_dtype=out[pas])
        rows = P.sample(c.shape[0], 8, rng)
        cols = P.sample(c.shape[1], 32, rng)
        got = P.to_numpy(c[torch.as_tensor(rows, device="cuda")][:, torch.as_tensor(cols, device="cuda")])
        del c
        want = _oracle_pass(bits, pas, wl.sign_mask, wl.seed, rows, cols)
        assert P.rel_fro(got, want) <= TOL[out[pas]], pas
