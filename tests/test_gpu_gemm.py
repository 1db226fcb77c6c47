"""GPU parity of the block-scaled 4-bit GEMMs (fwd_y, bwd_dx, bwd_dw; dense and grouped) against the
oracle's fp64 product of its own dequantized operands. Tolerances: relative Frobenius error <= 1e-5 for fp32
output and <= 4e-3 for bf16 output."""

import numpy as np
import pytest
import torch

from oracle import ufp4_oracle as O
from paper_2606_20381_amd import ufp4 as U
from paper_2606_20381_amd import workloads as WL
from tests import parity as P

pytestmark = pytest.mark.gpu

TOL = {torch.float32: 1e-5, torch.bfloat16: 4e-3}
RECIPE_RHT = {
    "ufp4": {k: True for k in P.OPERANDS},
    "e2m1": {"x": False, "w": False, "dy": False, "wt": False, "dyt": True, "xt": True},
}
# pass -> (left operand, right operand, gpu call)
PASSES = {
    "fwd_y": ("x", "w", U.gemm_fwd_y),
    "bwd_dx": ("dy", "wt", U.gemm_bwd_dx),
    "bwd_dw": ("dyt", "xt", U.gemm_bwd_dw),
}


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    U.lib()


def _layer_gpu(dev, fmt, rhts, mask, seed):
    q = {}
    for name, (layout, rnd, st) in P.OPERANDS.items():
        q[name] = P.gpu_operand(dev[P.SOURCE[name]], layout, fmt, rnd, rhts[name], mask, seed, st)
    return q


def _run_pass(q, pas, out_dtype):
    a, b, fn = PASSES[pas]
    return fn(q[a], q[b], out_dtype=out_dtype)


def _oracle_pass(bits, pas, fmt, rhts, mask, seed, rows=None, cols=None):
    """Oracle C[rows, cols] of one pass, quantizing only the operand rows it needs."""
    a, b, _ = PASSES[pas]
    la, ra, sa = P.OPERANDS[a]
    lb, rb, sb = P.OPERANDS[b]
    ia, sca = P.oracle_operand(bits[P.SOURCE[a]], la, fmt, ra, rhts[a], mask, seed, sa, rows)
    ib, scb = P.oracle_operand(bits[P.SOURCE[b]], lb, fmt, rb, rhts[b], mask, seed, sb, cols)
    return O.gemm_nt(ia, sca, ib, scb, fmt)


@pytest.mark.parametrize("recipe", ["ufp4", "e2m1"])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_tiny_layer_all_passes(recipe, out_dtype):
    wl = WL.tiny()
    fmt = O.UNIFORM if recipe == "ufp4" else O.E2M1
    rhts = RECIPE_RHT[recipe]
    bits = P.layer_bits(wl)
    dev = {k: getattr(wl, k).cuda() for k in ("x", "w", "dy")}
    q = _layer_gpu(dev, fmt, rhts, wl.sign_mask, wl.seed)
    for pas in PASSES:
        print(f"tiny {recipe} {pas} {out_dtype}", flush=True)
        got = P.to_numpy(_run_pass(q, pas, out_dtype))
        want = _oracle_pass(bits, pas, fmt, rhts, wl.sign_mask, wl.seed)
        assert got.shape == want.shape
        err = P.rel_fro(got, want)
        assert err <= TOL[out_dtype], (pas, err)


@pytest.mark.parametrize("mnk", [(200, 72, 48), (16, 16, 16), (1, 300, 400), (257, 129, 2064), (128, 128, 128)])
@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
def test_ragged_gemm_shapes(mnk, fmt):
    """Tiles of 128 x 128 with 8 K-blocks per stage: partial tiles on both axes, partial last stage."""
    m, n, k = mnk
    g = torch.Generator().manual_seed(m * 7 + n * 3 + k)
    x = torch.randn(m, k, generator=g).bfloat16()
    w = torch.randn(n, k, generator=g).bfloat16()
    xq = P.gpu_operand(x.cuda(), "rows", fmt, O.RTNE, True, 0x1111, 0, 0)
    wq = P.gpu_operand(w.cuda(), "rows", fmt, O.RTNE, True, 0x1111, 0, 0)
    got = P.to_numpy(U.gemm_fwd_y(xq, wq))
    ia, sa = P.oracle_operand(WL.bf16_bits(x), "rows", fmt, O.RTNE, True, 0x1111, 0, 0)
    ib, sb = P.oracle_operand(WL.bf16_bits(w), "rows", fmt, O.RTNE, True, 0x1111, 0, 0)
    want = O.gemm_nt(ia, sa, ib, sb, fmt)
    assert P.rel_fro(got, want) <= 1e-5


def test_zero_operand_and_output_stride():
    g = torch.Generator().manual_seed(3)
    x = torch.randn(64, 96, generator=g).bfloat16()
    x[:, 32:48] = 0  # a zero block column in every row
    w = torch.zeros(40, 96).bfloat16()
    xq = U.rht_quantize(x.cuda())
    wq = U.rht_quantize(w.cuda())
    out = torch.full((64, 48), 7.0, device="cuda")
    U.gemm_fwd_y(xq, wq, out=out[:, :40])
    o = out.cpu()
    assert torch.all(o[:, :40] == 0) and torch.all(o[:, 40:] == 7.0)


@pytest.mark.parametrize("kind", ["uniform", "e2m1", "mx"])
def test_empty_gemm_shapes(kind):
    """M = 0 and N = 0 give empty outputs; a zero-length reduction gives C = 0 (the kernels run no K-stage and
    still store every output, over a prefilled buffer)."""
    quant = {"uniform": U.rht_quantize, "e2m1": U.e2m1_quantize, "mx": U.mx_quantize}[kind]
    gemm = U.mx_gemm_fwd_y if kind == "mx" else U.gemm_fwd_y
    bf = dict(dtype=torch.bfloat16, device="cuda")
    for m, n, k in [(0, 40, 64), (70, 0, 64), (0, 0, 0), (300, 130, 0)]:
        print(f"empty gemm {kind} {m}x{n}x{k}", flush=True)
        xq, wq = quant(torch.randn(m, k, **bf)), quant(torch.randn(n, k, **bf))
        for odt in (torch.float32, torch.bfloat16):
            out = torch.full((m, n), 7.0, dtype=odt, device="cuda")
            y = gemm(xq, wq, out=out)
            torch.cuda.synchronize()
            assert y.shape == (m, n) and torch.all(y == 0)


def test_empty_reduction_grouped():
    """Grouped fwd_y over a zero-length reduction: every token row of every group is 0."""
    bf = dict(dtype=torch.bfloat16, device="cuda")
    off, _ = U.group_offsets([5, 0, 130])
    xq, wq = U.rht_quantize(torch.randn(135, 0, **bf)), U.rht_quantize(torch.randn(3 * 32, 0, **bf))
    out = torch.full((135, 32), 7.0, device="cuda")
    U.gemm_fwd_y_grouped(xq, wq, off, out=out)
    torch.cuda.synchronize()
    assert torch.all(out == 0)


def test_gemm_deterministic():
    wl = WL.tiny()
    xq = U.rht_quantize(wl.x.cuda(), sign_mask=wl.sign_mask)
    wq = U.rht_quantize(wl.w.cuda(), sign_mask=wl.sign_mask)
    a = U.gemm_fwd_y(xq, wq)
    b = U.gemm_fwd_y(xq, wq)
    assert torch.equal(a, b)


def _sampled_layer(wl, recipe, n=40, seed=0, out_dtype=torch.float32):
    fmt = O.UNIFORM if recipe == "ufp4" else O.E2M1
    rhts = RECIPE_RHT[recipe]
    rng = np.random.default_rng(seed)
    bits = P.layer_bits(wl)
    dev = {k: getattr(wl, k).cuda() for k in ("x", "w", "dy")}
    q = _layer_gpu(dev, fmt, rhts, wl.sign_mask, wl.seed)
    for pas in PASSES:
        print(f"{wl.name} {recipe} {pas}", flush=True)
        c = _run_pass(q, pas, out_dtype)
        rows = P.sample(c.shape[0], n, rng)
        cols = P.sample(c.shape[1], n, rng)
        got = P.to_numpy(c[torch.as_tensor(rows, device=c.device)][:, torch.as_tensor(cols, device=c.device)])
        del c
        want = _oracle_pass(bits, pas, fmt, rhts, wl.sign_mask, wl.seed, rows, cols)
        err = P.rel_fro(got, want)
        assert err <= TOL[out_dtype], (pas, err)


def test_dense_ffn_layer_sampled():
    wl = WL.dense_ffn()
    _sampled_layer(wl, "ufp4")
    _sampled_layer(wl, "ufp4", n=24, out_dtype=torch.bfloat16)
    _sampled_layer(wl, "e2m1", n=24)


def test_square_layer_sampled():
    wl = WL.square()
    _sampled_layer(wl, "ufp4", n=24)
    _sampled_layer(wl, "e2m1", n=16)


# ------------------------------------------------------------------------------------------------
# grouped (MoE) GEMMs
# ------------------------------------------------------------------------------------------------

def _grouped_case(x, w, dy, counts, mask, seed, fmt=O.UNIFORM, rows_per_group=None, cols=None, out_dtype=torch.float32,
                  rng=None):
    """Run the three grouped passes on the GPU and compare against the oracle on (sampled) outputs."""
    E, N, K = w.shape
    w2 = w.reshape(E * N, K)
    xb, w2b, dyb = WL.bf16_bits(x), WL.bf16_bits(w2), WL.bf16_bits(dy)
    off, red_total = U.group_offsets(counts)
    offs = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    xd, w2d, dyd = x.cuda(), w2.cuda(), dy.cuda()
    quant = U.rht_quantize if fmt == O.UNIFORM else U.e2m1_quantize
    xq = quant(xd, rht=True, sign_mask=mask)
    wq = quant(w2d, rht=True, sign_mask=mask)
    dyq = quant(dyd, rht=True, sign_mask=mask, rounding=U.SR, seed=seed, stream_id=0)
    eq, ered = U.group_offsets([N] * E)
    wtq = U.quantize_grouped_t(w2d, eq, ered, fmt=fmt, rht=True, sign_mask=mask)
    dytq = U.quantize_grouped_t(dyd, off, red_total, fmt=fmt, rht=True, sign_mask=mask, rounding=U.SR,
                                seed=seed, stream_id=1)
    xtq = U.quantize_grouped_t(xd, off, red_total, fmt=fmt, rht=True, sign_mask=mask)
    y = U.gemm_fwd_y_grouped(xq, wq, off, out_dtype=out_dtype)
    dx = U.gemm_bwd_dx_grouped(dyq, wtq, off, out_dtype=out_dtype)
    dw = U.gemm_bwd_dw_grouped(dytq, xtq, off, out_dtype=out_dtype)
    torch.cuda.synchronize()
    tol = TOL[out_dtype]
    rng = rng or np.random.default_rng(0)
    kc = np.arange(K) if cols is None else P.sample(K, len(cols), rng)
    nc = np.arange(N) if cols is None else P.sample(N, len(cols), rng)
    it, st, _ = P.oracle_operand_grouped(w2b, [N] * E, fmt, O.RTNE, True, mask, seed, 0, kc)
    yn, dxn = P.to_numpy(y), P.to_numpy(dx)
    for g, c in enumerate(counts):
        if c == 0:
            continue
        rows = np.arange(offs[g], offs[g + 1])
        if rows_per_group is not None:
            rows = rows[P.sample(len(rows), rows_per_group, rng)]
        # fwd_y: Y_g = Qx[rows] Qw[g*N + nc]^T
        ia, sa = P.oracle_operand(xb, "rows", fmt, O.RTNE, True, mask, seed, 0, rows)
        ib, sb = P.oracle_operand(w2b, "rows", fmt, O.RTNE, True, mask, seed, 0, g * N + nc)
        err = P.rel_fro(yn[np.ix_(rows, nc)], O.gemm_nt(ia, sa, ib, sb, fmt))
        assert err <= tol, ("fwd_y", g, err)
        # bwd_dx: dX_g = Qdy[rows] Qwt[kc, g*N:(g+1)*N]^T
        ia, sa = P.oracle_operand(dyb, "rows", fmt, O.SR, True, mask, seed, 0, rows)
        sl = slice(g * N, (g + 1) * N)
        err = P.rel_fro(dxn[np.ix_(rows, kc)], O.gemm_nt(ia, sa, it[:, sl], st[:, g * N // 16:(g + 1) * N // 16], fmt))
        assert err <= tol, ("bwd_dx", g, err)
    # bwd_dw: dW_g = Qdyt[nc, pad_g:pad_g+1] Qxt[kc, pad_g:pad_g+1]^T
    ida, sda, poffs = P.oracle_operand_grouped(dyb, counts, fmt, O.SR, True, mask, seed, 1, nc)
    ixa, sxa, _ = P.oracle_operand_grouped(xb, counts, fmt, O.RTNE, True, mask, seed, 0, kc)
    assert poffs[-1] == red_total
    dwn = P.to_numpy(dw)
    for g in range(len(counts)):
        cs = slice(int(poffs[g]), int(poffs[g + 1]))
        bs = slice(int(poffs[g]) // 16, int(poffs[g + 1]) // 16)
        want = O.gemm_nt(ida[:, cs], sda[:, bs], ixa[:, cs], sxa[:, bs], fmt)
        got = dwn[g][np.ix_(nc, kc)]
        if counts[g] == 0:
            assert np.all(got == 0)
        else:
            err = P.rel_fro(got, want)
            assert err <= tol, ("bwd_dw", g, err)


def test_grouped_offsets_past_and_short_of_the_rows():
    """Offsets are read on the device: a last offset beyond M_total computes exactly the rows that exist (the
    same bytes as the offsets that end at M_total), and output rows past a last offset below M_total are not
    written."""
    g = torch.Generator().manual_seed(21)
    E, N, K, M = 3, 48, 64, 200
    x = torch.randn(M, K, generator=g).bfloat16().cuda()
    w = (torch.randn(E * N, K, generator=g) * 0.05).bfloat16().cuda()
    xq, wq = U.rht_quantize(x, sign_mask=0x1234), U.rht_quantize(w, sign_mask=0x1234)
    dev = dict(dtype=torch.int64, device="cuda")
    ref = U.gemm_fwd_y_grouped(xq, wq, torch.tensor([0, 60, 160, 200], **dev))
    y = torch.full((M, N), 7.0, device="cuda")
    U.gemm_fwd_y_grouped(xq, wq, torch.tensor([0, 60, 160, 1000], **dev), out=y)
    torch.cuda.synchronize()
    assert torch.equal(y, ref)
    y = torch.full((M, N), 7.0, device="cuda")
    U.gemm_fwd_y_grouped(xq, wq, torch.tensor([0, 60, 100, 150], **dev), out=y)
    ref2 = U.gemm_fwd_y_grouped(xq, wq, torch.tensor([0, 60, 100, 200], **dev))
    torch.cuda.synchronize()
    assert torch.equal(y[:150], ref2[:150]) and torch.all(y[150:] == 7.0)


@pytest.mark.parametrize("counts", [[5, 16, 33, 0, 19], [300, 0, 7], [129, 127, 250, 1]])
@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
def test_grouped_small(counts, fmt):
    g = torch.Generator().manual_seed(len(counts) * 100 + sum(counts))
    E, N, K = len(counts), 48, 80
    x = torch.randn(sum(counts), K, generator=g).bfloat16()
    w = (torch.randn(E, N, K, generator=g) * 0.02).bfloat16()
    dy = (torch.randn(sum(counts), N, generator=g) * 1e-3).bfloat16()
    _grouped_case(x, w, dy, counts, 0x5A5A, 11, fmt=fmt)


@pytest.mark.parametrize("cfg,fmt", [("moe7.9b", O.UNIFORM), ("moe124b", O.UNIFORM), ("moe7.9b", O.E2M1)])
def test_moe_layer_sampled(cfg, fmt):
    wl = WL.CONFIGS[cfg]()
    print(f"{cfg} fmt {fmt} counts={wl.counts[:4]}.. total={sum(wl.counts)}", flush=True)
    _grouped_case(wl.x, wl.w, wl.dy, wl.counts, wl.sign_mask, wl.seed, fmt=fmt, rows_per_group=8,
                  cols=np.arange(24), rng=np.random.default_rng(4))
