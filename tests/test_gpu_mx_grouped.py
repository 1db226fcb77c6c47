"""GPU parity of the grouped (MoE) operands and GEMMs with power-of-two 1x32 scales, through the C ABI.

Operands: the grouped-rows form (each group of X's rows from a panel boundary, padding rows zero) equals, row for
row, the oracle's rowwise quantization of X (the SR counters use the row of X); the grouped-reduction form equals
the oracle's quantization of the transposed operand with each group's tokens zero-padded to 32. GEMMs: within
relative Frobenius error 1e-5 (fp32 output) / 4e-3 (bf16) of the oracle's fp64 products of its own dequantized
operands, per group; a group without tokens gets dW = 0."""

import numpy as np
import pytest
import torch

from oracle import ufp4_oracle as O
from paper_2606_20381_amd import ufp4 as U
from paper_2606_20381_amd import workloads as WL
from tests import parity as P

pytestmark = pytest.mark.gpu

TOL = {torch.float32: 1e-5, torch.bfloat16: 4e-3}


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    U.lib()


def _oracle_rows(bits, rounding, mask, seed, stream, rows):
    """Oracle rowwise power-of-two-scale quantization of rows `rows` of T (SR counters: those rows)."""
    rows = np.asarray(rows)
    return O.quantize_rows_mx(O.bf16_bits_to_f32(bits[rows]), rounding, True, mask, seed, stream, row_ids=rows)


def _oracle_cols(bits, rounding, mask, seed, stream, cols):
    """Oracle transposed operand rows `cols` (columns of T), reduction along all of T's rows."""
    cols = np.asarray(cols)
    a = np.ascontiguousarray(O.bf16_bits_to_f32(bits[:, cols]).T)
    return O.quantize_rows_mx(a, rounding, True, mask, seed, stream, row_ids=cols)


def _oracle_cols_grouped(bits, counts, rounding, mask, seed, stream, cols):
    """Oracle grouped-reduction operand rows `cols`: each group's tokens zero-padded to 32."""
    cols = np.asarray(cols)
    a, poff = O.operand_colwise_grouped(np.ascontiguousarray(bits[:, cols]), counts, block=32)
    idx, e8 = O.quantize_rows_mx(a, rounding, True, mask, seed, stream, row_ids=cols)
    return idx, e8, poff


def _assert_rows_equal(q, qrows, idx, e8, what):
    gc, gs = q.codes_rows(), q.scales_rows()
    sel = torch.as_tensor(np.asarray(qrows), dtype=torch.int64, device=gc.device)
    gc, gs = gc[sel].cpu().numpy(), gs[sel].cpu().numpy()
    assert np.array_equal(gc, O.pack_fp6(idx)), f"{what}: codes differ"
    assert np.array_equal(gs, e8), f"{what}: scales differ"


def _padded_row_starts(counts):
    return np.concatenate([[0], np.cumsum([-(-c // 128) * 128 for c in counts])]).astype(np.int64)


def _grouped_case(x, w, dy, counts, mask, seed, rows_per_group=None, cols=None, out_dtype=torch.float32, rng=None):
    E, N, K = w.shape
    M = sum(counts)
    w2 = w.reshape(E * N, K)
    xb, w2b, dyb = WL.bf16_bits(x), WL.bf16_bits(w2), WL.bf16_bits(dy)
    off, prow = U.group_offsets(counts, block=128)
    _, red32 = U.group_offsets(counts, block=32)
    offs = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    pstart = _padded_row_starts(counts)
    assert pstart[-1] == prow
    xd, w2d, dyd = x.cuda(), w2.cuda(), dy.cuda()
    xq = U.mx_quantize_grouped(xd, off, prow, transpose=False, sign_mask=mask)
    wq = U.mx_quantize(w2d, sign_mask=mask)
    dyq = U.mx_quantize_grouped(dyd, off, prow, transpose=False, sign_mask=mask, rounding=U.SR, seed=seed,
                                stream_id=0)
    wtq = U.mx_quantize(w2d, transpose=True, sign_mask=mask)
    dytq = U.mx_quantize_grouped(dyd, off, red32, transpose=True, sign_mask=mask, rounding=U.SR, seed=seed,
                                 stream_id=1)
    xtq = U.mx_quantize_grouped(xd, off, red32, transpose=True, sign_mask=mask)
    assert (xq.layout, dyq.layout, dytq.layout, xtq.layout) == (U.LAYOUT_GROUPED_ROWS,) * 2 + (U.LAYOUT_GROUPED_RED,) * 2
    y = U.mx_gemm_fwd_y_grouped(xq, wq, off, M, out_dtype=out_dtype)
    dx = U.mx_gemm_bwd_dx_grouped(dyq, wtq, off, M, out_dtype=out_dtype)
    dw = U.mx_gemm_bwd_dw_grouped(dytq, xtq, off, out_dtype=out_dtype)
    torch.cuda.synchronize()
    tol = TOL[out_dtype]
    rng = rng or np.random.default_rng(0)
    kc = np.arange(K) if cols is None else P.sample(K, len(cols), rng)
    nc = np.arange(N) if cols is None else P.sample(N, len(cols), rng)
    it, et = _oracle_cols(w2b, O.RTNE, mask, seed, 0, kc)  # W^T rows kc, reduction over all G*N
    yn, dxn = P.to_numpy(y), P.to_numpy(dx)
    for g, c in enumerate(counts):
        # padding rows of the grouped-rows operands are zero
        pad_rows = np.arange(pstart[g] + c, pstart[g + 1])
        if len(pad_rows):
            for q in (xq, dyq):
                sel = torch.as_tensor(pad_rows, dtype=torch.int64, device=q.codes.device)
                assert int(q.codes_rows()[sel].count_nonzero()) == 0 and int(q.scales_rows()[sel].count_nonzero()) == 0
        if c == 0:
            continue
        rows = np.arange(offs[g], offs[g + 1])
        if rows_per_group is not None:
            rows = rows[P.sample(len(rows), rows_per_group, rng)]
        qrows = pstart[g] + (rows - offs[g])
        # operands: the grouped rows are X's and dY's own rows, relocated
        ia, ea = _oracle_rows(xb, O.RTNE, mask, seed, 0, rows)
        _assert_rows_equal(xq, qrows, ia, ea, f"X group {g}")
        ida, eda = _oracle_rows(dyb, O.SR, mask, seed, 0, rows)
        _assert_rows_equal(dyq, qrows, ida, eda, f"dY group {g}")
        # fwd_y: Y_g = Qx[rows] Qw[g*N + nc]^T
        ib, eb = _oracle_rows(w2b, O.RTNE, mask, seed, 0, g * N + nc)
        err = P.rel_fro(yn[np.ix_(rows, nc)], O.gemm_nt_mx(ia, ea, ib, eb))
        assert err <= tol, ("fwd_y", g, err)
        # bwd_dx: dX_g = Qdy[rows] Qwt[kc, g*N:(g+1)*N]^T
        sl, bl = slice(g * N, (g + 1) * N), slice(g * N // 32, (g + 1) * N // 32)
        err = P.rel_fro(dxn[np.ix_(rows, kc)], O.gemm_nt_mx(ida, eda, it[:, sl], et[:, bl]))
        assert err <= tol, ("bwd_dx", g, err)
    # bwd_dw: dW_g = Qdyt[nc, pad_g:pad_{g+1}] Qxt[kc, pad_g:pad_{g+1}]^T
    idt, edt, poff = _oracle_cols_grouped(dyb, counts, O.SR, mask, seed, 1, nc)
    ixt, ext, _ = _oracle_cols_grouped(xb, counts, O.RTNE, mask, seed, 0, kc)
    assert poff[-1] == red32
    _assert_rows_equal(dytq, nc, idt, edt, "dY^T")
    _assert_rows_equal(xtq, kc, ixt, ext, "X^T")
    dwn = P.to_numpy(dw)
    for g in range(len(counts)):
        cs, bs = slice(int(poff[g]), int(poff[g + 1])), slice(int(poff[g]) // 32, int(poff[g + 1]) // 32)
        got = dwn[g][np.ix_(nc, kc)]
        if counts[g] == 0:
            assert np.all(got == 0)
        else:
            err = P.rel_fro(got, O.gemm_nt_mx(idt[:, cs], edt[:, bs], ixt[:, cs], ext[:, bs]))
            assert err <= tol, ("bwd_dw", g, err)


@pytest.mark.parametrize("counts", [[5, 16, 33, 0, 19], [300, 0, 7], [129, 127, 250, 1], [0, 256, 0]])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_mx_grouped_small(counts, out_dtype):
    g = torch.Generator().manual_seed(len(counts) * 100 + sum(counts))
    E, N, K = len(counts), 128, 96
    print(f"counts={counts} N={N} K={K} out={out_dtype}", flush=True)
    x = torch.randn(sum(counts), K, generator=g).bfloat16()
    w = (torch.randn(E, N, K, generator=g) * 0.02).bfloat16()
    dy = (torch.randn(sum(counts), N, generator=g) * 1e-3).bfloat16()
    _grouped_case(x, w, dy, counts, 0x5A3C, 11, out_dtype=out_dtype)


def test_mx_grouped_rows_past_the_last_group_are_zero():
    """Rows of a grouped-rows operand beyond the last group (a caller's larger buffer) are written as zeros."""
    counts = [3, 130]
    x = torch.randn(sum(counts), 64, generator=torch.Generator().manual_seed(5)).bfloat16().cuda()
    off, prow = U.group_offsets(counts, block=128)
    q = U.empty_qtensor_mx(prow + 256, 64)
    q.codes.fill_(0xFF)
    q.scales.fill_(0xFF)
    U.mx_quantize_grouped(x, off, prow + 256, transpose=False, sign_mask=0x77, out=q)
    torch.cuda.synchronize()
    assert q.rows == prow + 256
    assert int(q.codes_rows()[prow:].count_nonzero()) == 0 and int(q.scales_rows()[prow:].count_nonzero()) == 0
    assert int(q.codes_rows()[3:128].count_nonzero()) == 0  # padding of group 0


@pytest.mark.parametrize("cfg", ["moe7.9b", "moe124b"])
def test_mx_moe_layer_sampled(cfg):
    wl = WL.CONFIGS[cfg]()
    print(f"{cfg} counts={wl.counts[:4]}.. total={sum(wl.counts)}", flush=True)
    _grouped_case(wl.x, wl.w, wl.dy, wl.counts, wl.sign_mask, wl.seed, rows_per_group=4, cols=np.arange(16),
                  rng=np.random.default_rng(9))
