"""GPU parity of the fused RHT + quantization kernels against the oracle: codes, scales and SR decisions
bit-exact, called through the C ABI (ctypes binding)."""

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


def _check_operand(t_cpu, name, fmt, rht, mask, seed, rows=None, rounding=None, stream=None):
    layout, rnd, st = P.OPERANDS[name]
    rnd = rnd if rounding is None else rounding
    st = st if stream is None else stream
    bits = WL.bf16_bits(t_cpu)
    q = P.gpu_operand(t_cpu.cuda(), layout, fmt, rnd, rht, mask, seed, st)
    torch.cuda.synchronize()
    gc, gs = P.gpu_rows(q, rows)
    idx, sc = P.oracle_operand(bits, layout, fmt, rnd, rht, mask, seed, st, rows)
    P.assert_codes_equal(gc, gs, idx, sc, fmt, f"{name} fmt={fmt} rht={rht} rnd={rnd}")


# ------------------------------------------------------------------------------------------------
# tiny single linear layer (256x256, 512x256, 256x512), every operand, both grids
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("name", list(P.OPERANDS))
def test_tiny_ufp4_operands(name):
    wl = WL.tiny()
    print(f"tiny ufp4 {name} mask={wl.sign_mask:#06x}", flush=True)
    _check_operand(getattr(wl, P.SOURCE[name]), name, O.UNIFORM, True, wl.sign_mask, wl.seed)


@pytest.mark.parametrize("rht", [False, True])
@pytest.mark.parametrize("name", list(P.OPERANDS))
def test_tiny_e2m1_operands(name, rht):
    wl = WL.tiny()
    _check_operand(getattr(wl, P.SOURCE[name]), name, O.E2M1, rht, wl.sign_mask, wl.seed)


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
def test_tiny_no_rht(fmt, rounding):
    wl = WL.tiny()
    _check_operand(wl.x, "x", fmt, False, 0, 77, rounding=rounding, stream=5)
    _check_operand(wl.x, "xt", fmt, False, 0, 77, rounding=rounding, stream=5)


# ------------------------------------------------------------------------------------------------
# edge cases
# ------------------------------------------------------------------------------------------------

def _edge_tensor():
    """Zero blocks, a single huge outlier, tiny values, every uniform and E2M1 tie, values on the grid."""
    rows = []
    rows.append(np.zeros(64))
    r = np.zeros(64)
    r[17] = 3.0e4  # one outlier in an otherwise zero block
    r[32:48] = np.linspace(-1e-6, 1e-6, 16)
    rows.append(r)
    # uniform ties with amax 7 (scale 1, reciprocal 1): v = k + 1/2 exactly
    rows.append(np.array([7.0, -7.0] + [k + 0.5 for k in range(-7, 7)] + list(range(-7, 8)) + [0.0] * 33))
    # E2M1 ties with amax 6: bin edges 0.25 .. 5
    e = [6.0, 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, -0.25, -0.75, -1.25, -1.75, -2.5, -3.5, -5.0, -6.0]
    rows.append(np.array(e * 4))
    rng = np.random.default_rng(0)
    rows.append(rng.standard_normal(64) * 1e-30)
    rows.append(rng.standard_normal(64) * 1e30)
    t = torch.tensor(np.array(rows, dtype=np.float32)).bfloat16()
    return torch.cat([t, t.flip(0) * -1, t * 2.0], 0)  # 18 x 64


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
@pytest.mark.parametrize("rht", [False, True])
def test_edge_blocks_rowwise(fmt, rounding, rht):
    t = _edge_tensor()
    _check_operand(t, "x", fmt, rht, 0xA5A5, 3, rounding=rounding, stream=0)


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
def test_edge_blocks_transposed(fmt, rounding):
    t = _edge_tensor()[:16].t().contiguous()  # 64 x 16: transposed operand rows = 16 original rows
    _check_operand(t, "xt", fmt, True, 0x0F0F, 4, rounding=rounding, stream=1)


@pytest.mark.parametrize("shape", [(37, 400), (16, 16), (1, 2048), (130, 48)])
def test_ragged_rowwise(shape):
    g = torch.Generator().manual_seed(shape[0] * 1000 + shape[1])
    t = torch.randn(*shape, generator=g).bfloat16()
    _check_operand(t, "x", O.UNIFORM, True, 0x1357, 9)
    _check_operand(t, "dy", O.UNIFORM, True, 0x1357, 9)


@pytest.mark.parametrize("shape", [(272, 200), (16, 8), (128, 64), (400, 136), (48, 8), (272, 312), (48, 520)])
def test_ragged_transposed(shape):
    """Ragged tails on both axes. The transposed kernel's workgroups cover 256 operand rows (two panels): 312
    and 520 columns give 384 and 640 padded operand rows, so the last workgroup's second panel lies past the
    end and its stores must be skipped."""
    g = torch.Generator().manual_seed(shape[0] * 1000 + shape[1])
    t = torch.randn(*shape, generator=g).bfloat16()
    _check_operand(t, "xt", O.UNIFORM, True, 0x2468, 11)
    _check_operand(t, "dyt", O.UNIFORM, True, 0x2468, 11)
    _check_operand(t, "xt", O.E2M1, True, 0x2468, 11, rounding=O.SR, stream=2)


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
def test_panel_layout_padding_and_strides(fmt):
    """Panel layout: 200 rows -> 2 panels whose last 56 rows are zero; wider panel strides than needed are
    honoured (the gap is left untouched); both input layouts."""
    g = torch.Generator().manual_seed(17)
    t = torch.randn(200, 48, generator=g).bfloat16()
    bits = WL.bf16_bits(t)
    fn = U.rht_quantize if fmt == O.UNIFORM else U.e2m1_quantize
    for layout, src in (("rows", t), ("cols", t.t().contiguous())):
        qrows, red = 200, 48
        nkb = red // 16
        codes = torch.full((2, nkb * 1024 + 96), 0xAB, dtype=torch.uint8, device="cuda")
        scales = torch.full((2, nkb * 128 + 12), -5.0, dtype=torch.float32, device="cuda")
        q = U.QTensor(codes, scales, U.QDesc(codes=codes.data_ptr(), scales=scales.data_ptr(),
                                             code_panel_ld=codes.stride(0), scale_panel_ld=scales.stride(0), panels=2))
        print(f"panel layout fmt={fmt} layout={layout}", flush=True)
        fn(src.cuda(), transpose=(layout == "cols"), rht=True, sign_mask=0x1111, rounding=O.RTNE, seed=1, out=q)
        torch.cuda.synchronize()
        gc, gs = P.gpu_rows(q)
        idx, sc = P.oracle_operand(bits, "rows", fmt, O.RTNE, True, 0x1111, 1, 0)  # both give the operand t
        P.assert_codes_equal(gc, gs, idx, sc, fmt, f"panel layout {layout}")
        c = codes.cpu().numpy()
        sv = scales.cpu().numpy()
        pad = c[1, : nkb * 1024].reshape(nkb, 128, 8)[:, 200 - 128:, :]
        assert np.all(pad == 0), "padding rows of the last panel must be zero codes"
        assert np.all(sv[1, : nkb * 128].reshape(nkb, 128)[:, 200 - 128:] == 0.0)
        assert np.all(c[:, nkb * 1024:] == 0xAB) and np.all(sv[:, nkb * 128:] == -5.0), "gap between panels written"


def test_strided_input_rows_and_cols():
    g = torch.Generator().manual_seed(5)
    big = torch.randn(96, 200, generator=g).bfloat16().cuda()
    view = big[:, 8:168]  # ld 200, 160 columns, 16-byte aligned start
    bits = WL.bf16_bits(view.cpu())
    for layout, name in (("rows", "x"), ("cols", "xt")):
        q = P.gpu_operand(view, layout, O.UNIFORM, O.SR, True, 0xBEEF, 21, 3)
        gc, gs = P.gpu_rows(q)
        idx, sc = P.oracle_operand(bits, layout, O.UNIFORM, O.SR, True, 0xBEEF, 21, 3)
        P.assert_codes_equal(gc, gs, idx, sc, O.UNIFORM, name)


def test_seed_and_stream_change_sr_draws():
    wl = WL.tiny()
    x = wl.dy.cuda()
    a = U.rht_quantize(x, rounding=U.SR, seed=1, stream_id=0, sign_mask=wl.sign_mask)
    b = U.rht_quantize(x, rounding=U.SR, seed=2, stream_id=0, sign_mask=wl.sign_mask)
    c = U.rht_quantize(x, rounding=U.SR, seed=1, stream_id=1, sign_mask=wl.sign_mask)
    d = U.rht_quantize(x, rounding=U.SR, seed=1, stream_id=0, sign_mask=wl.sign_mask)
    assert not torch.equal(a.codes, b.codes) and not torch.equal(a.codes, c.codes)
    assert torch.equal(a.codes, d.codes) and torch.equal(a.scales, b.scales)


def test_empty_and_invalid_calls():
    L = U.lib()
    x = torch.zeros(32, 32, dtype=torch.bfloat16, device="cuda")
    q = U.empty_qtensor(32, 32)
    s = torch.cuda.current_stream().cuda_stream
    call = lambda *a: L.ufp4_rht_quantize(*a, q.ref(), s)
    # empty tensor: no launch, OK, and the descriptor records the empty operand
    assert call(x.data_ptr(), 0, 32, 32, 0, 1, 0, 0, 0, 0) == 0
    assert (q.rows, q.red, q.rht_block) == (0, 32, 16)
    # reduction length not a multiple of 16
    assert call(x.data_ptr(), 32, 24, 32, 0, 1, 0, 0, 0, 0) == 2
    # misaligned input
    assert call(x.data_ptr() + 2, 32, 16, 32, 0, 1, 0, 0, 0, 0) == 3
    # bad enum
    assert call(x.data_ptr(), 32, 32, 32, 0, 1, 0, 7, 0, 0) == 1
    # code panel stride too small
    q.desc.code_panel_ld = 8
    assert call(x.data_ptr(), 32, 32, 32, 0, 1, 0, 0, 0, 0) == 2
    torch.cuda.synchronize()


# ------------------------------------------------------------------------------------------------
# full-size workloads, sampled operand rows (the oracle computes them one by one)
# ------------------------------------------------------------------------------------------------

def _check_layer_sampled(wl, fmt, recipe_rht, n_rows=48, seed=0):
    rng = np.random.default_rng(seed)
    bits = P.layer_bits(wl)
    dev = {k: getattr(wl, k).cuda() for k in ("x", "w", "dy")}
    for name, (layout, rnd, st) in P.OPERANDS.items():
        rht = recipe_rht[name]
        src = P.SOURCE[name]
        b = bits[src]
        qrows = b.shape[0] if layout == "rows" else b.shape[1]
        rows = P.sample(qrows, n_rows, rng)
        print(f"{wl.name} {name} fmt={fmt} rht={rht} rows={len(rows)}", flush=True)
        q = P.gpu_operand(dev[src], layout, fmt, rnd, rht, wl.sign_mask, wl.seed, st)
        gc, gs = P.gpu_rows(q, rows)
        del q
        idx, sc = P.oracle_operand(b, layout, fmt, rnd, rht, wl.sign_mask, wl.seed, st, rows)
        P.assert_codes_equal(gc, gs, idx, sc, fmt, f"{wl.name} {name}")


UFP4_RHT = {k: True for k in P.OPERANDS}
E2M1_RHT = {"x": False, "w": False, "dy": False, "wt": False, "dyt": True, "xt": True}


def test_dense_ffn_operands_sampled():
    wl = WL.dense_ffn()
    _check_layer_sampled(wl, O.UNIFORM, UFP4_RHT)
    _check_layer_sampled(wl, O.E2M1, E2M1_RHT, n_rows=16)
    _check_layer_sampled(wl, O.E2M1, UFP4_RHT, n_rows=16)


def test_square_operands_sampled():
    wl = WL.square()
    _check_layer_sampled(wl, O.UNIFORM, UFP4_RHT, n_rows=24)


def test_1gib_quantizer_tensor_sampled():
    t = WL.quantizer_tensor()
    bits = WL.bf16_bits(t)
    dev = t.cuda()
    rng = np.random.default_rng(1)
    for layout, name in (("rows", "x"), ("cols", "xt")):
        qrows = bits.shape[0] if layout == "rows" else bits.shape[1]
        rows = P.sample(qrows, 16, rng)
        q = P.gpu_operand(dev, layout, O.UNIFORM, O.RTNE, True, 0x6A09, 5, 0)
        gc, gs = P.gpu_rows(q, rows)
        del q
        idx, sc = P.oracle_operand(bits, layout, O.UNIFORM, O.RTNE, True, 0x6A09, 5, 0, rows)
        P.assert_codes_equal(gc, gs, idx, sc, O.UNIFORM, f"1GiB {name}")


# ------------------------------------------------------------------------------------------------
# grouped (MoE) transposed quantization
# ------------------------------------------------------------------------------------------------

def _check_grouped(t_cpu, counts, fmt, rounding, rht, mask, seed, stream, rows=None):
    bits = WL.bf16_bits(t_cpu)
    off, red_total = U.group_offsets(counts)
    q = U.quantize_grouped_t(t_cpu.cuda(), off, red_total, fmt=fmt, rht=rht, sign_mask=mask,
                             rounding=rounding, seed=seed, stream_id=stream)
    gc, gs = P.gpu_rows(q, rows)
    idx, sc, po = P.oracle_operand_grouped(bits, counts, fmt, rounding, rht, mask, seed, stream, rows)
    assert po[-1] == red_total
    P.assert_codes_equal(gc, gs, idx, sc, fmt, f"grouped counts={counts[:4]}..")


@pytest.mark.parametrize("counts", [[5, 16, 33, 0, 19], [0, 0, 7], [300], [1] * 20, [129, 127, 250]])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
def test_grouped_small(counts, rounding):
    g = torch.Generator().manual_seed(sum(counts) + len(counts))
    t = torch.randn(sum(counts), 72, generator=g).bfloat16()
    _check_grouped(t, counts, O.UNIFORM, rounding, True, 0x3C3C, 8, 1)
    _check_grouped(t, counts, O.E2M1, rounding, True, 0x3C3C, 8, 1)


@pytest.mark.parametrize("cfg", ["moe7.9b", "moe124b"])
def test_moe_operands_sampled(cfg):
    wl = WL.CONFIGS[cfg]()
    rng = np.random.default_rng(2)
    E, N, K = wl.w.shape
    w2 = wl.w.reshape(E * N, K)
    # rowwise operands: X (along K), W (along K), dY (along N, SR)
    for name, t, rnd, st in (("x", wl.x, O.RTNE, 0), ("w", w2, O.RTNE, 0), ("dy", wl.dy, O.SR, 0)):
        rows = P.sample(t.shape[0], 32, rng)
        print(f"{cfg} {name}", flush=True)
        _check_operand(t, name, O.UNIFORM, True, wl.sign_mask, wl.seed, rows=rows, rounding=rnd, stream=st)
    # grouped transposed: X^T, dY^T over the ragged token groups; W^T over equal expert groups
    print(f"{cfg} xt/dyt/wt grouped", flush=True)
    _check_grouped(wl.x, wl.counts, O.UNIFORM, O.RTNE, True, wl.sign_mask, wl.seed, 0,
                   rows=P.sample(K, 24, rng))
    _check_grouped(wl.dy, wl.counts, O.UNIFORM, O.SR, True, wl.sign_mask, wl.seed, 1,
                   rows=P.sample(N, 24, rng))
    _check_grouped(w2, [N] * E, O.UNIFORM, O.RTNE, True, wl.sign_mask, wl.seed, 0, rows=P.sample(K, 24, rng))
