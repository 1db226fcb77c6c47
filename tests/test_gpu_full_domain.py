"""GPU parity on the whole finite bf16 range: blocks whose scale or RHT outputs are subnormal fp32 numbers, whose
amax lies below g / FLT_MAX (so g / amax is past the fp32 range), whose inputs are subnormal bf16 numbers, or whose
rotated values pass FLT_MAX -- in every layout and kernel: rowwise, transposed, two-operand, grouped transposed,
the statistics kernel, RHT blocks of 32-128, the fp32-input quantizer and the power-of-two-scale quantizer. Codes
and scales bit-exact against the oracle, called through the C ABI."""

import numpy as np
import pytest
import torch

from oracle import ufp4_oracle as O
from paper_2606_20381_amd import ufp4 as U
from paper_2606_20381_amd import workloads as WL
from tests import parity as P

pytestmark = pytest.mark.gpu

BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    U.lib()


def _edge_rows(width=64, seed=0):
    """[rows, width] fp32 (bf16-representable) rows, each of one magnitude class: amax at g 2^-126 and one bf16
    step either side for g = 7 and 6, amax below 7 / FLT_MAX, subnormal inputs, sums / 4 below 2^-126, a normal
    row, rows near the bf16 maximum (one aligned with a Hadamard row, so its rotated value passes FLT_MAX), and
    zeros mixed in."""
    rng = np.random.default_rng(seed)
    ulp = 2.0 ** -131  # bf16 step at 1.75 * 2^-124 = 7 * 2^-126
    rows = []
    for g in (7.0, 6.0):
        for a in (g * 2.0 ** -126 - ulp, g * 2.0 ** -126, g * 2.0 ** -126 + ulp):
            base = [a, -a / 3, a / 5, 0.0, -a, a / 7] + list(rng.uniform(-a, a, 10))
            rows.append(np.tile(base, width // 16))
    for a in (1.5e-38, 2.0e-38, 1.0e-38):  # 7 / FLT_MAX = 2.06e-38
        rows.append(np.concatenate([[a, -a], rng.uniform(-a, a, width - 2)]))
    for a in (9.2e-41, 3e-40, 5e-39):  # subnormal bf16
        rows.append(rng.uniform(-a, a, width))
    rows.append(np.tile([2.0 ** -124, 2.0 ** -125, -(2.0 ** -127), 2.0 ** -130] + [0.0] * 12, width // 16))
    rows.append(rng.standard_normal(width))
    eps = np.array([-1.0 if (0x6A09 >> j) & 1 else 1.0 for j in range(16)])
    rows.append(np.tile(eps * 2.0 ** 125, width // 16))  # eps x = 2^125 (1, ..., 1): sum 2^129 past FLT_MAX
    rows.append(np.concatenate([[BF16_MAX, -BF16_MAX], rng.uniform(-BF16_MAX, BF16_MAX, width - 2)]))
    rows.append(rng.uniform(-1, 1, width) * 2.0 ** 126)
    while len(rows) % 16:  # transposed uses need a leading dimension that is a multiple of 8
        rows.append(rng.standard_normal(width) * 10.0 ** rng.uniform(-37, 37))
    a = np.array(rows, dtype=np.float32)
    return O.bf16_bits_to_f32(O.f32_to_bf16_bits(a))  # bf16 values


def _outer_tensor(seed=1):
    """[96, 80] whose 16 x 16 tiles each hold one magnitude class (row class times column class, from 2^-133 up
    to 2^126), so both its row blocks and its column blocks are edge cases."""
    rng = np.random.default_rng(seed)
    m = 2.0 ** np.array([-60, -30, -3, 0, 30, 62])
    n = 2.0 ** np.array([-73, -66, -63, 0, 62])
    u = rng.uniform(0.5, 1.0, (96, 80)) * rng.choice([-1.0, 1.0], (96, 80))
    t = (np.repeat(m, 16)[:, None] * np.repeat(n, 16)[None, :] * u).astype(np.float32)
    t[16:32, 0:16] = 0.0
    return O.bf16_bits_to_f32(O.f32_to_bf16_bits(t))


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).bfloat16().cuda()


def _check(q, idx, sc, fmt, what):
    torch.cuda.synchronize()
    gc, gs = P.gpu_rows(q)
    P.assert_codes_equal(gc, gs, idx, sc, fmt, what)


def test_edge_rows_reach_every_case():
    """The edge tensor really contains what it claims (oracle side): subnormal scales, scales of blocks with amax
    below 7 / FLT_MAX, subnormal inputs, and RHT outputs past FLT_MAX."""
    a = _edge_rows()
    _, sc = O.quantize_rows(a, O.UNIFORM, O.RTNE, False)
    assert np.any((sc > 0) & (sc < np.float32(2.0 ** -126)))
    assert np.any((a != 0) & (np.abs(a) < np.float32(2.0 ** -126)))
    y = O.rht_blocks(a.reshape(len(a), -1, 16), 0x6A09)
    assert np.any(np.abs(y) > float(np.finfo(np.float32).max))
    assert np.any((y != 0) & (np.abs(y) < 2.0 ** -126))


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
@pytest.mark.parametrize("rht", [False, True])
def test_rowwise(fmt, rounding, rht):
    a = _edge_rows()
    print(f"full-domain rowwise fmt={fmt} rnd={rounding} rht={rht}", flush=True)
    q = P.gpu_operand(_dev(a), "rows", fmt, rounding, rht, 0x6A09, 21, 3)
    idx, sc = O.quantize_rows(a, fmt, rounding, rht, 0x6A09, 21, 3)
    _check(q, idx, sc, fmt, "rowwise")


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
@pytest.mark.parametrize("rht", [False, True])
def test_transposed(fmt, rounding, rht):
    a = _edge_rows()
    print(f"full-domain transposed fmt={fmt} rnd={rounding} rht={rht}", flush=True)
    q = P.gpu_operand(_dev(a.T), "cols", fmt, rounding, rht, 0x6A09, 22, 1)  # operand rows = rows of a
    idx, sc = O.quantize_rows(a, fmt, rounding, rht, 0x6A09, 22, 1)
    _check(q, idx, sc, fmt, "transposed")


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
def test_two_operand(fmt, rounding):
    t = _outer_tensor()
    print(f"full-domain two-operand fmt={fmt} rnd={rounding}", flush=True)
    qr, qc = U.quantize_dual(_dev(t), fmt=fmt, rht_rows=True, rht_cols=False, sign_mask_rows=0x6A09,
                             sign_mask_cols=0x1234, rounding=rounding, seed=23, stream_rows=4, stream_cols=5)
    bits = O.f32_to_bf16_bits(t)
    (ir, sr), (ic, scc) = O.quantize_both(bits, fmt, rounding, True, False, 0x6A09, 0x1234, 23, 4, 5)
    _check(qr, ir, sr, fmt, "two-operand rows")
    _check(qc, ic, scc, fmt, "two-operand cols")
    qr, qc = U.quantize_dual(_dev(t), fmt=fmt, rht_rows=False, rht_cols=True, sign_mask_rows=0x6A09,
                             sign_mask_cols=0x1234, rounding=rounding, seed=23, stream_rows=4, stream_cols=5)
    (ir, sr), (ic, scc) = O.quantize_both(bits, fmt, rounding, False, True, 0x6A09, 0x1234, 23, 4, 5)
    _check(qr, ir, sr, fmt, "two-operand rows (no RHT)")
    _check(qc, ic, scc, fmt, "two-operand cols (RHT)")


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
def test_grouped_transposed(fmt, rounding):
    a = _edge_rows()
    x = np.ascontiguousarray(a.T)  # tokens x channels: operand row c is a's row c
    counts = [5, 20, 0, 39]
    off, red = U.group_offsets(counts)
    print(f"full-domain grouped fmt={fmt} rnd={rounding}", flush=True)
    q = U.quantize_grouped_t(_dev(x), off, red, fmt=fmt, rht=True, sign_mask=0x6A09, rounding=rounding,
                             seed=24, stream_id=1)
    idx, sc, _ = P.oracle_operand_grouped(O.f32_to_bf16_bits(x), counts, fmt, rounding, True, 0x6A09, 24, 1)
    _check(q, idx, sc, fmt, "grouped transposed")


@pytest.mark.parametrize("n", [32, 64, 128])
@pytest.mark.parametrize("transpose", [False, True])
def test_rht_blocks(n, transpose):
    a = _edge_rows(width=128)
    mask = int.from_bytes(np.random.default_rng(n).bytes(n // 8), "little")
    print(f"full-domain rht block {n} transpose={transpose}", flush=True)
    src = a.T if transpose else a
    q = U.quantize_rht_block(_dev(src), O.UNIFORM, rht_block=n, sign_mask=mask, transpose=transpose)
    idx, sc = O.quantize_rows(a, O.UNIFORM, O.RTNE, True, mask, rht_block=n)
    _check(q, idx, sc, O.UNIFORM, f"rht block {n}")


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
def test_fp32_input(fmt, rounding):
    """The fp32-input quantizer (second half of the unfused form) on fp32 values down to the smallest subnormal and
    up to FLT_MAX."""
    rng = np.random.default_rng(5)
    fmax = float(np.finfo(np.float32).max)
    rows = [rng.uniform(-1, 1, 64) * s for s in (1e-45 * 8, 1e-40, 1.5e-38, 7 * 2.0 ** -126, 1.0, 1e38, fmax)]
    rows.append(np.tile([fmax, -fmax, 1e-45, 0.0] * 4, 4))
    a = np.array(rows, dtype=np.float32)
    print(f"full-domain fp32 input fmt={fmt} rnd={rounding}", flush=True)
    q = U.quantize_f32(torch.from_numpy(a).cuda(), fmt, rounding=rounding, seed=25, stream_id=2)
    idx, sc = O.quantize_rows(a, fmt, rounding, False, 0, 25, 2)
    _check(q, idx, sc, fmt, "fp32 input")


def test_unfused_rht_then_fp32_quantizer():
    """The unfused form on the edge rows whose rotated values stay inside the fp32 range (its fp32 intermediate
    cannot hold the others): same codes as the fused kernel."""
    a = _edge_rows()
    y = O.rht_blocks(a.reshape(len(a), -1, 16), 0x6A09).reshape(a.shape)
    keep = np.all(np.abs(y) <= float(np.finfo(np.float32).max), axis=1)
    a = a[keep]
    x = _dev(a)
    yd = U.rht(x, sign_mask=0x6A09)
    q = U.quantize_f32(yd, O.UNIFORM)
    torch.cuda.synchronize()
    assert np.array_equal(yd.cpu().numpy().view(np.uint32), y[keep].astype(np.float32).view(np.uint32))
    idx, sc = O.quantize_rows(a, O.UNIFORM, O.RTNE, True, 0x6A09)
    _check(q, idx, sc, O.UNIFORM, "unfused")


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rht", [False, True])
@pytest.mark.parametrize("transpose", [False, True])
def test_statistics_kernel(fmt, rht, transpose):
    """The statistics kernel quantizes as the quantizers do: its code histogram equals the oracle's on the edge
    rows (the fp64 sums are dominated by the large rows and agree to rounding)."""
    a = _edge_rows()
    src = a.T if transpose else a
    st = U.quant_stats(_dev(src), fmt, transpose=transpose, rht=rht, sign_mask=0x6A09, rounding=O.SR, seed=26,
                       stream_id=1)
    want = O.quant_stats(a, fmt, O.SR, rht, 0x6A09, 26, 1)
    assert list(st.hist) == list(want["hist"])
    for k in ("err2", "ref2", "cross"):
        assert abs(getattr(st, k) - want[k]) <= 1e-9 * abs(want[k]) + 1e-300, k


@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
@pytest.mark.parametrize("rht", [False, True])
@pytest.mark.parametrize("transpose", [False, True])
def test_power_of_two_scales(rounding, rht, transpose):
    a = _edge_rows()
    src = a.T if transpose else a
    print(f"full-domain mx rnd={rounding} rht={rht} transpose={transpose}", flush=True)
    q = U.mx_quantize(_dev(src), transpose=transpose, rht=rht, sign_mask=0x6A09, rounding=rounding, seed=27,
                      stream_id=2)
    idx, e8 = O.quantize_rows_mx(a, rounding, rht, 0x6A09, 27, 2)
    torch.cuda.synchronize()
    assert np.array_equal(q.codes_rows().cpu().numpy(), O.pack_fp6(idx))
    assert np.array_equal(q.scales_rows().cpu().numpy(), e8)
