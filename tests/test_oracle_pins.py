"""Pins for the CPU oracle: each test ties the oracle to something other than itself -- a value the paper
prints, a closed form, an invariant, a library routine or brute force on tiny inputs."""

import os
import shutil
import subprocess
import tempfile
from fractions import Fraction
from math import floor

import numpy as np
import pytest

from oracle import ufp4_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_table(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def _bf16_blocks(vals):
    return O.bf16_bits_to_f32(O.f32_to_bf16_bits(np.asarray(vals, dtype=np.float64).astype(np.float32)))


def _rand_bf16_bits(rng, shape, scale=1.0):
    x = (rng.standard_normal(shape) * scale).astype(np.float32)
    return O.f32_to_bf16_bits(x)


# ------------------------------------------------------------------------------------------------
# Hadamard / RHT (Sec. 2.2)
# ------------------------------------------------------------------------------------------------

def test_sylvester_recursion_equals_popcount_closed_form():
    h = O.hadamard_pm1(16)
    for i in range(16):
        for j in range(16):
            assert h[i, j] == (-1) ** bin(i & j).count("1")


@pytest.mark.parametrize("n", [2, 4, 8, 16, 32, 64])
def test_hadamard_orthogonality(n):
    h = O.hadamard_pm1(n)
    assert np.array_equal(h @ h.T, n * np.eye(n))
    hn = O.sylvester_hadamard(n)
    assert np.abs(hn.T @ hn - np.eye(n)).max() < 1e-14
    assert np.abs(hn - h / np.sqrt(n)).max() < 1e-15


@pytest.mark.parametrize("mask", [0, 1, 0x8000, 0xA5C3, 0xFFFF])
def test_rht_orthogonal_and_invertible(mask):
    eps = O.sign_vector(mask)
    m = np.diag(eps) @ O.hadamard_pm1(16)
    assert np.array_equal(m @ m.T, 16 * np.eye(16))
    rng = np.random.default_rng(mask)
    x = O.bf16_bits_to_f32(_rand_bf16_bits(rng, (50, 16))).astype(np.float64)
    y = O.rht_exact_f64(x, mask)
    # x S H / 4 = y  =>  x = 4 y H S / 16 = y H S / 4 (H symmetric, H H = 16 I)
    back = (y @ O.hadamard_pm1(16)) * eps * 0.25
    assert np.array_equal(back, x)


def test_sign_mask_bit_order():
    # bit j of the mask flips element j: a unit vector at j maps to eps_j * (row j of H) / 4
    for j in range(16):
        e = np.zeros((1, 16))
        e[0, j] = 1.0
        y_flip = O.rht_exact_f64(e, 1 << j)
        y_keep = O.rht_exact_f64(e, 0xFFFF ^ (1 << j))
        assert np.array_equal(y_flip[0], -O.hadamard_pm1(16)[j] / 4)
        assert np.array_equal(y_keep[0], O.hadamard_pm1(16)[j] / 4)


def test_rotation_invariance_all_three_gemms():
    """Sec. 2.2: Y = X W^T = (X H')(W H')^T along the shared dimension, for fwd_y, bwd_dx and bwd_dw."""
    rng = np.random.default_rng(7)
    m, n, k = 48, 32, 64
    x = rng.standard_normal((m, k))
    w = rng.standard_normal((n, k))
    dy = rng.standard_normal((m, n))
    mask = 0x3C5A

    def rot(a):  # rotate rows of a (reduction axis contiguous) blockwise
        r, c = a.shape
        return O.rht_exact_f64(a.reshape(r, c // 16, 16), mask).reshape(r, c)

    for a, b, ref in [(x, w, x @ w.T), (dy, w.T, dy @ w), (dy.T, x.T, dy.T @ x)]:
        got = rot(np.ascontiguousarray(a)) @ rot(np.ascontiguousarray(b)).T
        assert np.linalg.norm(got - ref) / np.linalg.norm(ref) < 1e-13


def _round_fraction_f32(q: Fraction) -> np.float32:
    """Correct IEEE binary32 round-half-even of an exact rational (independent of any float path)."""
    if q == 0:
        return np.float32(0.0)
    sign = -1 if q < 0 else 1
    a = abs(q)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    ulp_e = max(e - 23, -149)
    scaled = a / Fraction(2) ** ulp_e
    n = floor(scaled)
    rem = scaled - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    val = Fraction(n) * Fraction(2) ** ulp_e
    assert val < Fraction(2) ** 128
    return np.float32(sign * float(val))  # n < 2^25: exact in fp64 and in fp32


def test_rht_correctly_rounded_bruteforce():
    """y_i = RN32(1/4 sum_j H[i,j] eps_j x_j) against exact rational arithmetic, on blocks whose nonzero
    magnitudes span up to 2^41 (where fp64 sums are exact) and far beyond it (up to the whole bf16 range, where
    the oracle sums with integers), and on results in the subnormal range (gradual underflow)."""
    rng = np.random.default_rng(11)
    blocks = []
    for t in range(400):
        mant = rng.integers(-255, 256, size=16)
        spread = int(rng.integers(0, 42)) if t % 3 else int(rng.integers(42, 250))
        # every fourth block lies at the bottom of the bf16 range, where sums / 4 fall below 2^-126
        base = int(rng.integers(-133, -110)) if t % 4 == 0 else int(rng.integers(-120, 100))
        expo = base - rng.integers(0, spread + 1, size=16)
        vals = np.array([float(Fraction(int(mm)) * Fraction(2) ** int(ee - 7)) for mm, ee in zip(mant, expo)])
        if t % 7 == 0:
            vals[rng.integers(0, 16, size=5)] = 0.0
        blocks.append(O.bf16_bits_to_f32(O.f32_to_bf16_bits(vals.astype(np.float32))))
    keep = np.array(blocks)
    mask = 0x9E37
    got = O.rht_blocks(keep, mask)
    mag = np.abs(got)
    assert np.count_nonzero((mag > 0) & (mag < np.float32(2.0 ** -126))) > 200  # subnormal outputs are covered
    h = O.hadamard_pm1(16)
    eps = O.sign_vector(mask)
    for bi, b in enumerate(keep):
        xs = [Fraction(float(v)) for v in b]
        for i in range(16):
            s = sum(Fraction(int(h[i, j] * eps[j])) * xs[j] for j in range(16)) / 4
            want = _round_fraction_f32(s)
            assert np.float32(got[bi, i]).view(np.uint32) == want.view(np.uint32), (bi, i)


def test_rht_outputs_past_the_fp32_range_keep_24_bits():
    """Inputs near the bf16 maximum rotate to values beyond FLT_MAX: y is the exact value rounded to 24
    significant bits (no overflow), checked with exact rationals."""
    big = (2.0 - 2.0 ** -7) * 2.0 ** 127  # the largest bf16
    b = _bf16_blocks([[big, big, -big, big, big / 3, 0.0, big / 5, big] + [big / 7] * 8,
                      [big] * 16, [2.0 ** 125, 2.0 ** 126, -(2.0 ** 124)] + [0.0] * 13])
    mask = 0x0F0F
    got = O.rht_blocks(b, mask)
    assert np.any(np.abs(got) > float(np.finfo(np.float32).max))
    h, eps = O.hadamard_pm1(16), O.sign_vector(mask)
    for r in range(len(b)):
        xs = [Fraction(float(v)) for v in b[r]]
        for i in range(16):
            s = sum(Fraction(int(h[i, j] * eps[j])) * xs[j] for j in range(16)) / 4
            want = _round_fraction_sig(abs(s), 24) * (1 if s > 0 else -1) if s != 0 else Fraction(0)
            assert Fraction(float(got[r, i])) == want, (r, i)


def test_rht_beyond_the_fp64_exact_span():
    """Blocks whose terms span more than fp64 holds, built so that the large terms sum to an fp32 tie and only
    a tiny term decides the rounding (an fp64 evaluation would lose it and round the tie to even): each output
    equals the exact rational transform rounded once, for the 16-point RHT and for the 32/64/128-point ones."""
    b = np.zeros((7, 16))
    b[0, :3] = [1.0, 2.0 ** -24, 2.0 ** -100]      # tie broken upward / downward by 2^-100 per row of H
    b[1, :3] = [2.0 ** 100, 2.0 ** 76, -(2.0 ** -120)]
    b[2, :4] = [2.0 ** -60, 2.0 ** -84, 2.0 ** -133, 2.0 ** -130]  # subnormal tail terms
    b[3, [0, 5, 9]] = [3.0 * 2.0 ** 40, -(2.0 ** 16), 2.0 ** -90]
    b[4, :2] = [2.0 ** 20, 2.0 ** -22]              # spread 42: just past the fp64-exact domain
    b[5] = [2.0 ** (120 - 16 * k) * (1 + k / 128) for k in range(16)]  # every term in its own binade
    # exact ties on the integer path: the 2^-100 pair cancels in the odd rows of H, where 1 + 3 * 2^-24 remains,
    # the midpoint of 1 + 2^-23 and 1 + 2^-22 (rounds to the even one)
    b[6, [0, 2, 4, 5]] = [1.0, 3.0 * 2.0 ** -24, 2.0 ** -100, 2.0 ** -100]
    b = _bf16_blocks(b.tolist())
    assert not O._fp64_sums_exact(b).any()
    for mask in (0, 0x5A3C):
        got = O.rht_blocks(b, mask)
        h, eps = O.hadamard_pm1(16), O.sign_vector(mask)
        for r in range(len(b)):
            xs = [Fraction(float(v)) for v in b[r]]
            for i in range(16):
                s = sum(Fraction(int(h[i, j] * eps[j])) * xs[j] for j in range(16)) / 4
                assert Fraction(float(got[r, i])) == _round_fp32_no_overflow(s), (mask, r, i)
    # wider RHT blocks: n = 64 is one rounding of the exact transform (c = 1/8); n = 32 and 128 round the
    # exact product S * RN64(sqrt(1/n)) to fp64 first, then to fp32
    rng = np.random.default_rng(5)
    for n in (32, 64, 128):
        a = np.zeros((2, n))
        a[0, rng.choice(n, 5, replace=False)] = [1.0, 2.0 ** -24, -(2.0 ** -100), 2.0 ** 30, 2.0 ** -40]
        a[1, rng.choice(n, 3, replace=False)] = [2.0 ** 60, -(2.0 ** -70), 2.0 ** -126]
        a = _bf16_blocks(a.tolist())
        mask = (1 << n) - 1 - 0x1234
        got = O.rht_rows_n(a, mask, n)
        hn, en = O.hadamard_pm1(n), O.sign_vector(mask, n)
        c = Fraction(O.rht_norm(n))
        for r in range(2):
            xs = [Fraction(float(v)) for v in a[r]]
            for i in range(n):
                s = sum(Fraction(int(hn[i, j] * en[j])) * xs[j] for j in range(n))
                want = _round_fp32_no_overflow(s * c) if n == 64 else _round_fp32_no_overflow(Fraction(float(s * c)))
                assert Fraction(float(got[r, i])) == want, (n, r, i)


def _round_fraction_sig(q: Fraction, bits: int) -> Fraction:
    """Round-half-even of a positive rational to `bits` significant bits, with no exponent limit."""
    assert q > 0
    e = q.numerator.bit_length() - q.denominator.bit_length()
    while Fraction(2) ** e > q:
        e -= 1
    while Fraction(2) ** (e + 1) <= q:
        e += 1
    step = Fraction(2) ** (e - bits + 1)
    n = floor(q / step)
    rem = q / step - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return n * step


def _round_fp32_no_overflow(q: Fraction) -> Fraction:
    """fp32 rounding with gradual underflow below 2^-126 and 24 significant bits (no overflow) from 2^127 up."""
    if q == 0:
        return Fraction(0)
    if abs(q) >= Fraction(2) ** 127:
        return _round_fraction_sig(abs(q), 24) * (1 if q > 0 else -1)
    return Fraction(float(_round_fraction_f32(q)))


def _exact_quant_block(x, fmt, rounding, rht, mask, u16):
    """One 16-block quantized with exact rationals, step by step as Sec. 2.1 / 2.2 state it: y = RN32 of the
    exact RHT (or x), amax, s = RN32(amax / g) with gradual underflow, r = g / amax to 24 significant bits,
    v = RN32(y r), then the nearest level (ties to the even magnitude code) or the SR rule with the draws.
    Returns (signed level indices, scale as fp32)."""
    xs = [Fraction(float(v)) for v in x]
    if rht:
        h = O.hadamard_pm1(16)
        eps = O.sign_vector(mask)
        ys = [_round_fp32_no_overflow(sum(Fraction(int(h[i, j] * eps[j])) * xs[j] for j in range(16)) / 4)
              for i in range(16)]
    else:
        ys = xs
    g = Fraction(int(O.G_MAX[fmt]))
    amax = max(abs(t) for t in ys)
    if amax == 0:
        return [0] * 16, np.float32(0.0)
    q = amax / g
    s = np.float32(np.inf) if _round_fraction_sig(q, 24) >= Fraction(2) ** 128 else _round_fraction_f32(q)
    r = _round_fraction_sig(g / amax, 24)
    mags = [Fraction(float(m)) for m in O.GRID_MAGNITUDES[fmt]]
    levels = sorted({-m for m in mags} | set(mags))
    out = []
    for i, t in enumerate(ys):
        v = Fraction(float(_round_fraction_f32(t * r)))
        if rounding == O.RTNE:
            d = [abs(abs(v) - m) for m in mags]
            cand = [k for k, dd in enumerate(d) if dd == min(d)]
            k = [c for c in cand if c % 2 == 0][0] if len(cand) > 1 else cand[0]
            out.append(-k if v < 0 else k)
        else:
            vc = min(max(v, levels[0]), levels[-1])
            ia = max(k for k, L in enumerate(levels) if L <= vc)
            ga = levels[ia]
            if ia + 1 < len(levels) and Fraction(int(u16[i]), 65536) < (vc - ga) / (levels[ia + 1] - ga):
                ga = levels[ia + 1]
            k = mags.index(abs(ga))
            out.append(-k if ga < 0 else k)
    return out, s


def _edge_blocks():
    """Blocks at both ends of the fp32 range (bf16 values), each a case where plain fp32 arithmetic would break:
    amax at g * 2^-126 and one bf16 step either side (scale normal / subnormal), amax below g / FLT_MAX
    (g / amax beyond the fp32 range), subnormal bf16 inputs, RHT outputs in the subnormal range, a normal
    block for reference, and blocks near the bf16 maximum (RHT outputs beyond FLT_MAX)."""
    rng = np.random.default_rng(97)
    t = 2.0 ** -126
    ulp = 2.0 ** -131  # bf16 step at 7 * 2^-126 = 1.75 * 2^-124
    rows = []
    for g in (7.0, 6.0):
        for a in (g * t - ulp, g * t, g * t + ulp):
            rows.append([a, -a / 3, a / 5, 0.0, -a, a / 7] + list(rng.uniform(-a, a, 10)))
    for a in (1.5e-38, 2.0e-38, 1.0e-38, 1.2e-38):  # 7 / FLT_MAX = 2.06e-38: g / amax overflows fp32
        rows.append([a, -a, a / 2, 0.0] + list(rng.uniform(-a, a, 12)))
    for a in (9.2e-41, 3e-40, 1e-39, 5e-39):  # subnormal bf16 inputs (and subnormal RHT outputs)
        rows.append(list(rng.uniform(-a, a, 16)))
    rows.append([2.0 ** -124, 2.0 ** -125, -(2.0 ** -127), 2.0 ** -130] + [0.0] * 12)  # sums / 4 below 2^-126
    rows.append([2.0 ** -100, 2.0 ** -127, 2.0 ** -133] + list(rng.uniform(-1e-36, 1e-36, 13)))
    rows.append(list(rng.standard_normal(16)))
    big = (2.0 - 2.0 ** -7) * 2.0 ** 127  # the largest bf16: RHT outputs and E2M1 scales past FLT_MAX
    rows.append([big] * 16)
    rows.append([big, -big, big / 2, 0.0] + list(rng.uniform(-big, big, 12)))
    rows.append(list(rng.uniform(-1, 1, 16) * 2.0 ** 120))
    return _bf16_blocks(rows)


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
@pytest.mark.parametrize("rht", [False, True])
def test_quantizer_full_domain_against_exact_rationals(fmt, rounding, rht):
    """The whole finite bf16 range: tiny blocks (subnormal scales and RHT outputs, g / amax past FLT_MAX) and
    random blocks from 2^-133 to 2^120, every code and scale against `_exact_quant_block`."""
    rng = np.random.default_rng(101 + 4 * fmt + 2 * rounding + rht)
    rand = []
    for _ in range(60):
        base = int(rng.integers(-133, 121))
        e = base - rng.integers(0, 30, size=16)
        m = rng.integers(-255, 256, size=16)
        rand.append([float(Fraction(int(mm)) * Fraction(2) ** int(ee - 7)) for mm, ee in zip(m, e)])
    a = np.concatenate([_edge_blocks(), _bf16_blocks(rand)])
    a = a[np.isfinite(a).all(axis=1)]
    mask, seed = 0x6A09, 12345
    idx, sc = O.quantize_rows(a, fmt, rounding, rht, mask, seed=seed, stream=3)
    u = O.sr_draws(np.zeros((len(a), 1), np.int64), np.arange(len(a))[:, None], seed, 3)[:, 0]
    for r in range(len(a)):
        want, s = _exact_quant_block(a[r], fmt, rounding, rht, mask, u[r])
        assert list(idx[r]) == want, r
        assert sc[r, 0].view(np.uint32) == s.view(np.uint32), r
    assert np.any((sc > 0) & (sc < np.float32(2.0 ** -126)))  # subnormal scales occur


def test_reciprocal_is_rn24_and_equals_fp32_division_where_finite():
    rng = np.random.default_rng(103)
    amax = np.concatenate([np.abs(rng.standard_normal(2000) * 10.0 ** rng.integers(-37, 38, 2000)),
                           [2.0 ** -149, 1e-45, 1e-40, 1.5e-38, 2.0e-38, 2.06e-38, 2.1e-38, 7 * 2.0 ** -126]])
    amax = amax.astype(np.float32)
    amax = amax[amax > 0]
    for g in (7.0, 6.0, 4.0, 2.0):
        r = O.reciprocal_rn24(g, amax)
        for a, got in zip(amax.tolist(), r.tolist()):
            assert Fraction(got) == _round_fraction_sig(Fraction(int(g)) / Fraction(a), 24), (g, a)
        with np.errstate(over="ignore"):
            f32 = np.float32(g) / amax
        fin = np.isfinite(f32)
        assert np.array_equal(r[fin], f32[fin].astype(np.float64))
        assert not fin.all()  # the range contains amax below g / FLT_MAX


def test_tiny_block_codes_match_the_normal_block_they_scale():
    """RN commutes with powers of two: away from subnormal y and scale, a block scaled by 2^k has the same
    codes; scaling a normal block down to amax = 1.5e-38 (g / amax beyond FLT_MAX) keeps its codes."""
    rng = np.random.default_rng(107)
    base = _bf16_blocks(rng.standard_normal((8, 16)) * 4)
    for k in (-100, -120, -124):
        small = (base.astype(np.float64) * 2.0 ** k).astype(np.float32)
        assert np.array_equal(small.astype(np.float64) * 2.0 ** -k, base.astype(np.float64))  # exact scaling
        for fmt in (O.UNIFORM, O.E2M1):
            i0, s0 = O.quantize_rows(base, fmt, O.RTNE, False)
            i1, s1 = O.quantize_rows(small, fmt, O.RTNE, False)
            assert np.array_equal(i0, i1), (k, fmt)
            if k > -120:
                assert np.array_equal(s1.astype(np.float64), s0.astype(np.float64) * 2.0 ** k)


def test_mx_tiny_blocks_take_the_smallest_scale():
    """E8M0 stops at 2^-127: a block with amax < 2^-125 keeps byte 0 and its codes are RTNE(y * 2^127)."""
    rng = np.random.default_rng(109)
    a = _bf16_blocks(rng.uniform(-1, 1, (4, 32)) * np.array([[1e-38], [3e-39], [1e-40], [2.0 ** -124]]))
    idx, e8 = O.quantize_rows_mx(a, O.RTNE, False)
    assert np.all(e8[:3] == 0)
    for r in range(3):
        for i in range(32):
            v = Fraction(float(a[r, i])) * Fraction(2) ** 127
            lo = floor(v)
            k = lo + 1 if v - lo > Fraction(1, 2) or (v - lo == Fraction(1, 2) and lo % 2) else lo
            assert idx[r, i] == max(-7, min(7, k))
    codes, e = _mx_reference_block(a[3])
    assert list(idx[3]) == codes and e8[3, 0] == e


# ------------------------------------------------------------------------------------------------
# Rounding rules (Sec. 2.1) and Shrinkage Bias (Sec. 3.1)
# ------------------------------------------------------------------------------------------------

def test_uniform_rtne_is_rint_and_clip():
    rng = np.random.default_rng(3)
    v = np.concatenate([rng.uniform(-7.6, 7.6, 100000).astype(np.float32),
                        np.arange(-15, 16, dtype=np.float32) / 2,  # every tie
                        np.float32([7.0000005, -7.0000005, 0.0, -0.0])])
    got = O.round_nearest_even(v, O.UNIFORM)
    want = np.clip(np.rint(v.astype(np.float64)), -7, 7).astype(np.int64)
    assert np.array_equal(got, want)


def test_e2m1_rtne_ties_golden():
    rows = _read_table("e2m1_ties.txt")
    v = np.array([float(r[0]) for r in rows], dtype=np.float32)
    want = np.array([float(r[1]) for r in rows])
    got = O.level_values(O.round_nearest_even(v, O.E2M1), O.E2M1)
    assert np.array_equal(got, want)


def test_e2m1_rtne_matches_threshold_search():
    """Nearest level by searching the bin edges (midpoints) -- a different algorithm from the oracle's
    distance argmin; ties resolved by the golden tie table above."""
    mags = np.array([0, .5, 1, 1.5, 2, 3, 4, 6])
    mids = (mags[:-1] + mags[1:]) / 2
    rng = np.random.default_rng(5)
    v = rng.uniform(-7, 7, 200000).astype(np.float32)
    v = v[~np.isin(np.abs(v), mids)]
    idx = np.searchsorted(mids, np.abs(v.astype(np.float64)))
    want = np.where(v < 0, -mags[idx], mags[idx])
    got = O.level_values(O.round_nearest_even(v, O.E2M1), O.E2M1)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("row", _read_table("shrinkage_bias_bins.txt"))
def test_shrinkage_bias_per_bin(row):
    """Eq. (eq:bin-asymmetry-bias) by dense enumeration of a locally uniform density inside each bin."""
    fmt = O.E2M1 if row[0] == "e2m1" else O.UNIFORM
    lo, hi, want = float(row[2]), float(row[3]), float(row[4])
    n = 1 << 20
    t = lo + (hi - lo) * (np.arange(n) + 0.5) / n  # midpoint rule: strictly inside the open bin
    q = O.level_values(O.round_nearest_even(t, fmt), fmt)
    assert np.all(q == float(row[1]))
    assert abs(np.mean(q - t) - want) < 1e-9


def test_shrinkage_bias_uniform_inputs():
    """Uniform inputs over a range ending inside a bin: E2M1 shows a negative mean error, the uniform grid
    none. Over the full range [0, g_max] every grid has zero mean error (trapezoid identity), so the
    range stops at 5: the upper edge of E2M1's (3.5, 5) bin and the middle of the uniform (4.5, 5.5) bin."""
    n = 1 << 21
    t = 5.0 * (np.arange(n) + 0.5) / n
    b_e2m1 = np.mean(O.level_values(O.round_nearest_even(t, O.E2M1), O.E2M1) - t)
    b_uni = np.mean(O.level_values(O.round_nearest_even(t, O.UNIFORM), O.UNIFORM) - t)
    # closed form: the integral of (rho(t) - t) over each bin piece inside [0, 5], divided by 5
    pieces = [(0, 0.25, 0), (0.25, 0.75, .5), (0.75, 1.25, 1), (1.25, 1.75, 1.5), (1.75, 2.5, 2),
              (2.5, 3.5, 3), (3.5, 5.0, 4)]
    want_e2m1 = sum(q * (b - a) - (b * b - a * a) / 2 for a, b, q in pieces) / 5.0
    pieces_u = [(0, .5, 0), (.5, 1.5, 1), (1.5, 2.5, 2), (2.5, 3.5, 3), (3.5, 4.5, 4), (4.5, 5.0, 5)]
    want_uni = sum(q * (b - a) - (b * b - a * a) / 2 for a, b, q in pieces_u) / 5.0
    assert abs(want_uni) < 1e-15
    assert want_e2m1 < -0.05
    # the sample grid straddles bin edges (discontinuities), so the midpoint rule is accurate to ~1e-7
    assert abs(b_e2m1 - want_e2m1) < 1e-6
    assert abs(b_uni - want_uni) < 1e-6


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
def test_sr_exact_expectation(fmt):
    """Sec. 2.1: SR is unbiased. Enumerating all 65536 draws gives E[q] - v in [0, 2^-16 * width)."""
    rng = np.random.default_rng(9)
    g = O.G_MAX[fmt]
    # random values, values whose fraction f makes f * 2^16 an integer (the bias bound is tight there),
    # and tiny values around zero
    v = np.concatenate([rng.uniform(-g, g, 64), [0.3, -0.3, 1e-7, -1e-7, 0.5, -0.5, 0.25, 2.75, -3.125,
                                                 5.5, 1.0 + 2 ** -16]]).astype(np.float32)
    u = np.arange(65536, dtype=np.uint16)
    levels = O._signed_levels(fmt)
    for vi in v:
        q = O.level_values(O.round_stochastic(np.full(65536, vi, np.float32), u, fmt), fmt)
        ia = np.searchsorted(levels, float(vi), side="right") - 1
        ib = min(ia + 1, len(levels) - 1)
        width = levels[ib] - levels[ia] if ib > ia else 1.0
        assert set(np.unique(q)) <= {levels[ia], levels[ib]}
        bias = q.mean() - float(vi)
        assert 0.0 <= bias < width / 65536, (vi, bias)


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
def test_sr_keeps_grid_values(fmt):
    """A value already on the grid has probability 0 of moving (Sec. 2.1: Pr[q = g_b] = 0 at g_a)."""
    u = np.arange(65536, dtype=np.uint16)
    for lv in O._signed_levels(fmt):
        q = O.level_values(O.round_stochastic(np.full(65536, lv, np.float32), u, fmt), fmt)
        assert np.all(q == lv)


def test_philox_draw_bits_balanced():
    """Every bit of every draw position is a fair coin over many blocks (catches a lost or swapped bit
    in the extraction of 16-bit draws from the Philox words)."""
    u = O.sr_draws(np.arange(1 << 14)[:, None], np.arange(2)[None, :], seed=0x0123456789ABCDEF, stream=0)
    u = u.reshape(-1, 16).astype(np.uint32)
    n = u.shape[0]
    for bit in range(16):
        frac = ((u >> np.uint32(bit)) & np.uint32(1)).mean(axis=0)
        assert np.all(np.abs(frac - 0.5) < 5 * 0.5 / np.sqrt(n)), bit


def test_sr_statistical_mean_with_philox_draws():
    rng = np.random.default_rng(1)
    v = rng.uniform(-7, 7, 8).astype(np.float32)
    n_blocks = 1 << 13
    u = O.sr_draws(np.arange(n_blocks)[:, None], np.zeros((1, 1), np.int64), seed=1234, stream=3)
    u = u.reshape(-1)  # 131072 draws
    for vi in v:
        q = O.level_values(O.round_stochastic(np.full(u.size, vi, np.float32), u, O.UNIFORM), O.UNIFORM)
        f = float(vi) - np.floor(float(vi))
        sigma = np.sqrt(f * (1 - f) / u.size) + 1e-12
        assert abs(q.mean() - float(vi)) < 4.5 * sigma + 2 ** -16


def test_philox_draws_uniform_histogram():
    u = O.sr_draws(np.arange(4096)[:, None], np.arange(8)[None, :], seed=0xDEADBEEF12345678, stream=1)
    hist = np.bincount((u.reshape(-1) >> 12).astype(np.int64), minlength=16)
    expected = u.size / 16
    chi2 = np.sum((hist - expected) ** 2 / expected)
    assert chi2 < 60  # 15 degrees of freedom; p ~ 1e-7


def _build_rocrand_philox(tmp):
    src = os.path.join(tmp, "philox_ref.cpp")
    exe = os.path.join(tmp, "philox_ref")
    with open(src, "w") as f:
        f.write(
            "#include <hip/hip_runtime.h>\n#include <rocrand/rocrand_philox4x32_10.h>\n#include <cstdio>\n"
            "struct E : rocrand_device::philox4x32_10_engine {\n"
            "  uint4 raw(uint4 c, uint2 k) { return ten_rounds(c, k); } };\n"
            "int main() { E e; unsigned a[6];\n"
            "  while (scanf(\"%x %x %x %x %x %x\", a, a+1, a+2, a+3, a+4, a+5) == 6) {\n"
            "    uint4 o = e.raw(make_uint4(a[0], a[1], a[2], a[3]), make_uint2(a[4], a[5]));\n"
            "    printf(\"%08x %08x %08x %08x\\n\", o.x, o.y, o.z, o.w); } return 0; }\n")
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    subprocess.run(["g++", "-O1", "-D__HIP_PLATFORM_AMD__", f"-I{rocm}/include", src, "-o", exe],
                   check=True, capture_output=True)
    return exe


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.exists("/opt/rocm/include/rocrand"),
                    reason="needs g++ and the rocRAND headers")
def test_philox_matches_rocrand():
    """Philox4x32-10 against rocRAND's independent implementation (its engine's ten-round function)."""
    rng = np.random.default_rng(2024)
    ctr = rng.integers(0, 2 ** 32, size=(500, 4), dtype=np.uint64)
    key = rng.integers(0, 2 ** 32, size=(500, 2), dtype=np.uint64)
    ctr[0] = 0
    key[0] = 0
    ctr[1] = 0xFFFFFFFF
    key[1] = 0xFFFFFFFF
    with tempfile.TemporaryDirectory() as tmp:
        exe = _build_rocrand_philox(tmp)
        inp = "\n".join(" ".join(f"{int(v):x}" for v in list(c) + list(k)) for c, k in zip(ctr, key))
        out = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True).stdout.split()
    ref = np.array([int(w, 16) for w in out], dtype=np.uint64).reshape(-1, 4)
    for i in range(len(ctr)):
        got = O.philox4x32_10(ctr[i, 0], ctr[i, 1], ctr[i, 2], ctr[i, 3], key[i, 0], key[i, 1])
        assert [int(w) for w in got] == [int(w) for w in ref[i]], i


# ------------------------------------------------------------------------------------------------
# Quantizer (Sec. 2.1 display) -- invariants and brute force
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
@pytest.mark.parametrize("rht", [False, True])
def test_quantizer_invariants(fmt, rht):
    rng = np.random.default_rng(17)
    a = O.bf16_bits_to_f32(_rand_bf16_bits(rng, (64, 256)))
    a[3, 16:32] = 0.0  # a zero block
    idx, s = O.quantize_rows(a, fmt, O.RTNE, rht, 0x1234)
    g = O.G_MAX[fmt]
    y = O.rht_blocks(a.reshape(64, 16, 16), 0x1234) if rht else a.reshape(64, 16, 16)
    amax = np.abs(y).max(-1)
    assert np.array_equal(s, (amax / np.float32(g)).astype(np.float32))
    assert s[3, 1] == 0 and np.all(idx[3, 16:32] == 0)
    blocks = idx.reshape(64, 16, 16)
    lv = O.level_values(blocks, fmt)
    nz = amax > 0
    # the amax element carries the top level, with its sign
    am = np.abs(y).argmax(-1)
    top = np.take_along_axis(lv, am[..., None], -1)[..., 0]
    sgn = np.sign(np.take_along_axis(y, am[..., None], -1)[..., 0])
    assert np.all(top[nz] == g * sgn[nz])
    if fmt == O.UNIFORM:
        err = np.abs(lv * s[..., None].astype(np.float64) - y.astype(np.float64))
        assert np.all(err <= s[..., None] * (0.5 + 2 ** -20) + 1e-30)


def test_quantizer_bruteforce_tiny_blocks():
    """Every element's level is the nearest of all 15 signed levels to y/s, found with exact rationals."""
    rng = np.random.default_rng(23)
    for fmt in (O.UNIFORM, O.E2M1):
        levels = [Fraction(float(x)) for x in O._signed_levels(fmt)]
        mags = list(O.GRID_MAGNITUDES[fmt])
        for trial in range(40):
            a = O.bf16_bits_to_f32(_rand_bf16_bits(rng, (1, 16), scale=10.0 ** rng.uniform(-3, 3)))
            idx, s = O.quantize_rows(a, fmt, O.RTNE, trial % 2 == 1, trial * 977)
            y = O.rht_blocks(a.reshape(1, 1, 16), trial * 977)[0, 0] if trial % 2 else a[0]
            g = np.float32(O.G_MAX[fmt])
            r = g / np.abs(y).max()
            for i in range(16):
                v = Fraction(float(np.float32(y[i] * r)))
                d = [abs(v - L) for L in levels]
                best = min(d)
                cands = [L for L, dd in zip(levels, d) if dd == best]
                if len(cands) > 1:  # tie: even magnitude code
                    cands = [L for L in cands if mags.index(abs(float(L))) % 2 == 0]
                assert O.level_values(idx[0, i], fmt) == float(cands[0])


def test_sr_quantizer_uses_counter_draws_and_is_reproducible():
    rng = np.random.default_rng(29)
    a = O.bf16_bits_to_f32(_rand_bf16_bits(rng, (8, 64)))
    i1, s1 = O.quantize_rows(a, O.UNIFORM, O.SR, True, 0x55, seed=99, stream=0)
    i2, s2 = O.quantize_rows(a, O.UNIFORM, O.SR, True, 0x55, seed=99, stream=0)
    i3, _ = O.quantize_rows(a, O.UNIFORM, O.SR, True, 0x55, seed=99, stream=1)
    assert np.array_equal(i1, i2) and np.array_equal(s1, s2)
    assert not np.array_equal(i1, i3)
    # rows quantized alone, with their global row ids, give the same codes (counters are global)
    i4, _ = O.quantize_rows(a[5:7], O.UNIFORM, O.SR, True, 0x55, seed=99, stream=0, row_ids=[5, 6])
    assert np.array_equal(i4, i1[5:7])


def test_pack_unpack_roundtrip_and_bit_patterns():
    rng = np.random.default_rng(31)
    for fmt in (O.UNIFORM, O.E2M1):
        idx = rng.integers(-7, 8, size=(5, 32))
        p = O.pack_codes(idx, fmt)
        assert p.shape == (5, 16)
        assert np.array_equal(O.unpack_codes(p, fmt), idx)
    one = np.array([[-1, 7, -7, 0]])
    assert list(O.pack_codes(one, O.UNIFORM)[0]) == [0x79, 0x0F]  # -1 -> 0x9, 7 -> 0x7, -7 -> 0xF, 0 -> 0x0
    e = np.array([[-7, 7, -1, 0]])  # E2M1: -6 -> 0xF, 6 -> 0x7, -0.5 -> 0x9, 0 -> 0x0
    assert list(O.pack_codes(e, O.E2M1)[0]) == [0x7F, 0x09]


def test_colwise_is_rowwise_of_transpose():
    rng = np.random.default_rng(37)
    t = _rand_bf16_bits(rng, (64, 48))
    a = O.operand_colwise(t)
    b = O.bf16_bits_to_f32(np.ascontiguousarray(t.T))
    assert np.array_equal(a, b)
    i1, s1 = O.quantize_rows(a, O.UNIFORM, O.SR, True, 7, seed=5, stream=1)
    i2, s2 = O.quantize_rows(b, O.UNIFORM, O.SR, True, 7, seed=5, stream=1)
    assert np.array_equal(i1, i2) and np.array_equal(s1, s2)


@pytest.mark.parametrize("fmt", [O.UNIFORM, O.E2M1])
def test_both_operands_of_one_tensor(fmt):
    """quantize_both: a symmetric tensor gives the same operand both ways, and the transposed output of T
    is the rowwise output of T^T (with the settings swapped)."""
    rng = np.random.default_rng(41)
    a = rng.standard_normal((48, 48)).astype(np.float32)
    sym = O.f32_to_bf16_bits(a + a.T)
    (ir, sr), (ic, scol) = O.quantize_both(sym, fmt, O.SR, True, True, 0x1234, 0x1234, seed=9, stream_rows=3,
                                           stream_cols=3)
    assert np.array_equal(ir, ic) and np.array_equal(sr, scol)
    t = _rand_bf16_bits(rng, (32, 80))
    (ir, sr), (ic, scol) = O.quantize_both(t, fmt, O.SR, False, True, 0x00F0, 0xBEEF, seed=4, stream_rows=0,
                                           stream_cols=1)
    assert ir.shape == (32, 80) and ic.shape == (80, 32)
    tt = np.ascontiguousarray(t.T)
    (jr, tr), (jc, tc) = O.quantize_both(tt, fmt, O.SR, True, False, 0xBEEF, 0x00F0, seed=4, stream_rows=1,
                                         stream_cols=0)
    assert np.array_equal(ic, jr) and np.array_equal(scol, tr)
    assert np.array_equal(ir, jc) and np.array_equal(sr, tc)
    # different streams give different SR draws: the two outputs of a symmetric tensor then differ
    (ir, _), (ic, _) = O.quantize_both(sym, fmt, O.SR, True, True, 0x1234, 0x1234, seed=9, stream_rows=0,
                                       stream_cols=1)
    assert not np.array_equal(ir, ic)


# ------------------------------------------------------------------------------------------------
# GEMMs (Sec. 2.2)
# ------------------------------------------------------------------------------------------------

def test_gemm_integer_special_case():
    """Power-of-two scales: the dequantized product is an exactly representable integer matmul."""
    rng = np.random.default_rng(41)
    a = rng.integers(-7, 8, size=(24, 64))
    b = rng.integers(-7, 8, size=(40, 64))
    sa = (2.0 ** rng.integers(-6, 6, size=(24, 4))).astype(np.float32)
    sb = (2.0 ** rng.integers(-6, 6, size=(40, 4))).astype(np.float32)
    got = O.gemm_nt(a, sa, b, sb, O.UNIFORM)
    want = np.zeros((24, 40))
    for kb in range(4):
        blk = slice(16 * kb, 16 * kb + 16)
        want += (a[:, blk] @ b[:, blk].T) * np.outer(sa[:, kb], sb[:, kb])
    assert np.array_equal(got, want)


def test_gemm_bruteforce_fractions():
    rng = np.random.default_rng(43)
    for fmt in (O.UNIFORM, O.E2M1):
        a = rng.integers(-7, 8, size=(3, 32))
        b = rng.integers(-7, 8, size=(4, 32))
        sa = rng.uniform(0.01, 2, size=(3, 2)).astype(np.float32)
        sb = rng.uniform(0.01, 2, size=(4, 2)).astype(np.float32)
        got = O.gemm_nt(a, sa, b, sb, fmt)
        lv = {i: Fraction(float(O.level_values(np.array(i), fmt))) for i in range(-7, 8)}
        for i in range(3):
            for j in range(4):
                acc = sum(lv[a[i, k]] * Fraction(float(sa[i, k // 16])) * lv[b[j, k]] * Fraction(float(sb[j, k // 16]))
                          for k in range(32))
                assert abs(got[i, j] - float(acc)) <= 1e-14 * max(1.0, abs(float(acc)))


def test_grouped_padding_keeps_products():
    """Zero-padding each group's token axis to a multiple of 16 leaves X_g^T dY_g unchanged, with and
    without the rotation (Sec. 2.2 invariance)."""
    rng = np.random.default_rng(47)
    counts = [5, 16, 33, 0, 19]
    mtot = sum(counts)
    x = _rand_bf16_bits(rng, (mtot, 32))
    dy = _rand_bf16_bits(rng, (mtot, 24))
    ax, poff = O.operand_colwise_grouped(x, counts)
    ad, poff2 = O.operand_colwise_grouped(dy, counts)
    assert np.array_equal(poff, poff2) and list(np.diff(poff)) == [16, 16, 48, 0, 32]
    xf, df = O.bf16_bits_to_f32(x).astype(np.float64), O.bf16_bits_to_f32(dy).astype(np.float64)

    def rot(a):
        r, c = a.shape
        return O.rht_exact_f64(a.reshape(r, c // 16, 16).astype(np.float64), 0xBEEF).reshape(r, c)

    rx, rd = rot(ax), rot(ad)
    off = 0
    for gi, c in enumerate(counts):
        cols = slice(int(poff[gi]), int(poff[gi + 1]))
        ref = df[off:off + c].T @ xf[off:off + c]
        assert np.allclose(ad[:, cols].astype(np.float64) @ ax[:, cols].T.astype(np.float64), ref, rtol=0, atol=1e-12)
        if c:
            assert np.linalg.norm(rd[:, cols] @ rx[:, cols].T - ref) <= 1e-13 * np.linalg.norm(ref)
        off += c


@pytest.mark.parametrize("recipe", ["ufp4", "e2m1"])
def test_layer_gemms_approximate_exact_products(recipe):
    rng = np.random.default_rng(53)
    x = _rand_bf16_bits(rng, (64, 128))
    w = _rand_bf16_bits(rng, (96, 128))
    dy = _rand_bf16_bits(rng, (64, 96))
    q, out = O.layer_gemms(x, w, dy, recipe, sign_mask=0x2F1D, seed=3)
    xf, wf, df = (O.bf16_bits_to_f32(t).astype(np.float64) for t in (x, w, dy))
    for key, ref in (("y", xf @ wf.T), ("dx", df @ wf), ("dw", df.T @ xf)):
        assert out[key].shape == ref.shape
        assert O.sqnr_db(out[key], ref) > 12.0, key
    assert q["wt"][0].shape == (128, 96) and q["dyt"][0].shape == (96, 64) and q["xt"][0].shape == (128, 64)


@pytest.mark.parametrize("recipe", [r for r in O.RECIPES if r not in ("ufp4", "e2m1", "mxufp4")])
def test_recipe_variants(recipe):
    """Every ablation recipe still approximates the exact products, and its operands follow its switches:
    an operand is the plain quantization with the recipe's RHT flag, grid, rounding and stream."""
    rng = np.random.default_rng(57)
    x = _rand_bf16_bits(rng, (128, 128))
    w = _rand_bf16_bits(rng, (128, 128))
    dy = _rand_bf16_bits(rng, (128, 128))
    q, out = O.layer_gemms(x, w, dy, recipe, sign_mask=0x2F1D, seed=3)
    xf, wf, df = (O.bf16_bits_to_f32(t).astype(np.float64) for t in (x, w, dy))
    for key, ref in (("y", xf @ wf.T), ("dx", df @ wf), ("dw", df.T @ xf)):
        assert O.sqnr_db(out[key], ref) > 8.0, key
    cfg = O.RECIPES[recipe]
    rnd = O.SR if "dyt" in cfg.get("sr", ("dy", "dyt")) else O.RTNE
    n = cfg.get("rht_block", 16)
    mask = sum(0x2F1D << (16 * k) for k in range(n // 16))
    want = O.quantize_rows(O.operand_colwise(dy), cfg["fmt"], rnd, cfg["rht"][2], mask, 3, 1,
                           max_fpx=cfg.get("max_fpx"), rht_block=n)
    assert np.array_equal(q["dyt"][0], want[0]) and np.array_equal(q["dyt"][1], want[1])


def test_diagnostics_closed_forms():
    a = np.array([[1.0, 2.0], [3.0, 4.0]])
    assert O.operand_projection(0.9 * a, a) == pytest.approx(0.9)
    assert O.sqnr_db(1.1 * a, a) == pytest.approx(20.0)
    idx = np.array([[0, 1, 2, 3, 4, 5, 6, 7]])
    assert O.effective_bucket_ratio(idx, O.UNIFORM) == pytest.approx(1.0, abs=1e-9)
    assert O.effective_bucket_ratio(np.zeros((1, 8), np.int64), O.UNIFORM) == pytest.approx(1 / 8, abs=1e-9)


def _one_block(vals):
    row = np.zeros((1, 16), np.float32)
    row[0, :len(vals)] = vals
    return row


def test_quant_stats_hand_computed_blocks():
    """Sums worked out by hand for single 16-blocks (no RHT, scale 1 so that v = x)."""
    # uniform: 7, 3.375, -1.625 -> codes 7, 3, -2 (s = 7/7 = 1)
    st = O.quant_stats(_one_block([7.0, 3.375, -1.625]), O.UNIFORM, O.RTNE, False)
    assert st["err2"] == 0.28125 and st["ref2"] == 63.03125 and st["cross"] == 62.375
    assert st["hist"].tolist() == [13, 0, 1, 1, 0, 0, 0, 1]
    # E2M1: 6, 2.5, -0.75 -> 6, 2 (tie to the even code 4), -1 (tie to the even code 2)
    st = O.quant_stats(_one_block([6.0, 2.5, -0.75]), O.E2M1, O.RTNE, False)
    assert st["err2"] == 0.3125 and st["ref2"] == 42.8125 and st["cross"] == 41.75
    assert st["hist"].tolist() == [13, 0, 1, 0, 1, 0, 0, 1]
    # E2M1 cut at max_fpx = 2: s = 3, v = 2, 0.8333334, -0.25 -> 2 (code 4), 1 (code 2), 0 (tie to code 0)
    st = O.quant_stats(_one_block([6.0, 2.5, -0.75]), O.E2M1, O.RTNE, False, max_fpx=2)
    assert st["err2"] == 0.8125 and st["cross"] == 43.5
    assert st["hist"].tolist() == [14, 0, 1, 0, 1, 0, 0, 0]


def test_quant_stats_on_grid_input_is_lossless():
    """Blocks whose values are k * 2^e with max |k| = 7 quantize exactly: NMSE 0, alpha 1 (RTNE and SR)."""
    rng = np.random.default_rng(61)
    k = rng.integers(-7, 8, size=(24, 64)).astype(np.float64)
    k[:, ::16] = 7.0  # every block reaches the top level
    a = (k * np.exp2(rng.integers(-6, 7, size=(24, 4)).repeat(16, axis=1))).astype(np.float32)
    for rnd in (O.RTNE, O.SR):
        st = O.quant_stats(a, O.UNIFORM, rnd, False, seed=5)
        m = O.stats_metrics(st, O.UNIFORM)
        assert st["err2"] == 0.0 and m["alpha"] == 1.0
        assert st["hist"].tolist() == np.bincount(np.abs(k).astype(np.int64).ravel(), minlength=8).tolist()


def test_quant_stats_sums_are_consistent():
    """||q - r||^2 = ||q||^2 - 2 <q, r> + ||r||^2 with ||q||^2 taken from the dequantized operand; counts add up."""
    rng = np.random.default_rng(62)
    a = O.bf16_bits_to_f32(_rand_bf16_bits(rng, (48, 96)))
    for fmt, mf in ((O.UNIFORM, None), (O.E2M1, None), (O.E2M1, 4.0)):
        for rht in (False, True):
            st = O.quant_stats(a, fmt, O.SR, rht, 0x5A5A, seed=9, stream=1, max_fpx=mf)
            idx, sc = O.quantize_rows(a, fmt, O.SR, rht, 0x5A5A, 9, 1, max_fpx=mf)
            q2 = float(np.sum(O.dequantize(idx, sc, fmt) ** 2))
            assert st["err2"] == pytest.approx(q2 - 2 * st["cross"] + st["ref2"], rel=1e-9)
            assert int(st["hist"].sum()) == a.size


def test_stats_metrics_closed_forms():
    st = {"err2": 1.0, "ref2": 100.0, "cross": 90.0, "hist": np.array([4, 4, 4, 4, 4, 4, 4, 4])}
    m = O.stats_metrics(st, O.UNIFORM)
    assert m["nmse"] == 0.01 and m["sqnr_db"] == pytest.approx(20.0) and m["alpha"] == 0.9
    assert m["beff"] == pytest.approx(1.0, abs=1e-9)
    # the cut grid has K = 5 buckets; all mass in one of them gives 1/5
    st = {"err2": 0.0, "ref2": 1.0, "cross": 1.0, "hist": np.array([0, 0, 7, 0, 0, 0, 0, 0])}
    assert O.stats_metrics(st, O.E2M1, max_fpx=2)["beff"] == pytest.approx(1 / 5, abs=1e-9)
    assert O.delta_sqnr_db(0.01, 0.001) == pytest.approx(10.0)


# ------------------------------------------------------------------------------------------------
# Range-restricted E2M1 (Sec. 5 Q4: max_fpx in {2, 4, 6})
# ------------------------------------------------------------------------------------------------

def test_max_fpx_six_is_the_plain_e2m1_grid():
    rng = np.random.default_rng(63)
    a = O.bf16_bits_to_f32(_rand_bf16_bits(rng, (16, 64)))
    for rnd in (O.RTNE, O.SR):
        i0, s0 = O.quantize_rows(a, O.E2M1, rnd, True, 0x0F0F, 4, 0)
        i1, s1 = O.quantize_rows(a, O.E2M1, rnd, True, 0x0F0F, 4, 0, max_fpx=6)
        assert np.array_equal(i0, i1) and np.array_equal(s0, s1)


def test_max_fpx_levels_and_ties():
    assert O.grid_magnitudes(O.E2M1, 2).tolist() == [0.0, 0.5, 1.0, 1.5, 2.0]
    assert O.grid_magnitudes(O.E2M1, 4).tolist() == [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0]
    v = np.array([1.25, 1.75, -0.25, 2.6, 3.5, 5.0, -7.0], np.float32)
    assert O.round_nearest_even(v, O.E2M1, 2).tolist() == [2, 4, 0, 4, 4, 4, -4]
    assert O.round_nearest_even(v, O.E2M1, 4).tolist() == [2, 4, 0, 5, 6, 6, -6]
    assert O.round_nearest_even(v, O.E2M1).tolist() == [2, 4, 0, 5, 6, 6, -7]
    with pytest.raises(ValueError):
        O.grid_magnitudes(O.UNIFORM, 4)
    with pytest.raises(ValueError):
        O.grid_magnitudes(O.E2M1, 3)


def test_max_fpx_sr_is_exhaustively_unbiased_and_stays_on_the_cut_grid():
    """Over all 2^16 draws: the mean of SR equals v (v a multiple of 2^-16 of the bin), and no draw leaves
    the restricted grid, also 1 ulp above its top level."""
    u = np.arange(65536, dtype=np.uint32)
    for mf, v in ((4.0, 3.25), (4.0, -3.75), (2.0, 1.125), (2.0, -0.375)):
        q = O.level_values(O.round_stochastic(np.full(65536, v, np.float32), u, O.E2M1, mf), O.E2M1)
        assert q.mean() == v
    for mf in (2.0, 4.0):
        top = np.nextafter(np.float32(mf), np.float32(10.0))
        q = O.level_values(O.round_stochastic(np.full(65536, top, np.float32), u, O.E2M1, mf), O.E2M1)
        assert set(q.tolist()) == {mf}


def test_max_fpx_on_grid_block_is_reproduced():
    """A block on the cut grid with |x| reaching max_fpx * 2^e quantizes exactly with s = 2^e."""
    for mf in (2.0, 4.0):
        lv = O.grid_magnitudes(O.E2M1, mf)
        vals = np.concatenate([lv, -lv[1:]])[:16]
        row = np.zeros((1, 16), np.float32)
        row[0, :len(vals)] = vals * 0.125
        idx, sc = O.quantize_rows(row, O.E2M1, O.RTNE, False, max_fpx=mf)
        assert sc[0, 0] == np.float32(0.125)
        assert np.array_equal(O.dequantize(idx, sc, O.E2M1), row.astype(np.float64))


# ------------------------------------------------------------------------------------------------
# RHT blocks of 32 / 64 / 128 (Appendix search space: RHT block size)
# ------------------------------------------------------------------------------------------------

def _rn32(fr: Fraction) -> np.float32:
    """The fp32 number nearest to an exact rational, ties to the even significand."""
    c = np.float32(float(fr))
    cands = [np.nextafter(c, np.float32(-np.inf)), c, np.nextafter(c, np.float32(np.inf))]
    return min(cands, key=lambda v: (abs(Fraction(float(v)) - fr), int(np.float32(v).view(np.uint32)) & 1))


def test_rht_n_matrix_is_scipys_sylvester_hadamard():
    import scipy.linalg

    for n in O.RHT_BLOCKS:
        assert np.array_equal(O.hadamard_pm1(n), scipy.linalg.hadamard(n).astype(np.float64))
    assert O.rht_norm(16) == 0.25 and O.rht_norm(64) == 0.125


def test_rht_n_of_a_unit_vector_and_block_16():
    """e_0 without signs -> every output is RN32(1/sqrt(n)); n = 16 reduces to the block-16 RHT."""
    for n in (32, 64, 128):
        a = np.zeros((1, n), np.float32)
        a[0, 0] = 1.0
        y = O.rht_rows_n(a, 0, n)
        assert np.all(y == np.float32(1.0 / np.sqrt(n)))
        # a sign flip on position 0 flips every output
        assert np.all(O.rht_rows_n(a, 1, n) == -y)
    rng = np.random.default_rng(71)
    a = O.bf16_bits_to_f32(_rand_bf16_bits(rng, (8, 64)))
    assert np.array_equal(O.rht_rows_n(a, 0x9A3C, 16), O.rht_blocks(a.reshape(8, 4, 16), 0x9A3C).reshape(8, 64))


def test_rht_n_is_orthogonal_and_matches_exact_rationals():
    """Parseval within fp32 rounding; for n = 64 (power-of-two normalisation) every output equals the exact
    rational sum rounded once to fp32."""
    rng = np.random.default_rng(72)
    for n in (32, 64, 128):
        a = O.bf16_bits_to_f32(_rand_bf16_bits(rng, (6, 2 * n)))
        mask = int(rng.integers(0, 2 ** 62)) | (int(rng.integers(0, 2 ** 62)) << 62)
        mask &= (1 << n) - 1
        y = O.rht_rows_n(a, mask, n).astype(np.float64)
        xb = a.astype(np.float64).reshape(6, 2, n)
        yb = y.reshape(6, 2, n)
        assert np.allclose((yb ** 2).sum(-1), (xb ** 2).sum(-1), rtol=1e-6)
        if n == 64:
            for r in range(2):
                for i in (0, 5, 63):
                    tot = sum(Fraction(float(xb[r, 0, j])) * (-1 if (mask >> j) & 1 else 1)
                              * (-1 if bin(i & j).count("1") % 2 else 1) for j in range(n)) / 8
                    assert _rn32(tot) == np.float32(y[r, i])


def test_quantize_rows_with_rht_block_n():
    """rht_block = n quantizes the 16-blocks of the n-point transform; n = 16 is the default path."""
    rng = np.random.default_rng(73)
    a = O.bf16_bits_to_f32(_rand_bf16_bits(rng, (10, 128)))
    i16, s16 = O.quantize_rows(a, O.UNIFORM, O.SR, True, 0x77, 3, 0)
    j16, t16 = O.quantize_rows(a, O.UNIFORM, O.SR, True, 0x77, 3, 0, rht_block=16)
    assert np.array_equal(i16, j16) and np.array_equal(s16, t16)
    for n in (32, 64, 128):
        y = O.rht_rows_n(a, 0x123456789, n)
        want = O.quantize_rows(y, O.UNIFORM, O.RTNE, False)
        got = O.quantize_rows(a, O.UNIFORM, O.RTNE, True, 0x123456789, rht_block=n)
        assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])
    with pytest.raises(ValueError):
        O.quantize_rows(a[:, :48], O.UNIFORM, O.RTNE, True, 0, rht_block=32)


# ------------------------------------------------------------------------------------------------
# Uniform grid with power-of-two block scales (Sec. 4: scale hierarchy chosen for the hardware)
# ------------------------------------------------------------------------------------------------

def test_mx_scale_exponent_follows_the_ocp_shared_exponent_rule():
    """E = floor(log2 amax) - 2, checked with exact rationals: 4 * 2^E <= amax < 8 * 2^E."""
    rng = np.random.default_rng(51)
    amax = np.concatenate([
        (rng.standard_normal(4000) * 10.0 ** rng.integers(-30, 30, 4000)).astype(np.float32),
        np.float32([7.0, 3.5, 14.0, 1.0, 0.875, 4.0, 8.0, 7 * 2.0 ** -100, 3.4e38]),
        np.nextafter(np.float32([4.0, 8.0, 1.0]), np.float32(np.inf)),
        np.nextafter(np.float32([4.0, 8.0, 1.0]), np.float32(0)),
    ])
    amax = np.abs(amax)
    amax = amax[amax > 0]
    E = O.mx_scale_exponent(amax)
    for a, e in zip(amax.tolist(), E.tolist()):
        fa = Fraction(a)
        two_e = Fraction(2) ** e
        assert 4 * two_e <= fa < 8 * two_e, (a, e)
    assert O.mx_scale_exponent(np.float32([0.0]))[0] == -127


def test_e2m3_format_against_the_ocp_definition():
    # values fixed by the OCP Microscaling formats specification for FP6 E2M3
    assert O.e2m3_value(0b011111) == 7.5  # largest normal
    assert O.e2m3_value(0b001000) == 1.0
    assert O.e2m3_value(0b000001) == 0.125  # smallest subnormal
    assert O.e2m3_value(0b111111) == -7.5
    assert O.e2m3_value(0b010000) == 2.0
    k = np.arange(-7, 8)
    assert np.array_equal(O.e2m3_value(O.e2m3_codes(k)), k)
    assert O.e2m3_codes(np.array([0]))[0] == 0  # zero as +0


def test_fp6_packing_bit_positions_and_roundtrip():
    rng = np.random.default_rng(52)
    idx = rng.integers(-7, 8, size=(5, 96))
    p = O.pack_fp6(idx)
    assert p.shape == (5, 72)
    assert np.array_equal(O.unpack_fp6(p), idx)
    one = np.zeros((1, 32), dtype=np.int64)
    for j in (0, 1, 5, 21, 31):
        one[:] = 0
        one[0, j] = -1  # E2M3 -1 = 0b101000
        bits = int.from_bytes(O.pack_fp6(one)[0].tobytes(), "little")
        assert bits == 0b101000 << (6 * j)


def _mx_reference_block(y, u=None):
    """One 32-block by exact rationals: 2^E with 4 * 2^E <= amax < 8 * 2^E found by search, v = y / 2^E,
    then the nearest integer (ties to even) or the SR rule with 16-bit draws, clamped to [-7, 7]."""
    ys = [Fraction(float(t)) for t in y]
    amax = max(abs(t) for t in ys)
    if amax == 0:
        return [0] * len(ys), 0
    e = 0
    while 8 * Fraction(2) ** e <= amax:
        e += 1
    while 4 * Fraction(2) ** e > amax:
        e -= 1
    codes = []
    for i, t in enumerate(ys):
        v = min(max(t / Fraction(2) ** e, Fraction(-7)), Fraction(7))
        lo = floor(v)
        if u is None:
            frac = v - lo
            k = lo + 1 if frac > Fraction(1, 2) or (frac == Fraction(1, 2) and lo % 2 == 1) else lo
        else:
            k = lo + 1 if Fraction(int(u[i]), 65536) < v - lo else lo
        codes.append(max(-7, min(7, k)))
    return codes, e + 127


@pytest.mark.parametrize("rounding", [O.RTNE, O.SR])
def test_mx_quantizer_against_exact_rationals(rounding):
    rng = np.random.default_rng(53 + rounding)
    rows = 6
    a = (rng.standard_normal((rows, 64)) * np.exp(rng.standard_normal((rows, 1)) * 3)).astype(np.float32)
    a[1, :32] = 0.0  # a zero block
    a[2, 5] = 7.0 * 2.0 ** -3  # an exact top level
    a = O.bf16_bits_to_f32(O.f32_to_bf16_bits(a))
    idx, e8 = O.quantize_rows_mx(a, rounding, False, seed=7, stream=2)
    u = O.sr_draws(np.arange(4)[None, :], np.arange(rows)[:, None], 7, 2).reshape(rows, 2, 32)
    for r in range(rows):
        for b in range(2):
            codes, e = _mx_reference_block(a[r, 32 * b:32 * b + 32], None if rounding == O.RTNE else u[r, b])
            assert list(idx[r, 32 * b:32 * b + 32]) == codes, (r, b)
            if e:
                assert e8[r, b] == e


def test_mx_quantizer_invariants_with_rht():
    rng = np.random.default_rng(54)
    a = O.bf16_bits_to_f32(_rand_bf16_bits(rng, (16, 128), 3.0))
    idx, e8 = O.quantize_rows_mx(a, O.RTNE, True, sign_mask=0x5A5A)
    y = O.rht_blocks(a.reshape(16, 8, 16), 0x5A5A).reshape(16, 4, 32).astype(np.float64)
    s = np.ldexp(1.0, e8.astype(np.int64) - 127)
    top = np.abs(idx.reshape(16, 4, 32)).max(axis=-1)
    assert np.all((top >= 4) & (top <= 7))  # amax / 2^E lies in [4, 8): the top code is 4..7
    err = np.abs(idx.reshape(16, 4, 32) * s[..., None] - y)
    clipped = np.abs(y) > 7.5 * s[..., None]
    assert np.all(err[~clipped] <= s[..., None].repeat(32, -1)[~clipped] / 2)  # RTNE: within half a step
    assert np.all(err[clipped] <= s[..., None].repeat(32, -1)[clipped])  # clamped top values: within a step


def test_mx_gemm_special_cases():
    rng = np.random.default_rng(55)
    a = rng.integers(-7, 8, size=(5, 64))
    b = rng.integers(-7, 8, size=(3, 64))
    ones_a = np.full((5, 2), 127, np.uint8)
    ones_b = np.full((3, 2), 127, np.uint8)
    assert np.array_equal(O.gemm_nt_mx(a, ones_a, b, ones_b), (a @ b.T).astype(np.float64))
    ea = rng.integers(120, 135, size=(5, 2)).astype(np.uint8)
    eb = rng.integers(120, 135, size=(3, 2)).astype(np.uint8)
    c = O.gemm_nt_mx(a, ea, b, eb)
    for i in range(5):
        for j in range(3):
            want = sum(Fraction(int(a[i, k])) * Fraction(2) ** (int(ea[i, k // 32]) - 127) * int(b[j, k])
                       * Fraction(2) ** (int(eb[j, k // 32]) - 127) for k in range(64))
            assert c[i, j] == float(want)


def test_grouped_padding_to_32_for_power_of_two_scales():
    """With power-of-two 1x32 scales the token axis is padded per group to a multiple of 32: the padded lengths,
    no 32-block straddling two groups, zero padding, and per-group products unchanged by it."""
    rng = np.random.default_rng(48)
    counts = [5, 16, 33, 0, 19, 32]
    mtot = sum(counts)
    x = _rand_bf16_bits(rng, (mtot, 64))
    dy = _rand_bf16_bits(rng, (mtot, 32))
    ax, poff = O.operand_colwise_grouped(x, counts, block=32)
    ad, _ = O.operand_colwise_grouped(dy, counts, block=32)
    assert list(np.diff(poff)) == [32, 32, 64, 0, 32, 32] and all(p % 32 == 0 for p in poff)
    xf, df = O.bf16_bits_to_f32(x).astype(np.float64), O.bf16_bits_to_f32(dy).astype(np.float64)
    off = 0
    for gi, c in enumerate(counts):
        lo, hi = int(poff[gi]), int(poff[gi + 1])
        assert not np.any(ax[:, lo + c:hi]) and not np.any(ad[:, lo + c:hi])  # the padding is zero
        assert np.array_equal(ax[:, lo:lo + c], O.bf16_bits_to_f32(x)[off:off + c].T)
        ref = df[off:off + c].T @ xf[off:off + c]
        assert np.allclose(ad[:, lo:hi].astype(np.float64) @ ax[:, lo:hi].T.astype(np.float64), ref, rtol=0, atol=1e-12)
        off += c
    # quantized along the padded axis, a group's blocks hold only its own tokens: its product equals the one of
    # the group quantized alone (same values and the same draws up to the block numbering)
    idx, e8 = O.quantize_rows_mx(ax, O.RTNE, True, 0x1234)
    for gi, c in enumerate(counts):
        lo, hi = int(poff[gi]), int(poff[gi + 1])
        if hi == lo:
            continue
        alone = np.zeros((ax.shape[0], hi - lo), dtype=np.float32)
        alone[:, :c] = ax[:, lo:lo + c]
        i2, e2 = O.quantize_rows_mx(alone, O.RTNE, True, 0x1234)
        assert np.array_equal(idx[:, lo:hi], i2) and np.array_equal(e8[:, lo // 32:hi // 32], e2)


# ------------------------------------------------------------------------------------------------
# binary32 rounding, the scale quotient and the 4-bit code patterns, against their definitions
# ------------------------------------------------------------------------------------------------

def _rn24_exact(q: Fraction, subnormal_floor: bool = True) -> Fraction:
    """Round-half-even of an exact rational to 24 significant bits, on the binary32 grid below 2^-126 (gradual
    underflow) when `subnormal_floor`, with no upper exponent limit (the caller decides what overflows)."""
    if q == 0:
        return Fraction(0)
    sign = -1 if q < 0 else 1
    a = abs(q)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    ulp_e = max(e - 23, -149) if subnormal_floor else e - 23
    scaled = a / Fraction(2) ** ulp_e
    n = floor(scaled)
    rem = scaled - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return sign * Fraction(n) * Fraction(2) ** ulp_e


def test_round_to_fp32_against_exact_rounding():
    """RN onto the binary32 grid: ties to even in the normal range, gradual underflow with ties below 2^-126,
    and 24 significant bits kept past FLT_MAX (the RHT's largest outputs), against integer rounding."""
    vals = [1 + 2.0 ** -24, 1 + 3 * 2.0 ** -24, 1 + 2.0 ** -24 + 2.0 ** -60, -(1 + 2.0 ** -24),
            2.0 ** -150, 3 * 2.0 ** -150, 2.0 ** -150 + 2.0 ** -200, 5 * 2.0 ** -151, -(2.0 ** -149) * 1.5,
            2.0 ** -126 - 2.0 ** -150, 2.0 ** -126 - 2.0 ** -151,
            (2 - 2.0 ** -24) * 2.0 ** 127, (2 - 2.0 ** -23) * 2.0 ** 127, 2.0 ** 128 * (1 + 2.0 ** -24),
            3.9 * 2.0 ** 127, -(2.0 ** 129) * (1 + 3 * 2.0 ** -25), 0.0]
    rng = np.random.default_rng(12)
    mant = rng.integers(1 << 52, 1 << 53, size=300).astype(np.float64) * 2.0 ** -52
    expo = rng.integers(-160, 130, size=300)
    vals += list(np.where(rng.random(300) < 0.5, -1, 1) * mant * np.exp2(expo.astype(np.float64)))
    got = O.round_to_fp32(np.array(vals))
    for v, g in zip(vals, got):
        want = _rn24_exact(Fraction(float(v)))
        assert Fraction(float(g)) == want, (v, float(g), float(want))


@pytest.mark.parametrize("g", [7.0, 6.0, 4.0, 2.0])
def test_scale_quotient_against_exact_division(g):
    """s = RN32(amax/g) as IEEE binary32: subnormal for tiny amax, +inf where the rounded quotient reaches
    2^128, for amax from the smallest bf16 subnormal up to the RHT's largest output (4x the bf16 maximum)."""
    rng = np.random.default_rng(int(g))
    bf16_max = (2 - 2.0 ** -7) * 2.0 ** 127
    amax = [2.0 ** -133, 3 * 2.0 ** -133, 7 * 2.0 ** -126, 7 * 2.0 ** -126 * (1 - 2.0 ** -23), 1.0, 7.0, 6.0,
            bf16_max, 4 * bf16_max, g * (2 - 2.0 ** -24) * 2.0 ** 127, g * (2 - 2.0 ** -23) * 2.0 ** 127]
    m = rng.integers(1 << 23, 1 << 24, size=200).astype(np.float64) * 2.0 ** -23
    e = rng.integers(-133, 129, size=200).astype(np.float64)
    amax = np.array(amax + list(m * np.exp2(e)))
    amax = O.round_to_fp32(amax)  # amax is an fp32-precision value, possibly past FLT_MAX
    got = O.scale_rn32(amax, g)
    assert got.dtype == np.float32
    for a, s in zip(amax, got):
        q = _rn24_exact(Fraction(float(a)) / Fraction(g))
        if q >= Fraction(2) ** 128:
            assert np.isinf(s) and s > 0, (a, s)
        else:
            assert Fraction(float(s)) == q, (a, float(s), float(q))


def test_e2m1_nibbles_are_the_ocp_fp4_encoding():
    """Every E2M1 nibble decodes, by the OCP FP4 definition (sign bit 3, exponent bits 2-1 with bias 1,
    mantissa bit 0; exponent 0 is subnormal), to the level the oracle assigns to it; codes re-encode to the same
    nibble, except -0 which the quantizer never emits (zero is +0)."""
    nib = np.arange(16, dtype=np.uint8)
    idx = O.nibbles_to_idx(nib, O.E2M1)
    got = O.level_values(idx, O.E2M1)
    for n in range(16):
        s, ex, mt = (n >> 3) & 1, (n >> 1) & 3, n & 1
        mag = mt * 0.5 if ex == 0 else (1 + mt / 2) * 2.0 ** (ex - 1)
        assert got[n] == (-mag if s else mag), n
    back = O.code_nibbles(idx, O.E2M1)
    assert np.array_equal(back, np.where(nib == 8, 0, nib))


def test_grid_top_levels_and_block_padding():
    """g of each grid (Sec. 2.1: the largest level; Sec. 5 Q4's cut E2M1 grids) and the padding helper against
    brute force."""
    assert O.grid_gmax(O.UNIFORM) == 7.0 and O.grid_gmax(O.E2M1) == 6.0
    assert O.grid_gmax(O.E2M1, 4) == 4.0 and O.grid_gmax(O.E2M1, 2) == 2.0
    for block in (16, 32):
        for n in range(0, 200):
            want = next(m for m in range(0, n + block + 1, block) if m >= n)
            assert O.pad16(n, block) == want
