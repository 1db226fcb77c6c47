"""CPU oracle for the UFP4 hot path -- TEST INFRASTRUCTURE ONLY.

This is a plain, slow and deliberately obvious reference for the data-parallel hot path of the UFP4
recipe in "Rethinking Shrinkage Bias in LLM FP4 Pretraining" (arXiv 2606.20381):

  * the block-16 Random Hadamard Transform (RHT) of Sec. 2.2, applied along the reduction axis of a GEMM
    operand;
  * 1x16 block-scaled quantization (Sec. 2.1) to the uniform 4-bit grid of the recipe (Sec. 4, Table 1:
    codes -7..7) or to the E2M1 grid of the comparison recipe, with round-to-nearest-even (RTNE) or
    stochastic rounding (SR);
  * the quantized training GEMMs fwd_y, bwd_dx and bwd_dw (Sec. 2.2, last display and its closing
    sentence), evaluated as an fp64 product of the dequantized operands.

Who may use it: the tests, the smoke check and the CPU-baseline leg of the benchmark. The product (the
HIP library and its Python binding) never imports, links or runs anything here, and nothing here imports
the product package. Inputs are numpy arrays; bf16 tensors arrive as their raw uint16 bit patterns.

Readings of the paper that this oracle fixes (the paper states exact mathematics only):
  * RHT arithmetic: y = RN_fp32( (1/4) * sum_j H16[i,j] * eps_j * x_j ), the exact 16-term sum rounded
    once to fp32 precision ("correctly rounded"; gradual underflow below 2^-126, and no overflow: a rotated
    value past FLT_MAX keeps 24 significant bits), for every finite bf16 block. The sum is evaluated in fp64
    through an explicit 16x16 matrix product, which is exact when the nonzero magnitudes of a block span at
    most 2^41 (`_fp64_sums_exact`); the other blocks are summed with Python integers and rounded once.
  * Scale and reciprocal: s = RN32(amax / g), r = RN24(g / amax), v = RN32(y * r); g = 7 (uniform) or
    6 (E2M1). RN32 is IEEE binary32 rounding with gradual underflow (a tiny block gets a subnormal scale);
    RN24 rounds to 24 significant bits without an exponent limit, which is RN32 whenever g / amax is below
    the fp32 overflow threshold (every amax >= g / FLT_MAX) and keeps the reciprocal finite for the few
    normal and subnormal amax below it. A block with amax = 0 gets s = 0 and all codes 0.
  * RTNE tie rule: the level whose magnitude code is even (IEEE round-half-even on the 4-bit encoding).
  * SR: q = g_b with probability (v - g_a)/(g_b - g_a) over adjacent signed levels g_a <= v < g_b,
    realised with a 16-bit uniform draw U = u / 2^16: q = g_b iff U < (v - g_a)/(g_b - g_a).
    The draws come from Philox4x32-10 with key = seed and counter = (block, row, half, stream).
  * Codes outside the grid are clamped (|v| can exceed g by one fp32 ulp).
  * Packing: sign-magnitude nibbles for both grids -- sign in bit 3, magnitude code in bits 0-2 (for E2M1
    this is the OCP FP4 bit pattern), zero always encoded as +0; element 2j in the low nibble of byte j.
  * Range-restricted E2M1 (Sec. 5 Q4): the levels up to max_fpx are kept and g = max_fpx.
  * RHT blocks of 32/64/128 (Appendix search space): the exact fp64 sum times RN64(sqrt(1/n)), rounded once to
    fp32; the 16-blocks of the result are quantized as usual.
  * Diagnostics (Sec. 3.2): the reference of NMSE / alpha is the tensor the quantizer rounds (the fp32 RHT
    output, or x); B_eff counts the magnitude codes of the grid, zero included.
  * Recipes: per-GEMM RHT flags, the set of operands rounded stochastically (streams 0 and 1 for dY and dY^T,
    2-5 for X, W, W^T, X^T), max_fpx and the RHT block, for Table 1, Table 2's ablations, Sec. 5 Q4 and the
    Appendix search space.
"""

from __future__ import annotations

from fractions import Fraction
import math

import numpy as np

# ---------------------------------------------------------------------------------------------------
# Formats, rounding modes, constants (Sec. 2.1; Table 1)
# ---------------------------------------------------------------------------------------------------

UNIFORM = 0  # E1M2/INT4-style uniform grid, integer codes -7..7 (Sec. 4 recipe; Table 1)
E2M1 = 1  # FP4 E2M1 grid of the comparison recipe (Sec. 2.1, Fig. 1; Table 1)

RTNE = 0  # round to nearest, deterministic ties (Sec. 2.1)
SR = 1  # stochastic rounding (Sec. 2.1, second display)

BLOCK = 16  # 1x16 quantization block and RHT block (Table 1)

# Non-negative levels of each grid, in magnitude-code order (Sec. 2.1; Sec. 3.1 lists the E2M1 ones).
GRID_MAGNITUDES = {
    UNIFORM: np.arange(8, dtype=np.float64),  # 0..7; the E1M2 levels k/4 scaled by 4
    E2M1: np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]),
}
G_MAX = {UNIFORM: 7.0, E2M1: 6.0}  # g_max of Sec. 2.1

# Range-restricted E2M1 (Sec. 5 Q4, the max_fpx ablation; Appendix search space): keep only the levels up to
# max_fpx and use g = max_fpx. The kept levels are a prefix of the E2M1 list, so magnitude codes are unchanged.
E2M1_MAX_FPX = (2.0, 4.0, 6.0)


def grid_magnitudes(fmt: int, max_fpx=None) -> np.ndarray:
    """Non-negative levels of a grid in magnitude-code order; E2M1 optionally cut at max_fpx."""
    mags = GRID_MAGNITUDES[fmt]
    if max_fpx is None:
        return mags
    if fmt != E2M1 or float(max_fpx) not in E2M1_MAX_FPX:
        raise ValueError("max_fpx applies to E2M1 only and must be one of 2, 4, 6")
    return mags[mags <= float(max_fpx)]


def grid_gmax(fmt: int, max_fpx=None) -> float:
    """g of the scale s = amax/g: the top level of the (possibly restricted) grid."""
    return float(grid_magnitudes(fmt, max_fpx)[-1])


# ---------------------------------------------------------------------------------------------------
# bf16 helpers
# ---------------------------------------------------------------------------------------------------

def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact bf16 -> fp32 widening of raw uint16 bit patterns."""
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    u = u + np.uint64(0x7FFF) + lsb
    return (u >> np.uint64(16)).astype(np.uint16)


# ---------------------------------------------------------------------------------------------------
# Hadamard matrices and the RHT (Sec. 2.2)
# ---------------------------------------------------------------------------------------------------

def sylvester_hadamard(n: int) -> np.ndarray:
    """Normalised Sylvester Hadamard H_n by the recursion of Sec. 2.2 (H_1 = [1], factor 1/sqrt(2))."""
    if n < 1 or n & (n - 1):
        raise ValueError("n must be a power of two")
    h = np.ones((1, 1))
    while h.shape[0] < n:
        h = np.block([[h, h], [h, -h]]) / np.sqrt(2.0)
    return h


def hadamard_pm1(n: int = BLOCK) -> np.ndarray:
    """The same recursion without the 1/sqrt(2) factors: the +-1 matrix, H_n = hadamard_pm1(n)/sqrt(n).

    For n = 16 the collected normalisation is exactly 1/4 (Sec. 2.2 recursion, four levels).
    """
    if n < 1 or n & (n - 1):
        raise ValueError("n must be a power of two")
    h = np.ones((1, 1))
    while h.shape[0] < n:
        h = np.block([[h, h], [h, -h]])
    return h


def sign_vector(sign_mask: int, n: int = BLOCK) -> np.ndarray:
    """Diagonal of the random sign matrix S_n of Sec. 2.2: eps_j = -1 iff bit j of the mask is set."""
    return np.array([-1.0 if (int(sign_mask) >> j) & 1 else 1.0 for j in range(n)])


def _fp64_sums_exact(blocks: np.ndarray) -> np.ndarray:
    """Per block (last axis, n entries): whether the fp64 evaluation of every n-term signed sum is exact.

    Each term is a bf16 value (8 significant bits). With frexp exponents e_max and e_min over the nonzero
    entries of a block, the exact sum is a multiple of 2^(e_min - 8) below 2^(e_max + log2 n) in magnitude,
    so it fits the 53-bit fp64 significand when e_max - e_min <= 45 - log2 n (41 for n = 16).
    """
    mag = np.abs(blocks)
    nz = mag > 0
    _, e = np.frexp(np.where(nz, mag, 1.0))
    e_max = np.where(nz, e, np.iinfo(np.int32).min).max(axis=-1)
    e_min = np.where(nz, e, np.iinfo(np.int32).max).min(axis=-1)
    spread = np.where(nz.any(axis=-1), e_max - e_min, 0)
    return spread <= 45 - int(np.log2(blocks.shape[-1]))


def _exact_signed_sums(block: np.ndarray, eps: np.ndarray) -> tuple[list[int], int]:
    """The n sums sum_j H_n^pm1[i,j] eps_j x_j of one n-block exactly: integers m_i with sum_i = m_i * 2^e.

    Every x_j is a binary fraction p_j / 2^k_j (float.as_integer_ratio); over the common denominator 2^k the
    terms are integers and the sums are plain integer sums.
    """
    n = block.shape[-1]
    h = hadamard_pm1(n)
    ratios = [float(v).as_integer_ratio() for v in block]
    den = max(q for _, q in ratios)
    ints = [p * (den // q) for p, q in ratios]
    sums = [sum(int(h[i, j]) * int(eps[j]) * ints[j] for j in range(n)) for i in range(n)]
    return sums, -(den.bit_length() - 1)


def _round_int_to_fp32(m: int, e: int) -> float:
    """m * 2^e rounded onto the fp32 grid as `round_to_fp32` rounds: to nearest even, gradual underflow (the
    quantum never below 2^-149), and 24 significant bits with no exponent limit at the top. Returned as fp64."""
    if m == 0:
        return 0.0
    sign = -1.0 if m < 0 else 1.0
    m = abs(m)
    q = max(e + m.bit_length() - 24, -149)  # weight of the last kept bit
    if q > e:
        sh = q - e
        keep, rest, half = m >> sh, m & ((1 << sh) - 1), 1 << (sh - 1)
        if rest > half or (rest == half and keep & 1):
            keep += 1
        m, e = keep, q
    return sign * math.ldexp(m, e)


def rht_exact_f64(blocks: np.ndarray, sign_mask: int) -> np.ndarray:
    """Unrounded RHT of 16-element row blocks: each row vector x becomes x S_16 H_16 (Sec. 2.2).

    `blocks` has shape [..., 16]. H_16 is symmetric, so (x S H)_i = (1/4) sum_j H16pm1[i,j] eps_j x_j.
    Evaluated as an explicit matrix product in fp64; exact where `_fp64_sums_exact` holds.
    """
    blocks = np.asarray(blocks, dtype=np.float64)
    eps = sign_vector(sign_mask)
    return ((blocks * eps) @ hadamard_pm1(BLOCK)) * 0.25


def round_to_fp32(t: np.ndarray) -> np.ndarray:
    """Round to nearest even onto the binary32 grid, returned as fp64: gradual underflow below 2^-126 (IEEE), and
    no overflow -- a magnitude of 2^127 or more keeps 24 significant bits beyond the fp32 range. Only the RHT of
    inputs near the bf16 maximum reaches past it (|y| <= 4 max|x| for block 16)."""
    t = np.asarray(t, dtype=np.float64)
    big = np.abs(t) >= 2.0 ** 127
    low = np.where(big, 0.0, t).astype(np.float32).astype(np.float64)
    high = (np.where(big, t, 0.0) * 2.0 ** -64).astype(np.float32).astype(np.float64) * 2.0 ** 64
    return np.where(big, high, low)


def rht_blocks(blocks_f32: np.ndarray, sign_mask: int) -> np.ndarray:
    """RHT of bf16-valued 16-blocks, correctly rounded to fp32 precision (one rounding of the exact result,
    `round_to_fp32`: gradual underflow, no overflow). Returned as fp64 holding those values. Blocks whose fp64
    sums could round (nonzero magnitudes spanning more than 2^41) are summed exactly with integers."""
    b64 = np.asarray(blocks_f32, dtype=np.float64)
    y = round_to_fp32(rht_exact_f64(b64, sign_mask))
    wide = ~_fp64_sums_exact(b64)
    if wide.any():
        eps = sign_vector(sign_mask)
        for idx in zip(*np.nonzero(wide)):
            sums, e = _exact_signed_sums(b64[idx], eps)
            y[idx] = [_round_int_to_fp32(m, e - 2) for m in sums]  # the factor 1/4 of the 16-point RHT
    return y


# RHT blocks larger than the quantization block (the RHT block-size dimension of the E2M1 reference search,
# Appendix search-space table: 16 / 32 / 64 / 128). The transform of each n-block is x S_n H_n with the
# normalisation 1/sqrt(n) of the Sec. 2.2 recursion; the 16-blocks of its output are then quantized as usual.
RHT_BLOCKS = (16, 32, 64, 128)


def rht_norm(n: int) -> float:
    """fp64 normalisation of the n-point RHT: RN64(sqrt(1/n)); exactly 1/4 and 1/8 for n = 16 and 64."""
    return float(np.sqrt(1.0 / n))


def rht_rows_n(a_f32: np.ndarray, sign_mask: int, n: int) -> np.ndarray:
    """RHT of the n-blocks of every row of A [rows, red] (red % n == 0), as fp32.

    y = RN32( RN64( S * RN64(1/sqrt(n)) ) ) with S = sum_j H_n^pm1[i,j] eps_j x_j the exact sum (an explicit fp64
    matrix product where `_fp64_sums_exact` holds, integers elsewhere). For n = 16 and 64 the normalisation is a
    power of two and y is the correctly rounded transform; for n = 32 and 128 it is the correctly rounded fp64
    product, then rounded to fp32 precision (`round_to_fp32`; fp64 result). eps_j = -1 iff bit j of the n-bit
    `sign_mask` is set.
    """
    if n not in RHT_BLOCKS:
        raise ValueError("RHT block must be 16, 32, 64 or 128")
    a = np.asarray(a_f32, dtype=np.float64)
    rows, red = a.shape
    if red % n:
        raise ValueError("the reduction length must be a multiple of the RHT block")
    blocks = a.reshape(rows, red // n, n)
    eps = sign_vector(sign_mask, n)
    c = rht_norm(n)
    y = round_to_fp32(((blocks * eps) @ hadamard_pm1(n)) * c)
    wide = ~_fp64_sums_exact(blocks)
    for idx in zip(*np.nonzero(wide)):
        sums, e = _exact_signed_sums(blocks[idx], eps)
        if n in (16, 64):  # c = 2^-2 or 2^-3: one rounding of the exact transform
            y[idx] = [_round_int_to_fp32(m, e + int(math.log2(c))) for m in sums]
        else:  # the exact product S * c rounded to fp64 (Fraction -> float rounds correctly), then to fp32
            y[idx] = round_to_fp32(np.array([float(Fraction(m) * Fraction(2) ** e * Fraction(c)) for m in sums]))
    return y.reshape(rows, red)


# ---------------------------------------------------------------------------------------------------
# Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC'11)
# ---------------------------------------------------------------------------------------------------

PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
_MASK32 = np.uint64(0xFFFFFFFF)


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Philox4x32 with 10 rounds on arrays of 32-bit counters; returns the four 32-bit output words.

    One round: (hi0, lo0) = M0 * c0, (hi1, lo1) = M1 * c2 (64-bit products);
    (c0, c1, c2, c3) <- (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0); then the key is bumped by the Weyl
    constants (W0, W1) before the next round.
    """
    c0 = np.asarray(c0, dtype=np.uint64) & _MASK32
    c1 = np.asarray(c1, dtype=np.uint64) & _MASK32
    c2 = np.asarray(c2, dtype=np.uint64) & _MASK32
    c3 = np.asarray(c3, dtype=np.uint64) & _MASK32
    k0 = np.uint64(int(k0) & 0xFFFFFFFF)
    k1 = np.uint64(int(k1) & 0xFFFFFFFF)
    c0, c1, c2, c3 = np.broadcast_arrays(c0, c1, c2, c3)
    for _ in range(10):
        p0 = c0 * np.uint64(PHILOX_M0)
        p1 = c2 * np.uint64(PHILOX_M1)
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK32
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
        k0 = (k0 + np.uint64(PHILOX_W0)) & _MASK32
        k1 = (k1 + np.uint64(PHILOX_W1)) & _MASK32
    return tuple(w.astype(np.uint32) for w in (c0, c1, c2, c3))


def sr_draws(block_idx, row_idx, seed: int, stream: int) -> np.ndarray:
    """The sixteen 16-bit uniform draws of each quantization block, shape [..., 16] (uint16).

    Block (row r, block b) uses two Philox calls, counter (b, r, h, stream) for h = 0, 1 and key
    (seed low 32 bits, seed high 32 bits). Element j of the block takes the 16-bit half (j & 1) -- low
    half first -- of output word (j & 7) >> 1 of call h = j >> 3.
    """
    b = np.asarray(block_idx, dtype=np.uint64)
    r = np.asarray(row_idx, dtype=np.uint64)
    b, r = np.broadcast_arrays(b, r)
    k0, k1 = int(seed) & 0xFFFFFFFF, (int(seed) >> 32) & 0xFFFFFFFF
    out = np.empty(b.shape + (BLOCK,), dtype=np.uint16)
    for h in range(2):
        words = philox4x32_10(b, r, np.uint64(h), np.uint64(int(stream) & 0xFFFFFFFF), k0, k1)
        for w in range(4):
            out[..., 8 * h + 2 * w] = (words[w] & np.uint32(0xFFFF)).astype(np.uint16)
            out[..., 8 * h + 2 * w + 1] = (words[w] >> np.uint32(16)).astype(np.uint16)
    return out


# ---------------------------------------------------------------------------------------------------
# Rounding onto a grid (Sec. 2.1)
# ---------------------------------------------------------------------------------------------------

def round_nearest_even(v: np.ndarray, fmt: int, max_fpx=None) -> np.ndarray:
    """RTNE onto the signed grid: nearest level; on a tie, the level with the even magnitude code.

    Returns signed level *indices* (magnitude code with the sign of v; -0 becomes 0). Values beyond the
    largest level go to it (the nearest level). Brute force over every level of the grid (E2M1 cut at
    max_fpx when given).
    """
    mags = grid_magnitudes(fmt, max_fpx)
    a = np.abs(np.asarray(v, dtype=np.float64))
    dist = np.abs(a[..., None] - mags)  # exact: fp32 inputs, small dyadic levels
    best = dist.min(axis=-1, keepdims=True)
    cand = dist == best
    # among the (at most two) nearest levels prefer the even magnitude code
    even = (np.arange(len(mags)) % 2) == 0
    pick_even = cand & even
    idx = np.where(pick_even.any(axis=-1), pick_even.argmax(axis=-1), cand.argmax(axis=-1))
    return np.where(np.asarray(v) < 0, -idx, idx).astype(np.int64)


def _signed_levels(fmt: int, max_fpx=None) -> np.ndarray:
    mags = grid_magnitudes(fmt, max_fpx)
    return np.concatenate([-mags[:0:-1], mags])  # ascending, -g_max .. g_max


def round_stochastic(v: np.ndarray, u16: np.ndarray, fmt: int, max_fpx=None) -> np.ndarray:
    """SR onto the signed grid with 16-bit draws (Sec. 2.1, second display).

    For g_a <= v < g_b adjacent signed levels, q = g_b iff u/2^16 < (v - g_a)/(g_b - g_a); otherwise g_a.
    v on a level stays there; |v| beyond the largest level goes to it. Returns signed level indices.
    """
    levels = _signed_levels(fmt, max_fpx)
    v64 = np.asarray(v, dtype=np.float64)
    vc = np.clip(v64, levels[0], levels[-1])
    ia = np.searchsorted(levels, vc, side="right") - 1  # levels[ia] <= vc
    ia = np.clip(ia, 0, len(levels) - 1)
    ib = np.minimum(ia + 1, len(levels) - 1)
    ga, gb = levels[ia], levels[ib]
    width = np.where(ib > ia, gb - ga, 1.0)
    p_up = np.where(ib > ia, (vc - ga) / width, 0.0)  # exact: dyadic numbers, power-of-two widths
    u = np.asarray(u16, dtype=np.float64) / 65536.0
    q = np.where(u < p_up, gb, ga)
    # back to signed magnitude index
    mags = grid_magnitudes(fmt, max_fpx)
    idx = np.searchsorted(mags, np.abs(q))
    return np.where(q < 0, -idx, idx).astype(np.int64)


def level_values(signed_idx: np.ndarray, fmt: int) -> np.ndarray:
    """Signed level index -> level value (fp64)."""
    signed_idx = np.asarray(signed_idx)
    mags = GRID_MAGNITUDES[fmt]
    return np.sign(signed_idx) * mags[np.abs(signed_idx)]


# ---------------------------------------------------------------------------------------------------
# The blockwise quantizer Q_G of Sec. 2.1, with the RHT of Sec. 2.2 in front
# ---------------------------------------------------------------------------------------------------

def _check_block_domain(y: np.ndarray) -> None:
    """Inputs must be finite (Sec. 2.1 defines the quantizer for real-valued tensors)."""
    if not np.all(np.isfinite(y)):
        raise ValueError("non-finite input")


def scale_rn32(amax: np.ndarray, g: float) -> np.ndarray:
    """s = RN32(amax / g), the IEEE binary32 quotient: gradual underflow for tiny blocks, +inf past the fp32 range.
    amax holds fp32-precision values (fp64 array) that may exceed FLT_MAX (`round_to_fp32`); below 2^127 it is
    an fp32 number and one binary32 division gives s. Above, RN24(amax 2^-64 / g) 2^64 is that quotient with an
    unbounded exponent, and its cast to fp32 overflows exactly where the IEEE quotient does."""
    a = np.asarray(amax, dtype=np.float64)
    big = a >= 2.0 ** 127
    low = np.where(big, 0.0, a).astype(np.float32) / np.float32(g)
    q = (np.where(big, a, 0.0) * 2.0 ** -64).astype(np.float32) / np.float32(g)
    with np.errstate(over="ignore"):
        high = (q.astype(np.float64) * 2.0 ** 64).astype(np.float32)
    return np.where(big, high, low).astype(np.float32)


def reciprocal_rn24(g: float, amax: np.ndarray) -> np.ndarray:
    """r = g / amax rounded to nearest even at 24 significant bits, without an exponent limit (fp64 result).

    amax = m * 2^e with m in [0.5, 1) (exact); RN24(g / amax) = RN24(g / m) * 2^-e, and g / m in (g, 2g] is a
    normal fp32 quotient, so one IEEE binary32 division gives RN24(g / m). Equal to RN32(g / amax) whenever
    that is finite. amax = 0 gives 0.
    """
    a = np.asarray(amax, dtype=np.float64)
    m, e = np.frexp(a)
    r_m = np.float32(g) / np.where(a > 0, m, 1.0).astype(np.float32)
    return np.where(a > 0, r_m.astype(np.float64) * np.ldexp(1.0, -e), 0.0)


def quantize_rows(a_f32: np.ndarray, fmt: int, rounding: int, rht: bool, sign_mask: int = 0,
                  seed: int = 0, stream: int = 0, row_ids=None, block_base: int = 0, max_fpx=None,
                  rht_block: int = BLOCK):
    """Quantize an operand A [rows, red] along its contiguous (reduction) axis.

    Steps per 1x16 block B (Sec. 2.1 display; RHT of Sec. 2.2 applied first when `rht`):
      y = RHT(x) or x;  s = RN32(amax/g);  q_i = rho(y_i / s) with y_i/s taken as RN32(y_i * RN24(g/amax))
    (`reciprocal_rn24`).
    `row_ids` are the global row numbers used in the SR counters (default 0..rows-1); `block_base` is
    added to the block number (used for operands cut out of a longer reduction axis). `max_fpx` (E2M1
    only) restricts the grid to the levels up to it, with g = max_fpx. `rht_block` > 16 rotates n-blocks
    (`rht_rows_n`, with an n-bit sign mask) before the 1x16 quantization.
    Returns (signed level indices int64 [rows, red], scales fp32 [rows, red/16]).
    """
    a = np.asarray(a_f32, dtype=np.float32)
    rows, red = a.shape
    if red % BLOCK:
        raise ValueError("reduction length must be a multiple of 16")
    nb = red // BLOCK
    blocks = a.reshape(rows, nb, BLOCK)
    if rht and rht_block != BLOCK:
        y = rht_rows_n(a, sign_mask, rht_block).reshape(rows, nb, BLOCK)
    else:
        y = rht_blocks(blocks, sign_mask) if rht else blocks.astype(np.float64)
    _check_block_domain(y)
    g = grid_gmax(fmt, max_fpx)
    amax = np.abs(y).max(axis=-1)  # fp32 precision, held in fp64 (the RHT output may exceed FLT_MAX)
    nz = amax > 0
    scale = scale_rn32(amax, g)  # IEEE binary32: subnormal when tiny
    recip = reciprocal_rn24(g, amax)
    # one rounding per element: the fp64 product of two 24-bit significands is exact, then RN32
    v = (y * recip[..., None]).astype(np.float32)
    if rounding == RTNE:
        idx = round_nearest_even(v, fmt, max_fpx)
    elif rounding == SR:
        rid = np.arange(rows) if row_ids is None else np.asarray(row_ids)
        bidx = block_base + np.arange(nb)
        u = sr_draws(bidx[None, :], rid[:, None], seed, stream)
        idx = round_stochastic(v, u, fmt, max_fpx)
    else:
        raise ValueError("unknown rounding mode")
    idx = np.where(nz[..., None], idx, 0)
    return idx.reshape(rows, red), scale


# ---------------------------------------------------------------------------------------------------
# Operand views per GEMM (Sec. 2.2, closing sentence: the RHT axis is the reduction axis)
# ---------------------------------------------------------------------------------------------------

def operand_rowwise(t_bits: np.ndarray) -> np.ndarray:
    """Operand whose reduction axis is the contiguous axis of the stored tensor: A = T."""
    return bf16_bits_to_f32(t_bits)


def operand_colwise(t_bits: np.ndarray) -> np.ndarray:
    """Operand whose reduction axis is the strided axis: A = T^T (rows of A are columns of T)."""
    return np.ascontiguousarray(bf16_bits_to_f32(t_bits).T)


def quantize_both(t_bits: np.ndarray, fmt: int, rounding: int, rht_rows: bool, rht_cols: bool,
                  sign_mask_rows: int = 0, sign_mask_cols: int = 0, seed: int = 0, stream_rows: int = 0,
                  stream_cols: int = 0):
    """The two operands one stored tensor T [rows, cols] supplies to a training step (Sec. 2.2: the RHT and
    the quantization run along each GEMM's reduction axis, and T is reduced along its columns in one GEMM and
    along its rows in another): (Q(T) along cols, Q(T^T) along rows), two independent quantizations with
    their own RHT flag, sign mask and SR stream. Returns ((idx, scales) rowwise, (idx, scales) transposed).
    """
    return (quantize_rows(operand_rowwise(t_bits), fmt, rounding, rht_rows, sign_mask_rows, seed, stream_rows),
            quantize_rows(operand_colwise(t_bits), fmt, rounding, rht_cols, sign_mask_cols, seed, stream_cols))


def pad16(n: int, block: int = BLOCK) -> int:
    """n rounded up to a multiple of `block` (16: one quantization block; 32 for power-of-two scales)."""
    return -(-int(n) // block) * block


def operand_colwise_grouped(t_bits: np.ndarray, counts, block: int = BLOCK) -> tuple[np.ndarray, np.ndarray]:
    """Transposed operand of a grouped (MoE) tensor whose rows are split into consecutive groups.

    Group g owns rows [off_g, off_g + counts[g]) of T. Its block of A is T[group]^T with the reduction
    axis (the group's tokens) zero-padded to a multiple of `block` (the quantization block along that axis: 16,
    or 32 for power-of-two scales, so that no block straddles two groups); the padded groups are concatenated
    along the reduction axis. Zero padding keeps every group's GEMM unchanged ((XH')(WH')^T = XW^T).
    Returns (A [cols, sum of padded counts], padded offsets [G+1]).
    """
    t = bf16_bits_to_f32(t_bits)
    counts = [int(c) for c in counts]
    if sum(counts) != t.shape[0]:
        raise ValueError("group counts do not cover the rows")
    pads = [pad16(c, block) for c in counts]
    poff = np.concatenate([[0], np.cumsum(pads)]).astype(np.int64)
    a = np.zeros((t.shape[1], int(poff[-1])), dtype=np.float32)
    off = 0
    for g, c in enumerate(counts):
        a[:, poff[g]:poff[g] + c] = t[off:off + c].T
        off += c
    return a, poff


# ---------------------------------------------------------------------------------------------------
# Packing (codes -> bytes) and dequantization
# ---------------------------------------------------------------------------------------------------

def code_nibbles(idx: np.ndarray, fmt: int) -> np.ndarray:
    """4-bit code of each element: sign << 3 | magnitude code, zero as +0. For the uniform grid the
    magnitude code is |k|; for E2M1 it is the index of the magnitude, so the nibble is the OCP FP4 pattern."""
    idx = np.asarray(idx, dtype=np.int64)
    sign = (idx < 0).astype(np.int64)
    return ((sign << 3) | np.abs(idx)).astype(np.uint8)


def nibbles_to_idx(nib: np.ndarray, fmt: int) -> np.ndarray:
    nib = np.asarray(nib, dtype=np.int64)
    mag = nib & 7
    return np.where(nib & 8, -mag, mag)


def pack_codes(idx: np.ndarray, fmt: int) -> np.ndarray:
    """[rows, red] level indices -> [rows, red/2] bytes; element 2j in the low nibble of byte j."""
    nib = code_nibbles(idx, fmt)
    return (nib[:, 0::2] | (nib[:, 1::2] << np.uint8(4))).astype(np.uint8)


def unpack_codes(packed: np.ndarray, fmt: int) -> np.ndarray:
    packed = np.asarray(packed, dtype=np.uint8)
    rows, half = packed.shape
    nib = np.empty((rows, 2 * half), dtype=np.uint8)
    nib[:, 0::2] = packed & np.uint8(0xF)
    nib[:, 1::2] = packed >> np.uint8(4)
    return nibbles_to_idx(nib, fmt)


def dequantize(idx: np.ndarray, scales: np.ndarray, fmt: int) -> np.ndarray:
    """Q_G(T) as a numerical tensor (Sec. 2.1 footnote sentence): level value times block scale, fp64."""
    idx = np.asarray(idx)
    rows, red = idx.shape
    vals = level_values(idx, fmt).reshape(rows, red // BLOCK, BLOCK)
    return (vals * np.asarray(scales, dtype=np.float64)[..., None]).reshape(rows, red)


# ---------------------------------------------------------------------------------------------------
# Quantized GEMMs (Sec. 2.2: Y_hat = Q(XH') Q(WH')^T; all three training GEMMs in the same NT form)
# ---------------------------------------------------------------------------------------------------

def gemm_nt(a_idx, a_scales, b_idx, b_scales, fmt: int) -> np.ndarray:
    """C = deq(A) @ deq(B)^T in fp64; A [M, red], B [N, red] share the quantized reduction axis."""
    return dequantize(a_idx, a_scales, fmt) @ dequantize(b_idx, b_scales, fmt).T


# ---------------------------------------------------------------------------------------------------
# The uniform grid with power-of-two block scales (Sec. 4: the scale hierarchy is orthogonal to the grid
# and may follow the hardware). Quantization blocks of 32 along the reduction axis share one scale 2^E
# (OCP Microscaling rule), stored as an E8M0 byte E + 127; the RHT stays block-16 (two RHT blocks per scale
# block) and the codes are the uniform levels -7..7, stored as FP6 E2M3 numbers (every integer up to 7 is
# exact in E2M3).
# ---------------------------------------------------------------------------------------------------

MX_BLOCK = 32
E8M0_BIAS = 127


def mx_scale_exponent(amax) -> np.ndarray:
    """Per block, E = floor(log2 amax) - 2: the shared-exponent rule of the OCP Microscaling formats
    (floor(log2 amax) minus the exponent of the element format's largest binade) with the integer levels
    -7..7 read as FP6 E2M3 numbers, whose largest binade is [4, 8). Then amax / 2^E lies in [4, 8): the
    top element may exceed the top level 7 and is clamped to it (the rounding clamps, as for the fp32
    scales). E8M0 holds E >= -127 only: a block with amax < 2^-125 takes the smallest scale 2^-127 (byte 0),
    and then amax / 2^E < 4. amax = 0 gives E = -127 too; a zero block's codes are all 0 whatever the scale."""
    a = np.asarray(amax, dtype=np.float64)
    m, e = np.frexp(a)  # a = m * 2^e with 0.5 <= m < 1, so floor(log2 a) = e - 1
    return np.maximum(np.where(a > 0, e - 3, -E8M0_BIAS), -E8M0_BIAS).astype(np.int64)


def quantize_rows_mx(a_f32: np.ndarray, rounding: int, rht: bool, sign_mask: int = 0, seed: int = 0,
                     stream: int = 0, row_ids=None):
    """Quantize an operand A [rows, red] (red % 32 == 0) along its contiguous axis with power-of-two scales.

    Per 1x32 block: y = RHT16(x) on each half (or x); E = mx_scale_exponent(amax |y|); v = RN32(y * 2^-E) (|v| <
    8; a power of two, so exact unless below 2^-126); codes -7..7 by RTNE or SR with the draws of the two
    16-blocks it contains (the SR counters number 16-blocks, as in `quantize_rows`), |v| > 7 clamped to the top
    level. Returns (signed codes int64 [rows, red], E8M0 bytes uint8 [rows, red/32]).
    """
    a = np.asarray(a_f32, dtype=np.float32)
    rows, red = a.shape
    if red % MX_BLOCK:
        raise ValueError("reduction length must be a multiple of 32")
    n16, n32 = red // BLOCK, red // MX_BLOCK
    y16 = a.reshape(rows, n16, BLOCK)
    y16 = rht_blocks(y16, sign_mask) if rht else y16.astype(np.float64)
    _check_block_domain(y16)
    y = y16.reshape(rows, n32, MX_BLOCK)
    amax = np.abs(y).max(axis=-1)
    E = mx_scale_exponent(amax)
    v = (y * np.ldexp(1.0, -E)[..., None]).astype(np.float32)  # RN32: exact but below 2^-126 (as v of the 1x16 path)
    if rounding == RTNE:
        idx = round_nearest_even(v, UNIFORM)
    elif rounding == SR:
        rid = np.arange(rows) if row_ids is None else np.asarray(row_ids)
        u = sr_draws(np.arange(n16)[None, :], rid[:, None], seed, stream).reshape(rows, n32, MX_BLOCK)
        idx = round_stochastic(v, u, UNIFORM)
    else:
        raise ValueError("unknown rounding mode")
    return idx.reshape(rows, red), (E + E8M0_BIAS).astype(np.uint8)


def e2m3_value(bits) -> np.ndarray:
    """Value of a 6-bit FP6 E2M3 pattern (OCP MX formats): sign, 2 exponent bits (bias 1), 3 mantissa bits;
    exponent 0 is subnormal (m/8)."""
    b = np.asarray(bits, dtype=np.int64)
    s, e, m = (b >> 5) & 1, (b >> 3) & 3, b & 7
    mag = np.where(e == 0, m / 8.0, np.ldexp(1.0 + m / 8.0, e - 1))
    return np.where(s == 1, -mag, mag)


_E2M3_OF_INT = {int(e2m3_value(b)): b for b in range(32) if float(e2m3_value(b)).is_integer()}


def e2m3_codes(idx: np.ndarray) -> np.ndarray:
    """Signed integer codes -7..7 -> their E2M3 bit patterns (zero as +0), by search over the format."""
    idx = np.asarray(idx, dtype=np.int64)
    mag = np.vectorize(lambda k: _E2M3_OF_INT[int(k)])(np.abs(idx)) if idx.size else np.zeros(idx.shape, np.int64)
    return np.where(idx < 0, mag | 0x20, mag).astype(np.int64)


def pack_fp6(idx: np.ndarray) -> np.ndarray:
    """[rows, red] codes -> uint8 [rows, red * 3 / 4]: each 32-block as 24 bytes, element j of the block in
    bits 6j .. 6j + 5 of its little-endian 192-bit string (the operand layout of the scaled f8f6f4 MFMA)."""
    c = e2m3_codes(idx)
    rows, red = c.shape
    blocks = c.reshape(rows, red // MX_BLOCK, MX_BLOCK)
    out = np.zeros((rows, red // MX_BLOCK, 24), dtype=np.uint8)
    for j in range(MX_BLOCK):
        for bit in range(6):
            pos = 6 * j + bit
            out[..., pos // 8] |= (((blocks[..., j] >> bit) & 1) << (pos % 8)).astype(np.uint8)
    return out.reshape(rows, red // MX_BLOCK * 24)


def unpack_fp6(packed: np.ndarray) -> np.ndarray:
    """Inverse of pack_fp6: signed integer codes."""
    p = np.asarray(packed, dtype=np.uint8)
    rows, nbytes = p.shape
    blocks = p.reshape(rows, nbytes // 24, 24).astype(np.int64)
    bits = np.zeros((rows, nbytes // 24, MX_BLOCK), dtype=np.int64)
    for j in range(MX_BLOCK):
        for bit in range(6):
            pos = 6 * j + bit
            bits[..., j] |= ((blocks[..., pos // 8] >> (pos % 8)) & 1) << bit
    return e2m3_value(bits).astype(np.int64).reshape(rows, nbytes // 24 * MX_BLOCK)


def dequantize_mx(idx: np.ndarray, e8m0: np.ndarray) -> np.ndarray:
    """Codes and E8M0 block scales -> fp64 values k * 2^(e8m0 - 127)."""
    idx = np.asarray(idx, dtype=np.float64)
    rows, red = idx.shape
    sc = np.ldexp(1.0, np.asarray(e8m0, dtype=np.int64) - E8M0_BIAS)
    return (idx.reshape(rows, red // MX_BLOCK, MX_BLOCK) * sc[..., None]).reshape(rows, red)


def gemm_nt_mx(a_idx, a_e8m0, b_idx, b_e8m0) -> np.ndarray:
    """C = deq(A) @ deq(B)^T in fp64 for operands with power-of-two block scales."""
    return dequantize_mx(a_idx, a_e8m0) @ dequantize_mx(b_idx, b_e8m0).T


# ---------------------------------------------------------------------------------------------------
# One linear layer's three quantized GEMMs under a recipe (Sec. 4, Table 1; Sec. 2.2 closing sentence)
# ---------------------------------------------------------------------------------------------------

_T, _F = True, False
RECIPES = {
    # format, RHT on (fwd_y, bwd_dx, bwd_dw), SR on dY only (Table 1)
    "ufp4": dict(fmt=UNIFORM, rht=(_T, _T, _T)),
    "e2m1": dict(fmt=E2M1, rht=(_F, _F, _T)),
    # the UFP4 recipe with 1x32 power-of-two (E8M0) scales instead of 1x16 fp32 scales
    "mxufp4": dict(fmt=UNIFORM, rht=(_T, _T, _T), scales="e8m0x32"),
    # Table 2: RHT scope and SR under the uniform grid
    "ufp4-rht-none": dict(fmt=UNIFORM, rht=(_F, _F, _F)),
    "ufp4-rht-dw": dict(fmt=UNIFORM, rht=(_F, _F, _T)),
    "ufp4-rht-dx-dw": dict(fmt=UNIFORM, rht=(_F, _T, _T)),
    "ufp4-rht-y-dw": dict(fmt=UNIFORM, rht=(_T, _F, _T)),
    "ufp4-no-sr": dict(fmt=UNIFORM, rht=(_T, _T, _T), sr=()),
    # E2M1 variants (Sec. 5 Q4; Appendix search space)
    "e2m1-full-rht": dict(fmt=E2M1, rht=(_T, _T, _T)),
    "e2m1-max4": dict(fmt=E2M1, rht=(_T, _T, _T), max_fpx=4.0),
    "e2m1-max2": dict(fmt=E2M1, rht=(_T, _T, _T), max_fpx=2.0),
    "e2m1-sr-bwd": dict(fmt=E2M1, rht=(_F, _F, _T), sr=("dy", "dyt", "xt", "wt")),
    # RHT block (Appendix search space); the n-bit sign mask repeats the 16-bit one in every sub-block
    "ufp4-rht32": dict(fmt=UNIFORM, rht=(_T, _T, _T), rht_block=32),
    "ufp4-rht64": dict(fmt=UNIFORM, rht=(_T, _T, _T), rht_block=64),
    "ufp4-rht128": dict(fmt=UNIFORM, rht=(_T, _T, _T), rht_block=128),
}
# Philox stream (counter word 3) of each operand when it is rounded stochastically
SR_STREAMS = {"dy": 0, "dyt": 1, "x": 2, "w": 3, "wt": 4, "xt": 5}


def layer_gemms(x_bits, w_bits, dy_bits, recipe: str = "ufp4", sign_mask: int = 0, seed: int = 0,
                times: dict | None = None):
    """Quantize the six operands of one linear layer and run fwd_y, bwd_dx and bwd_dw.

    X [M, K], W [N, K], dY [M, N] (bf16 bit patterns). Operands:
      fwd_y : X, W rowwise along K (RTNE)              -> Y  [M, N]
      bwd_dx: dY rowwise along N (SR, stream 0),  W^T along N (RTNE)  -> dX [M, K]
      bwd_dw: dY^T along M (SR, stream 1),       X^T along M (RTNE)  -> dW [N, K]
    Returns a dict with the quantized operands (idx, scales) and the three fp64 outputs. If `times` is a dict,
    the wall-clock seconds of the six quantizations ("quantize") and of each GEMM ("fwd_y", "bwd_dx",
    "bwd_dw") are stored in it; this is bookkeeping only.
    """
    import time

    clock = [time.perf_counter()]

    def mark(name):
        now = time.perf_counter()
        if times is not None:
            times[name] = now - clock[0]
        clock[0] = now

    cfg = RECIPES[recipe]
    fmt = cfg["fmt"]
    r_y, r_dx, r_dw = cfg["rht"]
    q = {}
    if cfg.get("scales") == "e8m0x32":
        Q = quantize_rows_mx
        q["x"] = Q(operand_rowwise(x_bits), RTNE, r_y, sign_mask)
        q["w"] = Q(operand_rowwise(w_bits), RTNE, r_y, sign_mask)
        q["dy"] = Q(operand_rowwise(dy_bits), SR, r_dx, sign_mask, seed, 0)
        q["wt"] = Q(operand_colwise(w_bits), RTNE, r_dx, sign_mask)
        q["dyt"] = Q(operand_colwise(dy_bits), SR, r_dw, sign_mask, seed, 1)
        q["xt"] = Q(operand_colwise(x_bits), RTNE, r_dw, sign_mask)
        mark("quantize")
        out = {"y": gemm_nt_mx(*q["x"], *q["w"])}
        mark("fwd_y")
        out["dx"] = gemm_nt_mx(*q["dy"], *q["wt"])
        mark("bwd_dx")
        out["dw"] = gemm_nt_mx(*q["dyt"], *q["xt"])
        mark("bwd_dw")
        return q, out
    sr = set(cfg.get("sr", ("dy", "dyt")))
    n = cfg.get("rht_block", BLOCK)
    mask = sum((sign_mask & 0xFFFF) << (16 * k) for k in range(n // BLOCK))

    def quant(op, a, rht):
        rnd = SR if op in sr else RTNE
        return quantize_rows(a, fmt, rnd, rht, mask, seed, SR_STREAMS[op], max_fpx=cfg.get("max_fpx"), rht_block=n)

    q["x"] = quant("x", operand_rowwise(x_bits), r_y)
    q["w"] = quant("w", operand_rowwise(w_bits), r_y)
    q["dy"] = quant("dy", operand_rowwise(dy_bits), r_dx)
    q["wt"] = quant("wt", operand_colwise(w_bits), r_dx)
    q["dyt"] = quant("dyt", operand_colwise(dy_bits), r_dw)
    q["xt"] = quant("xt", operand_colwise(x_bits), r_dw)
    mark("quantize")
    out = {"y": gemm_nt(*q["x"], *q["w"], fmt)}
    mark("fwd_y")
    out["dx"] = gemm_nt(*q["dy"], *q["wt"], fmt)
    mark("bwd_dx")
    out["dw"] = gemm_nt(*q["dyt"], *q["xt"], fmt)
    mark("bwd_dw")
    return q, out


# ---------------------------------------------------------------------------------------------------
# Quality diagnostics (Sec. 3.2): SQNR, operand projection alpha, bucket entropy / effective ratio
# ---------------------------------------------------------------------------------------------------

def nmse(q: np.ndarray, ref: np.ndarray) -> float:
    """||Q - T||_F^2 / ||T||_F^2 (Sec. 3.2, NMSE)."""
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.sum((np.asarray(q, dtype=np.float64) - ref) ** 2) / np.sum(ref ** 2))


def sqnr_db(q: np.ndarray, ref: np.ndarray) -> float:
    return float(-10.0 * np.log10(nmse(q, ref)))


def operand_projection(q: np.ndarray, ref: np.ndarray) -> float:
    """alpha_A = <A_hat, A>_F / ||A||_F^2 (Sec. 3.2, operand projection)."""
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.sum(np.asarray(q, dtype=np.float64) * ref) / np.sum(ref * ref))


def effective_bucket_ratio(idx: np.ndarray, fmt: int, eps: float = 1e-12) -> float:
    """B_eff = exp(E)/K with E = -sum p_i log(p_i + eps) over the K magnitude buckets (Sec. 3.2)."""
    k = len(GRID_MAGNITUDES[fmt])
    mag = np.abs(np.asarray(idx)).ravel()
    p = np.bincount(mag, minlength=k)[:k] / mag.size
    ent = -np.sum(p * np.log(p + eps))
    return float(np.exp(ent) / k)


def quant_stats(a_f32: np.ndarray, fmt: int, rounding: int, rht: bool, sign_mask: int = 0, seed: int = 0,
                stream: int = 0, max_fpx=None) -> dict:
    """Sums behind the Sec. 3.2 diagnostics for one quantization of an operand A [rows, red].

    The reference is the tensor the quantizer rounds: ref = y, the RHT output rounded to fp32 (rht) or x
    itself; q = Q_G(ref) dequantized (level * scale, fp64). Returns
      err2 = ||q - ref||_F^2,  ref2 = ||ref||_F^2,  cross = <q, ref>_F,
      hist[m] = number of elements whose magnitude code is m (m = 0..7; bucket 0 is zero).
    NMSE = err2 / ref2 and alpha = cross / ref2 (Sec. 3.2); B_eff follows from hist.
    """
    a = np.asarray(a_f32, dtype=np.float32)
    rows, red = a.shape
    blocks = a.reshape(rows, red // BLOCK, BLOCK)
    y = rht_blocks(blocks, sign_mask) if rht else blocks.astype(np.float64)
    ref = y.reshape(rows, red)
    idx, sc = quantize_rows(a, fmt, rounding, rht, sign_mask, seed, stream, max_fpx=max_fpx)
    q = dequantize(idx, sc, fmt)
    return {
        "err2": float(np.sum((q - ref) ** 2)),
        "ref2": float(np.sum(ref * ref)),
        "cross": float(np.sum(q * ref)),
        "hist": np.bincount(np.abs(idx).ravel(), minlength=8)[:8].astype(np.int64),
    }


def stats_metrics(st: dict, fmt: int, max_fpx=None, eps: float = 1e-12) -> dict:
    """NMSE, SQNR (dB), alpha and B_eff (K = levels of the grid, zero included) from `quant_stats` sums."""
    k = len(grid_magnitudes(fmt, max_fpx))
    hist = np.asarray(st["hist"], dtype=np.float64)[:k]
    n = hist.sum()
    p = hist / n if n > 0 else hist
    ent = -np.sum(p * np.log(p + eps))
    ref2 = st["ref2"]
    nm = st["err2"] / ref2 if ref2 > 0 else float("nan")
    return {
        "nmse": nm,
        "sqnr_db": float(-10.0 * np.log10(nm)) if nm > 0 else float("inf"),
        "alpha": st["cross"] / ref2 if ref2 > 0 else float("nan"),
        "beff": float(np.exp(ent) / k),
    }


def delta_sqnr_db(nmse_raw: float, nmse_rht: float) -> float:
    """Delta SQNR = 10 log10(NMSE_I / NMSE_H16) (Sec. 3.2): positive when the rotation helps."""
    return float(10.0 * np.log10(nmse_raw / nmse_rht))
