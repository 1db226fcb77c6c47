// Fused block-16 RHT + 1x16 block-scaled 4-bit quantization (uniform grid -7..7, or the E2M1 baseline).
//
// What is computed per 16-element block of an operand's reduction axis (Sec. 2.1 quantizer display,
// Sec. 2.2 RHT, recipe of Sec. 4 / Table 1):
//   y    = RN32( x S_16 H_16 )            exact 16-term sum in fp64 (Sylvester butterfly), one rounding
//   s    = RN32(amax / g),  r = RN32(g / amax),  v = RN32(y * r)
//   code = RTNE(v) or SR(v; Philox draw)  onto the grid, clamped to +-g
// y is rounded with gradual underflow and without overflow (24 significant bits past FLT_MAX); s is the IEEE
// quotient (subnormal for tiny blocks, +inf past the fp32 range); r has 24 significant bits and no exponent
// limit (equal to RN32(g / amax) wherever that is finite).
//
// Fast path. The RHT's factor 1/4 is a power of two: the kernel keeps y' = 4y = RN32(unscaled sum), so amax' =
// 4 amax, RN32(g / amax') = r / 4, y' * RN32(g / amax') = y * r exactly, and s = RN32(amax' / g) / 4. For bf16
// inputs y' = 4y holds for every output (a sum below 2^-124 is a multiple of 2^-133 with at most 9 significant
// bits, so both it and a quarter of it are exact fp32 numbers); with amax' in [2^-121, 2^127) (or 0) the
// quotients are normal and these identities are exact (s by the FMA-corrected product, r by an IEEE division). Any other block takes the exact path (`quant_core`),
// which rescales the block by a power of two before the reciprocal. Real data never leaves the fast range; the
// check costs three instructions per block.
//
// Two input layouts: rowwise (reduction axis contiguous, one thread per block, 32-byte loads) and
// transposed (reduction axis strided: each thread loads a 16-row x 8-column sub-tile and builds its eight
// column blocks in registers). The transposed kernel also serves grouped (MoE) tensors whose token axis is
// cut into groups that are zero-padded to a multiple of 16. A third kernel produces both operands of one
// tensor (rowwise and transposed) from a single read of it.
//
// Output layout (panels): the quantized operand's rows are cut into panels of 128; within a panel, block b
// of all 128 rows is stored contiguously (codes: 128 x 8 bytes at b * 1024; scales: 128 floats at b * 128).
// Rows past the operand's last one in the final panel are written as zero codes and zero scales. This is the
// order in which the GEMM stages K-blocks, so its loads are contiguous runs.
//
// This translation unit is compiled with -ffp-contract=off: every fp32/fp64 operation above must round
// exactly once, as written.

#include "ufp4_device.h"
#include "ufp4_internal.h"

namespace ufp4 {

// ------------------------------------------------------------------------------------------------
// Per-element rounding onto the grid; returns the 4-bit code in the low bits.
// ------------------------------------------------------------------------------------------------

// Codes are sign-magnitude nibbles: sign in bit 3, |k| in bits 0-2, zero as +0.
//
// Uniform grid. 1.5 * 2^23 + 8 is an even integer with ulp 1: adding it to v (|v| <= 7.5) rounds v to the
// nearest integer k, ties to the even one (RTNE), and leaves the nibble k + 8 in bits 0-3 of the sum with
// bits 4-21 clear. No clamp is needed for RTNE: |v| = RN(|y| * RN(7/amax)) <= 7 (1 + 2^-23) rounds to 7.
constexpr float kMagic8 = 12582920.0f;

// Stochastic rounding between the integers lo = floor(v) and lo + 1: up iff lo + u/2^16 < v. Both sides
// are exact in fp32 (lo + u/2^16 needs at most 20 significant bits), so the decision is exact. Returns the
// chosen integer.
__device__ __forceinline__ float uniform_sr_level(float v, uint32_t u16) {
    const float vc = __builtin_fminf(__builtin_fmaxf(v, -7.0f), 7.0f);
    const float lo = floorf(vc);
    const float t = __builtin_fmaf((float)u16, 1.0f / 65536.0f, lo);
    return lo + ((t < vc) ? 1.0f : 0.0f);  // a zero level comes out as +0
}

// The same decision with the offset nibble as the result: lo + kMagic8 holds nibble lo + 8 in bits 0-3 (bits
// 4-21 clear), and the step up is added to that bit pattern as an integer (lo + 8 + 1 <= 15: no carry leaves
// the nibble, since lo = 7 only when the clamped v is 7, which never rounds up).
__device__ __forceinline__ uint32_t uniform_sr_offset(float v, uint32_t u16) {
    const float vc = __builtin_fminf(__builtin_fmaxf(v, -7.0f), 7.0f);
    const float lo = floorf(vc);
    const float t = __builtin_fmaf((float)u16, 1.0f / 65536.0f, lo);
    return __float_as_uint(lo + kMagic8) + ((t < vc) ? 1u : 0u);
}

// Eight words whose bits 0-3 hold a nibble and bits 4-21 are clear (higher bits arbitrary) -> one dword,
// element i in bits 4i .. 4i+3. Shifts by 12 and more push the arbitrary bits out of the word.
__device__ __forceinline__ uint32_t pack_nibbles(const uint32_t* t) {
    const uint32_t low = t[0] | (t[1] << 4) | (t[2] << 8);
    const uint32_t high = (t[3] << 12) | (t[4] << 16) | (t[5] << 20) | (t[6] << 24) | (t[7] << 28);
    return (low & 0xFFFu) | high;
}

// Offset nibbles n = k + 8 (k in -7..7, so n >= 1) -> sign-magnitude nibbles: n >= 8 gives n ^ 8 = k, n < 8
// gives (n ^ 15) + 1 = 16 - n = 8 | -k. Per nibble, without carries between nibbles.
__device__ __forceinline__ uint32_t offset_to_sign_magnitude(uint32_t x) {
    const uint32_t t = ~x & 0x88888888u;  // 8 in the nibbles with n < 8
    const uint32_t one = t >> 3;
    return (x ^ 0x88888888u ^ (t - one)) + one;
}

// E2M1 magnitude code of the nearest level, ties to the even code (levels 0,.5,1,1.5,2,3,4,6; the bin
// edges are the midpoints; an edge belongs to the even-coded side). For a >= 1 the levels are the fp32 values
// with one fraction bit, and the code is 2 (exponent - 126) + that bit: the significand is rounded to one
// fraction bit, ties to even, on the bit pattern. Below 1 the levels are 0, 0.5, 1: the code is RNE(2a), read
// off 2a + 2^23. Codes past 7 (a > 6 can only come from rounding) are cut to 7. Equal to the nearest-level
// search for every fp32 a in [0, 8] (checked exhaustively on the host).
__device__ __forceinline__ uint32_t e2m1_mag_rtne(float a) {
    const uint32_t b = __float_as_uint(a);
    const uint32_t r = b + 0x1FFFFFu + ((b >> 22) & 1u);
    const uint32_t hi = (r >> 22) - 252u;
    const uint32_t lo = __float_as_uint(__builtin_fmaf(a, 2.0f, 8388608.0f)) - 0x4B000000u;
    const uint32_t idx = a >= 1.0f ? hi : lo;
    return idx < 7u ? idx : 7u;
}

__device__ __forceinline__ uint32_t e2m1_rtne(float v) {
    const uint32_t idx = e2m1_mag_rtne(__builtin_fabsf(v));
    return idx | ((v < 0.0f && idx != 0u) ? 8u : 0u);
}

// SR over adjacent signed E2M1 levels g_a <= v < g_b (spacing d = g_b - g_a in {0.5, 1, 2}):
// q = g_b iff g_a + d * u/2^16 < v. For v >= 0 the bracket is [lower, upper) in magnitude, for v < 0 it
// is (-upper, -lower] mirrored, so that a value on a level never moves. `g` is the top level kept (the
// grid cut at max_fpx = 2, 4 or 6 keeps the levels up to it); v is clamped to it first.
__device__ __forceinline__ uint32_t e2m1_sr(float v, uint32_t u16, float g) {
    const float vc = __builtin_fminf(__builtin_fmaxf(v, -g), g);
    const float a = __builtin_fabsf(vc);
    const bool pos = vc >= 0.0f;
    // The bracket family: spacing d = 0.5 below 2 (codes 0-4), 1 below 4 (codes 4-6), 2 above (codes 6-7);
    // for v < 0 an edge value belongs to the family below it, so that a value on a level never moves.
    const bool s1 = pos ? a < 2.0f : a <= 2.0f;
    const bool s2 = pos ? a < 4.0f : a <= 4.0f;
    const float d = s1 ? 0.5f : (s2 ? 1.0f : 2.0f);
    const float inv = s1 ? 2.0f : (s2 ? 1.0f : 0.5f);  // 1/d: (a - base) * inv is exact
    const float base = s1 ? 0.0f : (s2 ? 2.0f : 4.0f);
    const int base_code = s1 ? 0 : (s2 ? 4 : 6);
    // |g_a| (v >= 0) or |g_a| of the mirrored bracket (v < 0) as base + j d, whose code is base_code + j
    const float r = (a - base) * inv;
    const float j = pos ? floorf(r) : ceilf(r);
    const float mag = base + j * d;
    const float ga = pos ? mag : -mag;
    const float t = __builtin_fmaf((float)u16 * (1.0f / 65536.0f), d, ga);
    const int code = base_code + (int)j;
    const int q = (t < vc) ? (pos ? code + 1 : code - 1) : code;  // g_b = g_a + d: one code up or down
    return (uint32_t)q | ((!pos && q != 0) ? 8u : 0u);
}

// RTNE needs no cut: |v| <= g (1 + 2^-23) for g = 2, 4, 6 already rounds to a level <= g.
template <int ROUND>
__device__ __forceinline__ uint32_t e2m1_code(float v, uint32_t u16, float g) {
    if constexpr (ROUND == kRoundSR) return e2m1_sr(v, u16, g);
    else return e2m1_rtne(v);
}

// ------------------------------------------------------------------------------------------------
// One 16-block: eight bf16 pairs in (element 2j in the low half of w[j]), packed codes + scale out.
// ------------------------------------------------------------------------------------------------
// The RHT of one 16-block: y' = 4y = RN32( sum_j H16[i,j] eps_j x_j ) (see the file header), or y = x.
// The exact sums sum_j H16pm1[i,j] eps_j x_j of one 16-block in fp64 (sx: the sign-bit XOR word per pair).
__device__ __forceinline__ void rht16_sums(const uint32_t* w, const uint32_t* sx, double* d) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const uint32_t p = w[j] ^ sx[j];  // eps_j = -1: flip the bf16 sign bit
        d[2 * j] = (double)bf16_lo(p);
        d[2 * j + 1] = (double)bf16_hi(p);
    }
    // Sylvester butterfly: after the four stages d = H16pm1 * (eps x), H16pm1[i][j] = (-1)^popcount(i&j).
#pragma unroll
    for (int h = 1; h < 16; h <<= 1) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            if (!(i & h)) {
                const double a = d[i], b = d[i + h];
                d[i] = a + b;
                d[i + h] = a - b;
            }
        }
    }
}

template <bool RHT>
__device__ __forceinline__ void rht16_unscaled(const uint32_t* w, const QuantArgs& qa, float* y) {
    if constexpr (RHT) {
        double d[16];
        rht16_sums(w, qa.sign_xor, d);
#pragma unroll
        for (int i = 0; i < 16; ++i) y[i] = (float)d[i];
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            y[2 * j] = bf16_lo(w[j]);
            y[2 * j + 1] = bf16_hi(w[j]);
        }
    }
}

// Block-n RHT, n = 16 m with m = 2, 4 or 8 (the RHT block larger than the quantization block). The Sylvester
// H_n is H_m (x) H_16 (outer factor on the high index bits), so after each thread's 16-point butterfly on its
// own 16-block -- sub-block `sub` of the n-block, with its 16 bits of the n-bit sign mask -- a butterfly over
// the m threads that hold the n-block (lanes `lane_step` apart, the partner of stage h at lane distance
// h * lane_step) completes the exact fp64 sums; then t = RN64(sum * RN64(sqrt(1/n))), whose rounding to fp32
// precision is y (`quant_wide`). Every lane must call this (inactive blocks with zero inputs): the exchange
// reads the partner lanes' registers.
__device__ __forceinline__ void rht_wide(const uint32_t (&w)[8], const QuantArgs& qa, uint32_t sub, int lane_step,
                                         double (&t)[16]) {
    const uint32_t mask = qa.sign_words[sub & (uint32_t)(qa.rht_m - 1)];  // this sub-block's 16 sign bits
    uint32_t sx[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) sx[j] = (((mask >> (2 * j)) & 1u) << 15) | (((mask >> (2 * j + 1)) & 1u) << 31);
    double d[16];
    rht16_sums(w, sx, d);
    for (int h = 1; h < qa.rht_m; h <<= 1) {
        const bool upper = (sub & (uint32_t)h) != 0u;  // this thread holds the "minus" half of the stage
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const double o = __shfl_xor(d[i], h * lane_step);
            d[i] = upper ? o - d[i] : d[i] + o;
        }
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) t[i] = d[i] * qa.rht_c;
}

// The fast path's amax range (see the file header), [2^-121, 2^127), as fp32 bit patterns.
constexpr uint32_t kFastLoBits = 0x03000000u;
constexpr uint32_t kFastEndBits = 0x7F000000u;

// amax (>= 0) outside {0} and [2^-121, 2^127) (infinity included): the block needs the exact path.
__device__ __forceinline__ bool needs_exact(float amax) {
    const uint32_t b = __float_as_uint(amax);
    return b - kFastLoBits >= kFastEndBits - kFastLoBits && b != 0u;
}

// Exact path (see the file header), for a block whose amax is outside the fast range: the block is rescaled in
// place by 2^64 (tiny) or 2^-64 (huge), and the fast arithmetic then runs on it. The power of two is exact on
// every element whose v can be nonzero, the reciprocal of the scaled amax is a normal fp32 number with the same
// 24-bit significand as g / amax, and (y_i 2^Q) r' is the same real product as y_i r, so one rounding still gives
// v_i. Only the stored scale is taken separately: s = RN32(amax / g) is one IEEE division of amax, an fp32
// number (for the folded RHT amax = amax' / 4 exactly). A folded or wide RHT output past FLT_MAX overflows y to
// infinity; then `exact_t` supplies the fp64 values t_i whose rounding to 24 bits is y_i, and the block is taken
// at 2^-64 (and s = RN32(amax 2^-64 / g) 2^64, +inf where amax / g is past the fp32 range).
//
// EXACT = false leaves the exact path out (its branch costs registers in the two-operand kernel): the result is
// then valid only when the function returns false, and the caller redoes the block with EXACT = true otherwise.
template <int FMT, int ROUND, bool FOLD, bool OVF, bool EXACT, typename TFn>
__device__ __forceinline__ bool quant_core(float (&y)[16], TFn&& exact_t, const QuantArgs& qa, uint32_t blk,
                                           uint32_t row, uint32_t& code_lo, uint32_t& code_hi, float& scale) {
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) amax = __builtin_fmaxf(amax, __builtin_fabsf(y[i]));
    const float g = FMT == kFmtUniform ? 7.0f : qa.e2m1_g;
    const bool exact = needs_exact(amax);
    float s_exact = 0.0f;
    if (EXACT && __builtin_expect(exact, 0)) {
        if (OVF && !(amax <= 0x1.fffffep127f)) {
            double t[16];
            exact_t(t);
            amax = 0.0f;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                y[i] = (float)(t[i] * 0x1p-64);  // y_i 2^-64: normal here, or too small to matter
                amax = __builtin_fmaxf(amax, __builtin_fabsf(y[i]));
            }
            s_exact = __fmul_rn(amax / g, 0x1p64f);
        } else {
            s_exact = (FOLD ? __fmul_rn(amax, 0.25f) : amax) / g;  // IEEE: subnormal for a tiny block
            const float q = amax < 1.0f ? 0x1p64f : 0x1p-64f;
#pragma unroll
            for (int i = 0; i < 16; ++i) y[i] = __fmul_rn(y[i], q);
            amax = __fmul_rn(amax, q);
        }
    }
    // RN(amax / g) as RN(amax * c) with c = RN(1/g), corrected by one FMA residual step: equal to the correctly
    // rounded quotient for every fp32 amax when g = 7 and for every normal quotient when g = 6 (both checked over
    // all fp32 inputs); for g = 2 and 4 the product is already exact. amax = 0 gives 0.
    const float c = FMT == kFmtUniform ? 1.0f / 7.0f : qa.e2m1_ginv;
    const float q0 = amax * c;
    const float sc = __builtin_fmaf(__builtin_fmaf(-q0, g, amax), c, q0);
    scale = EXACT && exact ? s_exact : (FOLD ? sc * 0.25f : sc);
    const float r = amax > 0.0f ? g / amax : 0.0f;  // IEEE division; zero block: all v = 0, codes 0
    float v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = __fmul_rn(y[i], r);

    uint32_t u[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if constexpr (ROUND == kRoundSR) {
        const Philox4 p0 = philox4x32_10(blk, row, 0u, qa.stream, qa.key0, qa.key1);
        const Philox4 p1 = philox4x32_10(blk, row, 1u, qa.stream, qa.key0, qa.key1);
        u[0] = p0.x; u[1] = p0.y; u[2] = p0.z; u[3] = p0.w;
        u[4] = p1.x; u[5] = p1.y; u[6] = p1.z; u[7] = p1.w;
    }
    if constexpr (FMT == kFmtUniform) {
        uint32_t tt[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            if constexpr (ROUND == kRoundSR) {
                const uint32_t u16 = (i & 1) ? (u[i >> 1] >> 16) : (u[i >> 1] & 0xFFFFu);
                tt[i] = uniform_sr_offset(v[i], u16);
            } else {
                tt[i] = __float_as_uint(v[i] + kMagic8);  // the rounding itself
            }
        }
        code_lo = offset_to_sign_magnitude(pack_nibbles(tt));
        code_hi = offset_to_sign_magnitude(pack_nibbles(tt + 8));
    } else {
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const uint32_t u16 = (i & 1) ? (u[i >> 1] >> 16) : (u[i >> 1] & 0xFFFFu);
            const uint32_t c = e2m1_code<ROUND>(v[i], u16, g);
            if (i < 8) lo |= c << (4 * i);
            else hi |= c << (4 * (i - 8));
        }
        code_lo = lo;
        code_hi = hi;
    }
    return exact;
}

// Values y given directly (no transform, or a transform already applied); finite, so they cannot overflow.
template <int FMT, int ROUND>
__device__ __forceinline__ void quant_y16(float (&y)[16], const QuantArgs& qa, uint32_t blk, uint32_t row,
                                          uint32_t& code_lo, uint32_t& code_hi, float& scale) {
    quant_core<FMT, ROUND, false, false, true>(y, [](double (&)[16]) {}, qa, blk, row, code_lo, code_hi, scale);
}

// The fp64 values y_i of the block-16 RHT before rounding (exact sums / 4), recomputed from the input words. The
// empty asm makes the words opaque, so the compiler recomputes the sums here instead of keeping the fast path's
// 32 registers of them alive until this rare branch.
__device__ __forceinline__ void rht16_exact(const uint32_t (&w)[8], const QuantArgs& qa, double (&t)[16]) {
    uint32_t wc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        wc[j] = w[j];
        asm volatile("" : "+v"(wc[j]));
    }
    rht16_sums(wc, qa.sign_xor, t);
#pragma unroll
    for (int i = 0; i < 16; ++i) t[i] *= 0.25;  // exact in fp64
}

// Makes a register tile opaque to the compiler in place (see the two-operand kernel's fix-up).
template <int R, int C>
__device__ __forceinline__ void opaque(uint32_t (&a)[R][C]) {
#pragma unroll
    for (int i = 0; i < R; ++i) {
#pragma unroll
        for (int j = 0; j < C; ++j) asm volatile("" : "+v"(a[i][j]));
    }
}

// One 16-block of bf16 pairs w (element 2j in the low half of w[j]), with the block-16 RHT when RHT. With EXACT
// = false the result is valid only if this returns false (see `quant_core`).
template <int FMT, int ROUND, bool RHT, bool EXACT = true>
__device__ __forceinline__ bool quant_block16(const uint32_t (&w)[8], const QuantArgs& qa, uint32_t blk, uint32_t row,
                                              uint32_t& code_lo, uint32_t& code_hi, float& scale) {
    float y[16];
    rht16_unscaled<RHT>(w, qa, y);
    if constexpr (RHT) {
        return quant_core<FMT, ROUND, true, true, EXACT>(y, [&](double (&t)[16]) { rht16_exact(w, qa, t); }, qa, blk,
                                                        row, code_lo, code_hi, scale);
    } else {
        return quant_core<FMT, ROUND, false, false, EXACT>(y, [](double (&)[16]) {}, qa, blk, row, code_lo, code_hi,
                                                          scale);
    }
}

// One block after a wider RHT (`rht_wide`): y = RN32(t), and t itself if that overflows.
template <int FMT, int ROUND>
__device__ __forceinline__ void quant_wide(const double (&t)[16], const QuantArgs& qa, uint32_t blk, uint32_t row,
                                           uint32_t& code_lo, uint32_t& code_hi, float& scale) {
    float y[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) y[i] = (float)t[i];
    quant_core<FMT, ROUND, false, true, true>(
        y, [&](double (&tt)[16]) {
#pragma unroll
            for (int i = 0; i < 16; ++i) tt[i] = t[i];
        },
        qa, blk, row, code_lo, code_hi, scale);
}

// ------------------------------------------------------------------------------------------------
// Rowwise: reduction axis contiguous. A workgroup of 512 threads quantizes a tile of 32 rows x 16 blocks
// through LDS: a wave reads 4 rows x 512 contiguous bytes, each thread quantizes one block, and the tile is
// written in panel order, each half-wave storing 32 rows x 8 bytes of one block. Consecutive workgroups take
// consecutive block tiles of the same rows. Padding rows of the last panel are written as zeros.
// ------------------------------------------------------------------------------------------------
constexpr int kRR = 32;    // tile rows
constexpr int kRB = 16;    // tile blocks
constexpr int kRT = 512;   // threads
constexpr int kRI = kRR * kRB / kRT;  // blocks per thread

// T = uint16_t: bf16 input (the fused kernel). T = float: fp32 input quantized without a transform, the
// second half of the unfused form (a standalone RHT writes y in fp32, see rht_rows_kernel).
template <int FMT, int ROUND, bool RHT, typename T = uint16_t, bool WIDE = false>
__global__ __launch_bounds__(kRT) void quant_rows_kernel(const T* __restrict__ x, int64_t ld, int64_t qrows,
                                                         int64_t nb, QuantArgs qa, uint8_t* __restrict__ codes,
                                                         int64_t code_pld, float* __restrict__ scales,
                                                         int64_t scale_pld) {
    constexpr int kVec = (int)sizeof(T) * kBlock / 16;  // 16-byte loads per block: 2 (bf16) or 4 (fp32)
    static_assert(sizeof(T) == 2 || !RHT, "the fp32-input kernel applies no transform");
    __shared__ uint2 s_codes[kRB][kRR];
    __shared__ float s_scales[kRB][kRR];
    const int t = threadIdx.x;
    const int64_t r0 = (int64_t)blockIdx.y * kRR;
    const int64_t b0 = (int64_t)blockIdx.x * kRB;

    // item k = t + kRT q: row k / 16, block k % 16 of the tile
    uint4 v[kRI][kVec];
#pragma unroll
    for (int q = 0; q < kRI; ++q) {
        const int k = t + kRT * q;
        const int64_t r = r0 + (k >> 4), b = b0 + (k & 15);
#pragma unroll
        for (int c = 0; c < kVec; ++c) v[q][c] = make_uint4(0, 0, 0, 0);
        if (r < qrows && b < nb) {
            const uint4* src = reinterpret_cast<const uint4*>(x + r * ld + b * kBlock);
#pragma unroll
            for (int c = 0; c < kVec; ++c) v[q][c] = src[c];
        }
    }
#pragma unroll
    for (int q = 0; q < kRI; ++q) {
        const int k = t + kRT * q;
        const int64_t r = r0 + (k >> 4), b = b0 + (k & 15);
        uint32_t lo = 0, hi = 0;
        float sc = 0.0f;
        if constexpr (WIDE) {
            // the 16 threads k .. of a tile row hold its 16 consecutive blocks: the n-block partners are lanes
            // h apart (n-blocks are aligned: b0 is a multiple of 16, nb of m)
            const uint32_t w[8] = {v[q][0].x, v[q][0].y, v[q][0].z, v[q][0].w,
                                   v[q][1].x, v[q][1].y, v[q][1].z, v[q][1].w};
            double tw[16];
            rht_wide(w, qa, (uint32_t)b, 1, tw);
            if (r < qrows && b < nb) quant_wide<FMT, ROUND>(tw, qa, (uint32_t)b, (uint32_t)r, lo, hi, sc);
        } else if (r < qrows && b < nb) {
            if constexpr (sizeof(T) == 2) {
                const uint32_t w[8] = {v[q][0].x, v[q][0].y, v[q][0].z, v[q][0].w,
                                       v[q][1].x, v[q][1].y, v[q][1].z, v[q][1].w};
                quant_block16<FMT, ROUND, RHT>(w, qa, (uint32_t)b, (uint32_t)r, lo, hi, sc);
            } else {
                float y[16];
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    y[4 * c] = __uint_as_float(v[q][c].x);
                    y[4 * c + 1] = __uint_as_float(v[q][c].y);
                    y[4 * c + 2] = __uint_as_float(v[q][c].z);
                    y[4 * c + 3] = __uint_as_float(v[q][c].w);
                }
                quant_y16<FMT, ROUND>(y, qa, (uint32_t)b, (uint32_t)r, lo, hi, sc);
            }
        }
        s_codes[k & 15][k >> 4] = make_uint2(lo, hi);
        s_scales[k & 15][k >> 4] = sc;
    }
    __syncthreads();
    // item k: block k / 32, row k % 32 (the 32 rows lie in one panel: r0 is a multiple of 32)
#pragma unroll
    for (int q = 0; q < kRI; ++q) {
        const int k = t + kRT * q;
        const int64_t r = r0 + (k % kRR), b = b0 + (k / kRR);
        if (b < nb) {
            const int64_t P = r >> 7, ri = r & 127;
            *reinterpret_cast<uint2*>(codes + P * code_pld + b * 1024 + ri * 8) = s_codes[k / kRR][k % kRR];
            scales[P * scale_pld + b * 128 + ri] = s_scales[k / kRR][k % kRR];
        }
    }
}

// ------------------------------------------------------------------------------------------------
// Transposed (and grouped-transposed): operand A = X^T, reduction along X's rows. A thread loads a
// 16-row x kXC-column bf16 sub-tile (one load of 2 kXC bytes per row) and quantizes its kXC column blocks
// from registers, so no LDS transposition and no barrier is needed. Its results are the kXC consecutive
// operand rows of its block, 8 kXC contiguous bytes of codes (stored directly, or through LDS so that the
// stores of a half-wave are contiguous; see the kernel). A workgroup of 256 threads covers 256 columns
// x 8 blocks; the 32 threads of one block read 512 contiguous bytes of each row. (Measured on the 1 GiB
// tensor: 64-column workgroups, 128 bytes per row, were 17% slower, wider ones no faster; 4 columns per
// thread performs within a few percent of 8; an LDS-transposed 128 x 64 tile was 12-20% slower.)
// ------------------------------------------------------------------------------------------------
// One row's kXC consecutive bf16 (kXC / 2 dwords) with a single 16- or 8-byte load.
template <int C>
__device__ __forceinline__ void load_row_chunk(const uint16_t* src, uint32_t (&d)[C / 2]) {
    if constexpr (C == 8) {
        const uint4 l = *reinterpret_cast<const uint4*>(src);
        d[0] = l.x; d[1] = l.y; d[2] = l.z; d[3] = l.w;
    } else {
        const uint2 l = *reinterpret_cast<const uint2*>(src);
        d[0] = l.x; d[1] = l.y;
    }
}

constexpr int kXC = 8;                     // columns (operand rows) per thread
constexpr int kMaxGroupsLds = 1024;

struct TGroups {
    const int64_t* off;  // token offsets [G+1] (device), nullptr for a dense tensor
    int32_t G;
};

// The token offsets of up to kMaxGroupsLds groups into s_off, and into s_poff the padded offsets: group lengths
// rounded up to multiples of PAD, prefix-summed. Thread t owns groups 4t .. 4t + 3 (read straight from global
// memory); the 256 partial sums are scanned with wave shuffles and one exchange of the four wave totals, so the
// whole call costs two barriers. Every thread of a 256-thread workgroup calls this; it ends with a barrier.
template <int PAD>
__device__ __forceinline__ void load_group_offsets(const TGroups& grp, int64_t* s_off, int64_t* s_poff) {
    __shared__ int64_t s_wave[4];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    int64_t o[5];
#pragma unroll
    for (int k = 0; k < 5; ++k) {
        const int g = 4 * t + k;
        o[k] = g <= grp.G ? grp.off[g] : 0;
    }
    int64_t part[4], run = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int g = 4 * t + k;
        const int64_t c = g < grp.G ? o[k + 1] - o[k] : 0;
        run += (c > 0 ? c + PAD - 1 : 0) / PAD * PAD;
        part[k] = run;
        if (g < grp.G) s_off[g] = o[k];
    }
    if (t == 0) {
        s_off[grp.G] = grp.off[grp.G];
        s_poff[0] = 0;
    }
    int64_t incl = run;  // inclusive scan over the wave
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int64_t v = __shfl_up(incl, d, 64);
        if (lane >= d) incl += v;
    }
    if (lane == 63) s_wave[wave] = incl;
    __syncthreads();
    int64_t base = incl - run;
    for (int w = 0; w < wave; ++w) base += s_wave[w];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int g = 4 * t + k;
        if (g < grp.G) s_poff[g + 1] = base + part[k];
    }
    __syncthreads();
}

// Last group g with s_poff[g] <= P (G >= 1).
__device__ __forceinline__ int find_group(const int64_t* s_poff, int G, int64_t P) {
    int lo = 0, hi = G - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (s_poff[mid] <= P) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// Column groups per workgroup. With 32 a wave reads 512 contiguous bytes of each row (two blocks of 256
// columns); the block-n RHT kernel keeps 8 so that the m blocks of an n-block lie in one wave.
constexpr int kXG = 64 / kXC;  // block-n RHT
constexpr int kXGD = 32;       // otherwise
static_assert(kXC == 8 || kXC == 4, "columns per thread");

template <int FMT, int ROUND, bool RHT, bool GROUPED, bool WIDE = false>
__global__ __launch_bounds__(256) void quant_cols_kernel(const uint16_t* __restrict__ x, int64_t rows,
                                                             int64_t cols, int64_t prows, int64_t ld,
                                                             int64_t red_total, TGroups grp, QuantArgs qa,
                                                             uint8_t* __restrict__ codes, int64_t code_pld,
                                                             float* __restrict__ scales, int64_t scale_pld) {
    __shared__ int64_t s_off[GROUPED ? kMaxGroupsLds + 1 : 1];
    __shared__ int64_t s_poff[GROUPED ? kMaxGroupsLds + 1 : 1];
    const int t = threadIdx.x;
    if constexpr (GROUPED) load_group_offsets<kBlock>(grp, s_off, s_poff);
    constexpr int XG = WIDE ? kXG : kXGD, XB = 256 / XG;  // column groups, blocks per workgroup
    // Staged stores (dense RTNE): each half-wave (32 threads, one block of 256 operand rows) puts its 2 KB of
    // codes and 1 KB of scales in its own LDS area in output order and reads them back so that every store
    // instruction writes 512 contiguous bytes instead of 16-byte pieces of 64-byte runs. Measured on the 1 GiB
    // tensor: 2% faster for uniform RTNE; SR, E2M1 and the grouped form would lose more to the extra registers
    // (past 128 VGPRs) than they gain, so they store directly.
    constexpr bool STAGE = !WIDE && !GROUPED && FMT == kFmtUniform && ROUND == kRoundRTNE && XG == 32 && kXC == 8;
    __shared__ uint4 s_stage[STAGE ? 8 : 1][STAGE ? 192 : 1];
    const int cg = t % XG, rb = t / XG;
    const int64_t cbase = (int64_t)blockIdx.x * (XG * kXC) + cg * kXC;  // first operand row of the thread
    // Without staging a thread past the last panel has nothing to do. With it, every thread stays: its (zero)
    // data fills its slot of the stage and stores to panels past the end are skipped.
    if (!STAGE && cbase >= prows) return;
    const int ncol = cols - cbase < kXC ? (int)(cols - cbase) : kXC;  // valid columns of the thread (<= 0: none)
    const int64_t nblk = red_total / kBlock;
    constexpr int kW = kXC / 2;  // dwords per row

    for (int64_t gb = (int64_t)blockIdx.y * XB + rb; gb < nblk; gb += (int64_t)gridDim.y * XB) {
        const int64_t P0 = gb * kBlock;
        // the 16 positions of a block lie in one group (group lengths are padded to multiples of 16): rows
        // src0 .. src0 + nvalid - 1 of X, the rest padding
        int64_t src0, nvalid;
        if constexpr (GROUPED) {
            const int lo = find_group(s_poff, grp.G, P0);
            const int64_t local0 = P0 - s_poff[lo];
            src0 = s_off[lo] + local0;
            nvalid = (s_off[lo + 1] - s_off[lo]) - local0;
        } else {
            src0 = P0;
            nvalid = kBlock;
        }
        if (src0 + nvalid > rows) nvalid = rows - src0;  // offsets beyond X are treated as padding
        if (src0 < 0 || nvalid < 0) nvalid = 0;

        uint32_t v[kBlock][kW];
        if (ncol == kXC && nvalid == kBlock) {  // the common case: a full 16 x kXC sub-tile, no per-row tests
#pragma unroll
            for (int j = 0; j < kBlock; ++j) load_row_chunk<kXC>(x + (src0 + j) * ld + cbase, v[j]);
        } else {
#pragma unroll
            for (int j = 0; j < kBlock; ++j) {
#pragma unroll
                for (int k = 0; k < kW; ++k) v[j][k] = 0;
                if (j < nvalid) {
                    const uint16_t* src = x + (src0 + j) * ld + cbase;
                    if (ncol == kXC) {
                        load_row_chunk<kXC>(src, v[j]);
                    } else if (ncol > 0) {  // ragged last columns: no read past column cols - 1
#pragma unroll
                        for (int k = 0; k < kXC; ++k)
                            if (k < ncol) v[j][k >> 1] |= (uint32_t)src[k] << (16 * (k & 1));
                    }
                }
            }
        }
        // Columns past `cols` and rows past a group's tokens hold zeros: such a block quantizes to zero codes
        // and a +0 scale, the padding value, so every block is quantized unconditionally.
        uint32_t clo[kXC], chi[kXC];
        float sc[kXC];
        uint32_t redo = 0;  // blocks outside the fast range (block-16 RHT or none), redone below
#pragma unroll
        for (int q = 0; q < kXC; ++q) {
            const uint32_t sel = (q & 1) ? 0x07060302u : 0x05040100u;  // high or low bf16 of each dword
            uint32_t w[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) w[j] = __builtin_amdgcn_perm(v[2 * j + 1][q >> 1], v[2 * j][q >> 1], sel);
            if constexpr (WIDE) {
                // consecutive blocks of the same columns are held by threads kXG apart (t = rb * kXG + cg)
                double tw[16];
                rht_wide(w, qa, (uint32_t)gb, kXG, tw);
                quant_wide<FMT, ROUND>(tw, qa, (uint32_t)gb, (uint32_t)(cbase + q), clo[q], chi[q], sc[q]);
                __builtin_amdgcn_sched_barrier(0);  // one column at a time: bounds the live fp64 sums
            } else {
                if (quant_block16<FMT, ROUND, RHT, false>(w, qa, (uint32_t)gb, (uint32_t)(cbase + q), clo[q], chi[q],
                                                          sc[q]))
                    redo |= 1u << q;
            }
        }
        // Rare: blocks outside the fast range are quantized again by the exact path. Kept out of the loop above,
        // where its branch would cost registers on every block; the inputs and the row are made opaque so that the
        // compiler recomputes here instead of keeping the loop's sums and draws alive.
        if (!WIDE && __builtin_expect(__builtin_amdgcn_ballot_w64(redo != 0u) != 0, 0)) {
            opaque(v);
            uint32_t row0 = (uint32_t)cbase;
            asm volatile("" : "+v"(row0));
#pragma unroll
            for (int q = 0; q < kXC; ++q) {
                if (redo & (1u << q)) {
                    const uint32_t sel = (q & 1) ? 0x07060302u : 0x05040100u;
                    uint32_t w[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) w[j] = __builtin_amdgcn_perm(v[2 * j + 1][q >> 1], v[2 * j][q >> 1], sel);
                    quant_block16<FMT, ROUND, RHT>(w, qa, (uint32_t)gb, row0 + q, clo[q], chi[q], sc[q]);
                }
            }
        }
        if constexpr (STAGE) {
            // half-wave area: codes of operand rows 0..255 of the block (8 bytes each, uint4 0..127), then their
            // scales (uint4 128..191); thread cg owns rows 8 cg .. 8 cg + 7
            uint4* st = s_stage[t >> 5];
            const int L = t & 31;
#pragma unroll
            for (int q = 0; q < 4; ++q) st[4 * L + q] = make_uint4(clo[2 * q], chi[2 * q], clo[2 * q + 1], chi[2 * q + 1]);
            st[128 + 2 * L] = make_uint4(__float_as_uint(sc[0]), __float_as_uint(sc[1]), __float_as_uint(sc[2]),
                                         __float_as_uint(sc[3]));
            st[129 + 2 * L] = make_uint4(__float_as_uint(sc[4]), __float_as_uint(sc[5]), __float_as_uint(sc[6]),
                                         __float_as_uint(sc[7]));
            // the half-wave reads what its own lanes wrote: LDS operations of a wave complete in order, the wait
            // and the compiler barrier keep the reads after the writes
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            const int64_t P0 = (int64_t)blockIdx.x * 2;  // the block's two panels
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int64_t P = P0 + (q >> 1);
                if (P * kPanelRows < prows)
                    *reinterpret_cast<uint4*>(codes + P * code_pld + gb * 1024 + (q & 1) * 512 + 16 * L) = st[32 * q + L];
            }
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                const int64_t P = P0 + q;
                if (P * kPanelRows < prows)
                    *reinterpret_cast<uint4*>(scales + P * scale_pld + gb * 128 + 4 * L) = st[128 + 32 * q + L];
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // reads done before the next iteration's writes
        } else {
            const int64_t P = cbase >> 7, ri = cbase & 127;  // the kXC rows lie in one panel
            uint4* dc = reinterpret_cast<uint4*>(codes + P * code_pld + gb * 1024 + ri * 8);
#pragma unroll
            for (int q = 0; q < kXC / 2; ++q) dc[q] = make_uint4(clo[2 * q], chi[2 * q], clo[2 * q + 1], chi[2 * q + 1]);
            float4* ds = reinterpret_cast<float4*>(scales + P * scale_pld + gb * 128 + ri);
#pragma unroll
            for (int q = 0; q < kXC / 4; ++q) ds[q] = make_float4(sc[4 * q], sc[4 * q + 1], sc[4 * q + 2], sc[4 * q + 3]);
        }
    }
}

// ------------------------------------------------------------------------------------------------
// Both operands of one tensor X [rows, cols] from one read of X: Q_r = Q(X) along cols (rowwise) and
// Q_c = Q(X^T) along rows (transposed), each with its own RHT flag, sign mask and SR stream; bit for bit the
// results of the two separate kernels. rows and cols are multiples of 16.
//
// A wave covers 256 columns x 2 row groups (512 contiguous bytes of each row it reads), a workgroup four
// waves stacked along the rows. The lanes l and l + 32 of a wave form a pair that owns a 16 x 16 sub-tile:
// rows 16 gb .. 16 gb + 15, columns col0 .. col0 + 15; lane l loads columns col0 .. col0 + 7 of all 16 rows,
// lane l + 32 the other eight. Each lane first quantizes its eight column blocks as the transposed kernel does. One
// v_permlane32_swap per dword then exchanges half of the sub-tile between the two lanes (lanes 0-31 give up
// rows 8-15 and receive columns 8-15 of rows 0-7, lanes 32-63 the converse), after which registers v[i]
// and v[8 + i] hold row 8h + i's full 16-column block in both lanes (h = l / 32). Each lane then quantizes
// eight row blocks and writes them as 64 contiguous bytes (eight consecutive rows of one block).
// Zero codes and scales fill the padding rows of both operands' last panels.
// ------------------------------------------------------------------------------------------------
constexpr int kDC = 16;       // 16-column chunks per wave: 512 contiguous bytes of each row
constexpr int kDB = 32 / kDC;  // 16-row groups per wave

template <int FMT, int ROUND, bool RHT_R, bool RHT_C>
__global__ __launch_bounds__(256) void quant_dual_kernel(const uint16_t* __restrict__ x, int64_t rows, int64_t cols,
                                                         int64_t ld, QuantArgs qr, QuantArgs qc,
                                                         uint8_t* __restrict__ codes_r, int64_t code_pld_r,
                                                         float* __restrict__ scales_r, int64_t scale_pld_r,
                                                         uint8_t* __restrict__ codes_c, int64_t code_pld_c,
                                                         float* __restrict__ scales_c, int64_t scale_pld_c) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int h = lane >> 5, chunk = lane % kDC, rbl = (lane & 31) / kDC;
    const int64_t col0 = (int64_t)blockIdx.x * (16 * kDC) + chunk * 16;  // first column of the pair's sub-tile
    const int64_t cbase = col0 + h * 8;                                  // first column of this lane
    const bool chunk_ok = col0 < cols;  // cols % 16 == 0: the 16 columns are all real or all padding
    if (col0 >= padded_rows(cols)) return;  // past Q_c's last panel (both lanes of the pair)
    const int64_t nblk = rows / kBlock;                 // reduction blocks of Q_c = 16-row groups of X
    const int64_t ngrp = padded_rows(rows) / kBlock;    // 16-row groups including Q_r's padding rows

    for (int64_t gb = (int64_t)blockIdx.y * (4 * kDB) + wave * kDB + rbl; gb < ngrp;
         gb += (int64_t)gridDim.y * (4 * kDB)) {
        const int64_t r0 = gb * kBlock + h * 8;  // first Q_r row of this lane
        const int64_t Pr = r0 >> 7, rir = r0 & 127;
        const int64_t bcol = col0 / kBlock;
        if (gb >= nblk) {  // padding rows of Q_r only
            if (chunk_ok) {
                uint4* dc = reinterpret_cast<uint4*>(codes_r + Pr * code_pld_r + bcol * 1024 + rir * 8);
#pragma unroll
                for (int q = 0; q < 4; ++q) dc[q] = make_uint4(0, 0, 0, 0);
                float4* ds = reinterpret_cast<float4*>(scales_r + Pr * scale_pld_r + bcol * 128 + rir);
                ds[0] = make_float4(0.f, 0.f, 0.f, 0.f);
                ds[1] = make_float4(0.f, 0.f, 0.f, 0.f);
            }
            continue;
        }
        uint32_t v[kBlock][4];
        if (chunk_ok) {
#pragma unroll
            for (int j = 0; j < kBlock; ++j) load_row_chunk<8>(x + (gb * kBlock + j) * ld + cbase, v[j]);
        } else {
#pragma unroll
            for (int j = 0; j < kBlock; ++j) v[j][0] = v[j][1] = v[j][2] = v[j][3] = 0;
        }
        // Q_c: the eight column blocks of this lane (operand rows cbase .. cbase + 7). Past `cols` the data is
        // zero, which quantizes to the padding value (zero codes, +0 scale).
        {
            uint32_t clo[8], chi[8];
            float sc[8];
            uint32_t redo = 0;  // blocks outside the fast range, redone below
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const uint32_t sel = (q & 1) ? 0x07060302u : 0x05040100u;
                uint32_t w[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) w[j] = __builtin_amdgcn_perm(v[2 * j + 1][q >> 1], v[2 * j][q >> 1], sel);
                if (quant_block16<FMT, ROUND, RHT_C, false>(w, qc, (uint32_t)gb, (uint32_t)(cbase + q), clo[q], chi[q],
                                                            sc[q]))
                    redo |= 1u << q;
            }
            const int64_t P = cbase >> 7, ri = cbase & 127;
            uint4* dc = reinterpret_cast<uint4*>(codes_c + P * code_pld_c + gb * 1024 + ri * 8);
#pragma unroll
            for (int q = 0; q < 4; ++q) dc[q] = make_uint4(clo[2 * q], chi[2 * q], clo[2 * q + 1], chi[2 * q + 1]);
            float4* ds = reinterpret_cast<float4*>(scales_c + P * scale_pld_c + gb * 128 + ri);
            ds[0] = make_float4(sc[0], sc[1], sc[2], sc[3]);
            ds[1] = make_float4(sc[4], sc[5], sc[6], sc[7]);
            // Rare: blocks outside the fast range are quantized again by the exact path and stored over the fast
            // results (the same thread wrote them: program order keeps the second store last). Kept out of the loop
            // above, where its branch would cost registers on every block.
            if (__builtin_expect(__builtin_amdgcn_ballot_w64(redo != 0u) != 0, 0)) {
                // inputs and row made opaque: otherwise the compiler reuses the loop's words, sums and draws here
                // and keeps them all alive through the loop
                opaque(v);
                uint32_t row0 = (uint32_t)cbase;
                asm volatile("" : "+v"(row0));
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    if (redo & (1u << q)) {
                        const uint32_t sel = (q & 1) ? 0x07060302u : 0x05040100u;
                        uint32_t w[8];
#pragma unroll
                        for (int j = 0; j < 8; ++j)
                            w[j] = __builtin_amdgcn_perm(v[2 * j + 1][q >> 1], v[2 * j][q >> 1], sel);
                        uint32_t lo, hi;
                        float s1;
                        quant_block16<FMT, ROUND, RHT_C>(w, qc, (uint32_t)gb, row0 + q, lo, hi, s1);
                        *reinterpret_cast<uint2*>(codes_c + P * code_pld_c + gb * 1024 + (ri + q) * 8) = make_uint2(lo, hi);
                        scales_c[P * scale_pld_c + gb * 128 + ri + q] = s1;
                    }
                }
            }
        }
        if (!chunk_ok) continue;  // no Q_r block for padding columns (the partner lane takes the same branch)
        __builtin_amdgcn_sched_barrier(0);  // keep the two phases apart: their temporaries would add up
        // exchange: afterwards v[i] = columns 0-7 and v[8 + i] = columns 8-15 of row 8h + i
#pragma unroll
        for (int i = 0; i < 8; ++i) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const auto r = __builtin_amdgcn_permlane32_swap(v[i][k], v[8 + i][k], false, false);
                v[i][k] = r[0];
                v[8 + i][k] = r[1];
            }
        }
        uint32_t rlo[8], rhi[8];
        float rs[8];
        uint32_t redo = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t w[8] = {v[i][0], v[i][1], v[i][2], v[i][3], v[8 + i][0], v[8 + i][1], v[8 + i][2], v[8 + i][3]};
            if (quant_block16<FMT, ROUND, RHT_R, false>(w, qr, (uint32_t)bcol, (uint32_t)(r0 + i), rlo[i], rhi[i], rs[i]))
                redo |= 1u << i;
        }
        uint4* dc = reinterpret_cast<uint4*>(codes_r + Pr * code_pld_r + bcol * 1024 + rir * 8);
#pragma unroll
        for (int q = 0; q < 4; ++q) dc[q] = make_uint4(rlo[2 * q], rhi[2 * q], rlo[2 * q + 1], rhi[2 * q + 1]);
        float4* ds = reinterpret_cast<float4*>(scales_r + Pr * scale_pld_r + bcol * 128 + rir);
        ds[0] = make_float4(rs[0], rs[1], rs[2], rs[3]);
        ds[1] = make_float4(rs[4], rs[5], rs[6], rs[7]);
        if (__builtin_expect(__builtin_amdgcn_ballot_w64(redo != 0u) != 0, 0)) {  // as for Q_c above
            opaque(v);
            uint32_t row0 = (uint32_t)r0;
            asm volatile("" : "+v"(row0));
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                if (redo & (1u << i)) {
                    const uint32_t w[8] = {v[i][0], v[i][1], v[i][2], v[i][3],
                                           v[8 + i][0], v[8 + i][1], v[8 + i][2], v[8 + i][3]};
                    uint32_t lo, hi;
                    float s1;
                    quant_block16<FMT, ROUND, RHT_R>(w, qr, (uint32_t)bcol, row0 + i, lo, hi, s1);
                    *reinterpret_cast<uint2*>(codes_r + Pr * code_pld_r + bcol * 1024 + (rir + i) * 8) = make_uint2(lo, hi);
                    scales_r[Pr * scale_pld_r + bcol * 128 + rir + i] = s1;
                }
            }
        }
    }
}

// ------------------------------------------------------------------------------------------------
// Power-of-two block scales (the scale hierarchy is free, Sec. 4): blocks of 32 along the reduction axis
// share one scale 2^E, E = floor(log2 amax) - 2 (the OCP Microscaling shared-exponent rule with the levels
// read as E2M3 numbers; |y| / 2^E < 8 and values past the top level are clamped to it), stored as the E8M0
// byte E + 127; the
// RHT stays block-16; codes are the uniform levels -7..7 stored as FP6 E2M3 numbers, 32 of them in 24 bytes
// (element j in bits 6j .. 6j + 5): the A/B operand format of v_mfma_scale_f32_32x32x64_f8f6f4. In a panel
// the 24 bytes of row i's block b are three 8-byte units, unit u at b * 3072 + u * 1024 + i * 8, so that
// consecutive rows' units are contiguous (conflict-free 8-byte LDS reads in the GEMM).
// ------------------------------------------------------------------------------------------------
constexpr int kMxBlock = 32;
typedef float fp6_v16 __attribute__((ext_vector_type(16)));
typedef uint32_t fp6_u6 __attribute__((ext_vector_type(6)));

// One 32-block: sixteen bf16 pairs in (element 2j in the low half of w[j]); 24 bytes of E2M3 codes and the
// E8M0 scale byte out. `blk16` numbers the block's first 16-block along the reduction axis (the SR counters
// count 16-blocks).
template <int ROUND, bool RHT>
__device__ __forceinline__ void quant_block32_mx(const uint32_t (&w)[16], const QuantArgs& qa, uint32_t blk16,
                                                 uint32_t row, uint32_t (&out)[6], uint32_t& e8m0) {
    float y[32];
    rht16_unscaled<RHT>(w, qa, y);
    rht16_unscaled<RHT>(w + 8, qa, y + 16);
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < 32; ++i) amax = __builtin_fmaxf(amax, __builtin_fabsf(y[i]));
    // floor(log2 amax) = (exponent field of amax) - 127 - P, with P = 2 for the folded RHT (y' = 4y) and P = 0
    // otherwise; the exact path (as for the fp32 scales) rescales a block outside the fast range in place by
    // 2^+-64 and adds it to P, so that amax is a normal number. E8M0 holds E >= -127: a tiny block takes the
    // smallest scale. v = y 2^-E is one multiplication by a power of two, exact but below 2^-126.
    int P = RHT ? 2 : 0;
    if (__builtin_expect(needs_exact(amax), 0)) {
        if (RHT && !(amax <= 0x1.fffffep127f)) {  // a rotated value past FLT_MAX: the fp64 sums at 2^-64
            amax = 0.0f;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const uint32_t wh[8] = {w[8 * h], w[8 * h + 1], w[8 * h + 2], w[8 * h + 3],
                                        w[8 * h + 4], w[8 * h + 5], w[8 * h + 6], w[8 * h + 7]};
                double t[16];
                rht16_exact(wh, qa, t);
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    y[16 * h + i] = (float)(t[i] * 0x1p-64);
                    amax = __builtin_fmaxf(amax, __builtin_fabsf(y[16 * h + i]));
                }
            }
            P = -64;
        } else {
            const float q = amax < 1.0f ? 0x1p64f : 0x1p-64f;
#pragma unroll
            for (int i = 0; i < 32; ++i) y[i] = __fmul_rn(y[i], q);
            P += amax < 1.0f ? 64 : -64;
            amax = __fmul_rn(amax, q);
        }
    }
    const int fl = (int)(__float_as_uint(amax) >> 23) - 127 - P;  // floor(log2 amax)
    const int E = fl - 2 > -127 ? fl - 2 : -127;
    e8m0 = amax > 0.0f ? (uint32_t)(E + 127) : 0u;
    const float mult = amax > 0.0f ? __uint_as_float((uint32_t)(127 - P - E) << 23) : 0.0f;  // 2^(-P-E), normal
    // levels as floats (integers -7..7, zero as +0), even elements in `ev`, odd ones in `od`: the E2M3
    // conversion instruction packs ev[i] at bits 12i and od[i] at bits 12i + 6 of its 192-bit result, and an
    // integer of magnitude <= 7 is exact in E2M3, so its rounding and the scale operand 1.0 change nothing
    fp6_v16 ev, od;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        uint32_t u[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        if constexpr (ROUND == kRoundSR) {
            const Philox4 p0 = philox4x32_10(blk16 + h, row, 0u, qa.stream, qa.key0, qa.key1);
            const Philox4 p1 = philox4x32_10(blk16 + h, row, 1u, qa.stream, qa.key0, qa.key1);
            u[0] = p0.x; u[1] = p0.y; u[2] = p0.z; u[3] = p0.w;
            u[4] = p1.x; u[5] = p1.y; u[6] = p1.z; u[7] = p1.w;
        }
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const float vi = __fmul_rn(y[16 * h + i], mult);  // |v| < 8: the top level 7 is the clamp
            float lv;
            if constexpr (ROUND == kRoundSR) {
                const uint32_t u16 = (i & 1) ? (u[i >> 1] >> 16) : (u[i >> 1] & 0xFFFFu);
                lv = uniform_sr_level(vi, u16);
            } else {
                lv = __builtin_rintf(__builtin_fminf(__builtin_fmaxf(vi, -7.0f), 7.0f)) + 0.0f;
            }
            if (i & 1) od[8 * h + (i >> 1)] = lv;
            else ev[8 * h + (i >> 1)] = lv;
        }
    }
    const fp6_u6 c = __builtin_amdgcn_cvt_scalef32_2xpk16_fp6_f32(ev, od, 1.0f);
#pragma unroll
    for (int k = 0; k < 6; ++k) out[k] = c[k];
}

// ------------------------------------------------------------------------------------------------
// Host-side launchers
// ------------------------------------------------------------------------------------------------
// ------------------------------------------------------------------------------------------------
// Quality statistics (Sec. 3.2 diagnostics). Every block is quantized as by the quantizers above, its codes
// are dequantized in registers (q = level * s, exact in fp64) and the kernel accumulates in fp64
// (q - ref)^2, ref^2 and q * ref, where ref is the value the quantizer rounds (the fp32 RHT output, or x),
// and counts the codes per magnitude code; nothing else is written. One thread per block in a grid-stride
// loop. Rowwise: consecutive threads take consecutive blocks of a row (32 contiguous bytes each).
// Transposed: consecutive threads take consecutive operand rows (columns of X) of one block, so each of
// the 16 row loads of a wave reads one contiguous 128-byte run.
// ------------------------------------------------------------------------------------------------
constexpr int kStatsThreads = 256;
constexpr int kStatsMaxGrid = 1024;  // few workgroups: one atomic per field and workgroup

template <int FMT>
__device__ __forceinline__ float level_of_nibble(uint32_t nib) {
    const uint32_t m = nib & 7u;
    float lv;
    if constexpr (FMT == kFmtUniform) lv = (float)m;
    else lv = m <= 4u ? 0.5f * (float)m : (m == 7u ? 6.0f : (float)(m - 2u));  // 0 .5 1 1.5 2 | 3 4 | 6
    return (nib & 8u) ? -lv : lv;
}

__global__ void stats_zero_kernel(QuantStats* out) {
    if (threadIdx.x == 0) {
        out->err2 = 0.0;
        out->ref2 = 0.0;
        out->cross = 0.0;
    }
    if (threadIdx.x < 8) out->hist[threadIdx.x] = 0ull;
}

template <int FMT, int ROUND, bool RHT, bool TRANS>
__global__ __launch_bounds__(kStatsThreads) void quant_stats_kernel(const uint16_t* __restrict__ x, int64_t ld,
                                                                    int64_t qrows, int64_t nb, QuantArgs qa,
                                                                    QuantStats* __restrict__ out) {
    double e2 = 0.0, r2 = 0.0, cr = 0.0;
    uint32_t hist[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    const int64_t total = qrows * nb;
    const int64_t step = (int64_t)gridDim.x * kStatsThreads;
    for (int64_t id = (int64_t)blockIdx.x * kStatsThreads + threadIdx.x; id < total; id += step) {
        int64_t r, b;
        uint32_t w[8];
        if constexpr (!TRANS) {
            r = id / nb;
            b = id - r * nb;
            const uint4* src = reinterpret_cast<const uint4*>(x + r * ld + b * kBlock);
            const uint4 v0 = src[0], v1 = src[1];
            w[0] = v0.x; w[1] = v0.y; w[2] = v0.z; w[3] = v0.w;
            w[4] = v1.x; w[5] = v1.y; w[6] = v1.z; w[7] = v1.w;
        } else {
            b = id / qrows;
            r = id - b * qrows;
            const uint16_t* src = x + b * kBlock * ld + r;
#pragma unroll
            for (int j = 0; j < 8; ++j) w[j] = (uint32_t)src[(2 * j) * ld] | ((uint32_t)src[(2 * j + 1) * ld] << 16);
        }
        uint32_t lo, hi;
        float sc;
        quant_block16<FMT, ROUND, RHT>(w, qa, (uint32_t)b, (uint32_t)r, lo, hi, sc);
        // ref = y: a quarter of y' under the RHT, unless y' overflowed (a rotated value past FLT_MAX: then the
        // fp64 sums give y with 24 significant bits)
        float y[16];
        rht16_unscaled<RHT>(w, qa, y);
        double ref[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) ref[i] = RHT ? 0.25 * (double)y[i] : (double)y[i];
        if (RHT) {
            float ym = 0.0f;
#pragma unroll
            for (int i = 0; i < 16; ++i) ym = __builtin_fmaxf(ym, __builtin_fabsf(y[i]));
            if (__builtin_expect(!(ym <= 0x1.fffffep127f), 0)) {
                double t[16];
                rht16_exact(w, qa, t);
#pragma unroll
                for (int i = 0; i < 16; ++i) ref[i] = (double)(float)(t[i] * 0x1p-64) * 0x1p64;
            }
        }
        const double s = (double)sc;
        uint64_t counts = 0;  // one byte per magnitude code: at most 16 per block
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const uint32_t nib = ((i < 8 ? lo : hi) >> (4 * (i & 7))) & 15u;
            const double q = (double)level_of_nibble<FMT>(nib) * s;  // a 4-bit level times an fp32 scale: exact
            const double d = q - ref[i];
            e2 = __builtin_fma(d, d, e2);
            r2 = __builtin_fma(ref[i], ref[i], r2);
            cr = __builtin_fma(q, ref[i], cr);
            counts += 1ull << (8 * (nib & 7u));
        }
#pragma unroll
        for (int m = 0; m < 8; ++m) hist[m] += (uint32_t)(counts >> (8 * m)) & 0xFFu;
    }
    // wave sums, then the four waves through LDS, then one atomic per field and workgroup
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        e2 += __shfl_xor(e2, o);
        r2 += __shfl_xor(r2, o);
        cr += __shfl_xor(cr, o);
#pragma unroll
        for (int m = 0; m < 8; ++m) hist[m] += __shfl_xor(hist[m], o);
    }
    __shared__ double s_sum[3][kStatsThreads / 64];
    __shared__ uint32_t s_hist[8][kStatsThreads / 64];
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        s_sum[0][wave] = e2;
        s_sum[1][wave] = r2;
        s_sum[2][wave] = cr;
#pragma unroll
        for (int m = 0; m < 8; ++m) s_hist[m][wave] = hist[m];
    }
    __syncthreads();
    if (threadIdx.x < 3) {
        double t = 0.0;
        for (int k = 0; k < kStatsThreads / 64; ++k) t += s_sum[threadIdx.x][k];
        atomicAdd(threadIdx.x == 0 ? &out->err2 : (threadIdx.x == 1 ? &out->ref2 : &out->cross), t);
    } else if (threadIdx.x >= 64 && threadIdx.x < 72) {
        const int m = threadIdx.x - 64;
        unsigned long long t = 0;
        for (int k = 0; k < kStatsThreads / 64; ++k) t += s_hist[m][k];
        if (t) atomicAdd(&out->hist[m], t);
    }
}

template <int FMT, int ROUND, bool RHT>
static hipError_t launch_stats_t(const StatsJob& j, hipStream_t s) {
    const int64_t nb = j.red / kBlock;
    const int64_t total = j.qrows * nb;
    const int64_t want = (total + kStatsThreads - 1) / kStatsThreads;
    const unsigned grid = (unsigned)(want < kStatsMaxGrid ? want : kStatsMaxGrid);
    if (grid == 0) return hipSuccess;
    const uint16_t* x = static_cast<const uint16_t*>(j.x);
    if (j.transpose) quant_stats_kernel<FMT, ROUND, RHT, true><<<grid, kStatsThreads, 0, s>>>(x, j.ld, j.qrows, nb, j.qa, j.stats);
    else quant_stats_kernel<FMT, ROUND, RHT, false><<<grid, kStatsThreads, 0, s>>>(x, j.ld, j.qrows, nb, j.qa, j.stats);
    return hipGetLastError();
}

template <int FMT>
static hipError_t dispatch_stats(const StatsJob& j, hipStream_t s) {
    if (j.rounding == kRoundSR) return j.rht ? launch_stats_t<FMT, kRoundSR, true>(j, s) : launch_stats_t<FMT, kRoundSR, false>(j, s);
    return j.rht ? launch_stats_t<FMT, kRoundRTNE, true>(j, s) : launch_stats_t<FMT, kRoundRTNE, false>(j, s);
}

hipError_t launch_quant_stats(const StatsJob& j, hipStream_t s) {
    stats_zero_kernel<<<1, 64, 0, s>>>(j.stats);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return j.format == kFmtE2M1 ? dispatch_stats<kFmtE2M1>(j, s) : dispatch_stats<kFmtUniform>(j, s);
}

template <int FMT, int ROUND, bool RHT, typename T = uint16_t, bool WIDE = false>
static hipError_t launch_rows_t(const QuantJob& j, hipStream_t s) {
    const int64_t nb = j.red / kBlock;
    const int64_t prows = padded_rows(j.qrows);
    if (nb == 0 || prows == 0) return hipSuccess;
    const dim3 grid((unsigned)((nb + kRB - 1) / kRB), (unsigned)(prows / kRR));
    quant_rows_kernel<FMT, ROUND, RHT, T, WIDE><<<grid, kRT, 0, s>>>(static_cast<const T*>(j.x), j.ld, j.qrows, nb,
                                                                    j.qa, static_cast<uint8_t*>(j.codes), j.code_pld,
                                                                    j.scales, j.scale_pld);
    return hipGetLastError();
}

// ------------------------------------------------------------------------------------------------
// Unfused form (Sec. 5 Q5 compares it with the fused kernel): a standalone block-16 RHT writes y =
// RN32(x S16 H16) in fp32 (one thread per block, 32 bytes in, 64 bytes out), then quant_rows_kernel<.., float>
// quantizes y without a transform. The fp32 intermediate holds y exactly, so both forms give the same codes.
// ------------------------------------------------------------------------------------------------
constexpr int kRhtThreads = 256;

__global__ __launch_bounds__(kRhtThreads) void rht_rows_kernel(const uint16_t* __restrict__ x, int64_t ld,
                                                               int64_t rows, int64_t nb, QuantArgs qa,
                                                               float* __restrict__ y, int64_t ldy) {
    const int64_t b = (int64_t)blockIdx.x * kRhtThreads + threadIdx.x;
    if (b >= nb) return;
    for (int64_t r = blockIdx.y; r < rows; r += gridDim.y) {
        const uint4* src = reinterpret_cast<const uint4*>(x + r * ld + b * kBlock);
        const uint4 v0 = src[0], v1 = src[1];
        const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
        double d[16];
        rht16_sums(w, qa.sign_xor, d);
        float yv[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) yv[i] = (float)(d[i] * 0.25);  // y = RN32(sum / 4); +-inf past FLT_MAX
        float4* dst = reinterpret_cast<float4*>(y + r * ldy + b * kBlock);
#pragma unroll
        for (int c = 0; c < 4; ++c) dst[c] = make_float4(yv[4 * c], yv[4 * c + 1], yv[4 * c + 2], yv[4 * c + 3]);
    }
}

hipError_t launch_rht(const RhtJob& j, hipStream_t s) {
    const int64_t nb = j.cols / kBlock;
    if (nb == 0 || j.rows == 0) return hipSuccess;
    const dim3 grid((unsigned)((nb + kRhtThreads - 1) / kRhtThreads), (unsigned)(j.rows < 65535 ? j.rows : 65535));
    rht_rows_kernel<<<grid, kRhtThreads, 0, s>>>(static_cast<const uint16_t*>(j.x), j.ld, j.rows, nb, j.qa, j.y, j.ldy);
    return hipGetLastError();
}

template <int FMT, int ROUND, bool RHT, bool GROUPED, bool WIDE = false>
static hipError_t launch_cols_t(const QuantJob& j, hipStream_t s) {
    const int64_t prows = padded_rows(j.qrows);
    const int64_t nblk = j.red / kBlock;
    constexpr int XG = WIDE ? kXG : kXGD, XB = 256 / XG;
    const int64_t gy = (nblk + XB - 1) / XB;
    if (prows == 0 || gy == 0) return hipSuccess;
    const dim3 grid((unsigned)((prows + XG * kXC - 1) / (XG * kXC)), (unsigned)(gy < 65535 ? gy : 65535));
    TGroups grp{j.group_off, j.num_groups};
    quant_cols_kernel<FMT, ROUND, RHT, GROUPED, WIDE><<<grid, 256, 0, s>>>(
        static_cast<const uint16_t*>(j.x), j.xrows, j.qrows, prows, j.ld, j.red, grp, j.qa,
        static_cast<uint8_t*>(j.codes), j.code_pld, j.scales, j.scale_pld);
    return hipGetLastError();
}

template <int FMT, int ROUND, bool RHT>
static hipError_t dispatch_layout(const QuantJob& j, hipStream_t s) {
    if (j.input_f32) {
        if constexpr (RHT) return hipErrorInvalidValue;  // rejected by the API layer
        else return launch_rows_t<FMT, ROUND, false, float>(j, s);
    }
    if (j.qa.rht_m > 1) {  // RHT block 32 / 64 / 128 (plain rowwise or transposed; checked by the API layer)
        if constexpr (!RHT) return hipErrorInvalidValue;
        else if (j.group_off) return hipErrorInvalidValue;
        else if (!j.transpose) return launch_rows_t<FMT, ROUND, false, uint16_t, true>(j, s);
        else return launch_cols_t<FMT, ROUND, false, false, true>(j, s);
    }
    if (!j.transpose) return launch_rows_t<FMT, ROUND, RHT>(j, s);
    if (j.group_off) return launch_cols_t<FMT, ROUND, RHT, true>(j, s);
    return launch_cols_t<FMT, ROUND, RHT, false>(j, s);
}

template <int FMT>
static hipError_t dispatch_fmt(const QuantJob& j, hipStream_t s) {
    if (j.rounding == kRoundSR) {
        return j.rht ? dispatch_layout<FMT, kRoundSR, true>(j, s) : dispatch_layout<FMT, kRoundSR, false>(j, s);
    }
    return j.rht ? dispatch_layout<FMT, kRoundRTNE, true>(j, s) : dispatch_layout<FMT, kRoundRTNE, false>(j, s);
}

hipError_t launch_quantize(const QuantJob& j, hipStream_t s) {
    return j.format == kFmtE2M1 ? dispatch_fmt<kFmtE2M1>(j, s) : dispatch_fmt<kFmtUniform>(j, s);
}

template <int FMT, int ROUND, bool RHT_R, bool RHT_C>
static hipError_t launch_dual_t(const DualJob& j, hipStream_t s) {
    const int64_t gx = (padded_rows(j.cols) + 16 * kDC - 1) / (16 * kDC);
    const int64_t gy = (padded_rows(j.rows) / kBlock + 4 * kDB - 1) / (4 * kDB);
    if (gx == 0 || gy == 0) return hipSuccess;
    const dim3 grid((unsigned)gx, (unsigned)(gy < 65535 ? gy : 65535));
    quant_dual_kernel<FMT, ROUND, RHT_R, RHT_C><<<grid, 256, 0, s>>>(
        static_cast<const uint16_t*>(j.x), j.rows, j.cols, j.ld, j.qr, j.qc, static_cast<uint8_t*>(j.codes_r),
        j.code_pld_r, j.scales_r, j.scale_pld_r, static_cast<uint8_t*>(j.codes_c), j.code_pld_c, j.scales_c,
        j.scale_pld_c);
    return hipGetLastError();
}

template <int FMT, int ROUND>
static hipError_t dispatch_dual_rht(const DualJob& j, hipStream_t s) {
    if (j.rht_r) return j.rht_c ? launch_dual_t<FMT, ROUND, true, true>(j, s) : launch_dual_t<FMT, ROUND, true, false>(j, s);
    return j.rht_c ? launch_dual_t<FMT, ROUND, false, true>(j, s) : launch_dual_t<FMT, ROUND, false, false>(j, s);
}

template <int FMT>
static hipError_t dispatch_dual_fmt(const DualJob& j, hipStream_t s) {
    return j.rounding == kRoundSR ? dispatch_dual_rht<FMT, kRoundSR>(j, s) : dispatch_dual_rht<FMT, kRoundRTNE>(j, s);
}

// Power-of-two-scale operands of X [rows, cols] by 32 x 256 tiles of X: Q_r along cols (DO_R; cols % 32 == 0)
// and Q_c = X^T along rows (DO_C; 32 tile rows per reduction block), one or both from a single read. Thread t
// loads 64 contiguous bytes of tile row t / 8 (the X row `src`, or zeros where src < 0), which are one 32-block of
// that row, and quantizes it for Q_r from its registers as row `qr_row` (SR counters: row src); for Q_c it
// leaves the words in LDS and, after one barrier, reads column t of the tile (32 values, block `qc_blk` of Q_c's
// row c0 + t) as bf16 pairs. Q_c's stores are consecutive operand rows (coalesced); Q_r's are 8-byte units of
// eight rows per block. Rows of Q_r below qr_prows past the data, and Q_c rows past the last column, are written
// as zero padding.
struct MxTileOut {
    uint8_t* codes_r;
    int64_t cpld_r;
    uint8_t* scales_r;
    int64_t spld_r;
    uint8_t* codes_c;
    int64_t cpld_c;
    uint8_t* scales_c;
    int64_t spld_c;
};

template <int ROUND, bool RHTR, bool RHTC, bool DO_R, bool DO_C>
__device__ __forceinline__ void mx_tile(const uint16_t* __restrict__ x, int64_t cols, int64_t ld, int64_t src,
                                        int64_t qr_row, int64_t qr_prows, int64_t qc_blk, int64_t c0,
                                        const QuantArgs& qr, const QuantArgs& qc, const MxTileOut& o,
                                        uint32_t* tile) {
    constexpr int kTW = 256 / 2 + 4;  // LDS words per tile row (16 bytes of padding)
    const int t = threadIdx.x, lr = t >> 3, lb = t & 7;
    const int64_t gc = c0 + 32 * lb;
    uint32_t w[16];
    const bool in = src >= 0 && gc + 32 <= cols;
    if (in) {
        const uint4* sp = reinterpret_cast<const uint4*>(x + src * ld + gc);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint4 l = sp[q];
            w[4 * q] = l.x; w[4 * q + 1] = l.y; w[4 * q + 2] = l.z; w[4 * q + 3] = l.w;
        }
    } else {
#pragma unroll
        for (int i = 0; i < 16; ++i) w[i] = 0;
        if (DO_C && !DO_R && src >= 0 && gc < cols) {  // Q_c alone allows any column count: a partial block
            const uint16_t* sp = x + src * ld;
            for (int i = 0; i < 16; ++i) {
                const int64_t k = gc + 2 * i;
                const uint32_t lo = k < cols ? sp[k] : 0u, hi = k + 1 < cols ? sp[k + 1] : 0u;
                w[i] = lo | (hi << 16);
            }
        }
    }
    if constexpr (DO_C) {
        uint4* const trow = reinterpret_cast<uint4*>(tile + lr * kTW + 16 * lb);
#pragma unroll
        for (int q = 0; q < 4; ++q) trow[q] = make_uint4(w[4 * q], w[4 * q + 1], w[4 * q + 2], w[4 * q + 3]);
    }
    if constexpr (DO_R) {
        if (qr_row < qr_prows && gc < cols) {
            uint32_t out[6] = {0, 0, 0, 0, 0, 0};
            uint32_t e8 = 0;
            const int64_t b = gc / kMxBlock;
            if (in) quant_block32_mx<ROUND, RHTR>(w, qr, (uint32_t)(2 * b), (uint32_t)src, out, e8);
            const int64_t P = qr_row >> 7, ri = qr_row & 127;
            uint8_t* dc = o.codes_r + P * o.cpld_r + b * 3072 + ri * 8;
#pragma unroll
            for (int q = 0; q < 3; ++q)
                *reinterpret_cast<uint2*>(dc + q * 1024) = make_uint2(out[2 * q], out[2 * q + 1]);
            o.scales_r[P * o.spld_r + b * 128 + ri] = (uint8_t)e8;
        }
    }
    if constexpr (DO_C) {
        __syncthreads();
        const int64_t cc = c0 + t;
        if (qc_blk >= 0 && cc < padded_rows(cols)) {
            uint32_t out[6] = {0, 0, 0, 0, 0, 0};
            uint32_t e8 = 0;
            if (cc < cols) {
                const uint32_t sel = (t & 1) ? 0x07060302u : 0x05040100u;
                uint32_t v[16];
#pragma unroll
                for (int j = 0; j < 16; ++j)
                    v[j] = __builtin_amdgcn_perm(tile[(2 * j + 1) * kTW + (t >> 1)], tile[2 * j * kTW + (t >> 1)], sel);
                quant_block32_mx<ROUND, RHTC>(v, qc, (uint32_t)(2 * qc_blk), (uint32_t)cc, out, e8);
            }
            const int64_t P = cc >> 7, ri = cc & 127;
            uint8_t* dc = o.codes_c + P * o.cpld_c + qc_blk * 3072 + ri * 8;
#pragma unroll
            for (int q = 0; q < 3; ++q)
                *reinterpret_cast<uint2*>(dc + q * 1024) = make_uint2(out[2 * q], out[2 * q + 1]);
            o.scales_c[P * o.spld_c + qc_blk * 128 + ri] = (uint8_t)e8;
        }
    }
}

constexpr int kMxTileWords = 32 * (256 / 2 + 4);

// Plain operands: workgroup L takes row tile L / n_ctiles and column tile L % n_ctiles (consecutive workgroups
// read adjacent spans of the same rows).
template <int ROUND, bool RHTR, bool RHTC, bool DO_R, bool DO_C>
__global__ __launch_bounds__(256) void mx_tile_kernel(const uint16_t* __restrict__ x, int64_t rows, int64_t cols,
                                                      int64_t ld, uint32_t n_ctiles, QuantArgs qr, QuantArgs qc,
                                                      MxTileOut o) {
    __shared__ uint4 tile4[DO_C ? kMxTileWords / 4 : 1];
    const uint32_t tr = blockIdx.x / n_ctiles, tc = blockIdx.x - tr * n_ctiles;
    const int64_t r0 = (int64_t)tr * 32, gr = r0 + (threadIdx.x >> 3);
    mx_tile<ROUND, RHTR, RHTC, DO_R, DO_C>(x, cols, ld, gr < rows ? gr : -1, gr, padded_rows(rows),
                                           r0 < rows ? r0 / kMxBlock : -1, (int64_t)tc * 256, qr, qc, o,
                                           reinterpret_cast<uint32_t*>(tile4));
}

// Grouped operands: workgroup (tr, y) takes tile row tr of the operand's grouped axis and column tiles
// kMxColChunk y .. kMxColChunk (y + 1) - 1, so that reading the group offsets is shared by a few tiles. GROWS
// (Q_r in grouped-rows form, for the ragged-M GEMMs): operand rows in panels, group g's rows X[off_g ..
// off_{g+1}) from row P_g = sum_{h<g} pad128(m_h), the rest zero; a tile's 32 rows lie in one group's padded
// range. Otherwise (Q_c with a grouped reduction, for bwd_dw): the reduction axis is each group's tokens padded
// to 32, so the tile's 32 positions are rows src0 .. src0 + nvalid - 1 of X and zero padding.
constexpr uint32_t kMxColChunk = 4;

template <int ROUND, bool RHT, bool GROWS>
__global__ __launch_bounds__(256) void mx_tile_grouped_kernel(const uint16_t* __restrict__ x, int64_t xrows,
                                                              int64_t cols, int64_t ld, uint32_t n_ctiles,
                                                              int64_t qr_prows, TGroups grp, QuantArgs qa,
                                                              MxTileOut o) {
    __shared__ int64_t s_off[kMaxGroupsLds + 1];
    __shared__ int64_t s_poff[kMaxGroupsLds + 1];
    __shared__ uint4 tile4[GROWS ? 1 : kMxTileWords / 4];
    load_group_offsets<GROWS ? kPanelRows : kMxBlock>(grp, s_off, s_poff);
    const int lr = threadIdx.x >> 3;
    const int64_t r0 = (int64_t)blockIdx.x * 32;
    const int g = find_group(s_poff, grp.G, r0);
    const int64_t cnt = s_off[g + 1] - s_off[g];
    int64_t src = -1;
    if constexpr (GROWS) {
        const int64_t local = r0 + lr - s_poff[g], sr = s_off[g] + local;
        if (local < cnt && sr >= 0 && sr < xrows) src = sr;
    } else {
        const int64_t local0 = r0 - s_poff[g], src0 = s_off[g] + local0;
        int64_t nvalid = cnt - local0;
        if (src0 + nvalid > xrows) nvalid = xrows - src0;  // offsets beyond X are treated as padding
        if (src0 < 0 || nvalid < 0) nvalid = 0;
        if (lr < nvalid) src = src0 + lr;
    }
    const uint32_t tc_end = min(n_ctiles, (blockIdx.y + 1) * kMxColChunk);
    for (uint32_t tc = blockIdx.y * kMxColChunk; tc < tc_end; ++tc) {
        mx_tile<ROUND, RHT, RHT, GROWS, !GROWS>(x, cols, ld, src, r0 + lr, qr_prows, GROWS ? -1 : r0 / kMxBlock,
                                                (int64_t)tc * 256, qa, qa, o, reinterpret_cast<uint32_t*>(tile4));
        if constexpr (!GROWS) __syncthreads();  // the tile's column reads before the next tile's writes
    }
}

// Tile counts of mx_tile_kernel's grid: Q_r needs the row tiles of its padded rows and the column tiles of the
// columns; Q_c the row tiles of the rows and the column tiles of its padded rows.
template <int ROUND, bool RHTR, bool RHTC, bool DO_R, bool DO_C>
static hipError_t launch_mx_tiles(const void* x, int64_t rows, int64_t cols, int64_t ld, const QuantArgs& qr,
                                  const QuantArgs& qc, const MxTileOut& o, hipStream_t s) {
    const int64_t n_rt = (DO_R ? padded_rows(rows) : rows) / 32;
    const int64_t n_ct = ((DO_C ? padded_rows(cols) : cols) + 255) / 256;
    if (n_rt == 0 || n_ct == 0) return hipSuccess;
    mx_tile_kernel<ROUND, RHTR, RHTC, DO_R, DO_C><<<dim3((unsigned)(n_rt * n_ct)), 256, 0, s>>>(
        static_cast<const uint16_t*>(x), rows, cols, ld, (uint32_t)n_ct, qr, qc, o);
    return hipGetLastError();
}

int64_t mx_tile_count(int64_t rows, int64_t cols, bool do_r, bool do_c) {
    return ((do_r ? padded_rows(rows) : rows) / 32) * (((do_c ? padded_rows(cols) : cols) + 255) / 256);
}

template <int ROUND, bool RHTR, bool RHTC>
static hipError_t launch_mx_dual_t(const MxDualJob& j, hipStream_t s) {
    const MxTileOut o{static_cast<uint8_t*>(j.codes_r), j.code_pld_r, static_cast<uint8_t*>(j.scales_r),
                      j.scale_pld_r, static_cast<uint8_t*>(j.codes_c), j.code_pld_c,
                      static_cast<uint8_t*>(j.scales_c), j.scale_pld_c};
    return launch_mx_tiles<ROUND, RHTR, RHTC, true, true>(j.x, j.rows, j.cols, j.ld, j.qr, j.qc, o, s);
}

template <int ROUND>
static hipError_t launch_mx_dual_r(const MxDualJob& j, hipStream_t s) {
    if (j.rht_r) return j.rht_c ? launch_mx_dual_t<ROUND, true, true>(j, s) : launch_mx_dual_t<ROUND, true, false>(j, s);
    return j.rht_c ? launch_mx_dual_t<ROUND, false, true>(j, s) : launch_mx_dual_t<ROUND, false, false>(j, s);
}

hipError_t launch_quantize_mx_dual(const MxDualJob& j, hipStream_t s) {
    return j.rounding == kRoundSR ? launch_mx_dual_r<kRoundSR>(j, s) : launch_mx_dual_r<kRoundRTNE>(j, s);
}

template <int ROUND, bool RHT, bool GR>
static hipError_t launch_mx_t(const MxQuantJob& j, hipStream_t s) {
    uint8_t* const c = static_cast<uint8_t*>(j.codes);
    uint8_t* const sc = static_cast<uint8_t*>(j.scales);
    const MxTileOut o = j.transpose ? MxTileOut{nullptr, 0, nullptr, 0, c, j.code_pld, sc, j.scale_pld}
                                    : MxTileOut{c, j.code_pld, sc, j.scale_pld, nullptr, 0, nullptr, 0};
    if constexpr (!GR) {  // the tile kernel with one output
        if (!j.transpose)
            return launch_mx_tiles<ROUND, RHT, false, true, false>(j.x, j.xrows, j.red, j.ld, j.qa, j.qa, o, s);
        return launch_mx_tiles<ROUND, false, RHT, false, true>(j.x, j.red, j.qrows, j.ld, j.qa, j.qa, o, s);
    } else {
        // grouped rows: Q_r [qrows, cols] with qrows the padded total; grouped reduction: Q_c [cols, red] with
        // red the padded token total; one workgroup per 32 positions of the grouped axis
        const int64_t cols = j.transpose ? j.qrows : j.red;
        const int64_t n_rt = (j.transpose ? j.red : j.qrows) / 32;
        const int64_t n_ct = ((j.transpose ? padded_rows(cols) : cols) + 255) / 256;
        if (n_rt == 0 || n_ct == 0) return hipSuccess;
        const TGroups grp{j.group_off, j.num_groups};
        const dim3 grid((unsigned)n_rt, (unsigned)((n_ct + kMxColChunk - 1) / kMxColChunk));
        if (j.transpose)
            mx_tile_grouped_kernel<ROUND, RHT, false><<<grid, 256, 0, s>>>(
                static_cast<const uint16_t*>(j.x), j.xrows, cols, j.ld, (uint32_t)n_ct, 0, grp, j.qa, o);
        else
            mx_tile_grouped_kernel<ROUND, RHT, true><<<grid, 256, 0, s>>>(
                static_cast<const uint16_t*>(j.x), j.xrows, cols, j.ld, (uint32_t)n_ct, j.qrows, grp, j.qa, o);
        return hipGetLastError();
    }
}

template <int ROUND, bool RHT>
static hipError_t launch_mx_g(const MxQuantJob& j, hipStream_t s) {
    return j.group_off ? launch_mx_t<ROUND, RHT, true>(j, s) : launch_mx_t<ROUND, RHT, false>(j, s);
}

hipError_t launch_quantize_mx(const MxQuantJob& j, hipStream_t s) {
    if (j.rounding == kRoundSR) return j.rht ? launch_mx_g<kRoundSR, true>(j, s) : launch_mx_g<kRoundSR, false>(j, s);
    return j.rht ? launch_mx_g<kRoundRTNE, true>(j, s) : launch_mx_g<kRoundRTNE, false>(j, s);
}

hipError_t launch_quantize_dual(const DualJob& j, hipStream_t s) {
    return j.format == kFmtE2M1 ? dispatch_dual_fmt<kFmtE2M1>(j, s) : dispatch_dual_fmt<kFmtUniform>(j, s);
}

int max_groups_quantize() { return kMaxGroupsLds; }

}  // namespace ufp4
