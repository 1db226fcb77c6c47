// Fused block-16 RHT + 1x16 block-scaled 4-bit quantization (uniform grid -7..7, or the E2M1 baseline).
//
// What is computed per 16-element block of an operand's reduction axis (Sec. 2.1 quantizer display,
// Sec. 2.2 RHT, recipe of Sec. 4 / Table 1):
//   y    = RN32( x S_16 H_16 )            exact 16-term sum in fp64 (Sylvester butterfly), one rounding
//   s    = RN32(amax / g),  r = RN32(g / amax),  v = RN32(y * r)
//   code = RTNE(v) or SR(v; Philox draw)  onto the grid, clamped to +-g
//
// Two layouts: rowwise (reduction axis contiguous, one thread per block, 32-byte loads) and transposed
// (reduction axis strided: a 128x64 tile is staged through LDS, each thread builds two column blocks
// from LDS, and the packed codes are restaged so that every output row is written in 64-byte runs).
// The transposed kernel also serves grouped (MoE) tensors whose token axis is cut into groups that are
// zero-padded to a multiple of 16.
//
// This translation unit is compiled with -ffp-contract=off: every fp32/fp64 operation above must round
// exactly once, as written.

#include "ufp4_device.h"
#include "ufp4_internal.h"

namespace ufp4 {

// ------------------------------------------------------------------------------------------------
// Per-element rounding onto the grid; returns the 4-bit code in the low bits.
// ------------------------------------------------------------------------------------------------

// 1.5 * 2^23: adding it to 0 <= x <= 2^22 rounds x to an integer (round-half-even in the current rounding
// mode) and leaves that integer in the low mantissa bits.
constexpr float kMagic = 12582912.0f;

// Codes are sign-magnitude nibbles: sign in bit 3, |k| in bits 0-2, zero as +0.
//
// RTNE: rounding is symmetric, so |k| = rint(|v|); k < 0 exactly when v < -1/2. No clamp is needed:
// |v| = RN(|y| * RN(7/amax)) <= 7 (1 + 2^-23), which still rounds to 7.
__device__ __forceinline__ uint32_t uniform_rtne(float v) {
    const uint32_t mag = __float_as_uint(__builtin_fabsf(v) + kMagic) & 0x7u;
    return mag | (v < -0.5f ? 8u : 0u);
}

// Stochastic rounding between the integers lo = floor(v) and lo + 1: up iff lo + u/2^16 < v. Both sides
// are exact in fp32 (lo + u/2^16 needs at most 20 significant bits), so the decision is exact.
__device__ __forceinline__ uint32_t uniform_sr(float v, uint32_t u16) {
    const float vc = __builtin_fminf(__builtin_fmaxf(v, -7.0f), 7.0f);
    const float lo = floorf(vc);
    const float t = __builtin_fmaf((float)u16, 1.0f / 65536.0f, lo);
    const float k = (t < vc) ? lo + 1.0f : lo;
    const uint32_t mag = __float_as_uint(__builtin_fabsf(k) + kMagic) & 0x7u;
    return mag | (k < 0.0f ? 8u : 0u);
}

// E2M1 magnitude code of the nearest level, ties to the even code (levels 0,.5,1,1.5,2,3,4,6; the bin
// edges are the midpoints; an edge belongs to the even-coded side).
__device__ __forceinline__ uint32_t e2m1_mag_rtne(float a) {
    return (uint32_t)(a > 0.25f) + (uint32_t)(a >= 0.75f) + (uint32_t)(a > 1.25f) + (uint32_t)(a >= 1.75f) +
           (uint32_t)(a > 2.5f) + (uint32_t)(a >= 3.5f) + (uint32_t)(a > 5.0f);
}

__device__ __forceinline__ uint32_t e2m1_rtne(float v) {
    const uint32_t idx = e2m1_mag_rtne(__builtin_fabsf(v));
    return idx | ((v < 0.0f && idx != 0u) ? 8u : 0u);
}

// E2M1 level (exact) -> magnitude code.
__device__ __forceinline__ uint32_t e2m1_code_of_level(float q) {
    const float m = __builtin_fabsf(q);
    const uint32_t idx = m <= 2.0f ? (uint32_t)(2.0f * m) : (m <= 4.0f ? (uint32_t)m + 2u : 7u);
    return idx | ((q < 0.0f && idx != 0u) ? 8u : 0u);
}

// SR over adjacent signed E2M1 levels g_a <= v < g_b (spacing d = g_b - g_a in {0.5, 1, 2}):
// q = g_b iff g_a + d * u/2^16 < v. For v >= 0 the bracket is [lower, upper) in magnitude, for v < 0 it
// is (-upper, -lower] mirrored, so that a value on a level never moves.
__device__ __forceinline__ uint32_t e2m1_sr(float v, uint32_t u16) {
    const float vc = __builtin_fminf(__builtin_fmaxf(v, -6.0f), 6.0f);
    const float a = __builtin_fabsf(vc);
    float ga, d;
    if (vc >= 0.0f) {
        d = a < 2.0f ? 0.5f : (a < 4.0f ? 1.0f : 2.0f);
        ga = floorf(a / d) * d;  // division by a power of two: exact
    } else {
        d = a <= 2.0f ? 0.5f : (a <= 4.0f ? 1.0f : 2.0f);
        ga = -(ceilf(a / d) * d);
    }
    const float t = __builtin_fmaf((float)u16 * (1.0f / 65536.0f), d, ga);
    const float q = (t < vc) ? ga + d : ga;
    return e2m1_code_of_level(q);
}

template <int FMT, int ROUND>
__device__ __forceinline__ uint32_t round_code(float v, uint32_t u16) {
    if constexpr (FMT == kFmtUniform) {
        if constexpr (ROUND == kRoundSR) return uniform_sr(v, u16);
        else return uniform_rtne(v);
    } else {
        if constexpr (ROUND == kRoundSR) return e2m1_sr(v, u16);
        else return e2m1_rtne(v);
    }
}

// ------------------------------------------------------------------------------------------------
// One 16-block: eight bf16 pairs in (element 2j in the low half of w[j]), packed codes + scale out.
// ------------------------------------------------------------------------------------------------
template <int FMT, int ROUND, bool RHT>
__device__ __forceinline__ void quant_block16(const uint32_t (&w)[8], const QuantArgs& qa, uint32_t blk, uint32_t row,
                                              uint32_t& code_lo, uint32_t& code_hi, float& scale) {
    float y[16];
    if constexpr (RHT) {
        double d[16];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t p = w[j] ^ qa.sign_xor[j];  // eps_j = -1: flip the bf16 sign bit
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
#pragma unroll
        for (int i = 0; i < 16; ++i) y[i] = (float)(d[i] * 0.25);
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            y[2 * j] = bf16_lo(w[j]);
            y[2 * j + 1] = bf16_hi(w[j]);
        }
    }
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) amax = __builtin_fmaxf(amax, __builtin_fabsf(y[i]));
    constexpr float g = FMT == kFmtUniform ? 7.0f : 6.0f;
    scale = amax / g;                               // IEEE-correct fp32 division
    const float r = amax > 0.0f ? g / amax : 0.0f;  // zero block: all v = 0, codes 0

    uint32_t u[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if constexpr (ROUND == kRoundSR) {
        const Philox4 p0 = philox4x32_10(blk, row, 0u, qa.stream, qa.key0, qa.key1);
        const Philox4 p1 = philox4x32_10(blk, row, 1u, qa.stream, qa.key0, qa.key1);
        u[0] = p0.x; u[1] = p0.y; u[2] = p0.z; u[3] = p0.w;
        u[4] = p1.x; u[5] = p1.y; u[6] = p1.z; u[7] = p1.w;
    }
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const float v = __fmul_rn(y[i], r);
        const uint32_t u16 = (i & 1) ? (u[i >> 1] >> 16) : (u[i >> 1] & 0xFFFFu);
        const uint32_t c = round_code<FMT, ROUND>(v, u16);
        if (i < 8) lo |= c << (4 * i);
        else hi |= c << (4 * (i - 8));
    }
    code_lo = lo;
    code_hi = hi;
}

// ------------------------------------------------------------------------------------------------
// Rowwise: reduction axis contiguous. One thread per 16-block.
// ------------------------------------------------------------------------------------------------
template <int FMT, int ROUND, bool RHT>
__global__ __launch_bounds__(256) void quant_rows_kernel(const uint16_t* __restrict__ x, int64_t ld, uint32_t total,
                                                         FastDiv nb, QuantArgs qa, uint8_t* __restrict__ codes,
                                                         int64_t code_ld, float* __restrict__ scales, int64_t scale_ld) {
    const uint32_t i = blockIdx.x * 256u + threadIdx.x;
    if (i >= total) return;
    const uint32_t r = fastdiv(i, nb);
    const uint32_t b = i - r * nb.d;
    const uint4* src = reinterpret_cast<const uint4*>(x + (int64_t)r * ld + (int64_t)b * kBlock);
    const uint4 v0 = src[0];
    const uint4 v1 = src[1];
    const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
    uint32_t lo, hi;
    float s;
    quant_block16<FMT, ROUND, RHT>(w, qa, b, r, lo, hi, s);
    *reinterpret_cast<uint2*>(codes + (int64_t)r * code_ld + (int64_t)b * 8) = make_uint2(lo, hi);
    scales[(int64_t)r * scale_ld + b] = s;
}

// ------------------------------------------------------------------------------------------------
// Transposed (and grouped-transposed): operand A = X^T, reduction along X's rows.
// Tile: 128 padded reduction positions (8 blocks) x 64 columns of X. 256 threads.
// ------------------------------------------------------------------------------------------------
constexpr int kTR = 128;               // tile rows (reduction positions), 8 blocks
constexpr int kTC = 64;                // tile columns (operand rows of A)
constexpr int kTStride = kTC / 2 + 4;  // LDS tile row stride in dwords (bf16 pairs), padded
constexpr int kMaxGroupsLds = 1024;

struct TGroups {
    const int64_t* off;   // token offsets [G+1] (device), nullptr for a dense tensor
    const int64_t* poff;  // padded offsets [G+1] (device)
    int32_t G;
};

template <int FMT, int ROUND, bool RHT, bool GROUPED>
__global__ __launch_bounds__(256) void quant_cols_kernel(const uint16_t* __restrict__ x, int64_t rows, int64_t cols,
                                                         int64_t ld, int64_t red_total, TGroups grp, QuantArgs qa,
                                                         uint8_t* __restrict__ codes, int64_t code_ld,
                                                         float* __restrict__ scales, int64_t scale_ld) {
    __shared__ uint32_t tile[kTR * kTStride];
    __shared__ int64_t src_row[kTR];
    __shared__ uint2 out_codes[kTC][kTR / kBlock + 1];
    __shared__ float out_scales[kTC][kTR / kBlock + 1];
    __shared__ int64_t s_off[GROUPED ? kMaxGroupsLds + 1 : 1];
    __shared__ int64_t s_poff[GROUPED ? kMaxGroupsLds + 1 : 1];

    const int t = threadIdx.x;
    const int64_t c0 = (int64_t)blockIdx.x * kTC;

    if constexpr (GROUPED) {
        for (int g = t; g <= grp.G; g += 256) {
            s_off[g] = grp.off[g];
            s_poff[g] = grp.poff[g];
        }
        __syncthreads();
    }

    for (int64_t p0 = (int64_t)blockIdx.y * kTR; p0 < red_total; p0 += (int64_t)gridDim.y * kTR) {
        // 1. source row of every tile row (-1: zero padding or past the end)
        if (t < kTR) {
            const int64_t P = p0 + t;
            int64_t sr = -1;
            if (P < red_total) {
                if constexpr (GROUPED) {
                    int lo = 0, hi = grp.G - 1;  // last group with poff[g] <= P
                    while (lo < hi) {
                        const int mid = (lo + hi + 1) >> 1;
                        if (s_poff[mid] <= P) lo = mid;
                        else hi = mid - 1;
                    }
                    const int64_t local = P - s_poff[lo];
                    // rows past the group's tokens are padding; offsets beyond X are treated as padding too
                    if (local < s_off[lo + 1] - s_off[lo] && s_off[lo] + local < rows) sr = s_off[lo] + local;
                } else {
                    sr = P;
                }
            }
            src_row[t] = sr;
        }
        __syncthreads();

        // 2. load the 128 x 64 bf16 tile (16 bytes per thread and pass, 8 threads per tile row)
        const bool full_cols = c0 + kTC <= cols;
#pragma unroll
        for (int pass = 0; pass < 4; ++pass) {
            const int chunk = t + 256 * pass;
            const int row = chunk >> 3, c8 = chunk & 7;
            const int64_t sr = src_row[row];
            uint4 v = make_uint4(0, 0, 0, 0);
            if (sr >= 0) {
                const uint16_t* src = x + sr * ld + c0 + c8 * 8;
                if (full_cols) {
                    v = *reinterpret_cast<const uint4*>(src);
                } else {
                    uint16_t e[8];
#pragma unroll
                    for (int k = 0; k < 8; ++k) e[k] = (c0 + c8 * 8 + k < cols) ? src[k] : (uint16_t)0;
                    v = make_uint4(e[0] | ((uint32_t)e[1] << 16), e[2] | ((uint32_t)e[3] << 16),
                                   e[4] | ((uint32_t)e[5] << 16), e[6] | ((uint32_t)e[7] << 16));
                }
            }
            uint32_t* dst = &tile[row * kTStride + c8 * 4];
            dst[0] = v.x;
            dst[1] = v.y;
            dst[2] = v.z;
            dst[3] = v.w;
        }
        __syncthreads();

        // 3. each thread: column pair (2p, 2p+1), block bl of the tile
        {
            const int p = t & 31, bl = t >> 5;
            uint32_t col_lo[8], col_hi[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const uint32_t a = tile[(bl * kBlock + 2 * j) * kTStride + p];
                const uint32_t b = tile[(bl * kBlock + 2 * j + 1) * kTStride + p];
                col_lo[j] = (a & 0xFFFFu) | (b << 16);
                col_hi[j] = (a >> 16) | (b & 0xFFFF0000u);
            }
            const uint32_t gblk = (uint32_t)(p0 / kBlock) + bl;
            const bool blk_ok = p0 + bl * kBlock < red_total;
            uint32_t lo, hi;
            float s;
            const int64_t ca = c0 + 2 * p, cb = ca + 1;
            if (blk_ok && ca < cols) {
                quant_block16<FMT, ROUND, RHT>(col_lo, qa, gblk, (uint32_t)ca, lo, hi, s);
                out_codes[2 * p][bl] = make_uint2(lo, hi);
                out_scales[2 * p][bl] = s;
            }
            if (blk_ok && cb < cols) {
                quant_block16<FMT, ROUND, RHT>(col_hi, qa, gblk, (uint32_t)cb, lo, hi, s);
                out_codes[2 * p + 1][bl] = make_uint2(lo, hi);
                out_scales[2 * p + 1][bl] = s;
            }
        }
        __syncthreads();

        // 4. write out: 64 operand rows x 8 blocks; 8 consecutive threads cover one row's 64 bytes
        const int64_t b0 = p0 / kBlock;
#pragma unroll
        for (int pass = 0; pass < 2; ++pass) {
            const int e = t + 256 * pass;
            const int cl = e >> 3, bl = e & 7;
            const int64_t c = c0 + cl;
            if (c < cols && p0 + bl * kBlock < red_total) {
                *reinterpret_cast<uint2*>(codes + c * code_ld + (b0 + bl) * 8) = out_codes[cl][bl];
                scales[c * scale_ld + b0 + bl] = out_scales[cl][bl];
            }
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------------------------------------
// Host-side launchers
// ------------------------------------------------------------------------------------------------
template <int FMT, int ROUND, bool RHT>
static hipError_t launch_rows_t(const QuantJob& j, hipStream_t s) {
    const uint32_t nb = (uint32_t)(j.red / kBlock);
    const uint32_t total = (uint32_t)(j.qrows * nb);
    const dim3 grid((total + 255) / 256);
    quant_rows_kernel<FMT, ROUND, RHT><<<grid, 256, 0, s>>>(static_cast<const uint16_t*>(j.x), j.ld, total,
                                                           make_fastdiv(nb), j.qa, static_cast<uint8_t*>(j.codes),
                                                           j.code_ld, j.scales, j.scale_ld);
    return hipGetLastError();
}

template <int FMT, int ROUND, bool RHT, bool GROUPED>
static hipError_t launch_cols_t(const QuantJob& j, hipStream_t s) {
    const int64_t gy = (j.red + kTR - 1) / kTR;
    const dim3 grid((unsigned)((j.qrows + kTC - 1) / kTC), (unsigned)(gy < 65535 ? gy : 65535));
    TGroups grp{j.group_off, j.group_poff, j.num_groups};
    quant_cols_kernel<FMT, ROUND, RHT, GROUPED><<<grid, 256, 0, s>>>(
        static_cast<const uint16_t*>(j.x), j.xrows, j.qrows, j.ld, j.red, grp, j.qa, static_cast<uint8_t*>(j.codes),
        j.code_ld, j.scales, j.scale_ld);
    return hipGetLastError();
}

template <int FMT, int ROUND, bool RHT>
static hipError_t dispatch_layout(const QuantJob& j, hipStream_t s) {
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

int max_groups_quantize() { return kMaxGroupsLds; }

}  // namespace ufp4
