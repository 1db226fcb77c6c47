// Block-scaled 4-bit NT GEMM on CDNA4 int8 MFMA (Sec. 2.2: Y_hat = Q(XH') Q(WH')^T; the three training
// GEMMs fwd_y, bwd_dx, bwd_dw all take this form once both operands are stored reduction-contiguous).
//
//   C[i, j] = sum_b  sA[i,b] * sB[j,b] * D_b[i, j],   D_b[i, j] = sum_{k in block b} A[i,k] * B[j,k]
//
// Every 16-element K-block has its own fp32 scale on both sides, so D_b is formed per block by one
// v_mfma_i32_32x32x16_i8 (K = 16 exactly) and folded into an fp32 accumulator by the VALU:
// acc += float(D_b) * (sA * sB). Codes are expanded to int8 through byte-permute tables: uniform codes to k,
// E2M1 codes to 2 * level (exact in int8; the factor 4 on D_b is undone at the end).
//
// Work split: 128 x 128 output tile per workgroup, 4 waves in 2 x 2, each wave 64 x 64 = 2 x 2 MFMA
// tiles. K is staged through LDS 8 blocks (128 codes) at a time, double-buffered: the next stage's
// global loads are in flight while the current one is computed. LDS holds codes as planes
// [block][half][row] (one dword = 8 codes per row and half), so the MFMA operand reads of a half-wave
// are 32 consecutive dwords; scales as planes [block][row].
//
// Grouped (MoE) problems: ragged M (fwd_y, bwd_dx: token rows split into groups) resolves its group
// from the tile index with a wave-wide prefix sum over the group sizes; ragged K (bwd_dw: the reduction
// runs over each group's padded token range) takes the group from blockIdx.z.

#include <cstdlib>
#include <cstring>

#include "ufp4_device.h"
#include "ufp4_internal.h"

namespace ufp4 {

typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128;
constexpr int SKB = 8;         // K-blocks per LDS stage
constexpr int CPL = BM + 2;    // dwords per code plane (row stride offset of 2 banks between planes)
constexpr int SPL = BM + 4;    // floats per scale plane
static_assert(BM == BN, "one plane stride for both operands");

struct alignas(16) GemmSmem {
    uint32_t a[2][SKB * 2 * CPL];
    uint32_t b[2][SKB * 2 * CPL];
    float as[2][SKB * SPL];
    float bs[2][SKB * SPL];
    int32_t grp[2];
};

// Per-byte sign masks: byte i of the result is 0xFF when bit 7 of byte i of x is set, else 0x00. The byte
// permute's selectors 8..11 replicate bits 15, 31, 47 and 63 of {x << 8, x}, i.e. bits 15, 31, 7, 23 of x.
__device__ __forceinline__ uint32_t byte_sign_mask(uint32_t x) {
    return __builtin_amdgcn_perm(x << 8, x, 0x090B080Au);
}

// 4 uniform sign-magnitude nibbles, one per byte (low 4 bits) -> 4 int8 holding the code k.
__device__ __forceinline__ uint32_t uniform_bytes_to_i8(uint32_t nib) {
    const uint32_t mag = nib & 0x07070707u;
    const uint32_t neg = __builtin_amdgcn_perm(0xF9FAFBFCu, 0xFDFEFF00u, mag);  // 0 -1 -2 .. -7
    const uint32_t m = byte_sign_mask(nib << 4);
    return (neg & m) | (mag & ~m);
}

// 8 packed uniform codes (one dword) -> 8 int8 lanes (even codes first, then odd).
__device__ __forceinline__ long expand_uniform(uint32_t d) {
    const uint32_t lo = uniform_bytes_to_i8(d & 0x0F0F0F0Fu);
    const uint32_t hi = uniform_bytes_to_i8((d >> 4) & 0x0F0F0F0Fu);
    return (long)(((uint64_t)hi << 32) | lo);
}

// 4 E2M1 nibbles, one per byte (low 4 bits) -> 4 int8 holding 2 * level.
__device__ __forceinline__ uint32_t e2m1_bytes_to_i8x2(uint32_t nib) {
    const uint32_t sel = nib & 0x07070707u;
    // magnitudes * 2: 0 1 2 3 4 6 8 12 and their negations
    const uint32_t pos = __builtin_amdgcn_perm(0x0C080604u, 0x03020100u, sel);
    const uint32_t neg = __builtin_amdgcn_perm(0xF4F8FAFCu, 0xFDFEFF00u, sel);
    const uint32_t m = ((nib >> 3) & 0x01010101u) * 0xFFu;
    return (pos & ~m) | (neg & m);
}

__device__ __forceinline__ long expand_e2m1(uint32_t d) {
    const uint32_t lo = e2m1_bytes_to_i8x2(d & 0x0F0F0F0Fu);
    const uint32_t hi = e2m1_bytes_to_i8x2((d >> 4) & 0x0F0F0F0Fu);
    return (long)(((uint64_t)hi << 32) | lo);
}

template <int FMT>
__device__ __forceinline__ long expand(uint32_t d) {
    if constexpr (FMT == kFmtUniform) return expand_uniform(d);
    else return expand_e2m1(d);
}

struct GemmArgs {
    GemmJob j;
};

// The problem one workgroup works on, with pointers already advanced to its tile / group.
struct Tile {
    const uint8_t* a;
    const float* as;
    const uint8_t* b;
    const float* bs;
    int mrows, nrows;  // valid rows of the tile in A and B
    int64_t nkb;       // reduction blocks
    int64_t c_off;     // element offset of the tile's (0, 0) in C
};

// Ragged-M: find the group owning global m-tile t. Wave 0 runs a prefix sum over per-group tile counts,
// 64 groups at a time; the result goes through LDS. Returns false for tiles past the last group.
__device__ bool resolve_ragged_m(const GemmJob& j, int32_t* grp, int64_t t, int& g_out, int64_t& local_tile) {
    const int tid = threadIdx.x;
    if (tid == 0) grp[0] = -1;
    __syncthreads();
    if (tid < 64) {
        int64_t base = 0;
        for (int g0 = 0; g0 < j.G; g0 += 64) {
            const int g = g0 + tid;
            int64_t cnt = 0;
            if (g < j.G) cnt = (j.offsets[g + 1] - j.offsets[g] + BM - 1) / BM;
            int64_t incl = cnt;
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const int64_t v = __shfl_up(incl, d, 64);
                if (tid >= d) incl += v;
            }
            const int64_t excl = incl - cnt;
            if (cnt > 0 && base + excl <= t && t < base + incl) {
                grp[0] = g;
                grp[1] = (int32_t)(t - base - excl);
            }
            base += __shfl(incl, 63, 64);
        }
    }
    __syncthreads();
    g_out = grp[0];
    local_tile = grp[1];
    return g_out >= 0;
}

// Write a workgroup's 128 x 128 fp32 accumulator tile (four waves, 2 x 2 MFMA tiles of 32 x 32 each; output
// row of register i in lane l: 8 (i / 4) + 4 (l / 32) + i % 4, column l % 32), scaled by `mul`.
template <int OUT>
__device__ __forceinline__ void store_tile(const GemmJob& j, const Tile& tl, const float (&acc)[2][2][16], float mul,
                                           int wm, int wn, int h, int l32) {
#pragma unroll
    for (int a = 0; a < 2; ++a) {
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int col = wn * 64 + b * 32 + l32;
            if (col >= tl.nrows) continue;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int row = wm * 64 + a * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
                if (row >= tl.mrows) continue;
                const float v = acc[a][b][i] * mul;
                const int64_t off = tl.c_off + (int64_t)row * j.ldc + col;
                if constexpr (OUT == kOutF32) {
                    static_cast<float*>(j.c)[off] = v;
                } else {
                    static_cast<uint16_t*>(j.c)[off] = (uint16_t)f32_to_bf16_bits(v);
                }
            }
        }
    }
}

// Resolve the workgroup's output tile (dense, ragged-M group or ragged-K group). Returns false when the
// workgroup has nothing to do (a ragged-M tile index past the last group); all threads agree.
__device__ bool resolve_tile(const GemmJob& j, int32_t* grp, Tile& tl) {
    const int64_t tn = blockIdx.x;
    if (j.mode == kGemmRaggedM) {
        int g;
        int64_t lt;
        if (!resolve_ragged_m(j, grp, blockIdx.y, g, lt)) return false;
        const int64_t r0 = j.offsets[g] + lt * BM;
        const int64_t end = j.offsets[g + 1] < j.M ? j.offsets[g + 1] : j.M;  // offsets past M_total: ignored
        const int64_t rows_g = end - r0;
        if (rows_g <= 0) return false;
        tl.a = j.a + r0 * j.lda;
        tl.as = j.as + r0 * j.ldas;
        const int64_t brow = g * j.b_group_rows + tn * BN;
        const int64_t bkb = g * j.b_group_kb;
        tl.b = j.b + brow * j.ldb + bkb * 8;
        tl.bs = j.bs + brow * j.ldbs + bkb;
        tl.mrows = (int)(rows_g < BM ? rows_g : BM);
        const int64_t nr = j.N - tn * BN;
        tl.nrows = (int)(nr < BN ? nr : BN);
        tl.nkb = j.nkb;
        tl.c_off = r0 * j.ldc + tn * BN;
    } else {
        const int64_t tm = blockIdx.y;
        int64_t kb0 = 0, c_base = 0;
        tl.nkb = j.nkb;
        if (j.mode == kGemmRaggedK) {
            const int g = blockIdx.z;
            // the group's padded token range, clamped to the operands' reduction length
            const int64_t p0 = j.offsets[g] < j.red_total ? j.offsets[g] : j.red_total;
            const int64_t p1 = j.offsets[g + 1] < j.red_total ? j.offsets[g + 1] : j.red_total;
            kb0 = p0 / 16;
            tl.nkb = p1 > p0 ? (p1 - p0) / 16 : 0;
            c_base = (int64_t)g * j.M * j.ldc;
        }
        tl.a = j.a + tm * BM * j.lda + kb0 * 8;
        tl.as = j.as + tm * BM * j.ldas + kb0;
        tl.b = j.b + tn * BN * j.ldb + kb0 * 8;
        tl.bs = j.bs + tn * BN * j.ldbs + kb0;
        const int64_t mr = j.M - tm * BM, nr = j.N - tn * BN;
        tl.mrows = (int)(mr < BM ? mr : BM);
        tl.nrows = (int)(nr < BN ? nr : BN);
        tl.c_off = c_base + tm * BM * j.ldc + tn * BN;
    }

    return true;
}

template <int FMT, int OUT>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs args) {
    __shared__ GemmSmem sm;
    const GemmJob& j = args.j;
    const int tid = threadIdx.x;

    Tile tl;
    if (!resolve_tile(j, sm.grp, tl)) return;

    // ---- main loop ----------------------------------------------------------------------------
    const int lane = tid & 63, h = lane >> 5, l32 = lane & 31;
    const int wave = tid >> 6, wm = wave >> 1, wn = wave & 1;

    float acc[2][2][16];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.0f;

    uint2 ra[4], rb[4];
    float rsa[4], rsb[4];
    const int64_t nstages = (tl.nkb + SKB - 1) / SKB;

    auto load_stage = [&](int64_t s) {
        const int64_t ks = s * SKB;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = tid + 256 * q;
            const int row = e >> 3, kb = e & 7;
            const bool kok = ks + kb < tl.nkb;
            const bool aok = kok && row < tl.mrows, bok = kok && row < tl.nrows;
            ra[q] = aok ? *reinterpret_cast<const uint2*>(tl.a + row * j.lda + (ks + kb) * 8) : make_uint2(0, 0);
            rsa[q] = aok ? tl.as[row * j.ldas + ks + kb] : 0.0f;
            rb[q] = bok ? *reinterpret_cast<const uint2*>(tl.b + row * j.ldb + (ks + kb) * 8) : make_uint2(0, 0);
            rsb[q] = bok ? tl.bs[row * j.ldbs + ks + kb] : 0.0f;
        }
    };
    auto store_stage = [&](int buf) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = tid + 256 * q;
            const int row = e >> 3, kb = e & 7;
            sm.a[buf][(kb * 2 + 0) * CPL + row] = ra[q].x;
            sm.a[buf][(kb * 2 + 1) * CPL + row] = ra[q].y;
            sm.b[buf][(kb * 2 + 0) * CPL + row] = rb[q].x;
            sm.b[buf][(kb * 2 + 1) * CPL + row] = rb[q].y;
            sm.as[buf][kb * SPL + row] = rsa[q];
            sm.bs[buf][kb * SPL + row] = rsb[q];
        }
    };

    if (nstages > 0) {
        load_stage(0);
        store_stage(0);
    }
    __syncthreads();

    for (int64_t s = 0; s < nstages; ++s) {
        const int buf = (int)(s & 1);
        if (s + 1 < nstages) load_stage(s + 1);
        const int64_t left = tl.nkb - s * SKB;
        const int kbn = (int)(left < SKB ? left : SKB);
#pragma unroll
        for (int kb = 0; kb < SKB; ++kb) {
            if (kb < kbn) {
                long aop[2], bop[2];
#pragma unroll
                for (int t2 = 0; t2 < 2; ++t2) {
                    aop[t2] = expand<FMT>(sm.a[buf][(kb * 2 + h) * CPL + wm * 64 + t2 * 32 + l32]);
                    bop[t2] = expand<FMT>(sm.b[buf][(kb * 2 + h) * CPL + wn * 64 + t2 * 32 + l32]);
                }
                v16i d[2][2];
#pragma unroll
                for (int a = 0; a < 2; ++a)
#pragma unroll
                    for (int b = 0; b < 2; ++b) {
                        const v16i z = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
                        d[a][b] = __builtin_amdgcn_mfma_i32_32x32x16_i8(aop[a], bop[b], z, 0, 0, 0);
                    }
                float sb[2];
#pragma unroll
                for (int b = 0; b < 2; ++b) sb[b] = sm.bs[buf][kb * SPL + wn * 64 + b * 32 + l32];
#pragma unroll
                for (int a = 0; a < 2; ++a) {
                    float sa[16];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const float4 v =
                            *reinterpret_cast<const float4*>(&sm.as[buf][kb * SPL + wm * 64 + a * 32 + 8 * q + 4 * h]);
                        sa[4 * q + 0] = v.x;
                        sa[4 * q + 1] = v.y;
                        sa[4 * q + 2] = v.z;
                        sa[4 * q + 3] = v.w;
                    }
#pragma unroll
                    for (int b = 0; b < 2; ++b)
#pragma unroll
                        for (int i = 0; i < 16; ++i)
                            acc[a][b][i] = __builtin_fmaf((float)d[a][b][i], sa[i] * sb[b], acc[a][b][i]);
                }
            }
        }
        if (s + 1 < nstages) store_stage(buf ^ 1);
        __syncthreads();
    }

    constexpr float kUndo = FMT == kFmtUniform ? 1.0f : 0.25f;
    store_tile<OUT>(j, tl, acc, kUndo, wm, wn, h, l32);
}

// ================================================================================================
// fp32-output variant (the default).
//
// The per-block dot product D_b comes out of the MFMA already in fp32 and a second MFMA forms the outer
// product sA[:, b] x sB[:, b] in the same register layout, so the VALU does one FMA per output and block:
// acc += D_b * (sA sB)_b.
//
//  * D_b: uniform codes become fp8 e4m3 subnormals (code k -> k * 2^-9, exact) while a stage is copied into
//    LDS and go through v_mfma_f32_32x32x16_fp8_fp8; E2M1 codes go straight into the scaled f8f6f4 MFMA as
//    FP4 operands (neutral E8M0 scales), the 16 codes of a block occupying 16 of its 64 K slots.
//  * (sA sB)_b: every fp32 scale is split exactly into three bf16 pieces s = s0 + s1 + s2 (top, middle and
//    low 8 significand bits) when staged; a v_mfma_f32_32x32x16_bf16 whose 16 K slots hold the nine
//    products a_i b_j (exact in fp32) sums them, i.e. sA sB up to fp32 accumulation rounding. The bf16
//    MFMA co-executes with the VALU FMAs; an fp32 MFMA would not.
//  * The MFMAs of one half of the wave's four tiles run while the VALU folds the other half (software
//    pipeline across K-blocks and stages).
// ================================================================================================

typedef float v16f __attribute__((ext_vector_type(16)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

constexpr int SKB2 = 4;          // K-blocks per LDS stage
constexpr int CPL2 = BM + 1;     // code plane stride in 8-byte entries
constexpr int SPL2 = BM + 2;     // scale plane stride in 8-byte entries

// 8 uniform codes (one packed dword of sign-magnitude nibbles) -> 8 fp8 e4m3 bytes. The byte s000 0mmm is an
// e4m3 subnormal worth (-1)^s * m * 2^-9, so the code k becomes k * 2^-9 exactly (the product of two codes
// carries 2^-18, undone once at the store). Even codes go to the low dword, odd codes to the high one.
__device__ __forceinline__ uint2 uniform_to_e4m3(uint32_t d) {
    const uint32_t lo = (d & 0x07070707u) | ((d << 4) & 0x80808080u);
    const uint32_t hi = ((d >> 4) & 0x07070707u) | (d & 0x80808080u);
    return make_uint2(lo, hi);
}

// Exact split of an fp32 value into three bf16 pieces x = s0 + s1 + s2 (truncations of the top, middle and
// low 8 significand bits; each difference is exact in fp32). Returned as {s0 | s1 << 16, s2}.
__device__ __forceinline__ uint2 split_bf16x3(float x) {
    const uint32_t hi = __float_as_uint(x) & 0xFFFF0000u;
    const float r1 = x - __uint_as_float(hi);
    const uint32_t mid = __float_as_uint(r1) & 0xFFFF0000u;
    const float r2 = r1 - __uint_as_float(mid);
    return make_uint2((hi >> 16) | mid, __float_as_uint(r2) >> 16);
}

// K-slot layout of the outer-product MFMA (slot t holds a_i * b_j): lanes 0-31 carry slots 0-7 =
// (0,0) (1,0) (2,0) (0,1) (1,1) (2,1) (0,2) (1,2), lanes 32-63 slot 8 = (2,2) and zeros. The byte-permute
// selectors pick each operand dword from the staged pair {s0 | s1 << 16, s2} (bytes 0-3 and 4-7).
struct SplitSel {
    uint32_t a[4], b[4];
};
__device__ __forceinline__ SplitSel make_split_sel(int h) {
    SplitSel s;
    if (h == 0) {
        s.a[0] = 0x03020100u; s.a[1] = 0x01000504u; s.a[2] = 0x05040302u; s.a[3] = 0x03020100u;  // a0a1 a2a0 a1a2 a0a1
        s.b[0] = 0x01000100u; s.b[1] = 0x03020100u; s.b[2] = 0x03020302u; s.b[3] = 0x05040504u;  // b0b0 b0b1 b1b1 b2b2
    } else {
        s.a[0] = s.b[0] = 0x07060504u;                                                              // s2 | 0
        s.a[1] = s.a[2] = s.a[3] = s.b[1] = s.b[2] = s.b[3] = 0x0C0C0C0Cu;                          // zeros
    }
    return s;
}
__device__ __forceinline__ v8bf split_operand(uint2 c, const uint32_t (&sel)[4]) {
    uint32_t d[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) d[i] = __builtin_amdgcn_perm(c.y, c.x, sel[i]);
    return __builtin_bit_cast(v8bf, d);
}

template <int FMT>
struct alignas(16) GemmSmem2 {
    // uniform: fp8 bytes (8 per row, block and half); E2M1: the raw packed codes in .x
    uint2 a[2][SKB2 * 2 * CPL2];
    uint2 b[2][SKB2 * 2 * CPL2];
    uint2 as[2][SKB2 * SPL2];  // split scales
    uint2 bs[2][SKB2 * SPL2];
    int32_t grp[2];
};

template <int FMT>
__device__ __forceinline__ v16f block_dot(uint2 a, uint2 b) {
    const v16f z = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
    if constexpr (FMT == kFmtUniform) {
        const long av = (long)(((uint64_t)a.y << 32) | a.x);
        const long bv = (long)(((uint64_t)b.y << 32) | b.x);
        return __builtin_amdgcn_mfma_f32_32x32x16_fp8_fp8(av, bv, z, 0, 0, 0);
    } else {
        const v8i av = {(int)a.x, 0, 0, 0, 0, 0, 0, 0};
        const v8i bv = {(int)b.x, 0, 0, 0, 0, 0, 0, 0};
        // A and B as FP4 E2M1 (format 4), E8M0 scales 127 = 2^0
        return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, z, 4, 4, 0, 127, 0, 127);
    }
}

__device__ __forceinline__ v16f scale_outer(v8bf a, v8bf b) {
    const v16f z = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, z, 0, 0, 0);
}

// VEC: the operands' rows are 16-byte aligned at every stage start (code row stride % 16 == 0, scale row
// stride % 4 == 0, first block % 4 == 0), so stages are fetched with 16-byte loads.
//
// Work split: 8 waves per 128 x 128 tile; wave (wm, wn) owns rows 64 wm .. +64 and columns 32 wn .. +32, i.e.
// two 32 x 32 MFMA tiles. At <= 128 VGPRs two workgroups share a CU (four waves per SIMD), which is what
// lets MFMAs and VALU FMAs of different waves overlap: a single wave issues neither back to back.
constexpr int kWaves2 = 8;

template <int FMT, int OUT, bool VEC>
__global__ __launch_bounds__(512, 2) void gemm_f32_kernel(GemmArgs args) {
    __shared__ GemmSmem2<FMT> sm;
    const GemmJob& j = args.j;
    const int tid = threadIdx.x;

    Tile tl;
    if (!resolve_tile(j, sm.grp, tl)) return;

    const int lane = tid & 63, h = lane >> 5, l32 = lane & 31;
    const int wave = tid >> 6, wm = wave >> 2, wn = wave & 3;
    const SplitSel sel = make_split_sel(h);

    float acc[2][16];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[a][i] = 0.0f;

    const int64_t nkb = tl.nkb;
    const int64_t nstages = (nkb + SKB2 - 1) / SKB2;

    // staging: threads 0-255 fetch A codes, 256-511 B codes (two threads per row, 16 bytes = two blocks
    // each); threads 0-127 fetch A scales, 128-255 B scales (one row, four blocks each)
    const bool c_is_a = tid < 256;
    const int crow = (tid & 255) >> 1, chalf = tid & 1;
    const bool has_s = tid < 256;
    const bool s_is_a = tid < 128;
    const int srow = tid & 127;
    uint4 qc, qs;

    auto load_stage = [&](int64_t s) {
        const int64_t ks = s * SKB2;
        {
            const uint8_t* base = c_is_a ? tl.a : tl.b;
            const int64_t ld = c_is_a ? j.lda : j.ldb;
            const int rows = c_is_a ? tl.mrows : tl.nrows;
            const int64_t kb = ks + 2 * chalf;
            qc = make_uint4(0, 0, 0, 0);
            if (crow < rows) {
                const uint8_t* p = base + crow * ld + kb * 8;
                if (VEC && kb + 1 < nkb) {
                    qc = *reinterpret_cast<const uint4*>(p);
                } else {
                    const uint2 u0 = kb < nkb ? *reinterpret_cast<const uint2*>(p) : make_uint2(0, 0);
                    const uint2 u1 = kb + 1 < nkb ? *reinterpret_cast<const uint2*>(p + 8) : make_uint2(0, 0);
                    qc = make_uint4(u0.x, u0.y, u1.x, u1.y);
                }
            }
        }
        qs = make_uint4(0, 0, 0, 0);
        if (has_s) {
            const float* base = s_is_a ? tl.as : tl.bs;
            const int64_t ld = s_is_a ? j.ldas : j.ldbs;
            const int rows = s_is_a ? tl.mrows : tl.nrows;
            if (srow < rows) {
                const float* p = base + srow * ld + ks;
                if (VEC && ks + 3 < nkb) {
                    qs = *reinterpret_cast<const uint4*>(p);
                } else {
                    uint32_t v[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) v[q] = ks + q < nkb ? __float_as_uint(p[q]) : 0u;
                    qs = make_uint4(v[0], v[1], v[2], v[3]);
                }
            }
        }
    };
    auto put_codes = [&](uint2* plane, uint32_t c, int kb, int half) {
        if constexpr (FMT == kFmtUniform) plane[(kb * 2 + half) * CPL2 + crow] = uniform_to_e4m3(c);
        else plane[(kb * 2 + half) * CPL2 + crow] = make_uint2(c, 0);
    };
    auto store_stage = [&](int buf) {
        uint2* cp = c_is_a ? sm.a[buf] : sm.b[buf];
        const int kb0 = 2 * chalf;
        put_codes(cp, qc.x, kb0, 0);
        put_codes(cp, qc.y, kb0, 1);
        put_codes(cp, qc.z, kb0 + 1, 0);
        put_codes(cp, qc.w, kb0 + 1, 1);
        if (has_s) {
            uint2* sp = s_is_a ? sm.as[buf] : sm.bs[buf];
            sp[0 * SPL2 + srow] = split_bf16x3(__uint_as_float(qs.x));
            sp[1 * SPL2 + srow] = split_bf16x3(__uint_as_float(qs.y));
            sp[2 * SPL2 + srow] = split_bf16x3(__uint_as_float(qs.z));
            sp[3 * SPL2 + srow] = split_bf16x3(__uint_as_float(qs.w));
        }
    };

    for (int64_t s = 0; s < nstages; ++s) {
        const int buf = (int)(s & 1);
        if (s == 0) {
            load_stage(0);
            store_stage(0);
            __syncthreads();
        }
        if (s + 1 < nstages) load_stage(s + 1);
        const int64_t left = nkb - s * SKB2;
        const int kbn = (int)(left < SKB2 ? left : SKB2);
#pragma unroll
        for (int kb = 0; kb < SKB2; ++kb) {
            if (kb < kbn) {
                const int pl = (kb * 2 + h) * CPL2;
                const uint2 b0 = sm.b[buf][pl + wn * 32 + l32];
                const v8bf vb = split_operand(sm.bs[buf][kb * SPL2 + wn * 32 + l32], sel.b);
#pragma unroll
                for (int a = 0; a < 2; ++a) {
                    const int ra = wm * 64 + a * 32 + l32;
                    const v16f d = block_dot<FMT>(sm.a[buf][pl + ra], b0);
                    const v16f w = scale_outer(split_operand(sm.as[buf][kb * SPL2 + ra], sel.a), vb);
#pragma unroll
                    for (int i = 0; i < 16; ++i) acc[a][i] = __builtin_fmaf(d[i], w[i], acc[a][i]);
                }
            }
        }
        if (s + 1 < nstages) store_stage(buf ^ 1);
        __syncthreads();
    }

    // uniform: the fp8 subnormal encoding scaled every product by 2^-18
    const float mul = FMT == kFmtUniform ? 262144.0f : 1.0f;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        const int col = wn * 32 + l32;
        if (col >= tl.nrows) continue;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int row = wm * 64 + a * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
            if (row >= tl.mrows) continue;
            const float v = acc[a][i] * mul;
            const int64_t off = tl.c_off + (int64_t)row * j.ldc + col;
            if constexpr (OUT == kOutF32) {
                static_cast<float*>(j.c)[off] = v;
            } else {
                static_cast<uint16_t*>(j.c)[off] = (uint16_t)f32_to_bf16_bits(v);
            }
        }
    }
}

// UFP4_GEMM_MFMA=i8 selects the int8-MFMA kernel (cvt + scale product + fma per output and block) instead of
// the default fp32-output kernel; both compute the same sums exactly up to fp32 accumulation order.
static bool use_i8_mfma() {
    static const bool v = [] {
        const char* e = getenv("UFP4_GEMM_MFMA");
        return e != nullptr && strcmp(e, "i8") == 0;
    }();
    return v;
}

template <int FMT, int OUT>
static hipError_t launch_t(const GemmJob& j, hipStream_t s) {
    dim3 grid((unsigned)((j.N + BN - 1) / BN), 1, 1);
    if (j.mode == kGemmRaggedM) {
        grid.y = (unsigned)((j.M + BM - 1) / BM + j.G);
    } else {
        grid.y = (unsigned)((j.M + BM - 1) / BM);
        if (j.mode == kGemmRaggedK) grid.z = (unsigned)j.G;
    }
    if (grid.x == 0 || grid.y == 0 || grid.z == 0) return hipSuccess;
    GemmArgs args{j};
    // 16-byte staging loads need every stage start of every row aligned; the ragged-K groups start at
    // arbitrary blocks, so they take the guarded 8-byte path.
    const bool vec = j.mode != kGemmRaggedK && j.lda % 16 == 0 && j.ldb % 16 == 0 && j.ldas % 4 == 0 &&
                     j.ldbs % 4 == 0 && (uintptr_t)j.a % 16 == 0 && (uintptr_t)j.b % 16 == 0 &&
                     (uintptr_t)j.as % 16 == 0 && (uintptr_t)j.bs % 16 == 0 &&
                     (j.mode != kGemmRaggedM || j.b_group_kb % 4 == 0);
    if (use_i8_mfma()) {
        gemm_kernel<FMT, OUT><<<grid, 256, 0, s>>>(args);
    } else if (vec) {
        gemm_f32_kernel<FMT, OUT, true><<<grid, 64 * kWaves2, 0, s>>>(args);
    } else {
        gemm_f32_kernel<FMT, OUT, false><<<grid, 64 * kWaves2, 0, s>>>(args);
    }
    return hipGetLastError();
}

hipError_t launch_gemm(const GemmJob& j, hipStream_t s) {
    if (j.format == kFmtE2M1) {
        return j.out_dtype == kOutBF16 ? launch_t<kFmtE2M1, kOutBF16>(j, s) : launch_t<kFmtE2M1, kOutF32>(j, s);
    }
    return j.out_dtype == kOutBF16 ? launch_t<kFmtUniform, kOutBF16>(j, s) : launch_t<kFmtUniform, kOutF32>(j, s);
}

}  // namespace ufp4
