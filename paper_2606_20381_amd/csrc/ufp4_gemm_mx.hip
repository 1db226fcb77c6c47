// Block-scaled 4-bit GEMM for the uniform grid with power-of-two 1x32 scales (the scale hierarchy of Sec. 4
// chosen for the hardware): C[i, j] = sum_k A[i,k] 2^(eA[i,k/32] - 127) B[j,k] 2^(eB[j,k/32] - 127), with the
// codes stored as FP6 E2M3 numbers and the scales as E8M0 bytes (quantizer: ufp4_quant.hip).
//
// The whole product runs on v_mfma_scale_f32_32x32x64_f8f6f4 with FP6 operands: each lane holds the 32 codes
// of one row and one 32-block (24 bytes, the storage format itself) and that block's E8M0 scale, and the
// matrix core applies both scales and accumulates in fp32. There is no per-block VALU work, unlike the fp32
// per-16 scales of the main recipe, so the kernel is bound by the matrix cores and by how fast operand tiles
// reach them.
//
// Tiling: a 128 x 128 output tile per 256-thread workgroup (4 waves of 64 x 64, 2 x 2 MFMA tiles of 32 x 32).
// K advances 128 (four 32-blocks) per stage. A stage of one operand is a contiguous 12 KiB run of its panel
// (the panel layout puts the 128 rows of a 32-block together) plus 512 scale bytes; it is fetched with 16-byte
// loads one stage ahead into registers and copied unchanged into double-buffered LDS.

#include "ufp4_internal.h"

namespace ufp4 {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef int v8i __attribute__((ext_vector_type(8)));

constexpr int kMxTile = 128;                    // rows of A and of B per tile (one panel each)
constexpr int kMxStageBlocks = 4;               // 32-blocks per stage
constexpr int kMxStageBytes = kMxStageBlocks * 3072;
constexpr int kMxStageChunks = kMxStageBytes / 16;  // 768 chunks of 16 bytes per operand
constexpr int kMxThreads = 256;
constexpr int kMxChunksPerThread = kMxStageChunks / kMxThreads;  // 3
static_assert(kMxStageChunks % kMxThreads == 0, "stage chunks");

struct MxSmem {
    uint8_t a[2][kMxStageBytes];
    uint8_t b[2][kMxStageBytes];
    uint32_t as[2][kMxStageBlocks * 32];  // 128 scale bytes per block
    uint32_t bs[2][kMxStageBlocks * 32];
};

struct MxStage {
    uint4 a[kMxChunksPerThread], b[kMxChunksPerThread];
    uint32_t s;  // one scale word: of A for threads 0-127, of B for threads 128-255
};

__device__ __forceinline__ v8i load_fp6_operand(const uint8_t* p) {  // 24 bytes, 8-byte aligned
    const uint2 x0 = *reinterpret_cast<const uint2*>(p);
    const uint2 x1 = *reinterpret_cast<const uint2*>(p + 8);
    const uint2 x2 = *reinterpret_cast<const uint2*>(p + 16);
    const v8i v = {(int)x0.x, (int)x0.y, (int)x1.x, (int)x1.y, (int)x2.x, (int)x2.y, 0, 0};
    return v;
}

template <int OUT>
__global__ __launch_bounds__(kMxThreads) void gemm_mx_kernel(MxGemmJob j) {
    __shared__ MxSmem sm;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h = lane >> 5, l32 = lane & 31;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t tm = blockIdx.y, tn = blockIdx.x;  // tile index = panel index of A and of B
    const uint8_t* ga = j.a + tm * j.a_pld;
    const uint8_t* gas = j.as + tm * j.as_pld;
    const uint8_t* gb = j.b + tn * j.b_pld;
    const uint8_t* gbs = j.bs + tn * j.bs_pld;
    const int nkb = (int)j.nkb;
    const int nst = (nkb + kMxStageBlocks - 1) / kMxStageBlocks;

    // Blocks past the reduction's end (last stage) are zero-filled: zero codes contribute nothing.
    auto load = [&](MxStage& r, int s) {
        const int kb0 = s * kMxStageBlocks;
#pragma unroll
        for (int i = 0; i < kMxChunksPerThread; ++i) {
            const int c = tid + kMxThreads * i;
            const bool ok = kb0 + c / 192 < nkb;  // 192 chunks per 32-block
            r.a[i] = ok ? reinterpret_cast<const uint4*>(ga + (int64_t)kb0 * 3072)[c] : make_uint4(0, 0, 0, 0);
            r.b[i] = ok ? reinterpret_cast<const uint4*>(gb + (int64_t)kb0 * 3072)[c] : make_uint4(0, 0, 0, 0);
        }
        const int w = tid & 127;  // scale word w of the stage: block w / 32
        const uint8_t* src = tid < 128 ? gas : gbs;
        r.s = kb0 + w / 32 < nkb ? reinterpret_cast<const uint32_t*>(src + (int64_t)kb0 * 128)[w] : 0u;
    };
    auto put = [&](int buf, const MxStage& r) {
#pragma unroll
        for (int i = 0; i < kMxChunksPerThread; ++i) {
            const int c = tid + kMxThreads * i;
            reinterpret_cast<uint4*>(sm.a[buf])[c] = r.a[i];
            reinterpret_cast<uint4*>(sm.b[buf])[c] = r.b[i];
        }
        if (tid < 128) sm.as[buf][tid] = r.s;
        else sm.bs[buf][tid - 128] = r.s;
    };

    v16f acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.0f;

    auto compute = [&](int buf) {
        const uint8_t* sas = reinterpret_cast<const uint8_t*>(sm.as[buf]);
        const uint8_t* sbs = reinterpret_cast<const uint8_t*>(sm.bs[buf]);
#pragma unroll
        for (int ks = 0; ks < kMxStageBlocks / 2; ++ks) {
            const int kk = 2 * ks + h;  // this lane's 32-block: lanes 0-31 hold K 0-31 of the step, 32-63 K 32-63
            v8i av[2], bv[2];
            int sa[2], sb[2];
#pragma unroll
            for (int a = 0; a < 2; ++a) {
                const int row = wm * 64 + a * 32 + l32;
                av[a] = load_fp6_operand(sm.a[buf] + kk * 3072 + row * 24);
                sa[a] = sas[kk * 128 + row];
            }
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const int col = wn * 64 + b * 32 + l32;
                bv[b] = load_fp6_operand(sm.b[buf] + kk * 3072 + col * 24);
                sb[b] = sbs[kk * 128 + col];
            }
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b)
                    // formats 2 = FP6 E2M3 for both operands; the scale bytes sit in byte 0 of sa / sb
                    acc[a][b] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av[a], bv[b], acc[a][b], 2, 2, 0,
                                                                                sa[a], 0, sb[b]);
        }
    };

    if (nst > 0) {
        MxStage r;
        load(r, 0);
        put(0, r);
        __syncthreads();
        for (int s = 0; s < nst; ++s) {
            const bool more = s + 1 < nst;
            if (more) load(r, s + 1);
            compute(s & 1);
            if (more) put((s + 1) & 1, r);
            __syncthreads();
        }
    }

#pragma unroll
    for (int a = 0; a < 2; ++a) {
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int64_t col = tn * kMxTile + wn * 64 + b * 32 + l32;
            if (col >= j.N) continue;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int64_t row = tm * kMxTile + wm * 64 + a * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
                if (row >= j.M) continue;
                const float v = acc[a][b][i];
                if constexpr (OUT == kOutF32) {
                    static_cast<float*>(j.c)[row * j.ldc + col] = v;
                } else {
                    static_cast<uint16_t*>(j.c)[row * j.ldc + col] = __builtin_bit_cast(uint16_t, (__bf16)v);  // RNE
                }
            }
        }
    }
}

hipError_t launch_gemm_mx(const MxGemmJob& j, hipStream_t s) {
    const dim3 grid((unsigned)((j.N + kMxTile - 1) / kMxTile), (unsigned)((j.M + kMxTile - 1) / kMxTile));
    if (grid.x == 0 || grid.y == 0) return hipSuccess;
    if (j.out_dtype == kOutBF16) gemm_mx_kernel<kOutBF16><<<grid, kMxThreads, 0, s>>>(j);
    else gemm_mx_kernel<kOutF32><<<grid, kMxThreads, 0, s>>>(j);
    return hipGetLastError();
}

}  // namespace ufp4
