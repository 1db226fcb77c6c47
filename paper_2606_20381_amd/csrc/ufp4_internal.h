// Internal interface between the C-ABI layer (ufp4_api.cpp) and the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ufp4 {

enum { kFmtUniform = 0, kFmtE2M1 = 1 };
enum { kRoundRTNE = 0, kRoundSR = 1 };
enum { kOutF32 = 0, kOutBF16 = 1 };

// Per-call constants of the quantizer.
struct QuantArgs {
    uint32_t sign_xor[8];  // XOR mask per bf16 pair: 0x8000 / 0x80000000 where eps_j = -1
    uint32_t key0, key1;   // Philox key = seed
    uint32_t stream;       // Philox counter word 3
};

// One quantization request, already validated.
struct QuantJob {
    int format, rounding, rht, transpose;
    const void* x;
    int64_t xrows, ld;  // X rows and leading dimension (elements)
    int64_t qrows;      // rows of the quantized operand
    int64_t red;        // reduction length of the quantized operand (padded total when grouped)
    const int64_t* group_off;   // grouped transposed only (device), else nullptr
    const int64_t* group_poff;  // grouped transposed only (device)
    int32_t num_groups;
    QuantArgs qa;
    void* codes;
    int64_t code_ld;
    float* scales;
    int64_t scale_ld;
};

hipError_t launch_quantize(const QuantJob& job, hipStream_t stream);
int max_groups_quantize();

// Block-scaled NT GEMM: C[i, j] = sum_b sA[i,b] sB[j,b] sum_{k in b} A[i,k] B[j,k] over `nkb` 16-blocks.
enum GemmMode { kGemmDense = 0, kGemmRaggedM = 1, kGemmRaggedK = 2 };

struct GemmJob {
    int format, out_dtype, mode;
    const uint8_t* a;  // codes of the left operand, row stride lda bytes
    int64_t lda;
    const float* as;  // its scales, row stride ldas floats
    int64_t ldas;
    const uint8_t* b;
    int64_t ldb;
    const float* bs;
    int64_t ldbs;
    int64_t M;    // rows of A: dense and ragged-K per problem; ragged-M the total over groups
    int64_t N;    // rows of B per problem
    int64_t nkb;  // reduction blocks (dense, ragged-M); unused for ragged-K (from the offsets)
    void* c;
    int64_t ldc;  // elements
    // grouped
    const int64_t* offsets;  // ragged-M: token offsets [G+1]; ragged-K: padded offsets [G+1]
    int32_t G;
    int64_t b_group_rows;  // ragged-M: B rows advanced per group (fwd_y: N)
    int64_t b_group_kb;    // ragged-M: B reduction blocks advanced per group (bwd_dx: N/16)
    int64_t red_total;     // ragged-K: reduction length of both operands (padded token total)
};

hipError_t launch_gemm(const GemmJob& job, hipStream_t stream);

}  // namespace ufp4
