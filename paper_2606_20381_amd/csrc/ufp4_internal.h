// Internal interface between the C-ABI layer (ufp4_api.cpp) and the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ufp4 {

enum { kFmtUniform = 0, kFmtE2M1 = 1 };

// Quantized operands are stored in panels of kPanelRows rows; within a panel, block b of every row sits at
// b * 1024 bytes (codes, 8 per row) and b * 128 floats (scales, 1 per row).
constexpr int64_t kPanelRows = 128;
constexpr int64_t kPanelBlockBytes = kPanelRows * 8;
constexpr int64_t kPanelBlockScales = kPanelRows;
__host__ __device__ constexpr int64_t padded_rows(int64_t rows) { return (rows + kPanelRows - 1) / kPanelRows * kPanelRows; }
enum { kRoundRTNE = 0, kRoundSR = 1 };
enum { kOutF32 = 0, kOutBF16 = 1 };

// Per-call constants of the quantizer.
struct QuantArgs {
    uint32_t sign_xor[8];  // XOR mask per bf16 pair: 0x8000 / 0x80000000 where eps_j = -1
    uint32_t key0, key1;   // Philox key = seed
    uint32_t stream;       // Philox counter word 3
    float e2m1_g;          // E2M1 top level max_fpx (2, 4 or 6) and RN(1 / max_fpx); unused by the uniform grid
    float e2m1_ginv;
    int32_t rht_m;          // RHT block = 16 * rht_m (1, 2, 4, 8); rht_m > 1 selects the wide-RHT kernels
    double rht_c;           // their normalisation RN64(sqrt(1 / (16 rht_m)))
    uint32_t sign_words[8]; // their sign mask: bits 16k .. 16k + 15 of the n-bit mask in word k
};

// One quantization request, already validated.
struct QuantJob {
    int format, rounding, rht, transpose;
    int input_f32;  // x is fp32 (rowwise, rht = 0): the quantizing half of the unfused form
    const void* x;
    int64_t xrows, ld;  // X rows and leading dimension (elements)
    int64_t qrows;      // rows of the quantized operand
    int64_t red;        // reduction length of the quantized operand (padded total when grouped)
    const int64_t* group_off;   // grouped transposed only: token offsets [G+1] (device), else nullptr
    int32_t num_groups;
    QuantArgs qa;
    void* codes;
    int64_t code_pld;  // bytes between panels
    float* scales;
    int64_t scale_pld;  // floats between panels
};

hipError_t launch_quantize(const QuantJob& job, hipStream_t stream);
int max_groups_quantize();

// Standalone block-16 RHT of X [rows, cols] along cols, y in fp32 (the unfused form).
struct RhtJob {
    const void* x;
    int64_t rows, cols, ld;
    QuantArgs qa;
    float* y;
    int64_t ldy;
};
hipError_t launch_rht(const RhtJob& job, hipStream_t stream);

// Quality statistics of one quantization (the operand is not stored): fp64 sums over the elements of
// (q - ref)^2, ref^2 and q * ref, where ref is the value the quantizer rounds (the fp32 RHT output, or x) and
// q the dequantized code, and the number of codes per magnitude code 0..7. Layout of the caller's output.
struct QuantStats {
    double err2, ref2, cross;
    unsigned long long hist[8];
};
// Same fields as QuantJob for a rowwise (transpose = 0) or transposed operand; no outputs but `stats`.
struct StatsJob {
    int format, rounding, rht, transpose;
    const void* x;
    int64_t ld;
    int64_t qrows, red;
    QuantArgs qa;
    QuantStats* stats;
};
hipError_t launch_quant_stats(const StatsJob& job, hipStream_t stream);

// Both quantized operands of one tensor X [rows, cols] (rows, cols multiples of 16) from one read: Q_r = X
// along cols ([rows, cols]) and Q_c = X^T along rows ([cols, rows]). Already validated.
struct DualJob {
    int format, rounding, rht_r, rht_c;
    const void* x;
    int64_t rows, cols, ld;
    QuantArgs qr, qc;  // sign masks and SR streams of Q_r and Q_c (same key)
    void* codes_r;
    int64_t code_pld_r;
    float* scales_r;
    int64_t scale_pld_r;
    void* codes_c;
    int64_t code_pld_c;
    float* scales_c;
    int64_t scale_pld_c;
};

hipError_t launch_quantize_dual(const DualJob& job, hipStream_t stream);

enum GemmMode { kGemmDense = 0, kGemmRaggedM = 1, kGemmRaggedK = 2 };

// Power-of-two block scales: the uniform grid with one E8M0 scale per 1x32 block and FP6 E2M3 codes.
// Operand [rows, red] (red % 32 == 0) in panels of 128 rows; within a panel, 32-block b of all 128 rows is
// contiguous: codes 128 x 24 bytes at b * 3072, scales 128 bytes at b * 128.
constexpr int64_t kMxPanelBlockBytes = kPanelRows * 24;
constexpr int64_t kMxPanelBlockScales = kPanelRows;

struct MxQuantJob {
    int rounding, rht, transpose;
    const void* x;
    int64_t xrows, ld;  // X rows and leading dimension (elements)
    int64_t qrows;      // rows of the quantized operand
    int64_t red;        // its reduction length (multiple of 32)
    // grouped: token offsets [G+1] on the device, else nullptr. Rowwise: groups of rows, each starting on a panel
    // boundary (qrows = the padded row count); transposed: the reduction axis padded to 32 per group (red = its
    // padded length)
    const int64_t* group_off;
    int32_t num_groups;
    QuantArgs qa;
    void* codes;
    int64_t code_pld;  // bytes between panels
    void* scales;
    int64_t scale_pld;  // bytes between panels
};

hipError_t launch_quantize_mx(const MxQuantJob& job, hipStream_t stream);

// Both operands with power-of-two scales from one read of X [rows, cols] (rows and cols multiples of 32).
struct MxDualJob {
    int rounding, rht_r, rht_c;
    const void* x;
    int64_t rows, cols, ld;
    QuantArgs qr, qc;  // per output: signs, SR stream
    void* codes_r;
    int64_t code_pld_r;
    void* scales_r;
    int64_t scale_pld_r;
    void* codes_c;
    int64_t code_pld_c;
    void* scales_c;
    int64_t scale_pld_c;
};

hipError_t launch_quantize_mx_dual(const MxDualJob& job, hipStream_t stream);
// Workgroups of the power-of-two-scale tile kernel (32 x 256 tiles) for the outputs asked for.
int64_t mx_tile_count(int64_t rows, int64_t cols, bool rows_out, bool cols_out);

// NT GEMM on two such operands: C[i, j] = sum_k A[i,k] 2^(eA[i,k/32]-127) B[j,k] 2^(eB[j,k/32]-127).
struct MxGemmJob {
    int out_dtype;
    const uint8_t* a;
    int64_t a_pld;
    const uint8_t* as;
    int64_t as_pld;
    const uint8_t* b;
    int64_t b_pld;
    const uint8_t* bs;
    int64_t bs_pld;
    int64_t M, N, nkb;  // rows of A, rows of B (ragged-M: per group), 32-blocks of the reduction
    int64_t a_rows, b_rows;  // rows stored in the A and B operands (their last panels)
    void* c;
    int64_t ldc;
    // grouped (mode kGemmRaggedM / kGemmRaggedK of GemmMode below): token offsets [G+1] on the device.
    // Ragged-M: A holds each group's rows from a panel boundary (row sum_{h<g} pad128(m_h)); B advances by
    // b_group_rows rows (fwd_y) or b_group_kb 32-blocks of the reduction (bwd_dx) per group; C rows are token rows.
    // Ragged-K: both operands' reduction is the token axis padded to 32 per group; C holds one [M, N] per group.
    int mode;
    const int64_t* offsets;
    int32_t G;
    int64_t m_tiles;       // ragged-M: bound on the number of 256-row tiles over all groups
    int64_t b_group_rows;
    int64_t b_group_kb;
};

hipError_t launch_gemm_mx(const MxGemmJob& job, hipStream_t stream);

// Block-scaled NT GEMM: C[i, j] = sum_b sA[i,b] sB[j,b] sum_{k in b} A[i,k] B[j,k] over `nkb` 16-blocks.

struct GemmJob {
    int format, out_dtype, mode;
    const uint8_t* a;  // codes of the left operand (panel layout), panel stride a_pld bytes
    int64_t a_pld;
    const float* as;  // its scales, panel stride as_pld floats
    int64_t as_pld;
    const uint8_t* b;
    int64_t b_pld;
    const float* bs;
    int64_t bs_pld;
    int64_t M;    // rows of A: dense and ragged-K per problem; ragged-M the total over groups
    int64_t N;    // rows of B per problem
    int64_t nkb;  // reduction blocks (dense, ragged-M); unused for ragged-K (from the offsets)
    void* c;
    int64_t ldc;  // elements
    // grouped
    const int64_t* offsets;  // token offsets [G+1] (ragged-K pads each group's count to a multiple of 16)
    int32_t G;
    int64_t b_group_rows;  // ragged-M: B rows advanced per group (fwd_y: N)
    int64_t b_group_kb;    // ragged-M: B reduction blocks advanced per group (bwd_dx: N/16)
    int64_t red_total;     // ragged-K: reduction length of both operands (padded token total)
};

hipError_t launch_gemm(const GemmJob& job, hipStream_t stream);

}  // namespace ufp4
