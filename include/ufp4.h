/*
 * ufp4.h -- C ABI of the UFP4 hot path on MI355X (gfx950).
 *
 * Implements the two data-parallel pieces of the UFP4 4-bit training recipe of "Rethinking Shrinkage
 * Bias in LLM FP4 Pretraining" (arXiv 2606.20381):
 *
 *   1. block-16 Random Hadamard Transform (Sec. 2.2) fused with 1x16 block-scaled quantization
 *      (Sec. 2.1) to the uniform 4-bit grid of the recipe (Sec. 4, Table 1), along the reduction axis
 *      of a GEMM operand -- rowwise (reduction axis contiguous) or transposed (reduction axis strided);
 *   2. the block-scaled 4-bit GEMMs fwd_y (Y = X W^T), bwd_dx (dX = dY W) and bwd_dw (dW = dY^T X) that
 *      consume those operands (Sec. 2.2, quantized GEMM display; RHT axis per GEMM in its last sentence).
 *
 * An E2M1 quantizer and the same GEMMs on E2M1 codes form the comparison baseline (Table 1).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - All pointers named *_dev are device pointers (HBM). Host pointers are named *_host. The caller owns
 *    every buffer; the library allocates, frees and synchronizes nothing, and keeps no state between calls.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream). Calls are asynchronous on it.
 *  - bf16 tensors are row-major with a leading dimension `ld` in elements (ld >= cols, ld % 8 == 0,
 *    base 16-byte aligned). A tensor with no element (rows or cols 0), input or GEMM output, is never
 *    accessed: its pointer may be NULL and its leading dimension is not checked.
 *  - A quantized operand Q is [rows, red] (red % 16 == 0, nkb = red/16 blocks of 16 along the reduction
 *    axis), described by a ufp4_qtensor (below) and stored in panels: rows 128p .. 128p+127 form panel p, and
 *    within a panel the data of block b of all 128 rows is contiguous -- the order in which the GEMMs stage
 *    K-blocks.
 *      codes : panel p at codes + p * code_panel_ld bytes; block b of row 128p + i at + b * 1024 + i * 8
 *              (8 bytes). Element 2j of the block is the low nibble of byte j. Each nibble is sign-magnitude:
 *              sign in bit 3, magnitude code in bits 0-2, zero always +0. Uniform grid: magnitude |k| of the
 *              code k in -7..7. E2M1: index of the magnitude in 0, .5, 1, 1.5, 2, 3, 4, 6 (the OCP FP4 bit
 *              pattern).
 *      scales: fp32; panel p at scales + p * scale_panel_ld floats; block b of row 128p + i at + b * 128 + i.
 *              Block b of row r dequantizes as level(code) * scale.
 *      code_panel_ld >= 1024 * nkb and a multiple of 16, scale_panel_ld >= 128 * nkb and a multiple of 4; both
 *      base pointers 16-byte aligned; the buffers hold `panels` >= ceil(rows / 128) whole panels
 *      (ufp4_qtensor_bytes gives the minimal layout). The quantizers write rows past `rows` in the last panel
 *      as zero codes and zero scales. Panel strides above 2^29 bytes (codes) or 2^27 floats (scales) return
 *      UFP4_ERR_UNSUPPORTED.
 *  - Quantizer arithmetic, per 16-block x (bf16):
 *      y_i  = the exact 1/4 * sum_j H16[i,j] * eps_j * x_j  rounded once to fp32 precision (rht != 0), else
 *             y = x; H16[i,j] = (-1)^popcount(i & j) (Sylvester, Sec. 2.2); eps_j = -1 iff bit j of sign_mask.
 *             Rounding: to nearest even, with gradual underflow below 2^-126 and no overflow (an output past
 *             FLT_MAX keeps 24 significant bits). The kernels sum in fp64: exact when the nonzero |x_j| of a
 *             block span at most 2^41; a block spanning more may lose its smallest terms, an error below
 *             2^-46 max|x_j| before the rounding to fp32 (y then need not be the correctly rounded value; a
 *             code may move to an adjacent level and a scale by an ulp where such a y decides them).
 *      amax = max |y_i|;  s = RN32(amax/g) (IEEE: subnormal for a tiny block, +inf past the fp32 range);
 *      r = g/amax rounded to 24 significant bits without an exponent limit (= RN32(g/amax) whenever that is
 *      finite);  v_i = RN32(y_i * r);  amax == 0 -> s = 0, codes 0.  Uniform grid g = 7, E2M1 g = 6.
 *      RTNE (Sec. 2.1): nearest level, ties to the level with the even magnitude code.
 *      SR   (Sec. 2.1): adjacent signed levels g_a <= v < g_b; q = g_b iff u/2^16 < (v - g_a)/(g_b - g_a),
 *             u a 16-bit Philox4x32-10 draw: key = (seed lo32, seed hi32), counter = (block, row, half,
 *             stream), element j takes 16-bit half (j & 1) of word (j & 7) >> 1 of call half = j >> 3.
 *             `block` is the block index along the reduction axis, `row` the operand row.
 *      |v| beyond the top level is clamped to it.
 *  - GEMMs: C[i, j] = sum_b sA[i,b] sB[j,b] sum_{k in block b} level(A[i,k]) level(B[j,k]) with fp32
 *    accumulation; output fp32 or bf16 (RNE), row-major with leading dimension ldc (elements). The output
 *    buffer must hold the product; the library cannot see its size.
 *
 * Errors: every call validates its arguments on the host before launching anything and returns
 * UFP4_OK or an error code (no launch happens on error). Device faults surface at the caller's next
 * synchronization. Inputs must be finite.
 */
#ifndef UFP4_H
#define UFP4_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    UFP4_OK = 0,
    UFP4_ERR_INVALID_ARG = 1, /* null pointer, negative size, unknown enum value                          */
    UFP4_ERR_SHAPE = 2,       /* reduction length not a multiple of 16, leading dimension or buffer too small */
    UFP4_ERR_ALIGN = 3,       /* pointer or leading dimension not aligned as required                      */
    UFP4_ERR_MISMATCH = 4,    /* the operands of a GEMM were quantized differently: grid, RHT block or sign */
                              /* mask, or reduction length (Sec. 2.2 needs the same H' on both operands)     */
    UFP4_ERR_UNSUPPORTED = 5, /* valid request outside the implemented limits or variants                   */
    UFP4_ERR_HIP = 6          /* kernel launch failed                                                      */
} ufp4_status;

enum { UFP4_FMT_UNIFORM = 0, UFP4_FMT_E2M1 = 1, UFP4_FMT_UNIFORM_MX32 = 2 };
enum { UFP4_ROUND_RTNE = 0, UFP4_ROUND_SR = 1 };
enum { UFP4_OUT_F32 = 0, UFP4_OUT_BF16 = 1 };
/* How a quantized operand's rows and reduction axis relate to the tensor it came from (ufp4_qtensor.layout):
 * PLAIN: row i and reduction position k are the tensor's; GROUPED_ROWS: the rows of expert groups, each group
 * starting on a panel boundary (ufp4_mx_quantize_grouped, transpose 0); GROUPED_RED: the reduction axis is the
 * groups' tokens, each group zero-padded to a multiple of the quantization block (ufp4_quantize_grouped_t,
 * ufp4_mx_quantize_grouped with transpose 1). */
enum { UFP4_LAYOUT_PLAIN = 0, UFP4_LAYOUT_GROUPED_ROWS = 1, UFP4_LAYOUT_GROUPED_RED = 2 };

/*
 * A quantized operand Q(A H') [rows, red] (Sec. 2.1: codes plus block scales). The caller sets the storage
 * fields and passes the descriptor to a quantizer, which checks that the operand fits them and records what it
 * wrote; the GEMMs read both and refuse operand pairs whose grid, RHT block, RHT signs or reduction length
 * differ (UFP4_ERR_MISMATCH): the rotation cancels in the product only when both operands carry the same H'
 * along the shared axis (Sec. 2.2).
 */
typedef struct {
    /* storage, set by the caller */
    void *codes;             /* device; panel layout above (UFP4_FMT_UNIFORM_MX32: see ufp4_mx_quantize) */
    void *scales;            /* device; fp32, or E8M0 bytes for UFP4_FMT_UNIFORM_MX32                   */
    int64_t code_panel_ld;   /* bytes from one panel of codes to the next                               */
    int64_t scale_panel_ld;  /* scale elements (floats, or bytes for E8M0) from one panel to the next   */
    int64_t panels;          /* whole panels the two buffers hold                                        */
    /* contents, written by the quantizer */
    int64_t rows;            /* operand rows                                                             */
    int64_t red;             /* reduction length                                                         */
    int32_t format;          /* UFP4_FMT_*                                                               */
    int32_t rht_block;       /* RHT along the reduction axis: 0 (none), 16, 32, 64 or 128                */
    uint16_t sign_words[8];  /* its signs: eps_j = -1 iff bit (j % 16) of word j / 16; unused words 0    */
    float max_fpx;           /* E2M1 grid cut at 2 or 4 (Sec. 5 Q4); 0 for the full grid                 */
    int32_t rounding;        /* UFP4_ROUND_* used (recorded only)                                        */
    int32_t layout;          /* UFP4_LAYOUT_*                                                            */
    int32_t reserved;        /* 0                                                                        */
} ufp4_qtensor;

/* Human-readable name of a status code (static string). */
const char *ufp4_status_string(int status);

/* Library version, "major.minor.patch". */
const char *ufp4_version(void);

/*
 * ufp4_qtensor_bytes -- the minimal storage of a [rows, red] operand of `format` (UFP4_FMT_*): panel count, panel
 * strides (code_panel_ld bytes; scale_panel_ld floats, or bytes for UFP4_FMT_UNIFORM_MX32) and the two buffer
 * sizes in bytes. Any output pointer may be NULL. red must be a multiple of 16 (32 for UFP4_FMT_UNIFORM_MX32);
 * an empty operand still has one panel. Host only.
 */
int ufp4_qtensor_bytes(int format, int64_t rows, int64_t red, int64_t *panels, int64_t *code_panel_ld,
                       int64_t *scale_panel_ld, size_t *codes_bytes, size_t *scales_bytes);

/*
 * ufp4_grouped_reduction -- the padded axis of a grouped operand: each group's tokens zero-padded to a multiple
 * of `block`, groups concatenated. block 16: the reduction of ufp4_quantize_grouped_t (bwd_dw of a MoE layer);
 * 32: that of ufp4_mx_quantize_grouped with transpose 1; 128: the rows of ufp4_mx_quantize_grouped with
 * transpose 0 (each group on whole panels). From host token offsets off_0 = 0 <= ... <= off_G: total = sum_g
 * block ceil((off_{g+1} - off_g) / block), and, if padded_offsets_host is not NULL, the G + 1 padded offsets
 * pad_0 = 0, pad_{g+1} = pad_g + block ceil((off_{g+1} - off_g) / block). Host only; other blocks return
 * UFP4_ERR_INVALID_ARG.
 */
int ufp4_grouped_reduction(const int64_t *group_offsets_host, int32_t num_groups, int32_t block,
                           int64_t *padded_offsets_host, int64_t *total);

/*
 * ufp4_rht_quantize -- fused RHT + uniform-grid quantization of one GEMM operand (Sec. 2.1, Sec. 2.2;
 * recipe of Sec. 4 / Table 1). Uniform grid, codes -7..7, g = 7.
 *
 *   x_dev      bf16 [rows, cols], leading dimension ld (elements).
 *   transpose  0: operand A = X, reduction along cols (cols % 16 == 0); Q is [rows, cols].
 *              1: operand A = X^T, reduction along rows (rows % 16 == 0); Q is [cols, rows].
 *   rht        nonzero: apply the block-16 RHT with sign_mask (bits 0..15) before quantizing.
 *   rounding   UFP4_ROUND_RTNE or UFP4_ROUND_SR (seed, stream_id select the Philox draws; ignored for RTNE).
 *   out        storage set by the caller; its contents fields are written.
 * Rowwise operands (transpose = 0) of more than 2097024 rows (16383 panels) return UFP4_ERR_UNSUPPORTED.
 */
int ufp4_rht_quantize(const void *x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht,
                      uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, ufp4_qtensor *out,
                      void *stream);

/* ufp4_e2m1_quantize -- the same operation on the E2M1 grid (g = 6, levels 0, .5, 1, 1.5, 2, 3, 4, 6),
 * the comparison baseline of Table 1. Arguments as ufp4_rht_quantize. */
int ufp4_e2m1_quantize(const void *x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht,
                       uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, ufp4_qtensor *out,
                       void *stream);

/*
 * ufp4_e2m1_quantize_range -- ufp4_e2m1_quantize on the E2M1 grid cut at max_fpx (Sec. 5 Q4, the
 * range-restricted E2M1 ablation): only the levels up to max_fpx are kept and g = max_fpx, so s = RN(amax /
 * max_fpx). max_fpx = 2 keeps 0, .5, 1, 1.5, 2; 4 keeps 0 .. 4; 6 is the full grid. The codes are the
 * E2M1 codes of the kept levels, so the E2M1 GEMMs consume the result unchanged. Other max_fpx values
 * (0 included) return UFP4_ERR_INVALID_ARG. Remaining arguments as ufp4_rht_quantize.
 */
int ufp4_e2m1_quantize_range(const void *x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht,
                             uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, float max_fpx,
                             ufp4_qtensor *out, void *stream);

/*
 * ufp4_quantize_rht_block -- RHT over blocks of n = 16, 32, 64 or 128 elements along the reduction axis, then
 * the usual 1x16 quantization of the result (the RHT block-size dimension of the paper's E2M1 reference
 * search, Appendix; the recipe itself uses 16). Per n-block: y = the fp32 rounding (as above) of
 * RN64( S * RN64(sqrt(1/n)) ) with S the exact sum_j H_n[i,j] eps_j x_j (H_n the Sylvester +-1 matrix, exact when a
 * block's nonzero |x| span at most 2^(45 - log2 n)); for n = 16 and 64 the factor is a power of two and y is
 * correctly rounded.
 *   rht_block        16, 32, 64 or 128; the reduction length must be a multiple of it.
 *   sign_words_host  host array of rht_block / 16 words: eps_j = -1 iff bit (j % 16) of word j / 16 is set.
 *   format           UFP4_FMT_UNIFORM or UFP4_FMT_E2M1 (full grid). Rowwise and plain transposed operands
 *                    (not grouped). rht_block = 16 is ufp4_rht_quantize / ufp4_e2m1_quantize with rht = 1.
 *   Remaining arguments as ufp4_rht_quantize. A GEMM's two operands must use the same block and signs.
 */
int ufp4_quantize_rht_block(int format, const void *x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose,
                            int rht_block, const uint16_t *sign_words_host, int rounding, uint64_t seed,
                            uint32_t stream_id, ufp4_qtensor *out, void *stream);

/*
 * ufp4_quant_stats -- quality statistics of one quantization, the sums behind the diagnostics of Sec. 3.2
 * (NMSE_A(G, T), SQNR, the operand projection alpha, the bucket entropy behind B_eff). The operand is
 * quantized exactly as ufp4_rht_quantize / ufp4_e2m1_quantize(_range) would quantize it, but nothing is
 * stored except the record below. For every element, ref is the value the quantizer rounds (the RHT output
 * y when rht != 0, else x) and q = level(code) * scale its dequantized value.
 *
 *   format, max_fpx  UFP4_FMT_UNIFORM with max_fpx = 0, or UFP4_FMT_E2M1 with max_fpx 0 (full grid), 2, 4, 6.
 *   stats_dev        device pointer (8-byte aligned) to one ufp4_quant_stats_t record, overwritten (zero for
 *                    an empty operand, whose x_dev may be NULL). fp64 sums are accumulated with atomics: their
 *                    last bits may differ between calls; the counts are exact.
 *   Other arguments as ufp4_rht_quantize. ufp4_quant_metrics turns the record into the Sec. 3.2 metrics.
 */
typedef struct {
    double err2;           /* sum of (q - ref)^2 */
    double ref2;           /* sum of ref^2 */
    double cross;          /* sum of q * ref */
    uint64_t hist[8];      /* elements whose magnitude code is m = 0..7 (m = 0: zero) */
} ufp4_quant_stats_t;

int ufp4_quant_stats(int format, float max_fpx, const void *x_dev, int64_t rows, int64_t cols, int64_t ld,
                     int transpose, int rht, uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id,
                     ufp4_quant_stats_t *stats_dev, void *stream);

/*
 * ufp4_quant_metrics -- the Sec. 3.2 diagnostics of one quantization from its ufp4_quant_stats_t record (host
 * copy): NMSE = err2 / ref2, SQNR = -10 log10 NMSE (dB; +inf when err2 = 0), the operand projection alpha =
 * cross / ref2 (NaN for an all-zero operand), and the bucket statistics over the K magnitude levels of the
 * grid, zero included (K = 8; the E2M1 grid cut at max_fpx 2 or 4 has K = 5 or 7): p_m = hist[m] / sum, the
 * entropy E = -sum_m p_m log(p_m + 1e-12) and B_eff = exp(E) / K. format and max_fpx as in ufp4_quant_stats.
 * Host only.
 */
typedef struct {
    double nmse;
    double sqnr_db;
    double alpha;
    double entropy;
    double beff;
} ufp4_quant_metrics_t;

int ufp4_quant_metrics(const ufp4_quant_stats_t *stats_host, int format, float max_fpx,
                       ufp4_quant_metrics_t *metrics_host);

/*
 * ufp4_rotation_gain -- Sec. 3.2's Delta SQNR of a rotation, 10 log10(NMSE without RHT / NMSE with RHT) in dB
 * (positive when the rotation lowers the quantization error), from the metrics of the two quantizations of
 * one operand; and the attenuation of a GEMM's coherent signal, eta = alpha_A * alpha_B, from the metrics of
 * its two operands. Either output pointer may be NULL. Host only.
 */
int ufp4_rotation_gain(const ufp4_quant_metrics_t *raw_host, const ufp4_quant_metrics_t *rotated_host,
                       double *delta_sqnr_db);
int ufp4_gemm_attenuation(const ufp4_quant_metrics_t *a_host, const ufp4_quant_metrics_t *b_host, double *eta);

/*
 * The unfused form of RHT + quantization (Sec. 5 Q5 measures it against the fused kernel): a standalone
 * transform that writes the rotated tensor, then a plain quantization of it. The intermediate is fp32, which
 * holds y exactly (unless a rotated value passes FLT_MAX, which only inputs within a factor 4 of the bf16
 * maximum produce), so ufp4_quantize_f32(ufp4_rht(x)) produces the same codes and scales as
 * ufp4_rht_quantize(x, rht = 1) (rowwise) bit for bit.
 *
 * ufp4_rht -- y = RN_fp32( x S_16 H_16 ) for every 16-block along the rows of x (Sec. 2.2; the arithmetic
 *   of the quantizer's transform, see the conventions above; +-inf past FLT_MAX). x_dev bf16 [rows, cols]
 *   (cols % 16 == 0, ld as for the quantizers); y_dev fp32 [rows, cols] with leading dimension ldy (ldy >= cols,
 *   ldy % 4 == 0, 16-byte aligned). sign_mask as for ufp4_rht_quantize.
 */
int ufp4_rht(const void *x_dev, int64_t rows, int64_t cols, int64_t ld, uint32_t sign_mask, float *y_dev,
             int64_t ldy, void *stream);

/*
 * ufp4_quantize_f32 -- rowwise quantization of an fp32 tensor without a transform (the second half of the
 *   unfused form): operand A = X [rows, cols] along cols, the arithmetic of ufp4_rht_quantize with rht = 0
 *   applied to fp32 values. format UFP4_FMT_UNIFORM or UFP4_FMT_E2M1 (full grid); ld >= cols, ld % 4 == 0,
 *   x_dev 16-byte aligned; inputs finite. rht, sign_mask: the block-16 RHT the input already carries (from
 *   ufp4_rht), recorded in `out` for the GEMMs' operand check; they do not change the arithmetic. Remaining
 *   arguments as ufp4_rht_quantize.
 */
int ufp4_quantize_f32(int format, const float *x_dev, int64_t rows, int64_t cols, int64_t ld, int rht,
                      uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, ufp4_qtensor *out,
                      void *stream);

/*
 * ufp4_quantize_grouped_t -- transposed quantization of an expert-grouped tensor (MoE), either grid.
 *
 *   x_dev              bf16 [rows, cols] (ld elements); rows are split into num_groups consecutive groups.
 *   group_offsets_dev  int64 [num_groups + 1] device array, 0 = off_0 <= ... <= off_G = rows.
 *   red_total          reduction length of Q, at least pad_G (ufp4_grouped_reduction) when the offsets are known
 *                      on the host, else any bound such as rows + 15 * num_groups; blocks past pad_G are zero.
 *   Q is [cols, red_total]: group g's block of Q is X[off_g:off_{g+1}]^T with its reduction (token) axis
 *   zero-padded to a multiple of 16, at reduction positions pad_g .. pad_{g+1} (the padded offsets are computed
 *   on the device from the token offsets). Block numbers in the SR counters count along the padded
 *   concatenated axis. Used for bwd_dw's dY^T and X^T and, with equal groups, for the per-expert W^T of bwd_dx.
 *   num_groups up to 1024.
 */
int ufp4_quantize_grouped_t(int format, const void *x_dev, int64_t rows, int64_t cols, int64_t ld,
                            const int64_t *group_offsets_dev, int32_t num_groups, int64_t red_total, int rht,
                            uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, ufp4_qtensor *out,
                            void *stream);

/*
 * ufp4_quantize_dual -- both quantized operands of one tensor from a single read of it (either grid):
 * Q_r = Q(X H') [rows, cols] along cols (transpose 0) and Q_c = Q(X^T H') [cols, rows] along rows
 * (transpose 1), as the fused RHT + quantize of Sec. 2.2 needs them for the two GEMMs a training step runs
 * on X (fwd_y and bwd_dw for X; bwd_dx and bwd_dw for dY; fwd_y and bwd_dx for W). Each output has its own
 * RHT flag, sign mask and SR stream; the results equal, bit for bit, ufp4_rht_quantize /
 * ufp4_e2m1_quantize called with transpose 0 and 1 and those arguments. The input is read from HBM once
 * (2 bytes per element instead of 4).
 *
 *   format             UFP4_FMT_UNIFORM or UFP4_FMT_E2M1.
 *   x_dev              bf16 [rows, cols], leading dimension ld; rows % 16 == 0 and cols % 16 == 0.
 *   rht_rows, sign_mask_rows, stream_rows   RHT and SR stream of Q_r; *_cols the same for Q_c.
 *   rounding, seed     as ufp4_rht_quantize, for both outputs.
 *   out_rows, out_cols Q_r and Q_c. The two outputs must not overlap each other or the input.
 */
int ufp4_quantize_dual(int format, const void *x_dev, int64_t rows, int64_t cols, int64_t ld, int rht_rows,
                       uint32_t sign_mask_rows, uint32_t stream_rows, int rht_cols, uint32_t sign_mask_cols,
                       uint32_t stream_cols, int rounding, uint64_t seed, ufp4_qtensor *out_rows,
                       ufp4_qtensor *out_cols, void *stream);

/*
 * Power-of-two block scales. The paper leaves the scale hierarchy open (Sec. 4: single-level, two-level or
 * block scales, chosen for the hardware); these calls pair the same uniform grid and RHT with one scale per
 * 1x32 block that gfx950's scaled matrix-core instruction applies itself.
 *
 * ufp4_mx_quantize -- fused RHT + quantization with power-of-two scales. Per 1x32 block along the reduction
 *   axis: y = RHT16 of each half as in ufp4_rht_quantize (or y = x); E = max(floor(log2 amax |y|) - 2, -127)
 *   (the OCP Microscaling shared-exponent rule, the levels read as FP6 E2M3 numbers; E8M0 stops at 2^-127);
 *   v = RN32(y * 2^-E) (|v| < 8); codes -7..7 by RTNE or SR (same rules and Philox draws, the counters numbering
 *   16-blocks), |v| > 7 clamped to the top level. Arguments as ufp4_rht_quantize, except:
 *     red % 32 == 0 (cols when transpose = 0, rows when transpose = 1); out->format becomes
 *     UFP4_FMT_UNIFORM_MX32;
 *     codes: FP6 E2M3 numbers (the integers -7..7 are exact), 32 per block in 24 bytes, element j in bits
 *            6j .. 6j + 5 of the block's little-endian 192-bit string;
 *     scales: uint8 E8M0 bytes E + 127 (0 for an all-zero block).
 *   Layout (panels of 128 rows, 32-blocks): the 24 code bytes of block b of row 128p + i are three 8-byte
 *   units, unit u (bytes 8u .. 8u + 7 of the string) at codes + p * code_panel_ld + b * 3072 + u * 1024
 *   + i * 8; its scale at scales + p * scale_panel_ld + b * 128 + i. code_panel_ld >= 3072 * red/32 and
 *   scale_panel_ld >= 128 * red/32, both multiples of 16; both pointers 16-byte aligned.
 *   Padding rows of the last panel are written as zero codes and scale byte 0. Rowwise operands of more than
 *   4194176 rows (32767 panels) return UFP4_ERR_UNSUPPORTED.
 */
int ufp4_mx_quantize(const void *x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht,
                     uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, ufp4_qtensor *out,
                     void *stream);

/*
 * ufp4_mx_quantize_dual -- both power-of-two-scale operands of one tensor from a single read of it: Q_r =
 *   Q(X H') [rows, cols] along cols and Q_c = Q(X^T H') [cols, rows] along rows, the pair the two GEMMs of a
 *   training step on X need (Sec. 2.2); equal, bit for bit, to ufp4_mx_quantize with transpose 0 and 1 and
 *   these arguments. rows % 32 == 0 and cols % 32 == 0; 2^31 rows or columns or more return
 *   UFP4_ERR_UNSUPPORTED. Each output has its own RHT flag, sign mask and SR stream; rounding and seed
 *   serve both. The outputs must not overlap each other or the input; the same descriptor for both returns
 *   UFP4_ERR_INVALID_ARG. Storage, padding rows and errors as ufp4_mx_quantize.
 */
int ufp4_mx_quantize_dual(const void *x_dev, int64_t rows, int64_t cols, int64_t ld, int rht_rows,
                          uint32_t sign_mask_rows, uint32_t stream_rows, int rht_cols, uint32_t sign_mask_cols,
                          uint32_t stream_cols, int rounding, uint64_t seed, ufp4_qtensor *out_rows,
                          ufp4_qtensor *out_cols, void *stream);

/*
 * ufp4_mx_gemm_fwd_y / _bwd_dx / _bwd_dw -- the three passes (operand roles as the ufp4_gemm_* calls below) on
 *   operands from ufp4_mx_quantize: C[i, j] = sum_k A[i,k] 2^(eA - 127) B[j,k] 2^(eB - 127) with the scales of
 *   each element's 32-block, accumulated in fp32 by the matrix core; output fp32 or bf16 (RNE) with leading
 *   dimension ldc. Outputs of 2^31 or more 128 x 128 tiles return UFP4_ERR_UNSUPPORTED; operands that are not
 *   UFP4_FMT_UNIFORM_MX32 or differ in RHT block, signs or reduction length return UFP4_ERR_MISMATCH.
 */
int ufp4_mx_gemm_fwd_y(const ufp4_qtensor *x, const ufp4_qtensor *w, void *y_dev, int64_t ldc, int out_dtype,
                       void *stream);
int ufp4_mx_gemm_bwd_dx(const ufp4_qtensor *dy, const ufp4_qtensor *wt, void *dx_dev, int64_t ldc, int out_dtype,
                        void *stream);
int ufp4_mx_gemm_bwd_dw(const ufp4_qtensor *dyt, const ufp4_qtensor *xt, void *dw_dev, int64_t ldc, int out_dtype,
                        void *stream);

/*
 * Grouped (MoE) operands and GEMMs with power-of-two scales. The GEMM stages whole 128-row panels, so an expert's
 * rows must start on a panel boundary: the ragged-M passes take A from the grouped-rows form below.
 *
 * ufp4_mx_quantize_grouped -- ufp4_mx_quantize over G groups of X's rows (device token offsets off_0 = 0 <= ...
 *   <= off_G <= rows, up to 1024 groups).
 *     transpose 0 (grouped rows; A of the grouped fwd_y and bwd_dx): Q is [padded_total, cols], cols % 32 == 0;
 *       group g's rows are X[off_g .. off_{g+1}) starting at row P_g = sum_{h<g} 128 ceil((off_{h+1} - off_h) /
 *       128), each quantized as ufp4_mx_quantize quantizes it (its SR counters use its row of X), the rows that
 *       pad a group to whole panels and any rows past the last group zero. padded_total >= P_G
 *       (ufp4_grouped_reduction with block 128).
 *     transpose 1 (grouped reduction; both operands of the grouped bwd_dw): Q is [cols, padded_total], the
 *       reduction axis being each group's tokens zero-padded to a multiple of 32 (no 32-block straddles two
 *       groups), groups concatenated; block numbers in the SR counters count along this axis. padded_total =
 *       ufp4_grouped_reduction with block 32.
 *   Other arguments and the storage as ufp4_mx_quantize; out->layout records the form.
 */
int ufp4_mx_quantize_grouped(const void *x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose,
                             const int64_t *group_offsets_dev, int32_t num_groups, int64_t padded_total, int rht,
                             uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, ufp4_qtensor *out,
                             void *stream);

/*
 * ufp4_mx_gemm_fwd_y_grouped -- Y[off_g .. off_{g+1}) = Q(X_g H') Q(W_g H')^T per group: x in grouped-rows form
 *   [*, K], w plain [G * N, K] (group g's weight rows g N .. g N + N - 1; N % 128 == 0), y [m_total, N] row-major
 *   with ldc >= N, m_total the rows of X (outputs past it are not written).
 * ufp4_mx_gemm_bwd_dx_grouped -- dX[off_g .. off_{g+1}) = Q(dY_g H') Q(W_g^T H')^T: dy in grouped-rows form [*, N]
 *   (N % 32 == 0), wt plain [K, G * N] (group g reduces over its positions g N .. g N + N - 1), dx [m_total, K].
 * ufp4_mx_gemm_bwd_dw_grouped -- dW[g] = Q(dY_g^T H') Q(X_g^T H')^T: dyt [N, R] and xt [K, R] in grouped-reduction
 *   form with the same offsets (R = the padded token axis), dw [G, N, K] (group g at dw + g N ldc; a group
 *   without tokens gets zeros). Up to 65535 groups.
 *   Operand forms other than these return UFP4_ERR_MISMATCH, as do the checks of the ungrouped calls.
 */
int ufp4_mx_gemm_fwd_y_grouped(const ufp4_qtensor *x, const ufp4_qtensor *w, const int64_t *group_offsets_dev,
                               int32_t num_groups, int64_t m_total, void *y_dev, int64_t ldc, int out_dtype,
                               void *stream);
int ufp4_mx_gemm_bwd_dx_grouped(const ufp4_qtensor *dy, const ufp4_qtensor *wt, const int64_t *group_offsets_dev,
                                int32_t num_groups, int64_t m_total, void *dx_dev, int64_t ldc, int out_dtype,
                                void *stream);
int ufp4_mx_gemm_bwd_dw_grouped(const ufp4_qtensor *dyt, const ufp4_qtensor *xt, const int64_t *group_offsets_dev,
                                int32_t num_groups, void *dw_dev, int64_t ldc, int out_dtype, void *stream);

/*
 * Block-scaled 4-bit GEMMs (Sec. 2.2). All three passes are NT products of two quantized operands that
 * share their reduction axis (the axis the RHT was applied along):
 *
 *   ufp4_gemm_fwd_y : Y  [M, N] = Q(X H')   [M, K] . Q(W H')   [N, K]^T
 *   ufp4_gemm_bwd_dx: dX [M, K] = Q(dY H')  [M, N] . Q(W^T H') [K, N]^T
 *   ufp4_gemm_bwd_dw: dW [N, K] = Q(dY^T H')[N, M] . Q(X^T H') [K, M]^T
 *
 * The shapes come from the descriptors (output rows = left operand's rows, columns = right operand's rows).
 * Both operands must be UFP4_FMT_UNIFORM or both UFP4_FMT_E2M1 with the same rht_block, sign words and
 * reduction length, else UFP4_ERR_MISMATCH. out_dtype UFP4_OUT_F32 or UFP4_OUT_BF16; out_dev row-major with
 * leading dimension ldc (elements).
 */
int ufp4_gemm_fwd_y(const ufp4_qtensor *x, const ufp4_qtensor *w, void *y_dev, int64_t ldc, int out_dtype,
                    void *stream);
int ufp4_gemm_bwd_dx(const ufp4_qtensor *dy, const ufp4_qtensor *wt, void *dx_dev, int64_t ldc, int out_dtype,
                     void *stream);
int ufp4_gemm_bwd_dw(const ufp4_qtensor *dyt, const ufp4_qtensor *xt, void *dw_dev, int64_t ldc, int out_dtype,
                     void *stream);

/*
 * Grouped (MoE) forms: num_groups experts, token rows expert-contiguous, group_offsets_dev the int64 token
 * offsets [num_groups + 1] on the device (0 = off_0 <= ... <= off_G).
 *
 *   fwd_y : Y_g  [m_g, N] = Qx[off_g:off_{g+1}, :K] . Qw[g*N:(g+1)*N, :K]^T         (Y  [M_total, N])
 *           Qx [M_total, K]; Qw [G*N, K] (its rows a multiple of num_groups).
 *   bwd_dx: dX_g [m_g, K] = Qdy[off_g:off_{g+1}, :N] . Qwt[:K, g*N:(g+1)*N]^T        (dX [M_total, K])
 *           Qdy [M_total, N]; Qwt [K, G*N] is the grouped-transposed quantization of W [G*N, K] with equal
 *           groups (its reduction length must be num_groups times Qdy's).
 *   bwd_dw: dW_g [N, K]  = Qdyt[:N, pad_g:pad_{g+1}] . Qxt[:K, pad_g:pad_{g+1}]^T    (dW [G, N, K], each
 *           [N, K] with leading dimension ldc, groups N * ldc apart). Qdyt [N, R], Qxt [K, R] from
 *           ufp4_quantize_grouped_t on the same offsets; the padded offsets pad_g are computed on the device.
 *
 * Offsets are read on the device: rows past M_total and reduction positions past R are ignored, output rows
 * past off_G (fwd_y, bwd_dx) are not written, groups with no tokens give dW_g = 0. Operand checks as for the dense calls; besides, fwd_y takes plain operands, bwd_dx a
 * plain Qdy and a plain or grouped-transposed Qwt (the same bytes: N is a multiple of 16), bwd_dw two
 * grouped-transposed operands (UFP4_LAYOUT_GROUPED_RED); other forms return UFP4_ERR_MISMATCH. num_groups up to
 * 65535.
 */
int ufp4_gemm_fwd_y_grouped(const ufp4_qtensor *x, const ufp4_qtensor *w, const int64_t *group_offsets_dev,
                            int32_t num_groups, void *y_dev, int64_t ldc, int out_dtype, void *stream);
int ufp4_gemm_bwd_dx_grouped(const ufp4_qtensor *dy, const ufp4_qtensor *wt, const int64_t *group_offsets_dev,
                             int32_t num_groups, void *dx_dev, int64_t ldc, int out_dtype, void *stream);
int ufp4_gemm_bwd_dw_grouped(const ufp4_qtensor *dyt, const ufp4_qtensor *xt, const int64_t *group_offsets_dev,
                             int32_t num_groups, void *dw_dev, int64_t ldc, int out_dtype, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* UFP4_H */
