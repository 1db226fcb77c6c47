// C ABI of libufp4: argument validation on the host, then one kernel launch on the caller's stream.
// Declarations and the meaning of every argument are in include/ufp4.h.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "../../include/ufp4.h"
#include "ufp4_internal.h"

using namespace ufp4;

static_assert(sizeof(ufp4_quant_stats_t) == sizeof(QuantStats), "statistics record layout");

namespace {

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

void fill_sign_xor(uint32_t mask, uint32_t (&sx)[8]) {
    for (int j = 0; j < 8; ++j) {
        sx[j] = (((mask >> (2 * j)) & 1u) ? 0x00008000u : 0u) | (((mask >> (2 * j + 1)) & 1u) ? 0x80000000u : 0u);
    }
}

int status_of(hipError_t e) { return e == hipSuccess ? UFP4_OK : UFP4_ERR_HIP; }

// Top level of the E2M1 grid: max_fpx 0 (the full grid, 6) or 2, 4, 6; the uniform grid takes 0 only.
bool valid_max_fpx(int format, float max_fpx) {
    if (max_fpx == 0.0f) return true;
    return format == UFP4_FMT_E2M1 && (max_fpx == 2.0f || max_fpx == 4.0f || max_fpx == 6.0f);
}

void fill_grid(float max_fpx, QuantArgs& qa) {
    const float g = max_fpx == 0.0f ? 6.0f : max_fpx;
    qa.e2m1_g = g;
    qa.e2m1_ginv = 1.0f / g;  // RN(1/g), as the kernels' constant for the uniform grid
    qa.rht_m = 1;             // block-16 RHT unless a caller asks for a wider one
    qa.rht_c = 0.25;
}

constexpr int64_t kMaxCodePanelLd = int64_t(1) << 29;   // bytes
constexpr int64_t kMaxScalePanelLd = int64_t(1) << 27;  // floats

// Panel-layout strides of a quantized operand with reduction length `red`.
int check_panels(const void* codes, int64_t code_pld, const float* scales, int64_t scale_pld, int64_t red) {
    const int64_t nkb = red / 16;
    if (code_pld < nkb * kPanelBlockBytes || scale_pld < nkb * kPanelBlockScales) return UFP4_ERR_SHAPE;
    if (code_pld % 16 != 0 || scale_pld % 4 != 0) return UFP4_ERR_ALIGN;
    if (!aligned(codes, 16) || !aligned(scales, 16)) return UFP4_ERR_ALIGN;
    if (code_pld > kMaxCodePanelLd || scale_pld > kMaxScalePanelLd) return UFP4_ERR_UNSUPPORTED;
    return UFP4_OK;
}

// Checks shared by the plain and grouped quantizers. `red` is the operand's reduction length, `qrows` its
// row count.
int check_quant_common(int format, const void* x, int64_t rows, int64_t cols, int64_t ld, int rht, uint32_t sign_mask,
                       int rounding, const void* codes, int64_t code_pld, const float* scales, int64_t scale_pld,
                       int64_t red, int64_t qrows) {
    if (format != UFP4_FMT_UNIFORM && format != UFP4_FMT_E2M1) return UFP4_ERR_INVALID_ARG;
    if (rounding != UFP4_ROUND_RTNE && rounding != UFP4_ROUND_SR) return UFP4_ERR_INVALID_ARG;
    if (rht != 0 && rht != 1) return UFP4_ERR_INVALID_ARG;
    if (sign_mask > 0xFFFFu) return UFP4_ERR_INVALID_ARG;
    if (rows < 0 || cols < 0 || red < 0 || qrows < 0) return UFP4_ERR_INVALID_ARG;
    if (!x || !codes || !scales) return UFP4_ERR_INVALID_ARG;
    if (ld < cols || ld % 8 != 0) return UFP4_ERR_SHAPE;
    if (red % 16 != 0) return UFP4_ERR_SHAPE;
    if (!aligned(x, 16)) return UFP4_ERR_ALIGN;
    const int st = check_panels(codes, code_pld, scales, scale_pld, red);
    if (st != UFP4_OK) return st;
    if (qrows >= (int64_t(1) << 31) || red / 16 >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    return UFP4_OK;
}

// rht_block 16 (with sign_mask) or 32 / 64 / 128 (with the n/16 words of `sign_words`).
int quantize_impl(int format, const void* x, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht,
                  uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, void* codes, int64_t code_pld,
                  float* scales, int64_t scale_pld, void* stream, float max_fpx = 0.0f, int rht_block = 16,
                  const uint16_t* sign_words = nullptr) {
    if (transpose != 0 && transpose != 1) return UFP4_ERR_INVALID_ARG;
    if (!valid_max_fpx(format, max_fpx)) return UFP4_ERR_INVALID_ARG;
    const int64_t red = transpose ? rows : cols;
    const int64_t qrows = transpose ? cols : rows;
    const int st = check_quant_common(format, x, rows, cols, ld, rht, sign_mask, rounding, codes, code_pld, scales,
                                      scale_pld, red, qrows);
    if (st != UFP4_OK) return st;
    // rowwise: one workgroup per 32 padded rows along the grid's y dimension
    if (!transpose && padded_rows(qrows) / 32 > 65535) return UFP4_ERR_UNSUPPORTED;
    if (rht_block != 16 && red % rht_block != 0) return UFP4_ERR_SHAPE;
    if (rows == 0 || cols == 0) return UFP4_OK;
    QuantJob j{};
    j.format = format;
    j.rounding = rounding;
    j.rht = rht;
    j.transpose = transpose;
    j.x = x;
    j.xrows = rows;
    j.ld = ld;
    j.qrows = qrows;
    j.red = red;
    j.group_off = nullptr;
    j.group_poff = nullptr;
    j.num_groups = 1;
    fill_sign_xor(sign_mask, j.qa.sign_xor);
    fill_grid(max_fpx, j.qa);
    j.qa.rht_m = rht_block / 16;
    j.qa.rht_c = sqrt(1.0 / rht_block);  // correctly rounded square root of an exact power of two
    for (int k = 0; k < rht_block / 16 && sign_words; ++k) j.qa.sign_words[k] = sign_words[k];
    j.qa.key0 = (uint32_t)seed;
    j.qa.key1 = (uint32_t)(seed >> 32);
    j.qa.stream = stream_id;
    j.codes = codes;
    j.code_pld = code_pld;
    j.scales = scales;
    j.scale_pld = scale_pld;
    return status_of(launch_quantize(j, static_cast<hipStream_t>(stream)));
}

// Panel layout of an operand with power-of-two 1x32 scales (reduction length `red`, a multiple of 32).
int check_panels_mx(const void* codes, int64_t code_pld, const void* scales, int64_t scale_pld, int64_t red) {
    const int64_t nkb = red / 32;
    if (code_pld < nkb * kMxPanelBlockBytes || scale_pld < nkb * kMxPanelBlockScales) return UFP4_ERR_SHAPE;
    if (code_pld % 16 != 0 || scale_pld % 16 != 0) return UFP4_ERR_ALIGN;
    if (!aligned(codes, 16) || !aligned(scales, 16)) return UFP4_ERR_ALIGN;
    if (code_pld > kMaxCodePanelLd || scale_pld > kMaxCodePanelLd) return UFP4_ERR_UNSUPPORTED;
    return UFP4_OK;
}

int mx_quantize_impl(const void* x, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht, uint32_t sign_mask,
                     int rounding, uint64_t seed, uint32_t stream_id, void* codes, int64_t code_pld, void* scales,
                     int64_t scale_pld, void* stream) {
    if (transpose != 0 && transpose != 1) return UFP4_ERR_INVALID_ARG;
    if (rounding != UFP4_ROUND_RTNE && rounding != UFP4_ROUND_SR) return UFP4_ERR_INVALID_ARG;
    if (rht != 0 && rht != 1) return UFP4_ERR_INVALID_ARG;
    if (sign_mask > 0xFFFFu) return UFP4_ERR_INVALID_ARG;
    if (rows < 0 || cols < 0) return UFP4_ERR_INVALID_ARG;
    if (!x || !codes || !scales) return UFP4_ERR_INVALID_ARG;
    const int64_t red = transpose ? rows : cols;
    const int64_t qrows = transpose ? cols : rows;
    if (ld < cols || ld % 8 != 0) return UFP4_ERR_SHAPE;
    if (red % 32 != 0) return UFP4_ERR_SHAPE;
    if (!aligned(x, 16)) return UFP4_ERR_ALIGN;
    const int st = check_panels_mx(codes, code_pld, scales, scale_pld, red);
    if (st != UFP4_OK) return st;
    if (qrows >= (int64_t(1) << 31) || red / 16 >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    if (!transpose && padded_rows(qrows) / 64 > 65535) return UFP4_ERR_UNSUPPORTED;  // one workgroup row per 64
    if (rows == 0 || cols == 0) return UFP4_OK;
    MxQuantJob j{};
    j.rounding = rounding;
    j.rht = rht;
    j.transpose = transpose;
    j.x = x;
    j.xrows = rows;
    j.ld = ld;
    j.qrows = qrows;
    j.red = red;
    fill_sign_xor(sign_mask, j.qa.sign_xor);
    j.qa.key0 = (uint32_t)seed;
    j.qa.key1 = (uint32_t)(seed >> 32);
    j.qa.stream = stream_id;
    j.codes = codes;
    j.code_pld = code_pld;
    j.scales = scales;
    j.scale_pld = scale_pld;
    return status_of(launch_quantize_mx(j, static_cast<hipStream_t>(stream)));
}

// NT product of two operands with power-of-two scales: A [rows_a, red], B [rows_b, red].
int mx_gemm_impl(const void* a, int64_t a_pld, const void* as, int64_t as_pld, const void* b, int64_t b_pld,
                 const void* bs, int64_t bs_pld, int64_t rows_a, int64_t rows_b, int64_t red, void* c, int64_t ldc,
                 int out_dtype, void* stream) {
    if (out_dtype != UFP4_OUT_F32 && out_dtype != UFP4_OUT_BF16) return UFP4_ERR_INVALID_ARG;
    if (rows_a < 0 || rows_b < 0 || red < 0) return UFP4_ERR_INVALID_ARG;
    if (!a || !as || !b || !bs || !c) return UFP4_ERR_INVALID_ARG;
    if (red % 32 != 0) return UFP4_ERR_SHAPE;
    int st = check_panels_mx(a, a_pld, as, as_pld, red);
    if (st == UFP4_OK) st = check_panels_mx(b, b_pld, bs, bs_pld, red);
    if (st != UFP4_OK) return st;
    if (ldc < rows_b) return UFP4_ERR_SHAPE;
    if (!aligned(c, out_dtype == UFP4_OUT_F32 ? 4 : 2)) return UFP4_ERR_ALIGN;
    // one workgroup per 128 x 128 output tile on a one-dimensional grid
    if (((rows_a + 127) / 128) * ((rows_b + 127) / 128) >= (int64_t(1) << 31) || red / 32 >= (int64_t(1) << 31))
        return UFP4_ERR_UNSUPPORTED;
    if (rows_a == 0 || rows_b == 0) return UFP4_OK;
    MxGemmJob j{};
    j.out_dtype = out_dtype;
    j.a = static_cast<const uint8_t*>(a);
    j.a_pld = a_pld;
    j.as = static_cast<const uint8_t*>(as);
    j.as_pld = as_pld;
    j.b = static_cast<const uint8_t*>(b);
    j.b_pld = b_pld;
    j.bs = static_cast<const uint8_t*>(bs);
    j.bs_pld = bs_pld;
    j.M = rows_a;
    j.N = rows_b;
    j.nkb = red / 32;
    j.c = c;
    j.ldc = ldc;
    return status_of(launch_gemm_mx(j, static_cast<hipStream_t>(stream)));
}

// Shared checks of the GEMM entry points. A is [rows_a, red], B is [rows_b, red] (reduction contiguous).
int check_gemm(const void* a, int64_t a_pld, const float* as, int64_t as_pld, const void* b, int64_t b_pld,
               const float* bs, int64_t bs_pld, int64_t rows_a, int64_t rows_b, int64_t red_a, int64_t red_b, int format,
               const void* c, int64_t ldc, int64_t c_cols, int out_dtype) {
    if (format != UFP4_FMT_UNIFORM && format != UFP4_FMT_E2M1) return UFP4_ERR_INVALID_ARG;
    if (out_dtype != UFP4_OUT_F32 && out_dtype != UFP4_OUT_BF16) return UFP4_ERR_INVALID_ARG;
    if (rows_a < 0 || rows_b < 0 || red_a < 0 || red_b < 0) return UFP4_ERR_INVALID_ARG;
    if (!a || !as || !b || !bs || !c) return UFP4_ERR_INVALID_ARG;
    if (red_a % 16 != 0 || red_b % 16 != 0) return UFP4_ERR_SHAPE;
    if (ldc < c_cols) return UFP4_ERR_SHAPE;
    int st = check_panels(a, a_pld, as, as_pld, red_a);
    if (st == UFP4_OK) st = check_panels(b, b_pld, bs, bs_pld, red_b);
    if (st != UFP4_OK) return st;
    if (!aligned(c, out_dtype == UFP4_OUT_F32 ? 4 : 2)) return UFP4_ERR_ALIGN;
    if (rows_a >= (int64_t(1) << 31) || rows_b >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    return UFP4_OK;
}

GemmJob make_job(int mode, const void* a, int64_t a_pld, const float* as, int64_t as_pld, const void* b,
                 int64_t b_pld, const float* bs, int64_t bs_pld, int64_t M, int64_t N, int64_t nkb, int format, void* c,
                 int64_t ldc, int out_dtype) {
    GemmJob j{};
    j.format = format;
    j.out_dtype = out_dtype;
    j.mode = mode;
    j.a = static_cast<const uint8_t*>(a);
    j.a_pld = a_pld;
    j.as = as;
    j.as_pld = as_pld;
    j.b = static_cast<const uint8_t*>(b);
    j.b_pld = b_pld;
    j.bs = bs;
    j.bs_pld = bs_pld;
    j.M = M;
    j.N = N;
    j.nkb = nkb;
    j.c = c;
    j.ldc = ldc;
    j.offsets = nullptr;
    j.G = 1;
    return j;
}

int gemm_dense(const void* a, int64_t a_pld, const float* as, int64_t as_pld, const void* b, int64_t b_pld,
               const float* bs, int64_t bs_pld, int64_t rows_a, int64_t rows_b, int64_t red, int format, void* c,
               int64_t ldc, int out_dtype, void* stream) {
    const int st = check_gemm(a, a_pld, as, as_pld, b, b_pld, bs, bs_pld, rows_a, rows_b, red, red, format, c, ldc,
                              rows_b, out_dtype);
    if (st != UFP4_OK) return st;
    if (rows_a == 0 || rows_b == 0) return UFP4_OK;
    const GemmJob j = make_job(kGemmDense, a, a_pld, as, as_pld, b, b_pld, bs, bs_pld, rows_a, rows_b, red / 16, format,
                               c, ldc, out_dtype);
    return status_of(launch_gemm(j, static_cast<hipStream_t>(stream)));
}

}  // namespace

extern "C" {

const char* ufp4_status_string(int status) {
    switch (status) {
        case UFP4_OK: return "ok";
        case UFP4_ERR_INVALID_ARG: return "invalid argument";
        case UFP4_ERR_SHAPE: return "bad shape or leading dimension";
        case UFP4_ERR_ALIGN: return "misaligned pointer or leading dimension";
        case UFP4_ERR_UNSUPPORTED: return "unsupported";
        case UFP4_ERR_HIP: return "HIP launch error";
        default: return "unknown status";
    }
}

const char* ufp4_version(void) { return "0.1.0"; }

int ufp4_rht_quantize(const void* x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht,
                      uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, void* codes_dev,
                      int64_t code_panel_ld, float* scales_dev, int64_t scale_panel_ld, void* stream) {
    return quantize_impl(UFP4_FMT_UNIFORM, x_dev, rows, cols, ld, transpose, rht, sign_mask, rounding, seed, stream_id,
                         codes_dev, code_panel_ld, scales_dev, scale_panel_ld, stream);
}

int ufp4_e2m1_quantize(const void* x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht,
                       uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, void* codes_dev,
                       int64_t code_panel_ld, float* scales_dev, int64_t scale_panel_ld, void* stream) {
    return quantize_impl(UFP4_FMT_E2M1, x_dev, rows, cols, ld, transpose, rht, sign_mask, rounding, seed, stream_id,
                         codes_dev, code_panel_ld, scales_dev, scale_panel_ld, stream);
}

int ufp4_e2m1_quantize_range(const void* x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht,
                             uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, float max_fpx,
                             void* codes_dev, int64_t code_panel_ld, float* scales_dev, int64_t scale_panel_ld,
                             void* stream) {
    if (max_fpx == 0.0f) return UFP4_ERR_INVALID_ARG;  // the full grid is ufp4_e2m1_quantize
    return quantize_impl(UFP4_FMT_E2M1, x_dev, rows, cols, ld, transpose, rht, sign_mask, rounding, seed, stream_id,
                         codes_dev, code_panel_ld, scales_dev, scale_panel_ld, stream, max_fpx);
}

int ufp4_quantize_rht_block(int format, const void* x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose,
                            int rht_block, const uint16_t* sign_words_host, int rounding, uint64_t seed,
                            uint32_t stream_id, void* codes_dev, int64_t code_panel_ld, float* scales_dev,
                            int64_t scale_panel_ld, void* stream) {
    if (rht_block != 16 && rht_block != 32 && rht_block != 64 && rht_block != 128) return UFP4_ERR_INVALID_ARG;
    if (!sign_words_host) return UFP4_ERR_INVALID_ARG;
    if (format != UFP4_FMT_UNIFORM && format != UFP4_FMT_E2M1) return UFP4_ERR_INVALID_ARG;
    if (rht_block == 16)
        return quantize_impl(format, x_dev, rows, cols, ld, transpose, 1, sign_words_host[0], rounding, seed, stream_id,
                             codes_dev, code_panel_ld, scales_dev, scale_panel_ld, stream);
    return quantize_impl(format, x_dev, rows, cols, ld, transpose, 1, 0, rounding, seed, stream_id, codes_dev,
                         code_panel_ld, scales_dev, scale_panel_ld, stream, 0.0f, rht_block, sign_words_host);
}

int ufp4_quant_stats(int format, float max_fpx, const void* x_dev, int64_t rows, int64_t cols, int64_t ld,
                     int transpose, int rht, uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id,
                     ufp4_quant_stats_t* stats_dev, void* stream) {
    if (format != UFP4_FMT_UNIFORM && format != UFP4_FMT_E2M1) return UFP4_ERR_INVALID_ARG;
    if (!valid_max_fpx(format, max_fpx)) return UFP4_ERR_INVALID_ARG;
    if (rounding != UFP4_ROUND_RTNE && rounding != UFP4_ROUND_SR) return UFP4_ERR_INVALID_ARG;
    if (transpose != 0 && transpose != 1) return UFP4_ERR_INVALID_ARG;
    if (rht != 0 && rht != 1) return UFP4_ERR_INVALID_ARG;
    if (sign_mask > 0xFFFFu) return UFP4_ERR_INVALID_ARG;
    if (rows < 0 || cols < 0) return UFP4_ERR_INVALID_ARG;
    const bool empty = rows == 0 || cols == 0;
    if ((!x_dev && !empty) || !stats_dev) return UFP4_ERR_INVALID_ARG;  // an empty operand may have no storage
    if (ld < cols || ld % 8 != 0) return UFP4_ERR_SHAPE;
    const int64_t red = transpose ? rows : cols;
    const int64_t qrows = transpose ? cols : rows;
    if (red % 16 != 0) return UFP4_ERR_SHAPE;
    if (!aligned(x_dev, 16) || !aligned(stats_dev, 8)) return UFP4_ERR_ALIGN;
    if (qrows >= (int64_t(1) << 31) || red / 16 >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    StatsJob j{};
    j.format = format;
    j.rounding = rounding;
    j.rht = rht;
    j.transpose = transpose;
    j.x = x_dev;
    j.ld = ld;
    j.qrows = empty ? 0 : qrows;
    j.red = red;
    fill_sign_xor(sign_mask, j.qa.sign_xor);
    fill_grid(max_fpx, j.qa);
    j.qa.key0 = (uint32_t)seed;
    j.qa.key1 = (uint32_t)(seed >> 32);
    j.qa.stream = stream_id;
    j.stats = reinterpret_cast<QuantStats*>(stats_dev);
    return status_of(launch_quant_stats(j, static_cast<hipStream_t>(stream)));
}

int ufp4_rht(const void* x_dev, int64_t rows, int64_t cols, int64_t ld, uint32_t sign_mask, float* y_dev, int64_t ldy,
             void* stream) {
    if (sign_mask > 0xFFFFu) return UFP4_ERR_INVALID_ARG;
    if (rows < 0 || cols < 0) return UFP4_ERR_INVALID_ARG;
    if (!x_dev || !y_dev) return UFP4_ERR_INVALID_ARG;
    if (cols % 16 != 0 || ld < cols || ld % 8 != 0 || ldy < cols || ldy % 4 != 0) return UFP4_ERR_SHAPE;
    if (!aligned(x_dev, 16) || !aligned(y_dev, 16)) return UFP4_ERR_ALIGN;
    if (cols / 16 / 256 >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    if (rows == 0 || cols == 0) return UFP4_OK;
    RhtJob j{};
    j.x = x_dev;
    j.rows = rows;
    j.cols = cols;
    j.ld = ld;
    fill_sign_xor(sign_mask, j.qa.sign_xor);
    fill_grid(0.0f, j.qa);
    j.y = y_dev;
    j.ldy = ldy;
    return status_of(launch_rht(j, static_cast<hipStream_t>(stream)));
}

int ufp4_quantize_f32(int format, const float* x_dev, int64_t rows, int64_t cols, int64_t ld, int rounding,
                      uint64_t seed, uint32_t stream_id, void* codes_dev, int64_t code_panel_ld, float* scales_dev,
                      int64_t scale_panel_ld, void* stream) {
    if (format != UFP4_FMT_UNIFORM && format != UFP4_FMT_E2M1) return UFP4_ERR_INVALID_ARG;
    if (rounding != UFP4_ROUND_RTNE && rounding != UFP4_ROUND_SR) return UFP4_ERR_INVALID_ARG;
    if (rows < 0 || cols < 0) return UFP4_ERR_INVALID_ARG;
    if (!x_dev || !codes_dev || !scales_dev) return UFP4_ERR_INVALID_ARG;
    if (cols % 16 != 0 || ld < cols || ld % 4 != 0) return UFP4_ERR_SHAPE;
    if (!aligned(x_dev, 16)) return UFP4_ERR_ALIGN;
    const int st = check_panels(codes_dev, code_panel_ld, scales_dev, scale_panel_ld, cols);
    if (st != UFP4_OK) return st;
    if (rows >= (int64_t(1) << 31) || padded_rows(rows) / 32 > 65535) return UFP4_ERR_UNSUPPORTED;
    if (rows == 0 || cols == 0) return UFP4_OK;
    QuantJob j{};
    j.format = format;
    j.rounding = rounding;
    j.rht = 0;
    j.transpose = 0;
    j.input_f32 = 1;
    j.x = x_dev;
    j.xrows = rows;
    j.ld = ld;
    j.qrows = rows;
    j.red = cols;
    j.num_groups = 1;
    fill_sign_xor(0, j.qa.sign_xor);
    fill_grid(0.0f, j.qa);
    j.qa.key0 = (uint32_t)seed;
    j.qa.key1 = (uint32_t)(seed >> 32);
    j.qa.stream = stream_id;
    j.codes = codes_dev;
    j.code_pld = code_panel_ld;
    j.scales = scales_dev;
    j.scale_pld = scale_panel_ld;
    return status_of(launch_quantize(j, static_cast<hipStream_t>(stream)));
}

int ufp4_quantize_grouped_t(int format, const void* x_dev, int64_t rows, int64_t cols, int64_t ld,
                            const int64_t* group_offsets_dev, const int64_t* padded_offsets_dev, int32_t num_groups,
                            int64_t red_total, int rht, uint32_t sign_mask, int rounding, uint64_t seed,
                            uint32_t stream_id, void* codes_dev, int64_t code_panel_ld, float* scales_dev,
                            int64_t scale_panel_ld, void* stream) {
    if (!group_offsets_dev || !padded_offsets_dev) return UFP4_ERR_INVALID_ARG;
    if (num_groups < 1 || num_groups > max_groups_quantize()) return num_groups < 1 ? UFP4_ERR_INVALID_ARG
                                                                                    : UFP4_ERR_UNSUPPORTED;
    if (red_total < rows) return UFP4_ERR_SHAPE;
    const int st = check_quant_common(format, x_dev, rows, cols, ld, rht, sign_mask, rounding, codes_dev, code_panel_ld,
                                      scales_dev, scale_panel_ld, red_total, cols);
    if (st != UFP4_OK) return st;
    if (red_total == 0 || cols == 0) return UFP4_OK;
    QuantJob j{};
    j.format = format;
    j.rounding = rounding;
    j.rht = rht;
    j.transpose = 1;
    j.x = x_dev;
    j.xrows = rows;
    j.ld = ld;
    j.qrows = cols;
    j.red = red_total;
    j.group_off = group_offsets_dev;
    j.group_poff = padded_offsets_dev;
    j.num_groups = num_groups;
    fill_sign_xor(sign_mask, j.qa.sign_xor);
    fill_grid(0.0f, j.qa);
    j.qa.key0 = (uint32_t)seed;
    j.qa.key1 = (uint32_t)(seed >> 32);
    j.qa.stream = stream_id;
    j.codes = codes_dev;
    j.code_pld = code_panel_ld;
    j.scales = scales_dev;
    j.scale_pld = scale_panel_ld;
    return status_of(launch_quantize(j, static_cast<hipStream_t>(stream)));
}

int ufp4_quantize_dual(int format, const void* x_dev, int64_t rows, int64_t cols, int64_t ld, int rht_rows,
                       uint32_t sign_mask_rows, uint32_t stream_rows, int rht_cols, uint32_t sign_mask_cols,
                       uint32_t stream_cols, int rounding, uint64_t seed, void* codes_r_dev, int64_t code_panel_ld_r,
                       float* scales_r_dev, int64_t scale_panel_ld_r, void* codes_c_dev, int64_t code_panel_ld_c,
                       float* scales_c_dev, int64_t scale_panel_ld_c, void* stream) {
    // Q_r = X [rows, cols] along cols; Q_c = X^T [cols, rows] along rows
    int st = check_quant_common(format, x_dev, rows, cols, ld, rht_rows, sign_mask_rows, rounding, codes_r_dev,
                                code_panel_ld_r, scales_r_dev, scale_panel_ld_r, cols, rows);
    if (st == UFP4_OK)
        st = check_quant_common(format, x_dev, rows, cols, ld, rht_cols, sign_mask_cols, rounding, codes_c_dev,
                                code_panel_ld_c, scales_c_dev, scale_panel_ld_c, rows, cols);
    if (st != UFP4_OK) return st;
    if (rows == 0 || cols == 0) return UFP4_OK;
    // grid: x over 64-column tiles of the padded columns, y over 32 groups of 16 rows (grid-stride beyond)
    if (padded_rows(cols) / 64 >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    DualJob j{};
    j.format = format;
    j.rounding = rounding;
    j.rht_r = rht_rows;
    j.rht_c = rht_cols;
    j.x = x_dev;
    j.rows = rows;
    j.cols = cols;
    j.ld = ld;
    fill_sign_xor(sign_mask_rows, j.qr.sign_xor);
    fill_sign_xor(sign_mask_cols, j.qc.sign_xor);
    fill_grid(0.0f, j.qr);
    fill_grid(0.0f, j.qc);
    j.qr.key0 = j.qc.key0 = (uint32_t)seed;
    j.qr.key1 = j.qc.key1 = (uint32_t)(seed >> 32);
    j.qr.stream = stream_rows;
    j.qc.stream = stream_cols;
    j.codes_r = codes_r_dev;
    j.code_pld_r = code_panel_ld_r;
    j.scales_r = scales_r_dev;
    j.scale_pld_r = scale_panel_ld_r;
    j.codes_c = codes_c_dev;
    j.code_pld_c = code_panel_ld_c;
    j.scales_c = scales_c_dev;
    j.scale_pld_c = scale_panel_ld_c;
    return status_of(launch_quantize_dual(j, static_cast<hipStream_t>(stream)));
}

int ufp4_mx_quantize(const void* x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht,
                     uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, void* codes_dev,
                     int64_t code_panel_ld, void* scales_dev, int64_t scale_panel_ld, void* stream) {
    return mx_quantize_impl(x_dev, rows, cols, ld, transpose, rht, sign_mask, rounding, seed, stream_id, codes_dev,
                            code_panel_ld, scales_dev, scale_panel_ld, stream);
}

int ufp4_mx_gemm_fwd_y(const void* x_codes_dev, int64_t x_code_panel_ld, const void* x_scales_dev,
                       int64_t x_scale_panel_ld, const void* w_codes_dev, int64_t w_code_panel_ld,
                       const void* w_scales_dev, int64_t w_scale_panel_ld, int64_t M, int64_t N, int64_t K, void* y_dev,
                       int64_t ldc, int out_dtype, void* stream) {
    return mx_gemm_impl(x_codes_dev, x_code_panel_ld, x_scales_dev, x_scale_panel_ld, w_codes_dev, w_code_panel_ld,
                        w_scales_dev, w_scale_panel_ld, M, N, K, y_dev, ldc, out_dtype, stream);
}

int ufp4_mx_gemm_bwd_dx(const void* dy_codes_dev, int64_t dy_code_panel_ld, const void* dy_scales_dev,
                        int64_t dy_scale_panel_ld, const void* wt_codes_dev, int64_t wt_code_panel_ld,
                        const void* wt_scales_dev, int64_t wt_scale_panel_ld, int64_t M, int64_t N, int64_t K,
                        void* dx_dev, int64_t ldc, int out_dtype, void* stream) {
    // dX [M, K] = dY [M, N] . (W^T [K, N])^T
    return mx_gemm_impl(dy_codes_dev, dy_code_panel_ld, dy_scales_dev, dy_scale_panel_ld, wt_codes_dev, wt_code_panel_ld,
                        wt_scales_dev, wt_scale_panel_ld, M, K, N, dx_dev, ldc, out_dtype, stream);
}

int ufp4_mx_gemm_bwd_dw(const void* dyt_codes_dev, int64_t dyt_code_panel_ld, const void* dyt_scales_dev,
                        int64_t dyt_scale_panel_ld, const void* xt_codes_dev, int64_t xt_code_panel_ld,
                        const void* xt_scales_dev, int64_t xt_scale_panel_ld, int64_t M, int64_t N, int64_t K,
                        void* dw_dev, int64_t ldc, int out_dtype, void* stream) {
    // dW [N, K] = dY^T [N, M] . (X^T [K, M])^T
    return mx_gemm_impl(dyt_codes_dev, dyt_code_panel_ld, dyt_scales_dev, dyt_scale_panel_ld, xt_codes_dev,
                        xt_code_panel_ld, xt_scales_dev, xt_scale_panel_ld, N, K, M, dw_dev, ldc, out_dtype, stream);
}

int ufp4_gemm_fwd_y(const void* x_codes_dev, int64_t x_code_panel_ld, const float* x_scales_dev, int64_t x_scale_panel_ld,
                    const void* w_codes_dev, int64_t w_code_panel_ld, const float* w_scales_dev, int64_t w_scale_panel_ld,
                    int64_t M, int64_t N, int64_t K, int format, void* y_dev, int64_t ldc, int out_dtype,
                    void* stream) {
    return gemm_dense(x_codes_dev, x_code_panel_ld, x_scales_dev, x_scale_panel_ld, w_codes_dev, w_code_panel_ld, w_scales_dev,
                      w_scale_panel_ld, M, N, K, format, y_dev, ldc, out_dtype, stream);
}

int ufp4_gemm_bwd_dx(const void* dy_codes_dev, int64_t dy_code_panel_ld, const float* dy_scales_dev, int64_t dy_scale_panel_ld,
                     const void* wt_codes_dev, int64_t wt_code_panel_ld, const float* wt_scales_dev, int64_t wt_scale_panel_ld,
                     int64_t M, int64_t N, int64_t K, int format, void* dx_dev, int64_t ldc, int out_dtype,
                     void* stream) {
    // dX [M, K] = dY [M, N] . (W^T [K, N])^T
    return gemm_dense(dy_codes_dev, dy_code_panel_ld, dy_scales_dev, dy_scale_panel_ld, wt_codes_dev, wt_code_panel_ld, wt_scales_dev,
                      wt_scale_panel_ld, M, K, N, format, dx_dev, ldc, out_dtype, stream);
}

int ufp4_gemm_bwd_dw(const void* dyt_codes_dev, int64_t dyt_code_panel_ld, const float* dyt_scales_dev,
                     int64_t dyt_scale_panel_ld, const void* xt_codes_dev, int64_t xt_code_panel_ld, const float* xt_scales_dev,
                     int64_t xt_scale_panel_ld, int64_t M, int64_t N, int64_t K, int format, void* dw_dev, int64_t ldc,
                     int out_dtype, void* stream) {
    // dW [N, K] = dY^T [N, M] . (X^T [K, M])^T
    return gemm_dense(dyt_codes_dev, dyt_code_panel_ld, dyt_scales_dev, dyt_scale_panel_ld, xt_codes_dev, xt_code_panel_ld,
                      xt_scales_dev, xt_scale_panel_ld, N, K, M, format, dw_dev, ldc, out_dtype, stream);
}

int ufp4_gemm_fwd_y_grouped(const void* x_codes_dev, int64_t x_code_panel_ld, const float* x_scales_dev, int64_t x_scale_panel_ld,
                            const void* w_codes_dev, int64_t w_code_panel_ld, const float* w_scales_dev, int64_t w_scale_panel_ld,
                            const int64_t* group_offsets_dev, int32_t num_groups, int64_t M_total, int64_t N, int64_t K,
                            int format, void* y_dev, int64_t ldc, int out_dtype, void* stream) {
    if (!group_offsets_dev || num_groups < 1) return UFP4_ERR_INVALID_ARG;
    const int st = check_gemm(x_codes_dev, x_code_panel_ld, x_scales_dev, x_scale_panel_ld, w_codes_dev, w_code_panel_ld, w_scales_dev,
                              w_scale_panel_ld, M_total, N * num_groups, K, K, format, y_dev, ldc, N, out_dtype);
    if (st != UFP4_OK) return st;
    if (M_total == 0 || N == 0) return UFP4_OK;
    GemmJob j = make_job(kGemmRaggedM, x_codes_dev, x_code_panel_ld, x_scales_dev, x_scale_panel_ld, w_codes_dev, w_code_panel_ld,
                         w_scales_dev, w_scale_panel_ld, M_total, N, K / 16, format, y_dev, ldc, out_dtype);
    j.offsets = group_offsets_dev;
    j.G = num_groups;
    j.b_group_rows = N;
    j.b_group_kb = 0;
    return status_of(launch_gemm(j, static_cast<hipStream_t>(stream)));
}

int ufp4_gemm_bwd_dx_grouped(const void* dy_codes_dev, int64_t dy_code_panel_ld, const float* dy_scales_dev,
                             int64_t dy_scale_panel_ld, const void* wt_codes_dev, int64_t wt_code_panel_ld,
                             const float* wt_scales_dev, int64_t wt_scale_panel_ld, const int64_t* group_offsets_dev,
                             int32_t num_groups, int64_t M_total, int64_t N, int64_t K, int format, void* dx_dev,
                             int64_t ldc, int out_dtype, void* stream) {
    if (!group_offsets_dev || num_groups < 1) return UFP4_ERR_INVALID_ARG;
    // A = dY [M_total, N]; B = W^T [K, G*N], group g uses reduction columns [g*N, (g+1)*N)
    const int st = check_gemm(dy_codes_dev, dy_code_panel_ld, dy_scales_dev, dy_scale_panel_ld, wt_codes_dev, wt_code_panel_ld,
                              wt_scales_dev, wt_scale_panel_ld, M_total, K, N, N * num_groups, format, dx_dev, ldc, K,
                              out_dtype);
    if (st != UFP4_OK) return st;
    if (M_total == 0 || K == 0) return UFP4_OK;
    GemmJob j = make_job(kGemmRaggedM, dy_codes_dev, dy_code_panel_ld, dy_scales_dev, dy_scale_panel_ld, wt_codes_dev, wt_code_panel_ld,
                         wt_scales_dev, wt_scale_panel_ld, M_total, K, N / 16, format, dx_dev, ldc, out_dtype);
    j.offsets = group_offsets_dev;
    j.G = num_groups;
    j.b_group_rows = 0;
    j.b_group_kb = N / 16;
    return status_of(launch_gemm(j, static_cast<hipStream_t>(stream)));
}

int ufp4_gemm_bwd_dw_grouped(const void* dyt_codes_dev, int64_t dyt_code_panel_ld, const float* dyt_scales_dev,
                             int64_t dyt_scale_panel_ld, const void* xt_codes_dev, int64_t xt_code_panel_ld,
                             const float* xt_scales_dev, int64_t xt_scale_panel_ld, const int64_t* padded_offsets_dev,
                             int32_t num_groups, int64_t red_total, int64_t N, int64_t K, int format, void* dw_dev,
                             int64_t ldc, int out_dtype, void* stream) {
    if (!padded_offsets_dev || num_groups < 1) return UFP4_ERR_INVALID_ARG;
    if (num_groups > 65535) return UFP4_ERR_UNSUPPORTED;
    // A = dY^T [N, red_total], B = X^T [K, red_total]; group g reduces over [pad_g, pad_{g+1}) of that axis
    const int st = check_gemm(dyt_codes_dev, dyt_code_panel_ld, dyt_scales_dev, dyt_scale_panel_ld, xt_codes_dev, xt_code_panel_ld,
                              xt_scales_dev, xt_scale_panel_ld, N, K, red_total, red_total, format, dw_dev, ldc, K,
                              out_dtype);
    if (st != UFP4_OK) return st;
    if (N == 0 || K == 0) return UFP4_OK;
    GemmJob j = make_job(kGemmRaggedK, dyt_codes_dev, dyt_code_panel_ld, dyt_scales_dev, dyt_scale_panel_ld, xt_codes_dev,
                         xt_code_panel_ld, xt_scales_dev, xt_scale_panel_ld, N, K, 0, format, dw_dev, ldc, out_dtype);
    j.offsets = padded_offsets_dev;
    j.G = num_groups;
    j.red_total = red_total;
    return status_of(launch_gemm(j, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
