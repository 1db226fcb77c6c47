// C ABI of libufp4: argument validation on the host, then one kernel launch on the caller's stream; plus the
// host-side arithmetic of the layout (ufp4_qtensor_bytes, ufp4_grouped_reduction) and of the Sec. 3.2 metrics.
// Declarations and the meaning of every argument are in include/ufp4.h.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "../../include/ufp4.h"
#include "ufp4_internal.h"

using namespace ufp4;

static_assert(sizeof(ufp4_quant_stats_t) == sizeof(QuantStats), "statistics record layout");
static_assert(sizeof(ufp4_qtensor) == 96, "descriptor layout (mirrored by the Python binding)");

namespace {

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

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

// Storage of `q` for a [rows, red] operand of `format`: pointers, panel strides, panel count.
int check_storage(const ufp4_qtensor* q, int format, int64_t rows, int64_t red) {
    if (!q) return UFP4_ERR_INVALID_ARG;
    if (!q->codes || !q->scales || q->panels < 0 || rows < 0 || red < 0) return UFP4_ERR_INVALID_ARG;
    const bool mx = format == UFP4_FMT_UNIFORM_MX32;
    const int64_t blk = mx ? 32 : 16;
    if (red % blk != 0) return UFP4_ERR_SHAPE;
    const int64_t nkb = red / blk;
    const int64_t cb = mx ? kMxPanelBlockBytes : kPanelBlockBytes;
    const int64_t sb = mx ? kMxPanelBlockScales : kPanelBlockScales;
    if (q->code_panel_ld < nkb * cb || q->scale_panel_ld < nkb * sb) return UFP4_ERR_SHAPE;
    if (q->panels < ceil_div(rows, kPanelRows)) return UFP4_ERR_SHAPE;
    if (q->code_panel_ld % 16 != 0 || q->scale_panel_ld % (mx ? 16 : 4) != 0) return UFP4_ERR_ALIGN;
    if (!aligned(q->codes, 16) || !aligned(q->scales, 16)) return UFP4_ERR_ALIGN;
    if (q->code_panel_ld > kMaxCodePanelLd || q->scale_panel_ld > (mx ? kMaxCodePanelLd : kMaxScalePanelLd))
        return UFP4_ERR_UNSUPPORTED;
    return UFP4_OK;
}

// What a quantizer wrote into `q`.
void record(ufp4_qtensor* q, int format, int64_t rows, int64_t red, int rht_block, const uint16_t* words,
            float max_fpx, int rounding, int layout = UFP4_LAYOUT_PLAIN) {
    q->rows = rows;
    q->red = red;
    q->format = format;
    q->rht_block = rht_block;
    for (int k = 0; k < 8; ++k) q->sign_words[k] = (words && k < rht_block / 16) ? words[k] : 0;
    q->max_fpx = max_fpx == 6.0f ? 0.0f : max_fpx;
    q->rounding = rounding;
    q->layout = layout;
    q->reserved = 0;
}

// An input tensor [rows, cols] with leading dimension ld (elements, a multiple of ld_mult) at x. An empty tensor
// (rows or cols 0) is read by nobody: it may have no storage and any leading dimension.
int check_input(const void* x, int64_t rows, int64_t cols, int64_t ld, int64_t ld_mult) {
    if (rows < 0 || cols < 0) return UFP4_ERR_INVALID_ARG;
    if (rows == 0 || cols == 0) return UFP4_OK;
    if (!x) return UFP4_ERR_INVALID_ARG;
    if (ld < cols || ld % ld_mult != 0) return UFP4_ERR_SHAPE;
    if (!aligned(x, 16)) return UFP4_ERR_ALIGN;
    return UFP4_OK;
}

// Checks shared by the bf16-input quantizers: the input tensor and the operand's storage.
int check_quant_common(int format, const void* x, int64_t rows, int64_t cols, int64_t ld, int rht, uint32_t sign_mask,
                       int rounding, const ufp4_qtensor* out, int64_t qrows, int64_t red) {
    if (format != UFP4_FMT_UNIFORM && format != UFP4_FMT_E2M1) return UFP4_ERR_INVALID_ARG;
    if (rounding != UFP4_ROUND_RTNE && rounding != UFP4_ROUND_SR) return UFP4_ERR_INVALID_ARG;
    if (rht != 0 && rht != 1) return UFP4_ERR_INVALID_ARG;
    if (sign_mask > 0xFFFFu) return UFP4_ERR_INVALID_ARG;
    if (rows < 0 || cols < 0 || red < 0 || qrows < 0) return UFP4_ERR_INVALID_ARG;
    const int si = check_input(x, rows, cols, ld, 8);
    if (si != UFP4_OK) return si;
    const int st = check_storage(out, format, qrows, red);
    if (st != UFP4_OK) return st;
    if (qrows >= (int64_t(1) << 31) || red / 16 >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    return UFP4_OK;
}

void fill_out(QuantJob& j, const ufp4_qtensor* out) {
    j.codes = out->codes;
    j.code_pld = out->code_panel_ld;
    j.scales = static_cast<float*>(out->scales);
    j.scale_pld = out->scale_panel_ld;
}

// rht_block 16 (with sign_mask) or 32 / 64 / 128 (with the n/16 words of `sign_words`).
int quantize_impl(int format, const void* x, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht,
                  uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, ufp4_qtensor* out, void* stream,
                  float max_fpx = 0.0f, int rht_block = 16, const uint16_t* sign_words = nullptr) {
    if (transpose != 0 && transpose != 1) return UFP4_ERR_INVALID_ARG;
    if (!valid_max_fpx(format, max_fpx)) return UFP4_ERR_INVALID_ARG;
    const int64_t red = transpose ? rows : cols;
    const int64_t qrows = transpose ? cols : rows;
    const int st = check_quant_common(format, x, rows, cols, ld, rht, sign_mask, rounding, out, qrows, red);
    if (st != UFP4_OK) return st;
    // rowwise: one workgroup per 32 padded rows along the grid's y dimension
    if (!transpose && padded_rows(qrows) / 32 > 65535) return UFP4_ERR_UNSUPPORTED;
    if (rht_block != 16 && red % rht_block != 0) return UFP4_ERR_SHAPE;
    const uint16_t mask16 = (uint16_t)sign_mask;
    record(out, format, qrows, red, rht ? rht_block : 0, rht_block == 16 ? &mask16 : sign_words, max_fpx, rounding);
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
    j.num_groups = 1;
    fill_sign_xor(sign_mask, j.qa.sign_xor);
    fill_grid(max_fpx, j.qa);
    j.qa.rht_m = rht_block / 16;
    j.qa.rht_c = sqrt(1.0 / rht_block);  // correctly rounded square root of an exact power of two
    for (int k = 0; k < rht_block / 16 && sign_words; ++k) j.qa.sign_words[k] = sign_words[k];
    j.qa.key0 = (uint32_t)seed;
    j.qa.key1 = (uint32_t)(seed >> 32);
    j.qa.stream = stream_id;
    fill_out(j, out);
    return status_of(launch_quantize(j, static_cast<hipStream_t>(stream)));
}

// The two operands of a GEMM: known formats (the power-of-two-scale one for `mx`, the others otherwise), the
// same format, RHT block and signs (Sec. 2.2: one H' for both), and storage that holds what they claim.
int check_operands(const ufp4_qtensor* a, const ufp4_qtensor* b, bool mx) {
    if (!a || !b) return UFP4_ERR_INVALID_ARG;
    for (const ufp4_qtensor* q : {a, b}) {
        if (q->format != UFP4_FMT_UNIFORM && q->format != UFP4_FMT_E2M1 && q->format != UFP4_FMT_UNIFORM_MX32)
            return UFP4_ERR_INVALID_ARG;
        if (q->rht_block != 0 && q->rht_block != 16 && q->rht_block != 32 && q->rht_block != 64 && q->rht_block != 128)
            return UFP4_ERR_INVALID_ARG;
        if ((q->format == UFP4_FMT_UNIFORM_MX32) != mx) return UFP4_ERR_MISMATCH;
    }
    if (a->format != b->format || a->rht_block != b->rht_block) return UFP4_ERR_MISMATCH;
    for (int k = 0; k < a->rht_block / 16; ++k)
        if (a->sign_words[k] != b->sign_words[k]) return UFP4_ERR_MISMATCH;
    int st = check_storage(a, a->format, a->rows, a->red);
    if (st == UFP4_OK) st = check_storage(b, b->format, b->rows, b->red);
    if (st != UFP4_OK) return st;
    if (a->rows >= (int64_t(1) << 31) || b->rows >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    return UFP4_OK;
}

// The output (c_cols columns per row, leading dimension ldc); an empty output may have no storage.
int check_output(const void* c, int64_t ldc, int64_t c_cols, int out_dtype, bool empty) {
    if (out_dtype != UFP4_OUT_F32 && out_dtype != UFP4_OUT_BF16) return UFP4_ERR_INVALID_ARG;
    if (empty) return UFP4_OK;
    if (!c) return UFP4_ERR_INVALID_ARG;
    if (ldc < c_cols) return UFP4_ERR_SHAPE;
    if (!aligned(c, out_dtype == UFP4_OUT_F32 ? 4 : 2)) return UFP4_ERR_ALIGN;
    return UFP4_OK;
}

GemmJob make_job(int mode, const ufp4_qtensor* a, const ufp4_qtensor* b, int64_t M, int64_t N, int64_t nkb, void* c,
                 int64_t ldc, int out_dtype) {
    GemmJob j{};
    j.format = a->format;
    j.out_dtype = out_dtype;
    j.mode = mode;
    j.a = static_cast<const uint8_t*>(a->codes);
    j.a_pld = a->code_panel_ld;
    j.as = static_cast<const float*>(a->scales);
    j.as_pld = a->scale_panel_ld;
    j.b = static_cast<const uint8_t*>(b->codes);
    j.b_pld = b->code_panel_ld;
    j.bs = static_cast<const float*>(b->scales);
    j.bs_pld = b->scale_panel_ld;
    j.M = M;
    j.N = N;
    j.nkb = nkb;
    j.c = c;
    j.ldc = ldc;
    j.offsets = nullptr;
    j.G = 1;
    return j;
}

// A [M, red] . B [N, red]^T for the three dense passes.
int gemm_dense(const ufp4_qtensor* a, const ufp4_qtensor* b, void* c, int64_t ldc, int out_dtype, void* stream) {
    int st = check_operands(a, b, false);
    if (st != UFP4_OK) return st;
    if (a->red != b->red) return UFP4_ERR_MISMATCH;
    st = check_output(c, ldc, b->rows, out_dtype, a->rows == 0 || b->rows == 0);
    if (st != UFP4_OK) return st;
    if (a->rows == 0 || b->rows == 0) return UFP4_OK;
    const GemmJob j = make_job(kGemmDense, a, b, a->rows, b->rows, a->red / 16, c, ldc, out_dtype);
    return status_of(launch_gemm(j, static_cast<hipStream_t>(stream)));
}

int mx_gemm_impl(const ufp4_qtensor* a, const ufp4_qtensor* b, void* c, int64_t ldc, int out_dtype, void* stream) {
    int st = check_operands(a, b, true);
    if (st != UFP4_OK) return st;
    if (a->red != b->red) return UFP4_ERR_MISMATCH;
    st = check_output(c, ldc, b->rows, out_dtype, a->rows == 0 || b->rows == 0);
    if (st != UFP4_OK) return st;
    // one workgroup per 256 x 256 output tile on a one-dimensional grid (the count of 128 x 128 tiles bounds it)
    if (ceil_div(a->rows, 128) * ceil_div(b->rows, 128) >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    if (a->rows == 0 || b->rows == 0) return UFP4_OK;
    MxGemmJob j{};
    j.out_dtype = out_dtype;
    j.a = static_cast<const uint8_t*>(a->codes);
    j.a_pld = a->code_panel_ld;
    j.as = static_cast<const uint8_t*>(a->scales);
    j.as_pld = a->scale_panel_ld;
    j.b = static_cast<const uint8_t*>(b->codes);
    j.b_pld = b->code_panel_ld;
    j.bs = static_cast<const uint8_t*>(b->scales);
    j.bs_pld = b->scale_panel_ld;
    j.M = a->rows;
    j.N = b->rows;
    j.nkb = a->red / 32;
    j.a_rows = a->rows;
    j.b_rows = b->rows;
    j.c = c;
    j.ldc = ldc;
    j.mode = kGemmDense;
    return status_of(launch_gemm_mx(j, static_cast<hipStream_t>(stream)));
}

MxGemmJob mx_job(const ufp4_qtensor* a, const ufp4_qtensor* b, void* c, int64_t ldc, int out_dtype) {
    MxGemmJob j{};
    j.out_dtype = out_dtype;
    j.a = static_cast<const uint8_t*>(a->codes);
    j.a_pld = a->code_panel_ld;
    j.as = static_cast<const uint8_t*>(a->scales);
    j.as_pld = a->scale_panel_ld;
    j.b = static_cast<const uint8_t*>(b->codes);
    j.b_pld = b->code_panel_ld;
    j.bs = static_cast<const uint8_t*>(b->scales);
    j.bs_pld = b->scale_panel_ld;
    j.a_rows = a->rows;
    j.b_rows = b->rows;
    j.c = c;
    j.ldc = ldc;
    return j;
}

int grid_levels(int format, float max_fpx) {
    if (format == UFP4_FMT_E2M1 && max_fpx == 2.0f) return 5;
    if (format == UFP4_FMT_E2M1 && max_fpx == 4.0f) return 7;
    return 8;
}

}  // namespace

extern "C" {

const char* ufp4_status_string(int status) {
    switch (status) {
        case UFP4_OK: return "ok";
        case UFP4_ERR_INVALID_ARG: return "invalid argument";
        case UFP4_ERR_SHAPE: return "bad shape, leading dimension or buffer size";
        case UFP4_ERR_ALIGN: return "misaligned pointer or leading dimension";
        case UFP4_ERR_MISMATCH: return "operands quantized differently (grid, RHT block, signs or reduction length)";
        case UFP4_ERR_UNSUPPORTED: return "unsupported";
        case UFP4_ERR_HIP: return "HIP launch error";
        default: return "unknown status";
    }
}

const char* ufp4_version(void) { return "0.3.0"; }

int ufp4_qtensor_bytes(int format, int64_t rows, int64_t red, int64_t* panels, int64_t* code_panel_ld,
                       int64_t* scale_panel_ld, size_t* codes_bytes, size_t* scales_bytes) {
    if (format != UFP4_FMT_UNIFORM && format != UFP4_FMT_E2M1 && format != UFP4_FMT_UNIFORM_MX32)
        return UFP4_ERR_INVALID_ARG;
    if (rows < 0 || red < 0) return UFP4_ERR_INVALID_ARG;
    const bool mx = format == UFP4_FMT_UNIFORM_MX32;
    const int64_t blk = mx ? 32 : 16;
    if (red % blk != 0) return UFP4_ERR_SHAPE;
    const int64_t nkb = red / blk;
    const int64_t p = rows > 0 ? ceil_div(rows, kPanelRows) : 1;
    // a zero-length reduction still gets 16 aligned bytes per panel
    const int64_t cld = nkb > 0 ? nkb * (mx ? kMxPanelBlockBytes : kPanelBlockBytes) : 16;
    const int64_t sld = nkb > 0 ? nkb * (mx ? kMxPanelBlockScales : kPanelBlockScales) : (mx ? 16 : 4);
    if (panels) *panels = p;
    if (code_panel_ld) *code_panel_ld = cld;
    if (scale_panel_ld) *scale_panel_ld = sld;
    if (codes_bytes) *codes_bytes = (size_t)(p * cld);
    if (scales_bytes) *scales_bytes = (size_t)(p * sld * (mx ? 1 : 4));
    return UFP4_OK;
}

int ufp4_grouped_reduction(const int64_t* group_offsets_host, int32_t num_groups, int32_t block,
                           int64_t* padded_offsets_host, int64_t* total) {
    if (!group_offsets_host || num_groups < 1) return UFP4_ERR_INVALID_ARG;
    if (block != 16 && block != 32 && block != 128) return UFP4_ERR_INVALID_ARG;
    if (group_offsets_host[0] != 0) return UFP4_ERR_INVALID_ARG;
    int64_t pad = 0;
    if (padded_offsets_host) padded_offsets_host[0] = 0;
    for (int32_t g = 0; g < num_groups; ++g) {
        const int64_t cnt = group_offsets_host[g + 1] - group_offsets_host[g];
        if (cnt < 0) return UFP4_ERR_INVALID_ARG;
        pad += ceil_div(cnt, block) * block;  // the group's tokens zero-padded to a multiple of the block
        if (padded_offsets_host) padded_offsets_host[g + 1] = pad;
    }
    if (total) *total = pad;
    return UFP4_OK;
}

int ufp4_rht_quantize(const void* x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht,
                      uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, ufp4_qtensor* out,
                      void* stream) {
    return quantize_impl(UFP4_FMT_UNIFORM, x_dev, rows, cols, ld, transpose, rht, sign_mask, rounding, seed, stream_id,
                         out, stream);
}

int ufp4_e2m1_quantize(const void* x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht,
                       uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, ufp4_qtensor* out,
                       void* stream) {
    return quantize_impl(UFP4_FMT_E2M1, x_dev, rows, cols, ld, transpose, rht, sign_mask, rounding, seed, stream_id,
                         out, stream);
}

int ufp4_e2m1_quantize_range(const void* x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht,
                             uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, float max_fpx,
                             ufp4_qtensor* out, void* stream) {
    if (max_fpx == 0.0f) return UFP4_ERR_INVALID_ARG;  // the full grid is ufp4_e2m1_quantize
    return quantize_impl(UFP4_FMT_E2M1, x_dev, rows, cols, ld, transpose, rht, sign_mask, rounding, seed, stream_id,
                         out, stream, max_fpx);
}

int ufp4_quantize_rht_block(int format, const void* x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose,
                            int rht_block, const uint16_t* sign_words_host, int rounding, uint64_t seed,
                            uint32_t stream_id, ufp4_qtensor* out, void* stream) {
    if (rht_block != 16 && rht_block != 32 && rht_block != 64 && rht_block != 128) return UFP4_ERR_INVALID_ARG;
    if (!sign_words_host) return UFP4_ERR_INVALID_ARG;
    if (format != UFP4_FMT_UNIFORM && format != UFP4_FMT_E2M1) return UFP4_ERR_INVALID_ARG;
    if (rht_block == 16)
        return quantize_impl(format, x_dev, rows, cols, ld, transpose, 1, sign_words_host[0], rounding, seed, stream_id,
                             out, stream);
    return quantize_impl(format, x_dev, rows, cols, ld, transpose, 1, 0, rounding, seed, stream_id, out, stream, 0.0f,
                         rht_block, sign_words_host);
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
    if (!stats_dev) return UFP4_ERR_INVALID_ARG;
    const int si = check_input(x_dev, rows, cols, ld, 8);
    if (si != UFP4_OK) return si;
    const bool empty = rows == 0 || cols == 0;
    const int64_t red = transpose ? rows : cols;
    const int64_t qrows = transpose ? cols : rows;
    if (red % 16 != 0) return UFP4_ERR_SHAPE;
    if (!aligned(stats_dev, 8)) return UFP4_ERR_ALIGN;
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

int ufp4_quant_metrics(const ufp4_quant_stats_t* s, int format, float max_fpx, ufp4_quant_metrics_t* m) {
    if (!s || !m) return UFP4_ERR_INVALID_ARG;
    if (format != UFP4_FMT_UNIFORM && format != UFP4_FMT_E2M1) return UFP4_ERR_INVALID_ARG;
    if (!valid_max_fpx(format, max_fpx)) return UFP4_ERR_INVALID_ARG;
    m->nmse = s->ref2 > 0.0 ? s->err2 / s->ref2 : NAN;
    m->sqnr_db = s->err2 > 0.0 ? -10.0 * log10(m->nmse) : INFINITY;
    m->alpha = s->ref2 > 0.0 ? s->cross / s->ref2 : NAN;
    const int k = grid_levels(format, max_fpx);
    double n = 0.0;
    for (int i = 0; i < k; ++i) n += (double)s->hist[i];
    double ent = 0.0;
    for (int i = 0; i < k && n > 0.0; ++i) {
        const double p = (double)s->hist[i] / n;
        ent -= p * log(p + 1e-12);
    }
    m->entropy = ent;
    m->beff = exp(ent) / k;
    return UFP4_OK;
}

int ufp4_rotation_gain(const ufp4_quant_metrics_t* raw, const ufp4_quant_metrics_t* rotated, double* delta_sqnr_db) {
    if (!raw || !rotated) return UFP4_ERR_INVALID_ARG;
    if (delta_sqnr_db) *delta_sqnr_db = 10.0 * log10(raw->nmse / rotated->nmse);
    return UFP4_OK;
}

int ufp4_gemm_attenuation(const ufp4_quant_metrics_t* a, const ufp4_quant_metrics_t* b, double* eta) {
    if (!a || !b) return UFP4_ERR_INVALID_ARG;
    if (eta) *eta = a->alpha * b->alpha;
    return UFP4_OK;
}

int ufp4_rht(const void* x_dev, int64_t rows, int64_t cols, int64_t ld, uint32_t sign_mask, float* y_dev, int64_t ldy,
             void* stream) {
    if (sign_mask > 0xFFFFu) return UFP4_ERR_INVALID_ARG;
    if (rows < 0 || cols < 0) return UFP4_ERR_INVALID_ARG;
    if (cols % 16 != 0) return UFP4_ERR_SHAPE;
    int si = check_input(x_dev, rows, cols, ld, 8);
    if (si == UFP4_OK) si = check_input(y_dev, rows, cols, ldy, 4);  // the output, checked like an input
    if (si != UFP4_OK) return si;
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

int ufp4_quantize_f32(int format, const float* x_dev, int64_t rows, int64_t cols, int64_t ld, int rht,
                      uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, ufp4_qtensor* out,
                      void* stream) {
    if (format != UFP4_FMT_UNIFORM && format != UFP4_FMT_E2M1) return UFP4_ERR_INVALID_ARG;
    if (rounding != UFP4_ROUND_RTNE && rounding != UFP4_ROUND_SR) return UFP4_ERR_INVALID_ARG;
    if (rht != 0 && rht != 1) return UFP4_ERR_INVALID_ARG;
    if (sign_mask > 0xFFFFu) return UFP4_ERR_INVALID_ARG;
    if (rows < 0 || cols < 0) return UFP4_ERR_INVALID_ARG;
    if (cols % 16 != 0) return UFP4_ERR_SHAPE;
    const int si = check_input(x_dev, rows, cols, ld, 4);
    if (si != UFP4_OK) return si;
    const int st = check_storage(out, format, rows, cols);
    if (st != UFP4_OK) return st;
    if (rows >= (int64_t(1) << 31) || padded_rows(rows) / 32 > 65535) return UFP4_ERR_UNSUPPORTED;
    const uint16_t mask16 = (uint16_t)sign_mask;
    record(out, format, rows, cols, rht ? 16 : 0, &mask16, 0.0f, rounding);
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
    fill_out(j, out);
    return status_of(launch_quantize(j, static_cast<hipStream_t>(stream)));
}

int ufp4_quantize_grouped_t(int format, const void* x_dev, int64_t rows, int64_t cols, int64_t ld,
                            const int64_t* group_offsets_dev, int32_t num_groups, int64_t red_total, int rht,
                            uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, ufp4_qtensor* out,
                            void* stream) {
    if (!group_offsets_dev) return UFP4_ERR_INVALID_ARG;
    if (num_groups < 1 || num_groups > max_groups_quantize()) return num_groups < 1 ? UFP4_ERR_INVALID_ARG
                                                                                    : UFP4_ERR_UNSUPPORTED;
    if (red_total < rows) return UFP4_ERR_SHAPE;
    const int st = check_quant_common(format, x_dev, rows, cols, ld, rht, sign_mask, rounding, out, cols, red_total);
    if (st != UFP4_OK) return st;
    const uint16_t mask16 = (uint16_t)sign_mask;
    record(out, format, cols, red_total, rht ? 16 : 0, &mask16, 0.0f, rounding, UFP4_LAYOUT_GROUPED_RED);
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
    j.num_groups = num_groups;
    fill_sign_xor(sign_mask, j.qa.sign_xor);
    fill_grid(0.0f, j.qa);
    j.qa.key0 = (uint32_t)seed;
    j.qa.key1 = (uint32_t)(seed >> 32);
    j.qa.stream = stream_id;
    fill_out(j, out);
    return status_of(launch_quantize(j, static_cast<hipStream_t>(stream)));
}

int ufp4_quantize_dual(int format, const void* x_dev, int64_t rows, int64_t cols, int64_t ld, int rht_rows,
                       uint32_t sign_mask_rows, uint32_t stream_rows, int rht_cols, uint32_t sign_mask_cols,
                       uint32_t stream_cols, int rounding, uint64_t seed, ufp4_qtensor* out_rows,
                       ufp4_qtensor* out_cols, void* stream) {
    // Q_r = X [rows, cols] along cols; Q_c = X^T [cols, rows] along rows
    int st = check_quant_common(format, x_dev, rows, cols, ld, rht_rows, sign_mask_rows, rounding, out_rows, rows,
                                cols);
    if (st == UFP4_OK)
        st = check_quant_common(format, x_dev, rows, cols, ld, rht_cols, sign_mask_cols, rounding, out_cols, cols,
                                rows);
    if (st != UFP4_OK) return st;
    if (out_rows == out_cols) return UFP4_ERR_INVALID_ARG;
    // grid: x over 64-column tiles of the padded columns, y over 32 groups of 16 rows (grid-stride beyond)
    if (padded_rows(cols) / 64 >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    const uint16_t mr = (uint16_t)sign_mask_rows, mc = (uint16_t)sign_mask_cols;
    record(out_rows, format, rows, cols, rht_rows ? 16 : 0, &mr, 0.0f, rounding);
    record(out_cols, format, cols, rows, rht_cols ? 16 : 0, &mc, 0.0f, rounding);
    if (rows == 0 || cols == 0) return UFP4_OK;
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
    j.codes_r = out_rows->codes;
    j.code_pld_r = out_rows->code_panel_ld;
    j.scales_r = static_cast<float*>(out_rows->scales);
    j.scale_pld_r = out_rows->scale_panel_ld;
    j.codes_c = out_cols->codes;
    j.code_pld_c = out_cols->code_panel_ld;
    j.scales_c = static_cast<float*>(out_cols->scales);
    j.scale_pld_c = out_cols->scale_panel_ld;
    return status_of(launch_quantize_dual(j, static_cast<hipStream_t>(stream)));
}

int ufp4_mx_quantize(const void* x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose, int rht,
                     uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, ufp4_qtensor* out,
                     void* stream) {
    if (transpose != 0 && transpose != 1) return UFP4_ERR_INVALID_ARG;
    if (rounding != UFP4_ROUND_RTNE && rounding != UFP4_ROUND_SR) return UFP4_ERR_INVALID_ARG;
    if (rht != 0 && rht != 1) return UFP4_ERR_INVALID_ARG;
    if (sign_mask > 0xFFFFu) return UFP4_ERR_INVALID_ARG;
    const int si = check_input(x_dev, rows, cols, ld, 8);
    if (si != UFP4_OK) return si;
    const int64_t red = transpose ? rows : cols;
    const int64_t qrows = transpose ? cols : rows;
    const int st = check_storage(out, UFP4_FMT_UNIFORM_MX32, qrows, red);
    if (st != UFP4_OK) return st;
    if (qrows >= (int64_t(1) << 31) || red / 16 >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    if (!transpose && padded_rows(qrows) / 64 > 65535) return UFP4_ERR_UNSUPPORTED;
    if (mx_tile_count(rows, cols, !transpose, transpose != 0) >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    const uint16_t mask16 = (uint16_t)sign_mask;
    record(out, UFP4_FMT_UNIFORM_MX32, qrows, red, rht ? 16 : 0, &mask16, 0.0f, rounding);
    if (rows == 0 || cols == 0) return UFP4_OK;
    MxQuantJob j{};
    j.rounding = rounding;
    j.rht = rht;
    j.transpose = transpose;
    j.x = x_dev;
    j.xrows = rows;
    j.ld = ld;
    j.qrows = qrows;
    j.red = red;
    fill_sign_xor(sign_mask, j.qa.sign_xor);
    j.qa.key0 = (uint32_t)seed;
    j.qa.key1 = (uint32_t)(seed >> 32);
    j.qa.stream = stream_id;
    j.codes = out->codes;
    j.code_pld = out->code_panel_ld;
    j.scales = out->scales;
    j.scale_pld = out->scale_panel_ld;
    return status_of(launch_quantize_mx(j, static_cast<hipStream_t>(stream)));
}

int ufp4_mx_quantize_dual(const void* x_dev, int64_t rows, int64_t cols, int64_t ld, int rht_rows,
                          uint32_t sign_mask_rows, uint32_t stream_rows, int rht_cols, uint32_t sign_mask_cols,
                          uint32_t stream_cols, int rounding, uint64_t seed, ufp4_qtensor* out_rows,
                          ufp4_qtensor* out_cols, void* stream) {
    // Q_r = X [rows, cols] along cols; Q_c = X^T [cols, rows] along rows
    if (rounding != UFP4_ROUND_RTNE && rounding != UFP4_ROUND_SR) return UFP4_ERR_INVALID_ARG;
    if ((rht_rows != 0 && rht_rows != 1) || (rht_cols != 0 && rht_cols != 1)) return UFP4_ERR_INVALID_ARG;
    if (sign_mask_rows > 0xFFFFu || sign_mask_cols > 0xFFFFu) return UFP4_ERR_INVALID_ARG;
    if (out_rows == out_cols) return UFP4_ERR_INVALID_ARG;
    const int si = check_input(x_dev, rows, cols, ld, 8);
    if (si != UFP4_OK) return si;
    int st = check_storage(out_rows, UFP4_FMT_UNIFORM_MX32, rows, cols);
    if (st == UFP4_OK) st = check_storage(out_cols, UFP4_FMT_UNIFORM_MX32, cols, rows);
    if (st != UFP4_OK) return st;
    if (rows >= (int64_t(1) << 31) || cols >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    if (mx_tile_count(rows, cols, true, true) >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;  // 1-D grid
    const uint16_t mr = (uint16_t)sign_mask_rows, mc = (uint16_t)sign_mask_cols;
    record(out_rows, UFP4_FMT_UNIFORM_MX32, rows, cols, rht_rows ? 16 : 0, &mr, 0.0f, rounding);
    record(out_cols, UFP4_FMT_UNIFORM_MX32, cols, rows, rht_cols ? 16 : 0, &mc, 0.0f, rounding);
    if (rows == 0 || cols == 0) return UFP4_OK;
    MxDualJob j{};
    j.rounding = rounding;
    j.rht_r = rht_rows;
    j.rht_c = rht_cols;
    j.x = x_dev;
    j.rows = rows;
    j.cols = cols;
    j.ld = ld;
    fill_sign_xor(sign_mask_rows, j.qr.sign_xor);
    fill_sign_xor(sign_mask_cols, j.qc.sign_xor);
    j.qr.key0 = j.qc.key0 = (uint32_t)seed;
    j.qr.key1 = j.qc.key1 = (uint32_t)(seed >> 32);
    j.qr.stream = stream_rows;
    j.qc.stream = stream_cols;
    j.codes_r = out_rows->codes;
    j.code_pld_r = out_rows->code_panel_ld;
    j.scales_r = out_rows->scales;
    j.scale_pld_r = out_rows->scale_panel_ld;
    j.codes_c = out_cols->codes;
    j.code_pld_c = out_cols->code_panel_ld;
    j.scales_c = out_cols->scales;
    j.scale_pld_c = out_cols->scale_panel_ld;
    return status_of(launch_quantize_mx_dual(j, static_cast<hipStream_t>(stream)));
}

int ufp4_mx_quantize_grouped(const void* x_dev, int64_t rows, int64_t cols, int64_t ld, int transpose,
                             const int64_t* group_offsets_dev, int32_t num_groups, int64_t padded_total, int rht,
                             uint32_t sign_mask, int rounding, uint64_t seed, uint32_t stream_id, ufp4_qtensor* out,
                             void* stream) {
    if (transpose != 0 && transpose != 1) return UFP4_ERR_INVALID_ARG;
    if (rounding != UFP4_ROUND_RTNE && rounding != UFP4_ROUND_SR) return UFP4_ERR_INVALID_ARG;
    if (rht != 0 && rht != 1) return UFP4_ERR_INVALID_ARG;
    if (sign_mask > 0xFFFFu) return UFP4_ERR_INVALID_ARG;
    if (padded_total < 0 || !group_offsets_dev) return UFP4_ERR_INVALID_ARG;
    if (num_groups < 1) return UFP4_ERR_INVALID_ARG;
    if (num_groups > max_groups_quantize()) return UFP4_ERR_UNSUPPORTED;
    const int si = check_input(x_dev, rows, cols, ld, 8);
    if (si != UFP4_OK) return si;
    // transpose 0: [padded_total, cols], groups of rows on whole panels; transpose 1: [cols, padded_total]
    const int64_t qrows = transpose ? cols : padded_total;
    const int64_t red = transpose ? padded_total : cols;
    if (transpose ? padded_total < rows : padded_total % kPanelRows != 0) return UFP4_ERR_SHAPE;
    const int st = check_storage(out, UFP4_FMT_UNIFORM_MX32, qrows, red);
    if (st != UFP4_OK) return st;
    if (qrows >= (int64_t(1) << 31) || red / 16 >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    if (!transpose && padded_rows(qrows) / 64 > 65535) return UFP4_ERR_UNSUPPORTED;
    // grid y: chunks of four 256-column tiles of X (its padded columns for the transposed form)
    if (((transpose ? padded_rows(cols) : cols) + 1023) / 1024 > 65535) return UFP4_ERR_UNSUPPORTED;
    const uint16_t mask16 = (uint16_t)sign_mask;
    record(out, UFP4_FMT_UNIFORM_MX32, qrows, red, rht ? 16 : 0, &mask16, 0.0f, rounding,
           transpose ? UFP4_LAYOUT_GROUPED_RED : UFP4_LAYOUT_GROUPED_ROWS);
    if (qrows == 0 || red == 0) return UFP4_OK;
    MxQuantJob j{};
    j.rounding = rounding;
    j.rht = rht;
    j.transpose = transpose;
    j.x = x_dev;
    j.xrows = rows;
    j.ld = ld;
    j.qrows = qrows;
    j.red = red;
    j.group_off = group_offsets_dev;
    j.num_groups = num_groups;
    fill_sign_xor(sign_mask, j.qa.sign_xor);
    j.qa.key0 = (uint32_t)seed;
    j.qa.key1 = (uint32_t)(seed >> 32);
    j.qa.stream = stream_id;
    j.codes = out->codes;
    j.code_pld = out->code_panel_ld;
    j.scales = out->scales;
    j.scale_pld = out->scale_panel_ld;
    return status_of(launch_quantize_mx(j, static_cast<hipStream_t>(stream)));
}

int ufp4_mx_gemm_fwd_y_grouped(const ufp4_qtensor* x, const ufp4_qtensor* w, const int64_t* group_offsets_dev,
                               int32_t num_groups, int64_t m_total, void* y_dev, int64_t ldc, int out_dtype,
                               void* stream) {
    if (!group_offsets_dev || num_groups < 1 || m_total < 0) return UFP4_ERR_INVALID_ARG;
    int st = check_operands(x, w, true);
    if (st != UFP4_OK) return st;
    if (x->layout != UFP4_LAYOUT_GROUPED_ROWS || w->layout != UFP4_LAYOUT_PLAIN) return UFP4_ERR_MISMATCH;
    if (x->red != w->red) return UFP4_ERR_MISMATCH;
    if (w->rows % num_groups != 0) return UFP4_ERR_SHAPE;
    const int64_t N = w->rows / num_groups;
    if (N % kPanelRows != 0) return UFP4_ERR_UNSUPPORTED;  // each group's weight rows start on a panel
    st = check_output(y_dev, ldc, N, out_dtype, m_total == 0 || N == 0);
    if (st != UFP4_OK) return st;
    if (m_total == 0 || N == 0 || x->rows == 0) return UFP4_OK;
    MxGemmJob j = mx_job(x, w, y_dev, ldc, out_dtype);
    j.mode = kGemmRaggedM;
    j.M = m_total;
    j.N = N;
    j.nkb = x->red / 32;
    j.offsets = group_offsets_dev;
    j.G = num_groups;
    j.m_tiles = ceil_div(x->rows, 256) + num_groups;
    j.b_group_rows = N;
    j.b_group_kb = 0;
    if (j.m_tiles * ceil_div(N, 256) >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    return status_of(launch_gemm_mx(j, static_cast<hipStream_t>(stream)));
}

int ufp4_mx_gemm_bwd_dx_grouped(const ufp4_qtensor* dy, const ufp4_qtensor* wt, const int64_t* group_offsets_dev,
                                int32_t num_groups, int64_t m_total, void* dx_dev, int64_t ldc, int out_dtype,
                                void* stream) {
    if (!group_offsets_dev || num_groups < 1 || m_total < 0) return UFP4_ERR_INVALID_ARG;
    int st = check_operands(dy, wt, true);
    if (st != UFP4_OK) return st;
    if (dy->layout != UFP4_LAYOUT_GROUPED_ROWS || wt->layout != UFP4_LAYOUT_PLAIN) return UFP4_ERR_MISMATCH;
    if (wt->red != dy->red * num_groups) return UFP4_ERR_MISMATCH;
    st = check_output(dx_dev, ldc, wt->rows, out_dtype, m_total == 0 || wt->rows == 0);
    if (st != UFP4_OK) return st;
    if (m_total == 0 || wt->rows == 0 || dy->rows == 0) return UFP4_OK;
    MxGemmJob j = mx_job(dy, wt, dx_dev, ldc, out_dtype);
    j.mode = kGemmRaggedM;
    j.M = m_total;
    j.N = wt->rows;
    j.nkb = dy->red / 32;
    j.offsets = group_offsets_dev;
    j.G = num_groups;
    j.m_tiles = ceil_div(dy->rows, 256) + num_groups;
    j.b_group_rows = 0;
    j.b_group_kb = dy->red / 32;
    if (j.m_tiles * ceil_div(j.N, 256) >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    return status_of(launch_gemm_mx(j, static_cast<hipStream_t>(stream)));
}

int ufp4_mx_gemm_bwd_dw_grouped(const ufp4_qtensor* dyt, const ufp4_qtensor* xt, const int64_t* group_offsets_dev,
                                int32_t num_groups, void* dw_dev, int64_t ldc, int out_dtype, void* stream) {
    if (!group_offsets_dev || num_groups < 1) return UFP4_ERR_INVALID_ARG;
    if (num_groups > 65535) return UFP4_ERR_UNSUPPORTED;
    int st = check_operands(dyt, xt, true);
    if (st != UFP4_OK) return st;
    if (dyt->layout != UFP4_LAYOUT_GROUPED_RED || xt->layout != UFP4_LAYOUT_GROUPED_RED) return UFP4_ERR_MISMATCH;
    if (dyt->red != xt->red) return UFP4_ERR_MISMATCH;
    st = check_output(dw_dev, ldc, xt->rows, out_dtype, dyt->rows == 0 || xt->rows == 0);
    if (st != UFP4_OK) return st;
    if (dyt->rows == 0 || xt->rows == 0) return UFP4_OK;
    if (ceil_div(dyt->rows, 256) * ceil_div(xt->rows, 256) >= (int64_t(1) << 31)) return UFP4_ERR_UNSUPPORTED;
    MxGemmJob j = mx_job(dyt, xt, dw_dev, ldc, out_dtype);
    j.mode = kGemmRaggedK;
    j.M = dyt->rows;
    j.N = xt->rows;
    j.nkb = dyt->red / 32;
    j.offsets = group_offsets_dev;
    j.G = num_groups;
    return status_of(launch_gemm_mx(j, static_cast<hipStream_t>(stream)));
}

int ufp4_mx_gemm_fwd_y(const ufp4_qtensor* x, const ufp4_qtensor* w, void* y_dev, int64_t ldc, int out_dtype,
                       void* stream) {
    return mx_gemm_impl(x, w, y_dev, ldc, out_dtype, stream);
}

int ufp4_mx_gemm_bwd_dx(const ufp4_qtensor* dy, const ufp4_qtensor* wt, void* dx_dev, int64_t ldc, int out_dtype,
                        void* stream) {
    return mx_gemm_impl(dy, wt, dx_dev, ldc, out_dtype, stream);  // dX [M, K] = dY [M, N] . (W^T [K, N])^T
}

int ufp4_mx_gemm_bwd_dw(const ufp4_qtensor* dyt, const ufp4_qtensor* xt, void* dw_dev, int64_t ldc, int out_dtype,
                        void* stream) {
    return mx_gemm_impl(dyt, xt, dw_dev, ldc, out_dtype, stream);  // dW [N, K] = dY^T [N, M] . (X^T [K, M])^T
}

int ufp4_gemm_fwd_y(const ufp4_qtensor* x, const ufp4_qtensor* w, void* y_dev, int64_t ldc, int out_dtype,
                    void* stream) {
    return gemm_dense(x, w, y_dev, ldc, out_dtype, stream);
}

int ufp4_gemm_bwd_dx(const ufp4_qtensor* dy, const ufp4_qtensor* wt, void* dx_dev, int64_t ldc, int out_dtype,
                     void* stream) {
    return gemm_dense(dy, wt, dx_dev, ldc, out_dtype, stream);  // dX [M, K] = dY [M, N] . (W^T [K, N])^T
}

int ufp4_gemm_bwd_dw(const ufp4_qtensor* dyt, const ufp4_qtensor* xt, void* dw_dev, int64_t ldc, int out_dtype,
                     void* stream) {
    return gemm_dense(dyt, xt, dw_dev, ldc, out_dtype, stream);  // dW [N, K] = dY^T [N, M] . (X^T [K, M])^T
}

int ufp4_gemm_fwd_y_grouped(const ufp4_qtensor* x, const ufp4_qtensor* w, const int64_t* group_offsets_dev,
                            int32_t num_groups, void* y_dev, int64_t ldc, int out_dtype, void* stream) {
    if (!group_offsets_dev || num_groups < 1) return UFP4_ERR_INVALID_ARG;
    int st = check_operands(x, w, false);
    if (st != UFP4_OK) return st;
    if (x->layout != UFP4_LAYOUT_PLAIN || w->layout != UFP4_LAYOUT_PLAIN) return UFP4_ERR_MISMATCH;
    if (x->red != w->red) return UFP4_ERR_MISMATCH;
    if (w->rows % num_groups != 0) return UFP4_ERR_SHAPE;
    const int64_t N = w->rows / num_groups;
    st = check_output(y_dev, ldc, N, out_dtype, x->rows == 0 || N == 0);
    if (st != UFP4_OK) return st;
    if (x->rows == 0 || N == 0) return UFP4_OK;
    GemmJob j = make_job(kGemmRaggedM, x, w, x->rows, N, x->red / 16, y_dev, ldc, out_dtype);
    j.offsets = group_offsets_dev;
    j.G = num_groups;
    j.b_group_rows = N;
    j.b_group_kb = 0;
    return status_of(launch_gemm(j, static_cast<hipStream_t>(stream)));
}

int ufp4_gemm_bwd_dx_grouped(const ufp4_qtensor* dy, const ufp4_qtensor* wt, const int64_t* group_offsets_dev,
                             int32_t num_groups, void* dx_dev, int64_t ldc, int out_dtype, void* stream) {
    if (!group_offsets_dev || num_groups < 1) return UFP4_ERR_INVALID_ARG;
    // A = dY [M_total, N]; B = W^T [K, G*N], group g uses reduction columns [g*N, (g+1)*N)
    int st = check_operands(dy, wt, false);
    if (st != UFP4_OK) return st;
    // dY's reduction (N) is a multiple of 16, so W^T's equal groups need no padding: its grouped-transposed
    // and plain transposed forms coincide and both are accepted
    if (dy->layout != UFP4_LAYOUT_PLAIN || wt->layout == UFP4_LAYOUT_GROUPED_ROWS) return UFP4_ERR_MISMATCH;
    if (wt->red != dy->red * num_groups) return UFP4_ERR_MISMATCH;
    st = check_output(dx_dev, ldc, wt->rows, out_dtype, dy->rows == 0 || wt->rows == 0);
    if (st != UFP4_OK) return st;
    if (dy->rows == 0 || wt->rows == 0) return UFP4_OK;
    GemmJob j = make_job(kGemmRaggedM, dy, wt, dy->rows, wt->rows, dy->red / 16, dx_dev, ldc, out_dtype);
    j.offsets = group_offsets_dev;
    j.G = num_groups;
    j.b_group_rows = 0;
    j.b_group_kb = dy->red / 16;
    return status_of(launch_gemm(j, static_cast<hipStream_t>(stream)));
}

int ufp4_gemm_bwd_dw_grouped(const ufp4_qtensor* dyt, const ufp4_qtensor* xt, const int64_t* group_offsets_dev,
                             int32_t num_groups, void* dw_dev, int64_t ldc, int out_dtype, void* stream) {
    if (!group_offsets_dev || num_groups < 1) return UFP4_ERR_INVALID_ARG;
    if (num_groups > 65535) return UFP4_ERR_UNSUPPORTED;
    // A = dY^T [N, R], B = X^T [K, R]; group g reduces over [pad_g, pad_{g+1}) of that axis
    int st = check_operands(dyt, xt, false);
    if (st != UFP4_OK) return st;
    // the kernel reduces each group over its tokens padded to 16, the layout ufp4_quantize_grouped_t writes
    if (dyt->layout != UFP4_LAYOUT_GROUPED_RED || xt->layout != UFP4_LAYOUT_GROUPED_RED) return UFP4_ERR_MISMATCH;
    if (dyt->red != xt->red) return UFP4_ERR_MISMATCH;
    st = check_output(dw_dev, ldc, xt->rows, out_dtype, dyt->rows == 0 || xt->rows == 0);
    if (st != UFP4_OK) return st;
    if (dyt->rows == 0 || xt->rows == 0) return UFP4_OK;
    GemmJob j = make_job(kGemmRaggedK, dyt, xt, dyt->rows, xt->rows, 0, dw_dev, ldc, out_dtype);
    j.offsets = group_offsets_dev;
    j.G = num_groups;
    j.red_total = dyt->red;
    return status_of(launch_gemm(j, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
