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
// Tiling: a 256 x 256 output tile per 512-thread workgroup (8 waves of 128 x 64, 4 x 2 MFMA tiles of 32 x 32,
// two waves per SIMD, one workgroup per CU). K advances 128 (four 32-blocks) per stage. A stage of one panel
// is a contiguous 12 KiB run (the panel layout puts the 128 rows of a 32-block together, each row's 24 bytes
// as three 8-byte units in three planes of 128 rows) plus 512 scale bytes; stages are copied unchanged from
// global memory into a three-deep LDS ring by direct-to-LDS loads issued two stages ahead, and a lane's
// operand is three 8-byte LDS reads that 32 consecutive rows make contiguous.

#include "ufp4_internal.h"

namespace ufp4 {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef int v8i __attribute__((ext_vector_type(8)));

constexpr int kMxTile = 256;                    // rows of A and of B per workgroup tile (two panels each)
constexpr int kMxStageBlocks = 4;               // 32-blocks per stage
constexpr int kMxStageBytes = kMxStageBlocks * 3072;  // one panel's codes per stage
constexpr int kMxThreads = 512;                 // 8 waves, two per SIMD, each a 128 x 64 tile
constexpr int kMxBufs = 3;                      // stages in LDS: the one computed and two in flight
constexpr int kMxLoadsPerStage = 7;             // per wave: 3 of A, 3 of B, 1 of scales (16 bytes per lane)

struct MxStageSmem {
    uint8_t a[2][kMxStageBytes];  // the tile's two panels of A
    uint8_t b[2][kMxStageBytes];
    uint8_t s[2][2][kMxStageBlocks * 128];  // scale bytes: [A, B][panel][block * 128 + row]
};

// The 24 bytes of one row's 32-block: three 8-byte units 1024 bytes apart (planar layout, see the file
// header), so 32 lanes reading consecutive rows touch 256 contiguous bytes per unit.
__device__ __forceinline__ v8i load_fp6_operand(const uint8_t* p) {
    const uint2 x0 = *reinterpret_cast<const uint2*>(p);
    const uint2 x1 = *reinterpret_cast<const uint2*>(p + 1024);
    const uint2 x2 = *reinterpret_cast<const uint2*>(p + 2048);
    const v8i v = {(int)x0.x, (int)x0.y, (int)x1.x, (int)x1.y, (int)x2.x, (int)x2.y, 0, 0};
    return v;
}

// 16 bytes per lane from global memory straight into LDS: lane i reads sbase + voff_i and its bytes land at
// lds_base + 16 i (sbase and lds_base wave-uniform, lds_base in M0). Written as inline assembly so that the
// compiler, which does not see these LDS writes, does not make every later LDS read wait for all of them; the
// kernel orders them itself (vmcnt waits and barriers).
__device__ __forceinline__ void dma16(uint32_t voff, const void* sbase, const void* lds_base) {
    const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)reinterpret_cast<uintptr_t>(lds_base));
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(m0)
                 : "memory", "m0");
}

// s_waitcnt immediates (gfx9 encoding): wait until at most n vector-memory operations are outstanding,
// and additionally for all LDS operations.
__device__ __forceinline__ void wait_vm_lgkm(int n) {
    switch (n) {
        case 0: __builtin_amdgcn_s_waitcnt(0x0070); break;
        default: __builtin_amdgcn_s_waitcnt(0x0070 | kMxLoadsPerStage); break;
    }
}

// Workgroup -> output tile. Workgroups are dealt to the 8 XCDs round robin (workgroup L to XCD L % 8) and each
// XCD has its own L2, so the first 8 * floor(T / 8) workgroups are renumbered to give XCD k the contiguous
// range of tiles [k T/8, (k + 1) T/8); tiles are then ordered in bands of kGroupRows tile rows, column by
// column within a band, so that the workgroups running together on one XCD share a few A and B panels.
constexpr int kGroupRows = 8;
__device__ __forceinline__ void tile_of(int64_t L, int64_t gy, int64_t gx, int64_t& tm, int64_t& tn) {
    const int64_t T = gx * gy, per = T / 8;
    const int64_t t = L < 8 * per ? (L % 8) * per + L / 8 : L;
    const int64_t band = t / (kGroupRows * gx);
    const int64_t first = band * kGroupRows;
    const int64_t rows = gy - first < kGroupRows ? gy - first : kGroupRows;
    const int64_t r = t - band * kGroupRows * gx;
    tm = first + r % rows;
    tn = r / rows;
}

constexpr int64_t kMxBlock32 = 32;  // reduction values per scale block

// Wave-uniform copy (SGPRs) of a value the compiler cannot prove uniform, e.g. one read back from LDS.
__device__ __forceinline__ int64_t uniform_i64_mx(int64_t v) {
    const uint64_t u = (uint64_t)v;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u), hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Ragged-M: the group and local tile of global m-tile t, with the group's padded row start (a multiple of 128)
// and its token rows. Wave 0 prefix-sums the per-group tile counts ceil(m_g / 256) and padded lengths
// pad128(m_g), 64 groups at a time; the result goes through LDS. Every thread calls this; false past the last tile.
struct MxGroupTile {
    int64_t g, lt, prow0, trow0, rows;
};
__device__ bool resolve_mx_ragged_m(const MxGemmJob& j, int64_t t, int64_t* slot, MxGroupTile& r) {
    const int tid = threadIdx.x;
    if (tid == 0) slot[0] = -1;
    __syncthreads();
    if (tid < 64) {
        int64_t tbase = 0, pbase = 0;
        for (int g0 = 0; g0 < j.G; g0 += 64) {
            const int g = g0 + tid;
            int64_t m = 0;
            if (g < j.G) m = j.offsets[g + 1] - j.offsets[g];
            if (m < 0) m = 0;
            const int64_t cnt = (m + kMxTile - 1) / kMxTile, pad = (m + 127) / 128 * 128;
            int64_t ti = cnt, pi = pad;
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const int64_t vt = __shfl_up(ti, d, 64), vp = __shfl_up(pi, d, 64);
                if (tid >= d) {
                    ti += vt;
                    pi += vp;
                }
            }
            const int64_t te = tbase + ti - cnt;  // first global tile of group g
            if (cnt > 0 && te <= t && t < te + cnt) {
                slot[0] = g;
                slot[1] = t - te;
                slot[2] = pbase + pi - pad;
                slot[3] = m;
            }
            tbase += __shfl(ti, 63, 64);
            pbase += __shfl(pi, 63, 64);
        }
    }
    __syncthreads();
    r.g = slot[0];
    if (r.g < 0) return false;
    r.lt = slot[1];
    r.prow0 = slot[2] + r.lt * kMxTile;
    r.trow0 = j.offsets[r.g] + r.lt * kMxTile;
    r.rows = slot[3] - r.lt * kMxTile;
    return true;
}

// Padded start of group g along a ragged reduction (token counts rounded up to 32, summed over h < g) and the
// group's padded length, by wave 0 through LDS; every thread calls this.
__device__ void mx_padded_range(const int64_t* off, int g, int64_t* slot, int64_t& start, int64_t& len) {
    const int tid = threadIdx.x;
    if (tid < 64) {
        int64_t sum = 0;
        for (int h = tid; h < g; h += 64) {
            const int64_t c = off[h + 1] - off[h];
            sum += (c > 0 ? c + kMxBlock32 - 1 : 0) / kMxBlock32 * kMxBlock32;
        }
#pragma unroll
        for (int d = 32; d > 0; d >>= 1) sum += __shfl_xor(sum, d, 64);
        if (tid == 0) slot[0] = sum;
    }
    __syncthreads();
    start = slot[0];
    const int64_t c = off[g + 1] - off[g];
    len = (c > 0 ? c + kMxBlock32 - 1 : 0) / kMxBlock32 * kMxBlock32;
}

template <int OUT>
__global__ __launch_bounds__(kMxThreads) void gemm_mx_kernel(MxGemmJob j) {
    // three separate LDS objects (not an array): the compiler then knows that loads in flight into one buffer
    // do not alias reads of another and does not make the reads wait for them
    __shared__ MxStageSmem sm0, sm1, sm2;
    __shared__ int64_t s_slot[4];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: load addresses stay scalar
    const int h = lane >> 5, l32 = lane & 31;
    const int wm = wave >> 2, wn = wave & 3;  // wave tile: rows wm * 128 .. + 127, cols wn * 64 .. + 63
    int64_t tm, tn;
    const int64_t gy = j.mode == kGemmRaggedM ? j.m_tiles : (j.M + kMxTile - 1) / kMxTile;
    tile_of(blockIdx.x, gy, (j.N + kMxTile - 1) / kMxTile, tm, tn);
    // What the tile covers: A panels from pa0, B panels from pb0, reduction blocks from a_kb0 / b_kb0 (nkb of
    // them), output rows out_row0 .. out_row0 + mrows - 1 (token rows for ragged-M) of the problem at c_base.
    int64_t pa0 = 2 * tm, pb0 = 2 * tn, a_kb0 = 0, b_kb0 = 0, nkb64 = j.nkb;
    int64_t out_row0 = tm * kMxTile, mrows = j.M - tm * kMxTile, c_base = 0;
    if (j.mode == kGemmRaggedM) {
        MxGroupTile r;
        if (!resolve_mx_ragged_m(j, tm, s_slot, r)) return;  // the whole workgroup agrees
        pa0 = r.prow0 / 128;
        out_row0 = r.trow0;
        mrows = r.rows < j.M - r.trow0 ? r.rows : j.M - r.trow0;  // token rows past the output are not stored
        pb0 = (r.g * j.b_group_rows) / 128 + 2 * tn;
        b_kb0 = r.g * j.b_group_kb;
    } else if (j.mode == kGemmRaggedK) {
        int64_t start, len;
        mx_padded_range(j.offsets, (int)blockIdx.y, s_slot, start, len);
        a_kb0 = b_kb0 = start / kMxBlock32;
        nkb64 = len / kMxBlock32;
        if (a_kb0 + nkb64 > j.nkb) nkb64 = j.nkb - a_kb0 > 0 ? j.nkb - a_kb0 : 0;  // clamped to the operands
        c_base = (int64_t)blockIdx.y * j.M * j.ldc;
    }
    pa0 = uniform_i64_mx(pa0);
    pb0 = uniform_i64_mx(pb0);
    a_kb0 = uniform_i64_mx(a_kb0);
    b_kb0 = uniform_i64_mx(b_kb0);
    nkb64 = uniform_i64_mx(nkb64);
    // The tile's two panels of each operand. A panel past the operand's last one (a tile over the edge) is
    // replaced by the last panel: those rows only feed outputs that are not stored.
    const int64_t pa_last = (j.a_rows - 1) / 128, pb_last = (j.b_rows - 1) / 128;
    if (pa0 > pa_last) pa0 = pa_last;  // only for offsets inconsistent with the operand: wrong values, no fault
    if (pb0 > pb_last) pb0 = pb_last;
    const int64_t pa1 = pa0 + 1 < pa_last ? pa0 + 1 : pa_last;
    const int64_t pb1 = pb0 + 1 < pb_last ? pb0 + 1 : pb_last;
    const uint8_t* const ga0 = j.a + pa0 * j.a_pld + a_kb0 * 3072;
    const uint8_t* const ga1 = j.a + pa1 * j.a_pld + a_kb0 * 3072;
    const uint8_t* const gb0 = j.b + pb0 * j.b_pld + b_kb0 * 3072;
    const uint8_t* const gb1 = j.b + pb1 * j.b_pld + b_kb0 * 3072;
    // this wave's scale run: chunks 16 w .. 16 w + 15 of [A panel 0, A panel 1, B panel 0, B panel 1] x 32
    const int sop = wave >> 2, sp = (wave >> 1) & 1;
    const uint8_t* const gs = sop == 0 ? j.as + (sp ? pa1 : pa0) * j.as_pld + a_kb0 * 128
                                       : j.bs + (sp ? pb1 : pb0) * j.bs_pld + b_kb0 * 128;
    const int64_t N = j.N, ldc = j.ldc;
    void* const cptr = j.c;
    const int nkb = (int)nkb64;
    const int nst = (nkb + kMxStageBlocks - 1) / kMxStageBlocks;
    const int kb_last = nkb - 1;

    // Stage s into a buffer with direct global-to-LDS loads: each wave instruction moves 64 x 16 bytes to
    // 1024 contiguous LDS bytes. Per operand a stage is 2 panels x 768 chunks; wave w copies chunks
    // i * 512 + w * 64 + lane (i < 3) of the pair, panel = chunk / 768, and scale chunks 16 w + lane (lanes
    // 0-15). Every wave issues the same 7 loads for every stage: blocks past the end of the reduction
    // (partial last stage) are read from the last block instead, and compute() gives them zero scales.
    const uint32_t voff = (uint32_t)lane * 16;
    auto issue = [&](int s, MxStageSmem& d) {
        const int kb0 = s * kMxStageBlocks;
#pragma unroll
        for (int i = 0; i < 3; ++i) {
            const int c0 = i * 512 + wave * 64;  // 64-chunk groups never straddle a panel or a block
            const int p = c0 / 768, cp0 = c0 - p * 768, blk = cp0 / 192;
            const int kb = kb0 + blk < kb_last ? kb0 + blk : kb_last;
            const int64_t off = (int64_t)kb * 3072 + (cp0 - blk * 192) * 16;
            dma16(voff, (p ? ga1 : ga0) + off, reinterpret_cast<uint4*>(d.a[p]) + cp0);
            dma16(voff, (p ? gb1 : gb0) + off, reinterpret_cast<uint4*>(d.b[p]) + cp0);
        }
        if (lane < 16) {
            const int cc = (wave & 1) * 16 + lane, blk = cc >> 3;  // chunk within the 32-chunk run
            const int kb = kb0 + blk < kb_last ? kb0 + blk : kb_last;
            dma16((uint32_t)(kb * 128 + (cc & 7) * 16), gs, reinterpret_cast<uint4*>(&d.s[0][0][0]) + wave * 16);
        }
    };

    v16f acc[4][2];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.0f;

    auto compute = [&](const MxStageSmem& d, int valid) {
#pragma unroll
        for (int ks = 0; ks < kMxStageBlocks / 2; ++ks) {
            const int kk = 2 * ks + h;  // this lane's 32-block: lanes 0-31 hold K 0-31 of the step, 32-63 K 32-63
            const bool live = kk < valid;  // blocks past the end get scale 2^-127 on both sides: products 0
            v8i av[4], bv[2];
            int sa[4], sb[2];
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const int col = wn * 64 + b * 32 + l32, p = col >> 7, r = col & 127;
                bv[b] = load_fp6_operand(d.b[p] + kk * 3072 + r * 8);
                sb[b] = live ? d.s[1][p][kk * 128 + r] : 0;
            }
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                const int r = a * 32 + l32;  // row within panel wm
                av[a] = load_fp6_operand(d.a[wm] + kk * 3072 + r * 8);
                sa[a] = live ? d.s[0][wm][kk * 128 + r] : 0;
#pragma unroll
                for (int b = 0; b < 2; ++b)
                    // formats 2 = FP6 E2M3 for both operands; the scale bytes sit in byte 0 of sa / sb
                    acc[a][b] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av[a], bv[b], acc[a][b], 2, 2, 0,
                                                                                sa[a], 0, sb[b]);
            }
        }
    };

    // Stage s is computed from buffer s % 3 while stages s + 1 and s + 2 are in flight. A wave's own loads
    // of stage s are complete once at most the 7 of stage s + 1 are outstanding; the barrier then makes every
    // wave's part visible, and it also orders the previous stage's reads of buffer (s + 2) % 3 before the
    // loads into it are issued.
    auto step = [&](int s, MxStageSmem& cur, MxStageSmem& next2) {
        wait_vm_lgkm(s + 1 < nst ? kMxLoadsPerStage : 0);
        __builtin_amdgcn_s_barrier();
        if (s + 2 < nst) issue(s + 2, next2);
        const int left = nkb - s * kMxStageBlocks;
        compute(cur, left < kMxStageBlocks ? left : kMxStageBlocks);
    };
    if (nst > 0) issue(0, sm0);
    if (nst > 1) issue(1, sm1);
    for (int s = 0; s < nst; s += 3) {
        step(s, sm0, sm2);
        if (s + 1 < nst) step(s + 1, sm1, sm0);
        if (s + 2 < nst) step(s + 2, sm2, sm1);
    }

    // Epilogue: lane (l32, h) holds rows 8q + 4h + t (q, t < 4) of column l32 of each 32 x 32 tile; a store
    // instruction writes two runs of 32 consecutive outputs. Tiles inside the output skip the bounds tests.
    const bool inside = mrows >= kMxTile && (tn + 1) * kMxTile <= N;
    auto store = [&](int64_t row, int64_t col, float v) {
        const int64_t off = c_base + row * ldc + col;
        if constexpr (OUT == kOutF32) {
            static_cast<float*>(cptr)[off] = v;
        } else {
            static_cast<uint16_t*>(cptr)[off] = __builtin_bit_cast(uint16_t, (__bf16)v);  // RNE
        }
    };
#pragma unroll
    for (int a = 0; a < 4; ++a) {
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int64_t col = tn * kMxTile + wn * 64 + b * 32 + l32;
            const int64_t lr0 = wm * 128 + a * 32 + 4 * h;  // tile row of acc element 0
            if (inside) {
#pragma unroll
                for (int i = 0; i < 16; ++i) store(out_row0 + lr0 + 8 * (i >> 2) + (i & 3), col, acc[a][b][i]);
            } else if (col < N) {
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int64_t lr = lr0 + 8 * (i >> 2) + (i & 3);
                    if (lr < mrows) store(out_row0 + lr, col, acc[a][b][i]);
                }
            }
        }
    }
}

hipError_t launch_gemm_mx(const MxGemmJob& j, hipStream_t s) {
    const int64_t gy = j.mode == kGemmRaggedM ? j.m_tiles : (j.M + kMxTile - 1) / kMxTile;
    const int64_t tiles = ((j.N + kMxTile - 1) / kMxTile) * gy;
    if (tiles == 0) return hipSuccess;
    const dim3 grid((unsigned)tiles, j.mode == kGemmRaggedK ? (unsigned)j.G : 1u);
    if (j.out_dtype == kOutBF16) gemm_mx_kernel<kOutBF16><<<grid, kMxThreads, 0, s>>>(j);
    else gemm_mx_kernel<kOutF32><<<grid, kMxThreads, 0, s>>>(j);
    return hipGetLastError();
}

}  // namespace ufp4
