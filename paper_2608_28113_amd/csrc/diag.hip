// Quality diagnostics of the paper's appendix behind the C ABI of
// include/hscale.h: the per-shift summary of the search statistics and the
// layer-output error of Eq. 3.

#include "common.h"

namespace {

// ---------------------------------------------------------------------------
// Selected-shift statistics (the paper's appendix on selected scale shifts):
// per shift d, the number of groups that chose it and the fp64 sums of their
// initial errors, chosen errors and relative reductions.  Deterministic: each
// block reduces a fixed chunk in a fixed order, then one wave per bin sums
// the block partials in a fixed order.
// ---------------------------------------------------------------------------

constexpr int kSumThreads = 256;
constexpr int kSumPerThread = 16;
constexpr int kSumChunk = kSumThreads * kSumPerThread;
constexpr int kSumOutside = 1 << 20;  // shift value standing for "no group"
static_assert(kSumThreads == 256, "the block reductions below combine exactly four waves");

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ int wave_min(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
    return v;
}

__device__ __forceinline__ int wave_max(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
    return v;
}

// Block b reduces groups [b * kSumChunk, (b + 1) * kSumChunk) into
// part[(b * K + k) * 3 + {0: init, 1: best, 2: rel}] and cnt[b * K + k] for
// every bin k = d + down (zeros for bins no group of the chunk chose).
__global__ __launch_bounds__(kSumThreads) void shift_summary_partial(const int8_t *__restrict__ shift,
                                                                     const float *__restrict__ err_best,
                                                                     const float *__restrict__ err_init,
                                                                     int64_t groups, int down, int up,
                                                                     double *__restrict__ part,
                                                                     uint32_t *__restrict__ cnt) {
    __shared__ double red[kSumThreads / 64][3];
    __shared__ uint32_t redc[kSumThreads / 64];
    __shared__ int lim[2][kSumThreads / 64];
    const int K = down + up + 1;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t base = (int64_t)blockIdx.x * kSumChunk;
    int d[kSumPerThread];
    float eb[kSumPerThread], ei[kSumPerThread];
    int lo = kSumOutside, hi = -kSumOutside;
#pragma unroll
    for (int e = 0; e < kSumPerThread; ++e) {
        const int64_t g = base + threadIdx.x + (int64_t)e * kSumThreads;
        d[e] = kSumOutside;
        eb[e] = ei[e] = 0.0f;
        if (g < groups) {
            const int v = shift[g];
            if (v >= -down && v <= up) {
                d[e] = v;
                eb[e] = err_best[g];
                ei[e] = err_init[g];
                lo = min(lo, v);
                hi = max(hi, v);
            }
        }
    }
    lo = wave_min(lo);
    hi = wave_max(hi);
    if (lane == 0) {
        lim[0][wave] = lo;
        lim[1][wave] = hi;
    }
    __syncthreads();
    lo = min(min(lim[0][0], lim[0][1]), min(lim[0][2], lim[0][3]));
    hi = max(max(lim[1][0], lim[1][1]), max(lim[1][2], lim[1][3]));
    double *bp = part + (size_t)blockIdx.x * K * 3;
    uint32_t *bc = cnt + (size_t)blockIdx.x * K;
    for (int k = threadIdx.x; k < K; k += kSumThreads) {
        if (k - down < lo || k - down > hi) {
            bp[3 * k] = bp[3 * k + 1] = bp[3 * k + 2] = 0.0;
            bc[k] = 0u;
        }
    }
    for (int v = lo; v <= hi; ++v) {  // block-uniform bounds
        double si = 0.0, sb = 0.0, sr = 0.0;
        uint32_t c = 0;
#pragma unroll
        for (int e = 0; e < kSumPerThread; ++e) {
            if (d[e] == v) {
                const double a = ei[e], b = eb[e];
                ++c;
                si += a;
                sb += b;
                sr += a > 0.0 ? (a - b) / a : 0.0;
            }
        }
        si = wave_sum(si);
        sb = wave_sum(sb);
        sr = wave_sum(sr);
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
        if (lane == 0) {
            red[wave][0] = si;
            red[wave][1] = sb;
            red[wave][2] = sr;
            redc[wave] = c;
        }
        __syncthreads();
        if (threadIdx.x < 3) {
            const int q = threadIdx.x;
            bp[3 * (v + down) + q] = (red[0][q] + red[1][q]) + (red[2][q] + red[3][q]);
        } else if (threadIdx.x == 3) {
            bc[v + down] = (redc[0] + redc[1]) + (redc[2] + redc[3]);
        }
        __syncthreads();
    }
}

// One wave per bin: lane l sums the partials of blocks l, l + 64, ... in
// order, then a fixed butterfly combines the lanes.
__global__ __launch_bounds__(64) void shift_summary_final(const double *__restrict__ part,
                                                          const uint32_t *__restrict__ cnt, int64_t blocks,
                                                          int K, uint64_t *__restrict__ count,
                                                          double *__restrict__ sum_init,
                                                          double *__restrict__ sum_best,
                                                          double *__restrict__ sum_rel) {
    const int k = blockIdx.x;
    double si = 0.0, sb = 0.0, sr = 0.0;
    uint64_t c = 0;
    for (int64_t b = threadIdx.x; b < blocks; b += 64) {
        const double *p = part + ((size_t)b * K + k) * 3;
        si += p[0];
        sb += p[1];
        sr += p[2];
        c += cnt[(size_t)b * K + k];
    }
    si = wave_sum(si);
    sb = wave_sum(sb);
    sr = wave_sum(sr);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
    if (threadIdx.x == 0) {
        count[k] = c;
        sum_init[k] = si;
        sum_best[k] = sb;
        sum_rel[k] = sr;
    }
}

// ---------------------------------------------------------------------------
// Layer-output error (Sec. 3.2, Eq. 3): L_r = sum_t (X dW^T)_tr^2 per output
// row r, with dW = W - W^ the rounding error of a stored NVFP4 tensor.
//
// dW is formed once in fp32 (w - v S[c], one rounding) and split into two
// bf16 planes hi + lo (|dW - hi - lo| <= 2^-18 |dW|), so X dW^T is two bf16
// MFMA products accumulated in fp32.  Each block computes a 384-token x
// 256-row tile of X dW^T in registers and reduces the squares of its columns
// in fp64; the tile is never written.  Per-tile column sums go to a
// workspace and a fixed-order tree adds them to row_err.
// ---------------------------------------------------------------------------

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Tile of X dW^T per block: kLfBM tokens x kLfBN weight rows, computed by
// kLfWM x kLfWN waves (each a 128 x 64 sub-tile of 32 x 32 MFMA
// accumulators, 128 registers).  Twelve waves, three per SIMD at up to 170
// registers each: the largest tile the register file holds, which keeps the
// bytes staged per MFMA flop low (the global -> LDS loads, not the matrix
// cores, bound this kernel).
constexpr int kLfBM = 384;
constexpr int kLfBN = 256;
constexpr int kLfWM = 3;
constexpr int kLfWN = 4;
constexpr int kLfBK = 32;  // k per LDS stage (two 16-deep MFMA steps)
constexpr int kLfThreads = 64 * kLfWM * kLfWN;
constexpr int kLfWaves = kLfThreads / 64;
constexpr int kLfMI = kLfBM / kLfWM / 32;  // accumulator tiles per wave, token direction
constexpr int kLfNJ = kLfBN / kLfWN / 32;  // accumulator tiles per wave, weight-row direction
constexpr int kLfRows = kLfBM + 2 * kLfBN;  // LDS rows of 64 bytes per stage (X, dW hi, dW lo)
constexpr int kLfStages = 2;                // LDS ring: one stage in flight while one is read
constexpr int kLfSlots = kLfRows / 16;      // 1 KB loads per stage, slot q issued by wave q % waves
constexpr int kLfLoadsPerWave = (kLfSlots + kLfWaves - 1) / kLfWaves;
static_assert(kLfBM % (kLfWM * 32) == 0 && kLfBN % (kLfWN * 32) == 0, "wave tiles of 32 x 32 accumulators");
static_assert(kLfStages * kLfRows * 64 <= 160 * 1024, "LDS ring exceeds the CU's 160 KB");
static_assert(kLfWM * kLfBN * 8 <= kLfRows * 64, "the epilogue's reduction fits in one stage buffer");
constexpr int64_t kLfMaxTilesPerPass = 1024;  // token tiles per tile launch (bounds the workspace)
// Buffer descriptors cover one tile's rows with 32-bit byte offsets: every
// tile spans less than 2^31 bytes for in <= 2^21.
constexpr int64_t kLfMaxIn = (int64_t)1 << 21;
constexpr int kLfXcdGroup = 4;  // row tiles grouped per token tile in the XCD-aware order
constexpr uint32_t kRawBufferWord3 = 0x00020000u;  // raw (untyped) buffer, 32-bit data format

__device__ __forceinline__ uint32_t bf16_bits_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;  // finite inputs
}

// dW of one 16-weight group, split into hi / lo bf16 planes of row stride
// ldd; groups beyond (out, in) in the padded planes are written as zeros.
__global__ __launch_bounds__(256) void delta_split_kernel(const u32x4 *__restrict__ W, int64_t out, int64_t in,
                                                          float s_g, const uint8_t *__restrict__ codes,
                                                          const uint2 *__restrict__ packed, int64_t rows_pad,
                                                          int64_t ldd, u32x4 *__restrict__ hi,
                                                          u32x4 *__restrict__ lo) {
    const int64_t Gp = ldd / kGroup, Gc = in / kGroup;
    const int64_t total = rows_pad * Gp;
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < total; q += stride) {
        const int64_t r = q / Gp, i = q % Gp;
        uint32_t hb[8], lb[8];
        if (r < out && i < Gc) {
            const int64_t g = r * Gc + i;
            float w[kGroup];
            load_group(W, g, w);
            const float S = s_g * e4m3fn_value(codes[g]);
            const uint2 p = packed[g];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const uint32_t src = k < 4 ? p.x : p.y;
                float2 v;
                switch (k & 3) {
                    case 0: { const auto t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(src, 1.0f, 0); v = make_float2(t[0], t[1]); break; }
                    case 1: { const auto t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(src, 1.0f, 1); v = make_float2(t[0], t[1]); break; }
                    case 2: { const auto t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(src, 1.0f, 2); v = make_float2(t[0], t[1]); break; }
                    default: { const auto t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(src, 1.0f, 3); v = make_float2(t[0], t[1]); break; }
                }
                const float d0 = fmaf(-v.x, S, w[2 * k]);
                const float d1 = fmaf(-v.y, S, w[2 * k + 1]);
                const uint32_t h0 = bf16_bits_rne(d0), h1 = bf16_bits_rne(d1);
                const uint32_t l0 = bf16_bits_rne(d0 - __uint_as_float(h0 << 16));
                const uint32_t l1 = bf16_bits_rne(d1 - __uint_as_float(h1 << 16));
                hb[k] = h0 | (h1 << 16);
                lb[k] = l0 | (l1 << 16);
            }
        } else {
#pragma unroll
            for (int k = 0; k < 8; ++k) hb[k] = lb[k] = 0u;
        }
        u32x4 *dh = hi + (r * ldd + i * kGroup) / 8;
        u32x4 *dl = lo + (r * ldd + i * kGroup) / 8;
        dh[0] = u32x4{hb[0], hb[1], hb[2], hb[3]};
        dh[1] = u32x4{hb[4], hb[5], hb[6], hb[7]};
        dl[0] = u32x4{lb[0], lb[1], lb[2], lb[3]};
        dl[1] = u32x4{lb[4], lb[5], lb[6], lb[7]};
    }
}

// LDS tiles hold rows of kLfBK bf16 (64 bytes = four 16-byte chunks); chunk c
// of row r lives at chunk position c ^ ((r >> 2) & 3).  A 16-byte operand
// read is served 16 lanes at a time over 64 four-byte banks (256 bytes); the
// 16 consecutive rows those lanes read then fall in 16 distinct bank groups
// (measured: no bank conflicts).
__device__ __forceinline__ int lf_lds_offset(int row, int chunk) {
    return row * 64 + ((chunk ^ ((row >> 2) & 3)) << 4);
}

// s_waitcnt immediate (gfx9 encoding) waiting until at most n vector memory
// operations of this wave are outstanding; the other counters are left free.
constexpr int waitcnt_vm(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

struct LfArgs {
    const u32x4 *X;      // [tokens, in] bf16
    int64_t tokens, in;  // of this pass
    const u32x4 *hi;     // [rows_pad, ldd] bf16 planes
    const u32x4 *lo;
    int64_t ldd;
    int64_t out;      // weight rows
    int64_t ntiles;   // rows_pad / kLfBN
    double *partial;  // [token tiles of the pass, out]
};

// The (token tile, row tile) of block b.  Blocks are dispatched to the 8
// XCDs round-robin (b % 8); XCD x takes a contiguous range of a linear order
// in which kLfXcdGroup row tiles of consecutive token tiles are adjacent, so
// the 32 blocks an XCD runs at once cover about 8 token tiles x 4 row tiles
// and share their X and dW k-slices in that XCD's L2.  Any order gives the
// same result; this one minimises the L2 misses of such a rectangle.
__device__ __forceinline__ void lf_tile_of_block(int64_t b, int64_t total, int64_t ntiles, int64_t &mt,
                                                 int64_t &nt) {
    const int64_t per = total / 8, rem = total % 8;
    const int64_t x = b % 8, slot = b / 8;
    const int64_t L = x * per + (x < rem ? x : rem) + slot;
    const int64_t MT = total / ntiles;
    const int64_t B = ntiles < kLfXcdGroup ? ntiles : kLfXcdGroup;
    const int64_t full = ntiles / B * B;
    const int64_t grp = L / (MT * B);
    if (grp * B < full) {
        const int64_t r = L - grp * MT * B;
        mt = r / B;
        nt = grp * B + r % B;
    } else {
        const int64_t Bt = ntiles - full;
        const int64_t r = L - full * MT;
        mt = r / Bt;
        nt = full + r % Bt;
    }
}

__global__ __launch_bounds__(kLfThreads, kLfWaves / 4) void lfull_tile_kernel(const LfArgs a) {
    __shared__ __attribute__((aligned(16))) uint8_t lds[kLfStages][kLfRows * 64];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: LDS addresses in SGPRs
    const int wm = wave % kLfWM, wn = wave / kLfWM;
    int64_t mt, nt;
    lf_tile_of_block(blockIdx.x, gridDim.x, a.ntiles, mt, nt);
    const int64_t t0 = mt * kLfBM, r0 = nt * kLfBN;
    const int stages = (int)(a.ldd / kLfBK);

    // A stage is loaded straight from global memory into LDS by buffer loads
    // (16 bytes per lane, 1 KB = 16 rows of the stage per load; lane l at row
    // 16 q + l / 4, position l % 4, fetching the chunk the swizzle stores
    // there).  One descriptor per block and operand: the token tile's X rows
    // (rows past `tokens` lie beyond the descriptor's range and read zeros),
    // the row tile's dW hi rows and lo rows (padded planes).  Per-lane
    // 32-bit offsets are fixed for the whole loop; a stage adds a uniform
    // offset.  X chunks past `in` (when in % 32 != 0) read the next row's
    // finite values or zeros, and meet zero dW columns.
    const int64_t xrow_bytes = a.in * 2, drow_bytes = a.ldd * 2;
    const int64_t valid_rows = a.tokens - t0 < kLfBM ? a.tokens - t0 : kLfBM;
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<u32x4 *>(a.X + t0 * (a.in / 8)), 0, (int)(valid_rows * xrow_bytes), kRawBufferWord3);
    const __amdgpu_buffer_rsrc_t rhi = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<u32x4 *>(a.hi + r0 * (a.ldd / 8)), 0, (int)(kLfBN * drow_bytes), kRawBufferWord3);
    const __amdgpu_buffer_rsrc_t rlo = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<u32x4 *>(a.lo + r0 * (a.ldd / 8)), 0, (int)(kLfBN * drow_bytes), kRawBufferWord3);
    uint32_t voff[kLfLoadsPerWave];
#pragma unroll
    for (int i = 0; i < kLfLoadsPerWave; ++i) {
        const int q = wave + i * kLfWaves;
        const int row = q * 16 + (lane >> 2);
        const int c = (lane & 3) ^ ((row >> 2) & 3);
        voff[i] = row < kLfBM ? (uint32_t)(row * xrow_bytes + c * 16)
                              : (uint32_t)(((row - kLfBM) % kLfBN) * drow_bytes + c * 16);
    }
    auto issue = [&](int s, int buf) {
        const uint32_t soff = (uint32_t)s * (kLfBK * 2);
#pragma unroll
        for (int i = 0; i < kLfLoadsPerWave; ++i) {
            const int q = wave + i * kLfWaves;
            if (q < kLfSlots) {
                auto *dst = (__attribute__((address_space(3))) void *)(lds[buf] + q * 1024);
                if (q < kLfBM / 16)
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, dst, 16, voff[i], soff, 0, 0);
                else if (q < (kLfBM + kLfBN) / 16)
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(rhi, dst, 16, voff[i], soff, 0, 0);
                else
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(rlo, dst, 16, voff[i], soff, 0, 0);
            }
        }
    };

    f32x16 acc[kLfMI][kLfNJ];
#pragma unroll
    for (int i = 0; i < kLfMI; ++i)
#pragma unroll
        for (int j = 0; j < kLfNJ; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

    // Two-buffer ring: stage s + 1 is issued once every wave has finished
    // reading stage s - 1 (the barrier), into that stage's buffer.  Each wave
    // first waits for its own loads of stage s (all its outstanding loads),
    // then the barrier makes all of stage s visible.  A plain s_barrier is
    // used: __syncthreads() adds a release fence that waits for every
    // outstanding load, the stage just issued included.
    issue(0, 0);
    for (int s = 0; s < stages; ++s) {
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
        asm volatile("s_barrier" ::: "memory");
        if (s + 1 < stages) issue(s + 1, (s + 1) % kLfStages);
        const uint8_t *base = lds[s % kLfStages];
#pragma unroll
        for (int kk = 0; kk < kLfBK / 16; ++kk) {
            const int c = 2 * kk + (lane >> 5);
            bf16x8 fa[kLfMI], fh[kLfNJ], fl[kLfNJ];
#pragma unroll
            for (int i = 0; i < kLfMI; ++i) {
                const int row = wm * (kLfBM / kLfWM) + i * 32 + (lane & 31);
                fa[i] = *reinterpret_cast<const bf16x8 *>(base + lf_lds_offset(row, c));
            }
#pragma unroll
            for (int j = 0; j < kLfNJ; ++j) {
                const int row = wn * (kLfBN / kLfWN) + j * 32 + (lane & 31);
                fh[j] = *reinterpret_cast<const bf16x8 *>(base + lf_lds_offset(kLfBM + row, c));
                fl[j] = *reinterpret_cast<const bf16x8 *>(base + lf_lds_offset(kLfBM + kLfBN + row, c));
            }
#pragma unroll
            for (int i = 0; i < kLfMI; ++i)
#pragma unroll
                for (int j = 0; j < kLfNJ; ++j) {
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fh[j], acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fl[j], acc[i][j], 0, 0, 0);
                }
        }
    }
    __syncthreads();

    // Column sums of squares: lane l holds column l % 32 of each 32x32
    // accumulator; lanes l and l + 32 share a column, and the kLfWM waves of
    // a column group share its columns (added in wm order).
    double sq[kLfNJ];
#pragma unroll
    for (int j = 0; j < kLfNJ; ++j) {
        double v = 0.0;
#pragma unroll
        for (int i = 0; i < kLfMI; ++i)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const double y = (double)acc[i][j][e];
                v = fma(y, y, v);
            }
        sq[j] = v + __shfl_xor(v, 32, 64);
    }
    double *red = reinterpret_cast<double *>(lds[0]);  // [kLfWM][kLfBN]
    if (lane < 32) {
#pragma unroll
        for (int j = 0; j < kLfNJ; ++j) red[wm * kLfBN + wn * (kLfBN / kLfWN) + j * 32 + lane] = sq[j];
    }
    __syncthreads();
    if (tid < kLfBN) {
        const int64_t col = r0 + tid;
        double v = red[tid];
#pragma unroll
        for (int w = 1; w < kLfWM; ++w) v += red[w * kLfBN + tid];
        if (col < a.out) a.partial[mt * a.out + col] = v;
    }
}

struct LfPlan {
    int64_t ldd = 0, rows_pad = 0, ntiles = 0, tiles_per_pass = 0;
    size_t plane_bytes = 0, partial_offset = 0, bytes = 0;
};

LfPlan lfull_plan(int64_t tokens, int64_t in, int64_t out) {
    LfPlan p;
    if (tokens <= 0 || in <= 0 || out <= 0) return p;
    p.ldd = (in + kLfBK - 1) / kLfBK * kLfBK;
    p.rows_pad = (out + kLfBN - 1) / kLfBN * kLfBN;
    p.ntiles = p.rows_pad / kLfBN;
    const int64_t tiles = (tokens + kLfBM - 1) / kLfBM;
    // A pass launches tiles_per_pass x ntiles blocks: at most kLfMaxTilesPerPass
    // token tiles, and never more blocks than a grid dimension holds.
    const int64_t grid_cap = INT_MAX / p.ntiles > 0 ? INT_MAX / p.ntiles : 1;
    const int64_t cap = grid_cap < kLfMaxTilesPerPass ? grid_cap : kLfMaxTilesPerPass;
    p.tiles_per_pass = tiles < cap ? tiles : cap;
    p.plane_bytes = round_up((size_t)p.rows_pad * (size_t)p.ldd * 2, 256);
    p.partial_offset = 2 * p.plane_bytes;
    p.bytes = p.partial_offset + (size_t)p.tiles_per_pass * (size_t)out * sizeof(double);
    return p;
}

int64_t summary_blocks(int64_t groups) { return groups > 0 ? (groups + kSumChunk - 1) / kSumChunk : 0; }

}  // namespace

extern "C" {

size_t hscale_shift_summary_workspace_bytes(int64_t groups, int32_t down, int32_t up) {
    if (groups <= 0 || down < 0 || up < 0 || down > kMaxWindow || up > kMaxWindow || groups > kMaxGroups) return 0;
    const size_t K = (size_t)(down + up + 1);
    return (size_t)summary_blocks(groups) * K * (3 * sizeof(double) + sizeof(uint32_t));
}

int hscale_shift_summary(const int8_t *shift, const float *err_best, const float *err_init, int64_t groups,
                         int32_t down, int32_t up, uint64_t *count, double *sum_init, double *sum_best,
                         double *sum_rel, void *workspace, size_t workspace_bytes, hipStream_t stream) {
    if (groups < 0 || groups > kMaxGroups) return HSCALE_ERR_SHAPE;
    if (down < 0 || up < 0 || down > kMaxWindow || up > kMaxWindow) return HSCALE_ERR_WINDOW;
    const int K = down + up + 1;
    if (!count || !sum_init || !sum_best || !sum_rel) return HSCALE_ERR_NULL;
    if (!aligned(count, 8) || !aligned(sum_init, 8) || !aligned(sum_best, 8) || !aligned(sum_rel, 8))
        return HSCALE_ERR_ALIGN;
    const size_t nk = (size_t)K * 8;
    const void *outs[4] = {count, sum_init, sum_best, sum_rel};
    for (int a = 0; a < 4; ++a)
        for (int b = a + 1; b < 4; ++b)
            if (overlaps(outs[a], nk, outs[b], nk)) return HSCALE_ERR_OVERLAP;
    const int64_t blocks = summary_blocks(groups);
    const size_t need = hscale_shift_summary_workspace_bytes(groups, down, up);
    if (groups > 0) {
        if (!shift || !err_best || !err_init) return HSCALE_ERR_NULL;
        if (!aligned(err_best, 4) || !aligned(err_init, 4)) return HSCALE_ERR_ALIGN;
        if (workspace_bytes < need) return HSCALE_ERR_WORKSPACE;
        if (!workspace) return HSCALE_ERR_NULL;
        if (!aligned(workspace, 8)) return HSCALE_ERR_ALIGN;
        const size_t g = (size_t)groups;
        const struct {
            const void *p;
            size_t n;
        } in_bufs[] = {{shift, g}, {err_best, g * 4}, {err_init, g * 4}, {workspace, need}};
        for (int a = 0; a < 4; ++a)
            for (const auto &b : in_bufs)
                if (overlaps(outs[a], nk, b.p, b.n)) return HSCALE_ERR_OVERLAP;
        for (int a = 0; a < 3; ++a)
            if (overlaps(workspace, need, in_bufs[a].p, in_bufs[a].n)) return HSCALE_ERR_OVERLAP;
    }
    double *part = static_cast<double *>(workspace);
    uint32_t *cnt = blocks > 0 ? reinterpret_cast<uint32_t *>(part + (size_t)blocks * K * 3) : nullptr;
    if (blocks > 0) {
        hipLaunchKernelGGL(shift_summary_partial, dim3((unsigned)blocks), dim3(kSumThreads), 0, stream, shift,
                           err_best, err_init, groups, down, up, part, cnt);
        if (launch_status() != HSCALE_OK) return HSCALE_ERR_HIP;
    }
    hipLaunchKernelGGL(shift_summary_final, dim3((unsigned)K), dim3(64), 0, stream, part, cnt, blocks, K, count,
                       sum_init, sum_best, sum_rel);
    return launch_status();
}

size_t hscale_output_error_workspace_bytes(int64_t tokens, int64_t in, int64_t out) {
    if (in % kGroup != 0 || in > kLfMaxIn || (in > 0 && out > kMaxGroups / (in / kGroup))) return 0;
    return lfull_plan(tokens, in, out).bytes;
}

int hscale_output_error(const void *X, int64_t tokens, int64_t in, const void *W, int64_t out, float global_scale,
                        const uint8_t *scale_codes, const uint8_t *packed_e2m1, double *row_err, void *workspace,
                        size_t workspace_bytes, hipStream_t stream) {
    if (tokens < 0 || in < 0 || out < 0 || in % kGroup != 0) return HSCALE_ERR_SHAPE;
    if (in > kLfMaxIn || (in > 0 && tokens > ((int64_t)1 << 46) / in)) return HSCALE_ERR_SHAPE;
    if (in > 0 && out > kMaxGroups / (in / kGroup)) return HSCALE_ERR_SHAPE;
    if (!scale_ok(global_scale)) return HSCALE_ERR_SCALE;
    if (tokens == 0 || in == 0 || out == 0) return HSCALE_OK;  // adds nothing
    if (!X || !W || !scale_codes || !packed_e2m1 || !row_err || !workspace) return HSCALE_ERR_NULL;
    if (!aligned(X, 16) || !aligned(W, 16) || !aligned(packed_e2m1, 8) || !aligned(row_err, 8) ||
        !aligned(workspace, 256))
        return HSCALE_ERR_ALIGN;
    const LfPlan p = lfull_plan(tokens, in, out);
    if (workspace_bytes < p.bytes) return HSCALE_ERR_WORKSPACE;
    const size_t nx = (size_t)tokens * (size_t)in * 2, nw = (size_t)out * (size_t)in * 2;
    const size_t nc = (size_t)out * (size_t)(in / kGroup), np = (size_t)out * (size_t)(in / 2);
    const size_t nr = (size_t)out * 8;
    const struct {
        const void *p;
        size_t n;
    } ins[] = {{X, nx}, {W, nw}, {scale_codes, nc}, {packed_e2m1, np}};
    for (const auto &b : ins)
        if (overlaps(row_err, nr, b.p, b.n) || overlaps(workspace, p.bytes, b.p, b.n)) return HSCALE_ERR_OVERLAP;
    if (overlaps(row_err, nr, workspace, p.bytes)) return HSCALE_ERR_OVERLAP;

    uint8_t *ws = static_cast<uint8_t *>(workspace);
    u32x4 *hi = reinterpret_cast<u32x4 *>(ws), *lo = reinterpret_cast<u32x4 *>(ws + p.plane_bytes);
    double *partial = reinterpret_cast<double *>(ws + p.partial_offset);
    hipLaunchKernelGGL(delta_split_kernel, dim3(grid_for(p.rows_pad * (p.ldd / kGroup), 256)), dim3(256), 0, stream,
                       static_cast<const u32x4 *>(W), out, in, global_scale, scale_codes,
                       reinterpret_cast<const uint2 *>(packed_e2m1), p.rows_pad, p.ldd, hi, lo);
    if (launch_status() != HSCALE_OK) return HSCALE_ERR_HIP;
    const int64_t pass_tokens = p.tiles_per_pass * kLfBM;
    for (int64_t t0 = 0; t0 < tokens; t0 += pass_tokens) {
        LfArgs a;
        a.tokens = tokens - t0 < pass_tokens ? tokens - t0 : pass_tokens;
        a.in = in;
        a.X = static_cast<const u32x4 *>(X) + t0 * (in / 8);
        a.hi = hi;
        a.lo = lo;
        a.ldd = p.ldd;
        a.out = out;
        a.ntiles = p.ntiles;
        a.partial = partial;
        const int64_t tiles = (a.tokens + kLfBM - 1) / kLfBM;
        hipLaunchKernelGGL(lfull_tile_kernel, dim3((unsigned)(tiles * p.ntiles)), dim3(kLfThreads), 0, stream, a);
        if (launch_status() != HSCALE_OK) return HSCALE_ERR_HIP;
        launch_tree<true>(partial, tiles, out, nullptr, row_err, stream);
        if (launch_status() != HSCALE_OK) return HSCALE_ERR_HIP;
    }
    return HSCALE_OK;
}

}  // extern "C"
