// H-Scale hot path for gfx950: the diagonal proxy h (Sec. 3.2, Eq. 4) and the
// per-group NVFP4 scale search (Sec. 3.3, Eq. 7, 9-13), behind the C ABI of
// include/hscale.h.
//
// Kernels
//   hdiag_partial  column sums of squares of bf16 X over one token slice.
//                  One wave covers 512 columns (16-byte loads, 8 columns per
//                  lane, a row segment of 1 KiB per wave); the four waves of
//                  a block interleave rows; 8 rows of loads are in flight per
//                  lane.  fp32 chains of at most 32 tokens fold into fp64; the
//                  block's four waves combine through LDS in a fixed order
//                  and one fp64 partial per (slice, column) goes to the
//                  caller's workspace.
//   hdiag_tree     fixed-order fp64 sum of the slice partials, one fp32 h per
//                  column.  No atomics: results are bit-identical run to run.
//   search         one 16-weight group per lane, lanes over consecutive
//                  groups (a wave reads 2 KiB of W contiguously and writes
//                  512 contiguous bytes of codes).  The 126-entry table of
//                  (S[c], R[c]) lives in LDS.  Per candidate: 16 fp32
//                  products w R, 8 hardware E2M1 down-conversions (packed
//                  nibbles with sign, round-to-nearest-even, saturating at 6),
//                  8 up-conversions back to grid values, 16 residual FMAs
//                  w - v S (one rounding each) and a 4x4 fp32 accumulation of
//                  h r^2.  The best candidate's packed nibbles are kept, so
//                  the final re-quantization costs nothing extra.
//
// The fp32 operations below are the fixed arithmetic of the header: IEEE
// round-to-nearest-even products, correctly rounded divisions (built with
// -fhip-fp32-correctly-rounded-divide-sqrt), explicit fmaf, and no implicit
// contraction (-ffp-contract=off).

#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstdint>
#include <cstring>

#include "hscale.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kGroup = 16;
constexpr int kMaxCode = 126;  // positive finite E4M3FN codes are 1..126
constexpr int kMaxWindow = 125;

// ---------------------------------------------------------------------------
// hdiag
// ---------------------------------------------------------------------------
constexpr int kHdThreads = 256;
constexpr int kHdWaves = kHdThreads / 64;
constexpr int kHdLaneCols = 8;                 // bf16 per 16-byte load
constexpr int kHdTileCols = 64 * kHdLaneCols;  // 512 columns per block
constexpr int kHdChunk = 32;                   // fp32 chain length per lane
constexpr int kHdUnroll = 8;                   // row loads in flight per lane
// Grid size: as many blocks as MI355X keeps resident at once (256 CUs x 7
// blocks of 4 waves at this kernel's 68 VGPRs), so the whole grid runs in
// one round with no tail.  The plan depends only on (tokens, in), which
// keeps results identical from run to run.
constexpr int kHdTargetBlocks = 1792;
constexpr int64_t kHdMinSliceTokens = 256;

struct HdiagPlan {
    int64_t tiles = 0;
    int64_t slices = 0;
    int64_t slice_tokens = 0;
};

HdiagPlan hdiag_plan(int64_t tokens, int64_t in) {
    HdiagPlan p;
    if (tokens <= 0 || in <= 0) return p;
    p.tiles = (in + kHdTileCols - 1) / kHdTileCols;
    int64_t slices = kHdTargetBlocks / p.tiles;
    int64_t max_slices = (tokens + kHdMinSliceTokens - 1) / kHdMinSliceTokens;
    if (slices > max_slices) slices = max_slices;
    if (slices < 1) slices = 1;
    p.slice_tokens = (tokens + slices - 1) / slices;
    p.slices = (tokens + p.slice_tokens - 1) / p.slice_tokens;
    return p;
}

__device__ __forceinline__ void hd_accumulate(float (&acc)[kHdLaneCols], const u32x4 &v) {
    const uint32_t d[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const float lo = __uint_as_float(d[k] << 16);
        const float hi = __uint_as_float(d[k] & 0xFFFF0000u);
        acc[2 * k] = fmaf(lo, lo, acc[2 * k]);
        acc[2 * k + 1] = fmaf(hi, hi, acc[2 * k + 1]);
    }
}

__device__ __forceinline__ void hd_fold(float (&acc)[kHdLaneCols], double (&acc64)[kHdLaneCols]) {
#pragma unroll
    for (int k = 0; k < kHdLaneCols; ++k) {
        acc64[k] += (double)acc[k];
        acc[k] = 0.0f;
    }
}

__global__ __launch_bounds__(kHdThreads) void hdiag_partial(const u32x4 *__restrict__ X, int64_t tokens,
                                                            int64_t in, int64_t slice_tokens,
                                                            double *__restrict__ partial) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t col = (int64_t)blockIdx.x * kHdTileCols + (int64_t)lane * kHdLaneCols;
    const int64_t slice = blockIdx.y;
    const int64_t t0 = slice * slice_tokens;
    int64_t t1 = t0 + slice_tokens;
    if (t1 > tokens) t1 = tokens;

    double acc64[kHdLaneCols];
    float acc[kHdLaneCols];
#pragma unroll
    for (int k = 0; k < kHdLaneCols; ++k) {
        acc64[k] = 0.0;
        acc[k] = 0.0f;
    }

    if (col < in) {
        const int64_t vec_per_row = in / kHdLaneCols;
        // This wave's rows: t0 + wave, t0 + wave + 4, ... < t1.
        const int64_t first = t0 + wave;
        const int64_t rows = first < t1 ? (t1 - first + kHdWaves - 1) / kHdWaves : 0;
        const u32x4 *p = X + (rows > 0 ? first * vec_per_row + col / kHdLaneCols : 0);
        const int64_t stride = (int64_t)kHdWaves * vec_per_row;
        int64_t r = 0;
        int since_fold = 0;
        for (; r + kHdUnroll <= rows; r += kHdUnroll) {
            u32x4 v[kHdUnroll];
#pragma unroll
            for (int u = 0; u < kHdUnroll; ++u) v[u] = __builtin_nontemporal_load(p + (r + u) * stride);
#pragma unroll
            for (int u = 0; u < kHdUnroll; ++u) hd_accumulate(acc, v[u]);
            since_fold += kHdUnroll;
            if (since_fold == kHdChunk) {
                hd_fold(acc, acc64);
                since_fold = 0;
            }
        }
        for (; r < rows; ++r) {
            const u32x4 v = __builtin_nontemporal_load(p + r * stride);
            hd_accumulate(acc, v);
        }
        hd_fold(acc, acc64);
    }

    // Combine the four waves' column sums in a fixed order.
    __shared__ double red[kHdWaves][kHdTileCols];
#pragma unroll
    for (int k = 0; k < kHdLaneCols; ++k) red[wave][lane * kHdLaneCols + k] = acc64[k];
    __syncthreads();
    const int c = threadIdx.x * 2;  // two columns per thread
    const int64_t gcol = (int64_t)blockIdx.x * kHdTileCols + c;
    if (gcol < in) {
        double2 s;
        s.x = ((red[0][c] + red[1][c]) + red[2][c]) + red[3][c];
        s.y = ((red[0][c + 1] + red[1][c + 1]) + red[2][c + 1]) + red[3][c + 1];
        *reinterpret_cast<double2 *>(partial + slice * in + gcol) = s;
    }
}

constexpr int kTreeCols = 64;
constexpr int kTreeLanes = 4;

// Sums the slice partials of each column in a fixed order: lane q of a
// column adds slices q, q + 4, ...; the four lane sums combine as
// ((s0 + s1) + s2) + s3.  kAccumulate adds the sum to an fp64 accumulator
// instead of writing fp32 h.
template <bool kAccumulate>
__global__ __launch_bounds__(kTreeCols *kTreeLanes) void hdiag_tree(const double *__restrict__ partial,
                                                                     int64_t slices, int64_t in,
                                                                     float *__restrict__ h,
                                                                     double *__restrict__ h64) {
    const int lane = threadIdx.x % kTreeCols;
    const int q = threadIdx.x / kTreeCols;
    const int64_t col = (int64_t)blockIdx.x * kTreeCols + lane;
    double s = 0.0;
    if (col < in) {
        for (int64_t k = q; k < slices; k += kTreeLanes) s += partial[k * in + col];
    }
    __shared__ double red[kTreeLanes][kTreeCols];
    red[q][lane] = s;
    __syncthreads();
    if (q == 0 && col < in) {
        const double total = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
        if (kAccumulate)
            h64[col] += total;
        else
            h[col] = (float)total;
    }
}

__global__ __launch_bounds__(256) void hdiag_finalize_kernel(const double *__restrict__ h64, int64_t in,
                                                             float *__restrict__ h) {
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (j < in) h[j] = (float)h64[j];
}

// ---------------------------------------------------------------------------
// Formats
// ---------------------------------------------------------------------------

// Value of a positive E4M3FN code byte c (1..126), exact in fp32:
// exponent field 0 is subnormal (m * 2^-9), otherwise (8 + m) * 2^(e - 10).
__device__ __forceinline__ float e4m3fn_value(int c) {
    const int e = c >> 3;
    const int m = c & 7;
    return e == 0 ? (float)m * 0x1p-9f : __uint_as_float((uint32_t)((e + 120) << 23) | ((uint32_t)m << 20));
}

// E4M3FN code of a non-negative fp32 t: round to nearest, ties to the even
// code, saturating at 448; then clipped to 1..126 (a zero or underflowing
// group starts at the smallest code).
__device__ __forceinline__ int e4m3fn_code_clipped(float t) {
    // Below 2^-6 the grid is the multiples of 2^-9: t * 512 is exact.
    const int sub = (int)__builtin_rintf(t * 512.0f);
    // Otherwise round the fp32 pattern to 3 mantissa bits (a carry moves into
    // the exponent) and rebias the exponent from 127 to 7.
    const uint32_t u = __float_as_uint(t);
    const int nrm = (int)((u + 0x7FFFFu + ((u >> 20) & 1u)) >> 20) - (120 << 3);
    const int c = t < 0x1p-6f ? sub : nrm;
    return min(max(c, 1), kMaxCode);
}

struct ScaleEntry {
    float S;  // fp32(s_g * l_c)
    float R;  // fp32(1 / S)
};

// The search indexes its table by c0 + d + kTabPad with no clamp: entries
// below kTabPad + 1 hold code 1 and entries above kTabPad + 126 hold code 126,
// which is the clip of Eq. 10.  c0 is in 1..126 and |d| <= 125, so the index
// stays in 1..376.
constexpr int kTabPad = kMaxWindow;
constexpr int kTabSize = 384;

// Fills a padded LDS table: tab[t] = (S, R) of code clip(t - kTabPad, 1, 126).
// The 126 distinct entries are computed once (one correctly rounded
// reciprocal each) into `uniq`, then copied out.  Needs blockDim.x >= 128.
__device__ __forceinline__ void build_scale_table(ScaleEntry *tab, ScaleEntry *uniq, float s_g) {
    const int c = threadIdx.x;
    if (c >= 1 && c <= kMaxCode) {
        const float S = s_g * e4m3fn_value(c);
        uniq[c] = ScaleEntry{S, 1.0f / S};
    }
    __syncthreads();
    for (int t = threadIdx.x; t < kTabSize; t += blockDim.x) tab[t] = uniq[min(max(t - kTabPad, 1), kMaxCode)];
    __syncthreads();
}

__device__ __forceinline__ void load_group(const u32x4 *__restrict__ W, int64_t g, float (&w)[kGroup]) {
    const u32x4 a = __builtin_nontemporal_load(W + 2 * g);
    const u32x4 b = __builtin_nontemporal_load(W + 2 * g + 1);
    const uint32_t d[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        w[2 * k] = __uint_as_float(d[k] << 16);
        w[2 * k + 1] = __uint_as_float(d[k] & 0xFFFF0000u);
    }
}

// Packed E2M1 codes of 16 weights at reciprocal scale R: two 32-bit words,
// element 2k in the low nibble of byte k.  The hardware conversion rounds to
// nearest even, saturates at 6 and keeps the sign (scale operand 1.0: no
// extra scaling).
__device__ __forceinline__ uint2 quantize_group(const float (&w)[kGroup], float R, uint2 old) {
    // Every byte of both words is overwritten, so `old` only saves a move.
    uint32_t p0 = old.x, p1 = old.y;
    p0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p0, w[0] * R, w[1] * R, 1.0f, 0);
    p0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p0, w[2] * R, w[3] * R, 1.0f, 1);
    p0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p0, w[4] * R, w[5] * R, 1.0f, 2);
    p0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p0, w[6] * R, w[7] * R, 1.0f, 3);
    p1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p1, w[8] * R, w[9] * R, 1.0f, 0);
    p1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p1, w[10] * R, w[11] * R, 1.0f, 1);
    p1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p1, w[12] * R, w[13] * R, 1.0f, 2);
    p1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p1, w[14] * R, w[15] * R, 1.0f, 3);
    return make_uint2(p0, p1);
}

// Adds the h-weighted squared residuals of elements 2K and 2K + 1 (byte K & 3
// of word `src`) to the chains e[(2K) & 3] and e[(2K + 1) & 3].  Residuals
// w - v S are single-rounding FMAs.
template <int K>
__device__ __forceinline__ void accumulate_pair(const float (&w)[kGroup], const float (&hh)[kGroup], uint32_t src,
                                                float S, float (&e)[4]) {
    const auto v = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(src, 1.0f, K & 3);
    constexpr int j0 = 2 * K, j1 = 2 * K + 1;
    const float r0 = fmaf(-v[0], S, w[j0]);
    const float r1 = fmaf(-v[1], S, w[j1]);
    e[j0 & 3] = fmaf(hh[j0] * r0, r0, e[j0 & 3]);
    e[j1 & 3] = fmaf(hh[j1] * r1, r1, e[j1 & 3]);
}

// h-weighted squared error sum_j h_j (w_j - v_j S)^2 of a packed group: the
// 16 terms go into 4 fp32 chains of 4 (j = q, q + 4, q + 8, q + 12),
// combined as (e0 + e1) + (e2 + e3).
__device__ __forceinline__ float group_error(const float (&w)[kGroup], const float (&hh)[kGroup], uint2 p,
                                             float S) {
    float e[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    accumulate_pair<0>(w, hh, p.x, S, e);
    accumulate_pair<1>(w, hh, p.x, S, e);
    accumulate_pair<2>(w, hh, p.x, S, e);
    accumulate_pair<3>(w, hh, p.x, S, e);
    accumulate_pair<4>(w, hh, p.y, S, e);
    accumulate_pair<5>(w, hh, p.y, S, e);
    accumulate_pair<6>(w, hh, p.y, S, e);
    accumulate_pair<7>(w, hh, p.y, S, e);
    return (e[0] + e[1]) + (e[2] + e[3]);
}

constexpr int kSearchThreads = 256;

// How the walk's initial code c0 is chosen (values of the C ABI's init_mode).
enum InitMode : int { kInitMaxAbs = 0, kInitFourOverSix = 1, kInitGiven = 2 };

// Adds the squared residuals of elements 2K and 2K + 1 to the plain-error
// chains (the 4over6 anchor score has no h).
template <int K>
__device__ __forceinline__ void accumulate_pair_plain(const float (&w)[kGroup], uint32_t src, float S,
                                                      float (&e)[4]) {
    const auto v = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(src, 1.0f, K & 3);
    constexpr int j0 = 2 * K, j1 = 2 * K + 1;
    const float r0 = fmaf(-v[0], S, w[j0]);
    const float r1 = fmaf(-v[1], S, w[j1]);
    e[j0 & 3] = fmaf(r0, r0, e[j0 & 3]);
    e[j1 & 3] = fmaf(r1, r1, e[j1 & 3]);
}

// Plain squared error sum_j (w_j - v_j S)^2 of a packed group: single-rounding
// residuals, 4 fp32 chains of 4.
__device__ __forceinline__ float group_plain_error(const float (&w)[kGroup], uint2 p, float S) {
    float e[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    accumulate_pair_plain<0>(w, p.x, S, e);
    accumulate_pair_plain<1>(w, p.x, S, e);
    accumulate_pair_plain<2>(w, p.x, S, e);
    accumulate_pair_plain<3>(w, p.x, S, e);
    accumulate_pair_plain<4>(w, p.y, S, e);
    accumulate_pair_plain<5>(w, p.y, S, e);
    accumulate_pair_plain<6>(w, p.y, S, e);
    accumulate_pair_plain<7>(w, p.y, S, e);
    return (e[0] + e[1]) + (e[2] + e[3]);
}

// Initial code of Eq. 7 from max|w| and an anchor (6 for max-abs; 4 or 6 for
// 4over6): fp32(amax / anchor), then fp32(. / s_g), then Q_fp8 and the clip.
__device__ __forceinline__ int anchor_code(float amax, float anchor, float s_g) {
    const float s_init = amax / anchor;
    return e4m3fn_code_clipped(s_init / s_g);
}

// Eq. 7 and 9-13 for one group held in registers: the initial code (by the
// rule kInit; `given` is the caller's code for kInitGiven), then the walk
// d = -down..up in pairs, keeping the first minimum.  With kStats it also
// reports the chosen shift, its error and the error at d = 0.
template <int kInit, bool kStats>
__device__ __forceinline__ void search_group(const float (&w)[kGroup], const float (&hh)[kGroup],
                                             const ScaleEntry *tab, int down, int up, float s_g, int given,
                                             int &code, uint2 &best_p, int &shift, float &err_best,
                                             float &err_init) {
    int c0;
    if (kInit == kInitGiven) {
        c0 = min(max(given, 1), kMaxCode);
    } else {
        float amax = 0.0f;
#pragma unroll
        for (int j = 0; j < kGroup; ++j) amax = fmaxf(amax, fabsf(w[j]));
        c0 = anchor_code(amax, 6.0f, s_g);
        if (kInit == kInitFourOverSix) {
            // Anchor 4 (amax / 4 is exact) against anchor 6 by plain squared
            // error; anchor 4 on a tie.
            const int c4 = anchor_code(amax, 4.0f, s_g);
            const ScaleEntry e4 = tab[c4 + kTabPad];
            const ScaleEntry e6 = tab[c0 + kTabPad];
            const float l4 = group_plain_error(w, quantize_group(w, e4.R, make_uint2(0u, 0u)), e4.S);
            const float l6 = group_plain_error(w, quantize_group(w, e6.R, make_uint2(0u, 0u)), e6.S);
            if (l4 <= l6) c0 = c4;
        }
    }
    const ScaleEntry *col = tab + (c0 + kTabPad);  // col[d] is candidate c0 + d, clipped
    float best_e = 0.0f, e_init = 0.0f;
    int best_d = -down;
    best_p = make_uint2(0u, 0u);
    // Scratch words the conversions rewrite in place (all 8 bytes each time),
    // carried across iterations so no register copies are needed.
    uint2 pa = best_p, pb = best_p;
    int d = -down;
    for (; d < up; d += 2) {
        const ScaleEntry sa = col[d];
        const ScaleEntry sb = col[d + 1];
        pa = quantize_group(w, sa.R, pa);
        pb = quantize_group(w, sb.R, pb);
        const float ea = group_error(w, hh, pa, sa.S);
        const float eb = group_error(w, hh, pb, sb.S);
        if (kStats) {
            if (d == 0) e_init = ea;
            if (d + 1 == 0) e_init = eb;
        }
        if (d == -down || ea < best_e) {
            best_e = ea;
            best_d = d;
            best_p = pa;
        }
        if (eb < best_e) {
            best_e = eb;
            best_d = d + 1;
            best_p = pb;
        }
    }
    if (d == up) {  // odd candidate count: the last one
        const ScaleEntry se = col[d];
        pa = quantize_group(w, se.R, pa);
        const float e = group_error(w, hh, pa, se.S);
        if (kStats && d == 0) e_init = e;
        if (d == -down || e < best_e) {
            best_e = e;
            best_d = d;
            best_p = pa;
        }
    }
    code = min(max(c0 + best_d, 1), kMaxCode);
    shift = best_d;
    err_best = best_e;
    err_init = e_init;
}

// Arguments of a search over a block of `rows` x (16 Gc) weights inside
// larger row-major arrays.  Group (r, i) reads W at r * ldw + 16 i bf16
// elements (ldw_vec counts 16-byte vectors), h at 16 i, the initial code at
// r * ldi + i, and writes its code at r * ldc + i and its packed nibbles at
// r * ldp + 8 i bytes (ldp_vec counts 8-byte words).
struct SearchArgs {
    const u32x4 *W;
    uint64_t ldw_vec;
    const float4 *h;
    uint32_t num_groups;  // rows * Gc
    uint32_t Gc;          // groups per row
    int down, up;
    float s_g;
    const uint8_t *init;
    uint64_t ldi;
    uint8_t *codes;
    uint64_t ldc;
    uint2 *packed;
    uint64_t ldp_vec;
    int8_t *shift;    // statistics, [rows * Gc] at index g (kStats only)
    float *err_best;
    float *err_init;
};

// One group per lane over the flat index g = r * Gc + i of the block, so the
// lanes of a wave cover consecutive groups of a row (contiguous loads and
// stores) and a lane's h slice is h[16 i .. 16 i + 15].  A launch normally
// covers every group once; larger problems loop with a grid stride.
template <int kInit, bool kStats>
__global__ __launch_bounds__(kSearchThreads) void search_kernel(const SearchArgs a) {
    __shared__ ScaleEntry tab[kTabSize];
    __shared__ ScaleEntry uniq[kMaxCode + 1];
    build_scale_table(tab, uniq, a.s_g);

    const uint32_t stride = gridDim.x * kSearchThreads;
    const uint32_t first = blockIdx.x * kSearchThreads;  // wave-uniform
    uint32_t g = first + threadIdx.x;
    if (g >= a.num_groups) return;
    // (r, i) of g from the uniform block offset: at most one wrap per row
    // crossed inside the block.
    uint32_t r = first / a.Gc;
    uint32_t i = first % a.Gc + threadIdx.x;
    while (i >= a.Gc) {
        i -= a.Gc;
        ++r;
    }
    const uint32_t step_r = stride / a.Gc, step_i = stride % a.Gc;

    for (;;) {
        float w[kGroup];
        const u32x4 *src = a.W + (uint64_t)r * a.ldw_vec + 2 * (uint64_t)i;
        load_group(src, 0, w);
        float hh[kGroup];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 v = a.h[4 * (uint64_t)i + q];
            hh[4 * q] = v.x;
            hh[4 * q + 1] = v.y;
            hh[4 * q + 2] = v.z;
            hh[4 * q + 3] = v.w;
        }
        const int given = kInit == kInitGiven ? (int)a.init[(uint64_t)r * a.ldi + i] : 0;
        int code, shift;
        uint2 best_p;
        float e_best, e_init;
        search_group<kInit, kStats>(w, hh, tab, a.down, a.up, a.s_g, given, code, best_p, shift, e_best, e_init);
        a.codes[(uint64_t)r * a.ldc + i] = (uint8_t)code;
        a.packed[(uint64_t)r * a.ldp_vec + i] = best_p;
        if (kStats) {
            a.shift[g] = (int8_t)shift;
            a.err_best[g] = e_best;
            a.err_init[g] = e_init;
        }

        if (a.num_groups - g <= stride) break;
        g += stride;
        r += step_r;
        i += step_i;
        if (i >= a.Gc) {
            i -= a.Gc;
            ++r;
        }
    }
}

__global__ __launch_bounds__(kSearchThreads) void quantize_kernel(const u32x4 *__restrict__ W,
                                                                  int64_t num_groups, float s_g,
                                                                  const uint8_t *__restrict__ codes,
                                                                  uint2 *__restrict__ packed) {
    __shared__ ScaleEntry tab[kTabSize];
    __shared__ ScaleEntry uniq[kMaxCode + 1];
    build_scale_table(tab, uniq, s_g);
    const int64_t stride = (int64_t)gridDim.x * kSearchThreads;
    for (int64_t g = (int64_t)blockIdx.x * kSearchThreads + threadIdx.x; g < num_groups; g += stride) {
        float w[kGroup];
        load_group(W, g, w);
        const int c = min(max((int)codes[g], 1), kMaxCode);
        packed[g] = quantize_group(w, tab[c + kTabPad].R, make_uint2(0u, 0u));
    }
}

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
// MFMA products accumulated in fp32.  Each block computes a 256-token x
// 128-row tile of X dW^T in registers and reduces the squares of its columns
// in fp64; the tile is never written.  Per-tile column sums go to a
// workspace and a fixed-order tree adds them to row_err.
// ---------------------------------------------------------------------------

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Tile of X dW^T per block: kLfBM tokens x kLfBN weight rows, computed by
// kLfWM x kLfWN waves (each a (kLfBM / kLfWM) x (kLfBN / kLfWN) sub-tile of
// 32 x 32 MFMA accumulators).
constexpr int kLfBM = 256;
constexpr int kLfBN = 256;
constexpr int kLfWM = 2;
constexpr int kLfWN = 4;
constexpr int kLfBK = 32;  // k per LDS stage (two 16-deep MFMA steps)
constexpr int kLfThreads = 64 * kLfWM * kLfWN;
constexpr int kLfMI = kLfBM / kLfWM / 32;  // accumulator tiles per wave, token direction
constexpr int kLfNJ = kLfBN / kLfWN / 32;  // accumulator tiles per wave, weight-row direction
constexpr int kLfRows = kLfBM + 2 * kLfBN;  // LDS rows of 64 bytes per stage (X, dW hi, dW lo)
constexpr int kLfStages = 3;                // LDS ring depth: two stages in flight while one is used
constexpr int kLfWaves = kLfThreads / 64;
constexpr int kLfDmaPerWave = kLfRows / 16 / kLfWaves;  // 1 KB direct-to-LDS loads per wave per stage
static_assert(kLfRows % (16 * kLfWaves) == 0 && kLfBM % 16 == 0 && kLfBN % 16 == 0, "stage split");
static_assert(kLfStages * kLfRows * 64 <= 160 * 1024, "LDS ring exceeds the CU's 160 KB");
constexpr int64_t kLfMaxTilesPerPass = 1024;  // token tiles per tile launch (bounds the workspace)

__device__ __forceinline__ uint32_t bf16_bits_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;  // finite inputs
}

// dW of one 16-weight group, split into hi / lo bf16 planes of row stride
// ldd; groups beyond (out, in) in the padded planes are written as zeros, and
// so are the 256 bytes at `zero` (the source of out-of-range X chunks).
__global__ __launch_bounds__(256) void delta_split_kernel(const u32x4 *__restrict__ W, int64_t out, int64_t in,
                                                          float s_g, const uint8_t *__restrict__ codes,
                                                          const uint2 *__restrict__ packed, int64_t rows_pad,
                                                          int64_t ldd, u32x4 *__restrict__ hi,
                                                          u32x4 *__restrict__ lo, u32x4 *__restrict__ zero) {
    if (blockIdx.x == 0 && threadIdx.x < 16) zero[threadIdx.x] = u32x4{0u, 0u, 0u, 0u};
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
    double *partial;    // [token tiles of the pass, out]
    const u32x4 *zero;  // 16 zero bytes, read for chunks outside X
};

__global__ __launch_bounds__(kLfThreads) void lfull_tile_kernel(const LfArgs a) {
    __shared__ __attribute__((aligned(16))) uint8_t lds[kLfStages][kLfRows * 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % kLfWM, wn = wave / kLfWM;
    const int64_t mt = blockIdx.x / a.ntiles, nt = blockIdx.x % a.ntiles;
    const int64_t t0 = mt * kLfBM, r0 = nt * kLfBN;
    const int64_t xrow_vec = a.in / 8, drow_vec = a.ldd / 8;
    const int stages = (int)(a.ldd / kLfBK);

    // A stage is filled straight from global memory into LDS: each wave
    // issues kLfDmaPerWave 16-byte-per-lane loads, each landing in 1 KB
    // (16 rows) of the stage, lane l at row 16 kb + l / 4, position l % 4;
    // the lane fetches the chunk that the swizzle stores at that position.
    // Rows below kLfBM are X (out-of-range chunks read zeros), then dW hi,
    // dW lo (padded planes, always in range).
    auto issue = [&](int s, int buf) {
        const int64_t kvec = (int64_t)s * (kLfBK / 8);
#pragma unroll
        for (int i = 0; i < kLfDmaPerWave; ++i) {
            const int kb = wave + i * kLfWaves;
            const int row = kb * 16 + (lane >> 2);
            const int c = (lane & 3) ^ ((row >> 2) & 3);
            const u32x4 *src;
            if (kb < kLfBM / 16) {
                const int64_t t = t0 + row, kv = kvec + c;
                src = (t < a.tokens && kv < xrow_vec) ? a.X + t * xrow_vec + kv : a.zero;
            } else {
                const int rb = row - kLfBM;
                const u32x4 *plane = rb < kLfBN ? a.hi : a.lo;
                src = plane + (r0 + rb % kLfBN) * drow_vec + kvec + c;
            }
            __builtin_amdgcn_global_load_lds(static_cast<const void *>(src),
                                             (__attribute__((address_space(3))) void *)(lds[buf] + kb * 1024), 16,
                                             0, 0);
        }
    };

    f32x16 acc[kLfMI][kLfNJ];
#pragma unroll
    for (int i = 0; i < kLfMI; ++i)
#pragma unroll
        for (int j = 0; j < kLfNJ; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

    // Ring of kLfStages buffers: stage s + 2 is issued once every wave has
    // finished reading stage s - 1 (the barrier), into that stage's buffer.
    // Each wave first waits for its own loads of stage s (vmcnt counts them in
    // issue order; the kLfDmaPerWave loads of stage s + 1 may stay in
    // flight); the barrier then makes all of stage s visible.  A plain
    // s_barrier is used: __syncthreads() adds a release fence that waits for
    // every outstanding load, stage s + 1's included.
    issue(0, 0);
    if (stages > 1) issue(1, 1);
    for (int s = 0; s < stages; ++s) {
        if (s + 1 < stages)
            __builtin_amdgcn_s_waitcnt(waitcnt_vm(kLfDmaPerWave));
        else
            __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
        asm volatile("s_barrier" ::: "memory");
        if (s + 2 < stages) issue(s + 2, (s + 2) % kLfStages);
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

// ---------------------------------------------------------------------------
// Host side: validation and launch
// ---------------------------------------------------------------------------

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

bool overlaps(const void *a, size_t na, const void *b, size_t nb) {
    if (na == 0 || nb == 0) return false;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + nb && b0 < a0 + na;
}

// True when s_g keeps every S[c] a finite normal fp32 with a finite
// reciprocal: s_g * 2^-9 >= 2^-126 and s_g * 448 < 2^128.
bool scale_ok(float s_g) {
    if (!std::isfinite(s_g) || !(s_g > 0.0f)) return false;
    const double lo = (double)s_g * std::ldexp(1.0, -9);
    const double hi = (double)s_g * 448.0;
    return lo >= std::ldexp(1.0, -126) && hi < std::ldexp(1.0, 128) * (1.0 - std::ldexp(1.0, -25));
}

// The search indexes groups with 32-bit arithmetic.
constexpr int64_t kMaxGroups = ((int64_t)1 << 32) - 1;

int grid_for(int64_t groups) {
    // Enough blocks to fill every CU several times over; the grid-stride loop
    // covers the rest and amortises the per-block table.
    int64_t blocks = (groups + kSearchThreads - 1) / kSearchThreads;
    const int64_t cap = 65536;
    if (blocks > cap) blocks = cap;
    if (blocks < 1) blocks = 1;
    return (int)blocks;
}

int launch_status() { return hipGetLastError() == hipSuccess ? HSCALE_OK : HSCALE_ERR_HIP; }

// Bytes spanned by `rows` rows of `width` elements at a row stride of `ld`
// elements of `elem` bytes each.
size_t span(int64_t rows, int64_t ld, int64_t width, size_t elem) {
    if (rows <= 0 || width <= 0) return 0;
    return ((size_t)(rows - 1) * (size_t)ld + (size_t)width) * elem;
}

int search_block(const void *W, int64_t ldw, int64_t out, int64_t cols, const float *h, int32_t down, int32_t up,
                 float s_g, int32_t init_mode, const uint8_t *init_codes, int64_t ldi, uint8_t *codes, int64_t ldc,
                 uint8_t *packed, int64_t ldp, hipStream_t stream, int8_t *shift = nullptr,
                 float *err_best = nullptr, float *err_init = nullptr) {
    const bool stats = shift || err_best || err_init;
    if (out < 0 || cols < 0 || cols % kGroup != 0) return HSCALE_ERR_SHAPE;
    const int64_t Gc = cols / kGroup;
    if (out > 0 && cols > 0 && out > kMaxGroups / Gc) return HSCALE_ERR_SHAPE;
    if (init_mode < kInitMaxAbs || init_mode > kInitGiven) return HSCALE_ERR_SHAPE;
    if (down < 0 || up < 0 || down > kMaxWindow || up > kMaxWindow) return HSCALE_ERR_WINDOW;
    if (!scale_ok(s_g)) return HSCALE_ERR_SCALE;
    if (out == 0 || cols == 0) return HSCALE_OK;
    if (ldw < cols || ldc < Gc || ldp < cols / 2 || (init_mode == kInitGiven && ldi < Gc)) return HSCALE_ERR_SHAPE;
    if (!W || !h || !codes || !packed || (init_mode == kInitGiven && !init_codes)) return HSCALE_ERR_NULL;
    if (stats && (!shift || !err_best || !err_init)) return HSCALE_ERR_NULL;
    if (!aligned(W, 16) || ldw % 8 != 0 || !aligned(h, 16) || !aligned(packed, 8) || ldp % 8 != 0)
        return HSCALE_ERR_ALIGN;
    if (stats && (!aligned(err_best, 4) || !aligned(err_init, 4))) return HSCALE_ERR_ALIGN;
    const size_t nw = span(out, ldw, cols, 2), nh = (size_t)cols * 4;
    const size_t nc = span(out, ldc, Gc, 1), np = span(out, ldp, cols / 2, 1);
    if (overlaps(codes, nc, W, nw) || overlaps(codes, nc, h, nh) || overlaps(packed, np, W, nw) ||
        overlaps(packed, np, h, nh) || overlaps(codes, nc, packed, np))
        return HSCALE_ERR_OVERLAP;
    if (init_mode == kInitGiven) {
        // The codes may be refined in place (init_codes == scale_codes with
        // the same stride: each group reads its own byte before writing it).
        const size_t ni = span(out, ldi, Gc, 1);
        const bool in_place = init_codes == codes && ldi == ldc;
        if ((!in_place && overlaps(init_codes, ni, codes, nc)) || overlaps(init_codes, ni, packed, np))
            return HSCALE_ERR_OVERLAP;
    }
    if (stats) {
        // Every statistics array is written: none may overlap another buffer.
        const size_t groups = (size_t)out * (size_t)Gc;
        const struct {
            const void *p;
            size_t n;
        } in_bufs[] = {{W, nw}, {h, nh}, {codes, nc}, {packed, np},
                       {init_codes, init_mode == kInitGiven ? span(out, ldi, Gc, 1) : 0}},
          st[] = {{shift, groups}, {err_best, groups * 4}, {err_init, groups * 4}};
        for (const auto &a : st) {
            for (const auto &b : in_bufs)
                if (b.n && overlaps(a.p, a.n, b.p, b.n)) return HSCALE_ERR_OVERLAP;
        }
        if (overlaps(shift, groups, err_best, groups * 4) || overlaps(shift, groups, err_init, groups * 4) ||
            overlaps(err_best, groups * 4, err_init, groups * 4))
            return HSCALE_ERR_OVERLAP;
    }
    SearchArgs a;
    a.W = static_cast<const u32x4 *>(W);
    a.ldw_vec = (uint64_t)ldw / 8;
    a.h = reinterpret_cast<const float4 *>(h);
    a.num_groups = (uint32_t)(out * Gc);
    a.Gc = (uint32_t)Gc;
    a.down = down;
    a.up = up;
    a.s_g = s_g;
    a.init = init_codes;
    a.ldi = (uint64_t)ldi;
    a.codes = codes;
    a.ldc = (uint64_t)ldc;
    a.packed = reinterpret_cast<uint2 *>(packed);
    a.ldp_vec = (uint64_t)ldp / 8;
    a.shift = shift;
    a.err_best = err_best;
    a.err_init = err_init;
    const dim3 grid(grid_for(out * Gc)), block(kSearchThreads);
    if (!stats) {
        switch (init_mode) {
            case kInitMaxAbs: hipLaunchKernelGGL((search_kernel<kInitMaxAbs, false>), grid, block, 0, stream, a); break;
            case kInitFourOverSix:
                hipLaunchKernelGGL((search_kernel<kInitFourOverSix, false>), grid, block, 0, stream, a);
                break;
            default: hipLaunchKernelGGL((search_kernel<kInitGiven, false>), grid, block, 0, stream, a); break;
        }
    } else {
        switch (init_mode) {
            case kInitMaxAbs: hipLaunchKernelGGL((search_kernel<kInitMaxAbs, true>), grid, block, 0, stream, a); break;
            case kInitFourOverSix:
                hipLaunchKernelGGL((search_kernel<kInitFourOverSix, true>), grid, block, 0, stream, a);
                break;
            default: hipLaunchKernelGGL((search_kernel<kInitGiven, true>), grid, block, 0, stream, a); break;
        }
    }
    return launch_status();
}

struct LfPlan {
    int64_t ldd = 0, rows_pad = 0, ntiles = 0, tiles_per_pass = 0;
    size_t plane_bytes = 0, zero_offset = 0, partial_offset = 0, bytes = 0;
};

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

LfPlan lfull_plan(int64_t tokens, int64_t in, int64_t out) {
    LfPlan p;
    if (tokens <= 0 || in <= 0 || out <= 0) return p;
    p.ldd = (in + kLfBK - 1) / kLfBK * kLfBK;
    p.rows_pad = (out + kLfBN - 1) / kLfBN * kLfBN;
    p.ntiles = p.rows_pad / kLfBN;
    const int64_t tiles = (tokens + kLfBM - 1) / kLfBM;
    p.tiles_per_pass = tiles < kLfMaxTilesPerPass ? tiles : kLfMaxTilesPerPass;
    p.plane_bytes = round_up((size_t)p.rows_pad * (size_t)p.ldd * 2, 256);
    p.zero_offset = 2 * p.plane_bytes;
    p.partial_offset = p.zero_offset + 256;
    p.bytes = p.partial_offset + (size_t)p.tiles_per_pass * (size_t)out * sizeof(double);
    return p;
}

int64_t summary_blocks(int64_t groups) { return groups > 0 ? (groups + kSumChunk - 1) / kSumChunk : 0; }

int hdiag_run(const void *X, int64_t tokens, int64_t in, float *h, double *h64, void *workspace,
              size_t workspace_bytes, hipStream_t stream) {
    if (tokens < 0 || in < 0 || in % kGroup != 0) return HSCALE_ERR_SHAPE;
    if (in > ((int64_t)1 << 40) || (in > 0 && tokens > ((int64_t)1 << 46) / in)) return HSCALE_ERR_SHAPE;
    if (in == 0) return HSCALE_OK;
    const bool accumulate = h64 != nullptr;
    if (!accumulate && !h) return HSCALE_ERR_NULL;
    if (!accumulate && !aligned(h, 4)) return HSCALE_ERR_ALIGN;
    if (accumulate && !aligned(h64, 8)) return HSCALE_ERR_ALIGN;
    const HdiagPlan p = hdiag_plan(tokens, in);
    const size_t need = hscale_hdiag_workspace_bytes(tokens, in);
    const size_t nout = accumulate ? (size_t)in * 8 : (size_t)in * 4;
    const void *out = accumulate ? (const void *)h64 : (const void *)h;
    if (tokens > 0) {
        if (!X) return HSCALE_ERR_NULL;
        if (!aligned(X, 16)) return HSCALE_ERR_ALIGN;
        if (workspace_bytes < need) return HSCALE_ERR_WORKSPACE;
        if (!workspace) return HSCALE_ERR_NULL;
        if (!aligned(workspace, 16)) return HSCALE_ERR_ALIGN;
        const size_t nx = (size_t)tokens * (size_t)in * 2;
        if (overlaps(out, nout, X, nx) || overlaps(workspace, need, X, nx) || overlaps(workspace, need, out, nout))
            return HSCALE_ERR_OVERLAP;
        dim3 grid((unsigned)p.tiles, (unsigned)p.slices);
        hipLaunchKernelGGL(hdiag_partial, grid, dim3(kHdThreads), 0, stream, static_cast<const u32x4 *>(X),
                           tokens, in, p.slice_tokens, static_cast<double *>(workspace));
        if (launch_status() != HSCALE_OK) return HSCALE_ERR_HIP;
    } else if (accumulate) {
        return HSCALE_OK;  // nothing to add
    }
    const unsigned tree_blocks = (unsigned)((in + kTreeCols - 1) / kTreeCols);
    if (accumulate)
        hipLaunchKernelGGL(hdiag_tree<true>, dim3(tree_blocks), dim3(kTreeCols * kTreeLanes), 0, stream,
                           static_cast<const double *>(workspace), p.slices, in, (float *)nullptr, h64);
    else
        hipLaunchKernelGGL(hdiag_tree<false>, dim3(tree_blocks), dim3(kTreeCols * kTreeLanes), 0, stream,
                           static_cast<const double *>(workspace), p.slices, in, h, (double *)nullptr);
    return launch_status();
}

}  // namespace

extern "C" {

const char *hscale_status_string(int status) {
    switch (status) {
        case HSCALE_OK: return "HSCALE_OK";
        case HSCALE_ERR_NULL: return "HSCALE_ERR_NULL: a required pointer is NULL";
        case HSCALE_ERR_SHAPE: return "HSCALE_ERR_SHAPE: negative size, in % 16 != 0, or too large";
        case HSCALE_ERR_ALIGN: return "HSCALE_ERR_ALIGN: a pointer is misaligned";
        case HSCALE_ERR_WINDOW: return "HSCALE_ERR_WINDOW: window outside 0..125";
        case HSCALE_ERR_SCALE: return "HSCALE_ERR_SCALE: global_scale not finite, not > 0, or out of range";
        case HSCALE_ERR_WORKSPACE: return "HSCALE_ERR_WORKSPACE: workspace too small";
        case HSCALE_ERR_HIP: return "HSCALE_ERR_HIP: the HIP runtime rejected a launch";
        case HSCALE_ERR_OVERLAP: return "HSCALE_ERR_OVERLAP: an output overlaps an input";
        default: return "unknown hscale status";
    }
}

size_t hscale_hdiag_workspace_bytes(int64_t tokens, int64_t in) {
    if (tokens <= 0 || in <= 0 || in % kGroup != 0) return 0;
    const HdiagPlan p = hdiag_plan(tokens, in);
    return (size_t)p.slices * (size_t)in * sizeof(double);
}

int hscale_hdiag(const void *X, int64_t tokens, int64_t in, float *h, void *workspace, size_t workspace_bytes,
                 hipStream_t stream) {
    return hdiag_run(X, tokens, in, h, nullptr, workspace, workspace_bytes, stream);
}

int hscale_hdiag_accumulate(const void *X, int64_t tokens, int64_t in, double *h64, void *workspace,
                            size_t workspace_bytes, hipStream_t stream) {
    if (in > 0 && !h64) return HSCALE_ERR_NULL;
    return hdiag_run(X, tokens, in, nullptr, h64, workspace, workspace_bytes, stream);
}

int hscale_hdiag_finalize(const double *h64, int64_t in, float *h, hipStream_t stream) {
    if (in < 0 || in % kGroup != 0) return HSCALE_ERR_SHAPE;
    if (in == 0) return HSCALE_OK;
    if (!h64 || !h) return HSCALE_ERR_NULL;
    if (!aligned(h64, 8) || !aligned(h, 4)) return HSCALE_ERR_ALIGN;
    if (overlaps(h64, (size_t)in * 8, h, (size_t)in * 4)) return HSCALE_ERR_OVERLAP;
    hipLaunchKernelGGL(hdiag_finalize_kernel, dim3((unsigned)((in + 255) / 256)), dim3(256), 0, stream, h64, in, h);
    return launch_status();
}

int hscale_search_block(const void *W, int64_t ldw, int64_t out, int64_t cols, const float *h, int32_t down,
                        int32_t up, float global_scale, int32_t init_mode, const uint8_t *init_codes, int64_t ldi,
                        uint8_t *scale_codes, int64_t ldc, uint8_t *packed_e2m1, int64_t ldp, hipStream_t stream) {
    return search_block(W, ldw, out, cols, h, down, up, global_scale, init_mode, init_codes, ldi, scale_codes, ldc,
                        packed_e2m1, ldp, stream);
}

int hscale_search_du(const void *W, int64_t out, int64_t in, const float *h, int32_t down, int32_t up,
                     float global_scale, uint8_t *scale_codes, uint8_t *packed_e2m1, hipStream_t stream) {
    return search_block(W, in, out, in, h, down, up, global_scale, kInitMaxAbs, nullptr, 0, scale_codes,
                        in / kGroup, packed_e2m1, in / 2, stream);
}

int hscale_search(const void *W, int64_t out, int64_t in, const float *h, int32_t window, float global_scale,
                  uint8_t *scale_codes, uint8_t *packed_e2m1, hipStream_t stream) {
    return hscale_search_du(W, out, in, h, window, window, global_scale, scale_codes, packed_e2m1, stream);
}

int hscale_search_4over6(const void *W, int64_t out, int64_t in, const float *h, int32_t down, int32_t up,
                         float global_scale, uint8_t *scale_codes, uint8_t *packed_e2m1, hipStream_t stream) {
    return search_block(W, in, out, in, h, down, up, global_scale, kInitFourOverSix, nullptr, 0, scale_codes,
                        in / kGroup, packed_e2m1, in / 2, stream);
}

int hscale_search_from(const void *W, int64_t out, int64_t in, const float *h, int32_t down, int32_t up,
                       float global_scale, const uint8_t *init_codes, uint8_t *scale_codes, uint8_t *packed_e2m1,
                       hipStream_t stream) {
    return search_block(W, in, out, in, h, down, up, global_scale, kInitGiven, init_codes, in / kGroup,
                        scale_codes, in / kGroup, packed_e2m1, in / 2, stream);
}

int hscale_search_stats(const void *W, int64_t out, int64_t in, const float *h, int32_t down, int32_t up,
                        float global_scale, int32_t init_mode, const uint8_t *init_codes, uint8_t *scale_codes,
                        uint8_t *packed_e2m1, int8_t *shift, float *err_best, float *err_init, hipStream_t stream) {
    if (out > 0 && in > 0 && (!shift || !err_best || !err_init)) return HSCALE_ERR_NULL;
    return search_block(W, in, out, in, h, down, up, global_scale, init_mode, init_codes, in / kGroup, scale_codes,
                        in / kGroup, packed_e2m1, in / 2, stream, shift, err_best, err_init);
}

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
    if (in % kGroup != 0 || in > ((int64_t)1 << 40) || (in > 0 && out > kMaxGroups / (in / kGroup))) return 0;
    return lfull_plan(tokens, in, out).bytes;
}

int hscale_output_error(const void *X, int64_t tokens, int64_t in, const void *W, int64_t out, float global_scale,
                        const uint8_t *scale_codes, const uint8_t *packed_e2m1, double *row_err, void *workspace,
                        size_t workspace_bytes, hipStream_t stream) {
    if (tokens < 0 || in < 0 || out < 0 || in % kGroup != 0) return HSCALE_ERR_SHAPE;
    if (in > ((int64_t)1 << 40) || (in > 0 && tokens > ((int64_t)1 << 46) / in)) return HSCALE_ERR_SHAPE;
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
    hipLaunchKernelGGL(delta_split_kernel, dim3(grid_for(p.rows_pad * (p.ldd / kGroup))), dim3(256), 0, stream,
                       static_cast<const u32x4 *>(W), out, in, global_scale, scale_codes,
                       reinterpret_cast<const uint2 *>(packed_e2m1), p.rows_pad, p.ldd, hi, lo,
                       reinterpret_cast<u32x4 *>(ws + p.zero_offset));
    if (launch_status() != HSCALE_OK) return HSCALE_ERR_HIP;
    const int64_t pass_tokens = p.tiles_per_pass * kLfBM;
    const unsigned tree_blocks = (unsigned)((out + kTreeCols - 1) / kTreeCols);
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
        a.zero = reinterpret_cast<const u32x4 *>(ws + p.zero_offset);
        const int64_t tiles = (a.tokens + kLfBM - 1) / kLfBM;
        hipLaunchKernelGGL(lfull_tile_kernel, dim3((unsigned)(tiles * p.ntiles)), dim3(kLfThreads), 0, stream, a);
        if (launch_status() != HSCALE_OK) return HSCALE_ERR_HIP;
        hipLaunchKernelGGL(hdiag_tree<true>, dim3(tree_blocks), dim3(kTreeCols * kTreeLanes), 0, stream,
                           static_cast<const double *>(partial), tiles, out, (float *)nullptr, row_err);
        if (launch_status() != HSCALE_OK) return HSCALE_ERR_HIP;
    }
    return HSCALE_OK;
}

int hscale_quantize(const void *W, int64_t out, int64_t in, float global_scale, const uint8_t *scale_codes,
                    uint8_t *packed_e2m1, hipStream_t stream) {
    if (out < 0 || in < 0 || in % kGroup != 0) return HSCALE_ERR_SHAPE;
    if (out > 0 && in > 0 && out > kMaxGroups / (in / kGroup)) return HSCALE_ERR_SHAPE;
    if (!scale_ok(global_scale)) return HSCALE_ERR_SCALE;
    if (out == 0 || in == 0) return HSCALE_OK;
    if (!W || !scale_codes || !packed_e2m1) return HSCALE_ERR_NULL;
    if (!aligned(W, 16) || !aligned(packed_e2m1, 8)) return HSCALE_ERR_ALIGN;
    const size_t nw = (size_t)out * (size_t)in * 2, nc = (size_t)out * (size_t)(in / kGroup);
    const size_t np = (size_t)out * (size_t)(in / 2);
    if (overlaps(packed_e2m1, np, W, nw) || overlaps(packed_e2m1, np, scale_codes, nc)) return HSCALE_ERR_OVERLAP;
    const int64_t groups = out * (in / kGroup);
    hipLaunchKernelGGL(quantize_kernel, dim3(grid_for(groups)), dim3(kSearchThreads), 0, stream,
                       static_cast<const u32x4 *>(W), groups, global_scale, scale_codes,
                       reinterpret_cast<uint2 *>(packed_e2m1));
    return launch_status();
}

}  // extern "C"
