// Shared definitions of the H-Scale HIP library (include/hscale.h): number
// formats, the per-tensor scale table, group loads, the fixed-order column
// tree, and host-side argument checks.  Each translation unit gets its own
// internal copy (anonymous namespace).
//
// The fp32 operations of the library are the fixed arithmetic of the header:
// IEEE round-to-nearest-even products, correctly rounded divisions (built
// with -fhip-fp32-correctly-rounded-divide-sqrt), explicit fmaf, and no
// implicit contraction (-ffp-contract=off).
#pragma once

#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <type_traits>

#include "hscale.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kGroup = 16;
constexpr int kMaxCode = 126;  // positive finite E4M3FN codes are 1..126
constexpr int kMaxWindow = 125;

constexpr int kTreeThreads = 256;

// Sums the slice partials of each column in a fixed order: kLanes lanes per
// column, lane q adding slices q, q + kLanes, ... in order, then the lane
// sums added in lane order.  kAccumulate adds the sum to an fp64 accumulator
// instead of writing fp32 h.  The lane count is chosen from the slice count
// alone (tree_lanes), so a given problem always sums in the same order.
template <bool kAccumulate, int kLanes>
__global__ __launch_bounds__(kTreeThreads) void hdiag_tree(const double *__restrict__ partial, int64_t slices,
                                                           int64_t in, float *__restrict__ h,
                                                           double *__restrict__ h64) {
    constexpr int kCols = kTreeThreads / kLanes;
    const int lane = threadIdx.x % kCols;
    const int q = threadIdx.x / kCols;
    const int64_t col = (int64_t)blockIdx.x * kCols + lane;
    double s = 0.0;
    if (col < in) {
#pragma unroll 8
        for (int64_t k = q; k < slices; k += kLanes) s += partial[k * in + col];
    }
    __shared__ double red[kLanes][kCols];
    red[q][lane] = s;
    __syncthreads();
    if (q == 0 && col < in) {
        double total = red[0][lane];
#pragma unroll
        for (int l = 1; l < kLanes; ++l) total += red[l][lane];
        if (kAccumulate)
            h64[col] += total;
        else
            h[col] = (float)total;
    }
}

// Lanes per column for summing `slices` partials: about 16 or fewer slices
// per lane, so the per-lane chains stay short and small column counts still
// spread over many blocks.
inline int tree_lanes(int64_t slices) { return slices <= 64 ? 4 : slices <= 256 ? 16 : 64; }

// Launches the fixed-order column sum of slices x in partials.
template <bool kAccumulate>
inline void launch_tree(const double *partial, int64_t slices, int64_t in, float *h, double *h64,
                        hipStream_t stream) {
    const int lanes = tree_lanes(slices);
    const unsigned blocks = (unsigned)((in + kTreeThreads / lanes - 1) / (kTreeThreads / lanes));
    if (lanes == 4)
        hipLaunchKernelGGL((hdiag_tree<kAccumulate, 4>), dim3(blocks), dim3(kTreeThreads), 0, stream, partial, slices,
                           in, h, h64);
    else if (lanes == 16)
        hipLaunchKernelGGL((hdiag_tree<kAccumulate, 16>), dim3(blocks), dim3(kTreeThreads), 0, stream, partial,
                           slices, in, h, h64);
    else
        hipLaunchKernelGGL((hdiag_tree<kAccumulate, 64>), dim3(blocks), dim3(kTreeThreads), 0, stream, partial,
                           slices, in, h, h64);
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

// The 16 bf16 weights of a group (two 16-byte words) as exact fp32 values.
__device__ __forceinline__ void unpack_group(const u32x4 a, const u32x4 b, float (&w)[kGroup]) {
    const uint32_t d[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        w[2 * k] = __uint_as_float(d[k] << 16);
        w[2 * k + 1] = __uint_as_float(d[k] & 0xFFFF0000u);
    }
}

__device__ __forceinline__ void load_group(const u32x4 *__restrict__ W, int64_t g, float (&w)[kGroup]) {
    unpack_group(__builtin_nontemporal_load(W + 2 * g), __builtin_nontemporal_load(W + 2 * g + 1), w);
}

// ---------------------------------------------------------------------------
// Host side: argument checks shared by the entry points
// ---------------------------------------------------------------------------

inline bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

inline bool overlaps(const void *a, size_t na, const void *b, size_t nb) {
    if (na == 0 || nb == 0) return false;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + nb && b0 < a0 + na;
}

// True when s_g keeps every S[c] a finite normal fp32 with a finite
// reciprocal: s_g * 2^-9 >= 2^-126 and s_g * 448 < 2^128.
inline bool scale_ok(float s_g) {
    if (!std::isfinite(s_g) || !(s_g > 0.0f)) return false;
    const double lo = (double)s_g * std::ldexp(1.0, -9);
    const double hi = (double)s_g * 448.0;
    return lo >= std::ldexp(1.0, -126) && hi < std::ldexp(1.0, 128) * (1.0 - std::ldexp(1.0, -25));
}

// The search indexes groups with 32-bit arithmetic.
constexpr int64_t kMaxGroups = ((int64_t)1 << 32) - 1;

// Blocks of `threads` lanes for a grid-stride loop over `groups` items, one
// item per lane: enough to fill every CU many times over, capped at 65536.
inline int grid_for(int64_t groups, int threads) {
    int64_t blocks = (groups + threads - 1) / threads;
    const int64_t cap = 65536;
    if (blocks > cap) blocks = cap;
    if (blocks < 1) blocks = 1;
    return (int)blocks;
}

inline int launch_status() { return hipGetLastError() == hipSuccess ? HSCALE_OK : HSCALE_ERR_HIP; }

// Bytes spanned by `rows` rows of `width` elements at a row stride of `ld`
// elements of `elem` bytes each.
inline size_t span(int64_t rows, int64_t ld, int64_t width, size_t elem) {
    if (rows <= 0 || width <= 0) return 0;
    return ((size_t)(rows - 1) * (size_t)ld + (size_t)width) * elem;
}

inline size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace
