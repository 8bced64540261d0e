// The per-group NVFP4 scale search (Sec. 3.3, Eq. 7, 9-13) and the final
// re-quantization, behind the C ABI of include/hscale.h.
//
//   search  one 16-weight group per lane, lanes over consecutive groups (a
//           wave reads 2 KiB of W contiguously and writes 512 contiguous
//           bytes of codes).  The 126-entry table of (S[c], R[c]) lives in
//           LDS.  Per candidate: 16 fp32 products w R, 8 hardware E2M1
//           down-conversions (packed nibbles with sign, round-to-nearest-
//           even, saturating at 6), 8 up-conversions back to grid values, 16
//           residual FMAs w - v S (one rounding each) and a 4x4 fp32
//           accumulation of h r^2.  The best candidate's packed nibbles are
//           kept, so the final re-quantization costs nothing extra.

#include "common.h"

namespace {

// fp32 products, FMAs and adds in the 64-bit VOP3 encoding.  The compiler
// prefers the 32-bit VOP2 forms, which on gfx950 issue markedly slower when
// interleaved with the FP4 conversions (measured at down_proj +-4: the
// search loop runs 15% faster with these forms).  The arithmetic is the
// same IEEE fp32 operation either way; only the encoding differs.
__device__ __forceinline__ float mul_e64(float a, float b) {
    float d;
    asm("v_mul_f32_e64 %0, %1, %2" : "=v"(d) : "v"(a), "v"(b));
    return d;
}
__device__ __forceinline__ float fma_e64(float a, float b, float c) {
    float d;
    asm("v_fma_f32 %0, %1, %2, %3" : "=v"(d) : "v"(a), "v"(b), "v"(c));
    return d;
}
__device__ __forceinline__ float add_e64(float a, float b) {
    float d;
    asm("v_add_f32_e64 %0, %1, %2" : "=v"(d) : "v"(a), "v"(b));
    return d;
}

// Packed E2M1 codes of 16 weights at reciprocal scale R: two 32-bit words,
// element 2k in the low nibble of byte k.  The hardware conversion rounds to
// nearest even, saturates at 6 and keeps the sign (scale operand 1.0: no
// extra scaling).
__device__ __forceinline__ uint2 quantize_group(const float (&w)[kGroup], float R, uint2 old) {
    // Every byte of both words is overwritten, so `old` only saves a move.
    uint32_t p0 = old.x, p1 = old.y;
    p0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p0, mul_e64(w[0], R), mul_e64(w[1], R), 1.0f, 0);
    p0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p0, mul_e64(w[2], R), mul_e64(w[3], R), 1.0f, 1);
    p0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p0, mul_e64(w[4], R), mul_e64(w[5], R), 1.0f, 2);
    p0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p0, mul_e64(w[6], R), mul_e64(w[7], R), 1.0f, 3);
    p1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p1, mul_e64(w[8], R), mul_e64(w[9], R), 1.0f, 0);
    p1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p1, mul_e64(w[10], R), mul_e64(w[11], R), 1.0f, 1);
    p1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p1, mul_e64(w[12], R), mul_e64(w[13], R), 1.0f, 2);
    p1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p1, mul_e64(w[14], R), mul_e64(w[15], R), 1.0f, 3);
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
    e[j0 & 3] = fma_e64(mul_e64(hh[j0], r0), r0, e[j0 & 3]);
    e[j1 & 3] = fma_e64(mul_e64(hh[j1], r1), r1, e[j1 & 3]);
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
    return add_e64(add_e64(e[0], e[1]), add_e64(e[2], e[3]));
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
    e[j0 & 3] = fma_e64(r0, r0, e[j0 & 3]);
    e[j1 & 3] = fma_e64(r1, r1, e[j1 & 3]);
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
    return add_e64(add_e64(e[0], e[1]), add_e64(e[2], e[3]));
}

// Initial code of Eq. 7 from max|w| and an anchor (6 for max-abs; 4 or 6 for
// 4over6): fp32(amax / anchor), then fp32(. / s_g), then Q_fp8 and the clip.
__device__ __forceinline__ int anchor_code(float amax, float anchor, float s_g) {
    const float s_init = amax / anchor;
    return e4m3fn_code_clipped(s_init / s_g);
}


// Packed E2M1 codes of one group for up to three candidates whose reciprocal
// scales are R, R / 2 and R / 4 (codes c, c + 8, c + 16, all normal and
// unclipped, so S and R scale by exact powers of two): each product w R is
// formed once, and the conversion's power-of-two scale operand divides it by
// 2 or 4 before rounding, which equals converting w (R / 2) or w (R / 4)
// (checked bit for bit on the hardware, midpoints included).
template <int kM, int K>
__device__ __forceinline__ void convert_pair_multi(const float (&w)[kGroup], float R, uint2 (&p)[3]) {
    const float x0 = mul_e64(w[2 * K], R), x1 = mul_e64(w[2 * K + 1], R);
    if constexpr (K < 4) {
        p[0].x = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p[0].x, x0, x1, 1.0f, K);
        if constexpr (kM > 1) p[1].x = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p[1].x, x0, x1, 2.0f, K);
        if constexpr (kM > 2) p[2].x = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p[2].x, x0, x1, 4.0f, K);
    } else {
        p[0].y = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p[0].y, x0, x1, 1.0f, K - 4);
        if constexpr (kM > 1) p[1].y = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p[1].y, x0, x1, 2.0f, K - 4);
        if constexpr (kM > 2) p[2].y = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p[2].y, x0, x1, 4.0f, K - 4);
    }
}

template <int kM>
__device__ __forceinline__ void quantize_group_multi(const float (&w)[kGroup], float R, uint2 (&p)[3]) {
    convert_pair_multi<kM, 0>(w, R, p);
    convert_pair_multi<kM, 1>(w, R, p);
    convert_pair_multi<kM, 2>(w, R, p);
    convert_pair_multi<kM, 3>(w, R, p);
    convert_pair_multi<kM, 4>(w, R, p);
    convert_pair_multi<kM, 5>(w, R, p);
    convert_pair_multi<kM, 6>(w, R, p);
    convert_pair_multi<kM, 7>(w, R, p);
}

// Windows of at least this many candidates walk residue classes (below);
// for smaller windows one or two shared classes do not pay for the lost
// candidate pairing (measured: the paper's 16-candidate window gains 6%,
// the 9-candidate one loses 4%).
constexpr int kClassMinCandidates = 16;

// The initial code of Eq. 7 by the rule kInit (`given` is the caller's code
// for kInitGiven), in 1..126.
template <int kInit>
__device__ __forceinline__ int initial_code(const float (&w)[kGroup], const ScaleEntry *tab, float s_g, int given) {
    if (kInit == kInitGiven) return min(max(given, 1), kMaxCode);
    float amax = 0.0f;
#pragma unroll
    for (int j = 0; j < kGroup; ++j) amax = fmaxf(amax, fabsf(w[j]));
    int c0 = anchor_code(amax, 6.0f, s_g);
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
    return c0;
}

// Eq. 7 and 9-13 for one group held in registers: the initial code, then the
// walk d = -down..up, keeping the first minimum.  With kStats it also
// reports the chosen shift, its error and the error at d = 0.
template <int kInit, bool kStats>
__device__ __forceinline__ void search_group(const float (&w)[kGroup], const float (&hh)[kGroup],
                                             const ScaleEntry *tab, int down, int up, float s_g, int given,
                                             int &code, uint2 &best_p, int &shift, float &err_best,
                                             float &err_init) {
    const int c0 = initial_code<kInit>(w, tab, s_g, given);
    const ScaleEntry *col = tab + (c0 + kTabPad);  // col[d] is candidate c0 + d, clipped
    const int K = down + up + 1;
    if (K >= kClassMinCandidates && K <= 24 && __all(c0 - down >= 8 && c0 + up <= kMaxCode)) {
        // Every candidate of every lane in the wave is a normal, unclipped
        // code: walk the 8 residue classes c mod 8, each member c + 8 m
        // sharing the products of its class base.  Candidates are then
        // visited out of order, so ties keep the smaller shift.  The first
        // candidate visited always replaces the start state (best_d is above
        // every shift), so even when every score is +Inf (an fp32 overflow)
        // the result is a real candidate: the smallest shift, as in the
        // plain walk.
        float best_e = INFINITY, e_init = 0.0f;
        int best_d = INT_MAX;
        best_p = make_uint2(0u, 0u);
        uint2 p[3] = {best_p, best_p, best_p};
        const int nb = K < 8 ? K : 8;
        for (int b = 0; b < nb; ++b) {
            const int d0 = -down + b;
            const int members = 1 + (d0 + 8 <= up) + (d0 + 16 <= up);  // wave-uniform
            const float R = col[d0].R;
            if (members == 1)
                quantize_group_multi<1>(w, R, p);
            else if (members == 2)
                quantize_group_multi<2>(w, R, p);
            else
                quantize_group_multi<3>(w, R, p);
#pragma unroll
            for (int m = 0; m < 3; ++m) {
                if (m < members) {
                    const int d = d0 + 8 * m;
                    const float e = group_error(w, hh, p[m], col[d].S);
                    if (kStats && d == 0) e_init = e;
                    if (e < best_e || (e == best_e && d < best_d)) {
                        best_e = e;
                        best_d = d;
                        best_p = p[m];
                    }
                }
            }
        }
        code = c0 + best_d;
        shift = best_d;
        err_best = best_e;
        err_init = e_init;
        return;
    }
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

// Pointer `byte_off` bytes past `base`, with a 32-bit offset: the loads and
// stores then take the uniform base from scalar registers and one 32-bit
// offset per lane, instead of 64-bit address arithmetic per lane.
template <typename T>
__device__ __forceinline__ T *at_byte(T *base, uint32_t byte_off) {
    using B = typename std::conditional<std::is_const<T>::value, const char, char>::type;
    return reinterpret_cast<T *>(reinterpret_cast<B *>(base) + byte_off);
}

// One group per lane over the flat index g = r * Gc + i of the block, so the
// lanes of a wave cover consecutive groups of a row (contiguous loads and
// stores) and a lane's h slice is h[16 i .. 16 i + 15].  A launch normally
// covers every group once; larger problems loop with a grid stride.
// kFlat: every array is contiguous (row strides equal the row widths) and
// W's byte span fits in 32 bits, so group g sits at byte 32 g of W, 8 g of
// the packed codes and g of the scale codes.
template <int kInit, bool kStats, bool kFlat>
__global__ __launch_bounds__(kSearchThreads) void search_kernel(const SearchArgs a) {
    __shared__ ScaleEntry tab[kTabSize];
    __shared__ ScaleEntry uniq[kMaxCode + 1];
    const bool single = a.down == 0 && a.up == 0;  // wave-uniform
    // A single candidate under the max-abs or given rule needs one scale per
    // lane, computed directly (the same fp32 product and correctly rounded
    // reciprocal as the table's entry); every other search reads the block's
    // table.
    const bool direct = !kStats && single && kInit != kInitFourOverSix;
    if (!direct) build_scale_table(tab, uniq, a.s_g);

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
        if (kFlat) {
            const u32x4 *src = at_byte(a.W, g << 5);
            unpack_group(__builtin_nontemporal_load(src), __builtin_nontemporal_load(src + 1), w);
        } else {
            load_group(a.W + (uint64_t)r * a.ldw_vec + 2 * (uint64_t)i, 0, w);
        }
        int given = 0;
        if (kInit == kInitGiven) given = kFlat ? (int)*at_byte(a.init, g) : (int)a.init[(uint64_t)r * a.ldi + i];
        int code, shift = 0;
        uint2 best_p;
        float e_best = 0.0f, e_init = 0.0f;
        if (!kStats && single) {
            // One candidate is its own first minimum: it needs no score, so
            // h is not read (the RTN code of Eq. 7 and its quantization).
            code = initial_code<kInit>(w, tab, a.s_g, given);
            const float R = direct ? 1.0f / (a.s_g * e4m3fn_value(code)) : tab[code + kTabPad].R;
            best_p = quantize_group(w, R, make_uint2(0u, 0u));
        } else {
            float hh[kGroup];
            const float4 *hsrc = kFlat ? at_byte(a.h, i << 6) : a.h + 4 * (uint64_t)i;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float4 v = hsrc[q];
                hh[4 * q] = v.x;
                hh[4 * q + 1] = v.y;
                hh[4 * q + 2] = v.z;
                hh[4 * q + 3] = v.w;
            }
            search_group<kInit, kStats>(w, hh, tab, a.down, a.up, a.s_g, given, code, best_p, shift, e_best,
                                        e_init);
        }
        if (kFlat) {
            *at_byte(a.codes, g) = (uint8_t)code;
            *at_byte(a.packed, g << 3) = best_p;
        } else {
            a.codes[(uint64_t)r * a.ldc + i] = (uint8_t)code;
            a.packed[(uint64_t)r * a.ldp_vec + i] = best_p;
        }
        if (kStats) {
            *at_byte(a.shift, g) = (int8_t)shift;
            *at_byte(a.err_best, g << 2) = e_best;
            *at_byte(a.err_init, g << 2) = e_init;
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

// Several independent layers searched by one launch, with the same shift
// set and initial-code rule.  The layers' arrays are contiguous.  Each block
// covers 256 consecutive groups of one layer and finds that layer among the
// kernel arguments by its first block (a uniform scan over at most
// kMaxBatchLayers entries), then proceeds as the single-layer search.
constexpr int kMaxBatchLayers = 32;

struct BatchLayer {
    const u32x4 *W;
    const float4 *h;
    const uint8_t *init;
    uint8_t *codes;
    uint2 *packed;
    uint32_t Gc;      // groups per row
    uint32_t groups;  // rows * Gc
    uint32_t block0;  // first block of the layer in the launch
    float s_g;
};

struct BatchArgs {
    BatchLayer layer[kMaxBatchLayers];
    int count;
    int down, up;
};

// kFlat: every layer's W spans less than 4 GiB, so 32-bit byte offsets from
// the scalar bases address all of its arrays.
template <int kInit, bool kFlat>
__global__ __launch_bounds__(kSearchThreads) void search_layers_kernel(const BatchArgs a) {
    int L = 0;
#pragma unroll
    for (int k = 1; k < kMaxBatchLayers; ++k)
        if (k < a.count && blockIdx.x >= a.layer[k].block0) L = k;
    const BatchLayer ly = a.layer[L];
    __shared__ ScaleEntry tab[kTabSize];
    __shared__ ScaleEntry uniq[kMaxCode + 1];
    const bool single = a.down == 0 && a.up == 0;
    const bool direct = single && kInit != kInitFourOverSix;  // as in search_kernel
    if (!direct) build_scale_table(tab, uniq, ly.s_g);

    const uint32_t first = (blockIdx.x - ly.block0) * kSearchThreads;  // wave-uniform
    const uint32_t g = first + threadIdx.x;
    if (g >= ly.groups) return;
    uint32_t i = first % ly.Gc + threadIdx.x;
    while (i >= ly.Gc) i -= ly.Gc;

    float w[kGroup];
    if (kFlat) {
        const u32x4 *src = at_byte(ly.W, g << 5);
        unpack_group(__builtin_nontemporal_load(src), __builtin_nontemporal_load(src + 1), w);
    } else {
        load_group(ly.W, g, w);
    }
    int given = 0;
    if (kInit == kInitGiven) given = kFlat ? (int)*at_byte(ly.init, g) : (int)ly.init[g];
    int code;
    uint2 best_p;
    if (single) {  // one candidate: no score, h not read
        code = initial_code<kInit>(w, tab, ly.s_g, given);
        const float R = direct ? 1.0f / (ly.s_g * e4m3fn_value(code)) : tab[code + kTabPad].R;
        best_p = quantize_group(w, R, make_uint2(0u, 0u));
    } else {
        float hh[kGroup];
        const float4 *hsrc = kFlat ? at_byte(ly.h, i << 6) : ly.h + 4 * (uint64_t)i;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 v = hsrc[q];
            hh[4 * q] = v.x;
            hh[4 * q + 1] = v.y;
            hh[4 * q + 2] = v.z;
            hh[4 * q + 3] = v.w;
        }
        int shift;
        float e_best, e_init;
        search_group<kInit, false>(w, hh, tab, a.down, a.up, ly.s_g, given, code, best_p, shift, e_best, e_init);
    }
    if (kFlat) {
        *at_byte(ly.codes, g) = (uint8_t)code;
        *at_byte(ly.packed, g << 3) = best_p;
    } else {
        ly.codes[g] = (uint8_t)code;
        ly.packed[g] = best_p;
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

template <bool kFlat>
void launch_search(int init_mode, bool stats, dim3 grid, dim3 block, hipStream_t stream, const SearchArgs &a) {
    if (!stats) {
        switch (init_mode) {
            case kInitMaxAbs:
                hipLaunchKernelGGL((search_kernel<kInitMaxAbs, false, kFlat>), grid, block, 0, stream, a);
                break;
            case kInitFourOverSix:
                hipLaunchKernelGGL((search_kernel<kInitFourOverSix, false, kFlat>), grid, block, 0, stream, a);
                break;
            default: hipLaunchKernelGGL((search_kernel<kInitGiven, false, kFlat>), grid, block, 0, stream, a); break;
        }
    } else {
        switch (init_mode) {
            case kInitMaxAbs:
                hipLaunchKernelGGL((search_kernel<kInitMaxAbs, true, kFlat>), grid, block, 0, stream, a);
                break;
            case kInitFourOverSix:
                hipLaunchKernelGGL((search_kernel<kInitFourOverSix, true, kFlat>), grid, block, 0, stream, a);
                break;
            default: hipLaunchKernelGGL((search_kernel<kInitGiven, true, kFlat>), grid, block, 0, stream, a); break;
        }
    }
}

// Host-side checks of a search over a block of `out` x `cols` weights inside
// row-major arrays with the given row strides (statistics arrays optional):
// HSCALE_OK when the arguments are valid, an empty problem included.
int check_search(const void *W, int64_t ldw, int64_t out, int64_t cols, const float *h, int32_t down, int32_t up,
                 float s_g, int32_t init_mode, const uint8_t *init_codes, int64_t ldi, const uint8_t *codes,
                 int64_t ldc, const uint8_t *packed, int64_t ldp, const int8_t *shift, const float *err_best,
                 const float *err_init) {
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
    return HSCALE_OK;
}

int search_block(const void *W, int64_t ldw, int64_t out, int64_t cols, const float *h, int32_t down, int32_t up,
                 float s_g, int32_t init_mode, const uint8_t *init_codes, int64_t ldi, uint8_t *codes, int64_t ldc,
                 uint8_t *packed, int64_t ldp, hipStream_t stream, int8_t *shift = nullptr,
                 float *err_best = nullptr, float *err_init = nullptr) {
    const int status = check_search(W, ldw, out, cols, h, down, up, s_g, init_mode, init_codes, ldi, codes, ldc,
                                    packed, ldp, shift, err_best, err_init);
    if (status != HSCALE_OK || out == 0 || cols == 0) return status;
    const bool stats = shift || err_best || err_init;
    const int64_t Gc = cols / kGroup;
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
    // The flat form needs contiguous arrays and 32-bit byte offsets: W spans
    // 32 bytes per group (the largest array) and h 4 bytes per column.
    const int64_t groups = out * Gc;
    const bool flat = ldw == cols && ldc == Gc && ldp == cols / 2 && (init_mode != kInitGiven || ldi == Gc) &&
                      groups <= ((int64_t)1 << 27) && cols <= ((int64_t)1 << 28);
    const dim3 grid(grid_for(groups, kSearchThreads)), block(kSearchThreads);
    if (flat)
        launch_search<true>(init_mode, stats, grid, block, stream, a);
    else
        launch_search<false>(init_mode, stats, grid, block, stream, a);
    return launch_status();
}

// Launches one batch of at most kMaxBatchLayers non-empty, checked layers.
template <int kInit>
void launch_layers(const BatchArgs &a, uint32_t blocks, bool flat, hipStream_t stream) {
    if (flat)
        hipLaunchKernelGGL((search_layers_kernel<kInit, true>), dim3(blocks), dim3(kSearchThreads), 0, stream, a);
    else
        hipLaunchKernelGGL((search_layers_kernel<kInit, false>), dim3(blocks), dim3(kSearchThreads), 0, stream, a);
}

int search_layers(const hscale_layer *layers, int32_t count, int32_t down, int32_t up, int32_t init_mode,
                  hipStream_t stream) {
    if (count < 0) return HSCALE_ERR_SHAPE;
    if (init_mode < kInitMaxAbs || init_mode > kInitGiven) return HSCALE_ERR_SHAPE;
    if (down < 0 || up < 0 || down > kMaxWindow || up > kMaxWindow) return HSCALE_ERR_WINDOW;
    if (count == 0) return HSCALE_OK;
    if (!layers) return HSCALE_ERR_NULL;
    for (int32_t k = 0; k < count; ++k) {
        const hscale_layer &l = layers[k];
        const int status = check_search(l.W, l.in, l.out, l.in, l.h, down, up, l.global_scale, init_mode,
                                        l.init_codes, l.in / kGroup, l.scale_codes, l.in / kGroup, l.packed_e2m1,
                                        l.in / 2, nullptr, nullptr, nullptr);
        if (status != HSCALE_OK) return status;
    }
    // The layers run concurrently: no layer's outputs may overlap another
    // layer's inputs or outputs.
    auto spans = [&](const hscale_layer &l, size_t &nw, size_t &nh, size_t &nc, size_t &np) {
        const bool empty = l.out == 0 || l.in == 0;
        nw = empty ? 0 : (size_t)l.out * (size_t)l.in * 2;
        nh = empty ? 0 : (size_t)l.in * 4;
        nc = empty ? 0 : (size_t)l.out * (size_t)(l.in / kGroup);
        np = empty ? 0 : (size_t)l.out * (size_t)(l.in / 2);
    };
    for (int32_t x = 0; x < count; ++x) {
        size_t xw, xh, xc, xp;
        spans(layers[x], xw, xh, xc, xp);
        for (int32_t y = 0; y < count; ++y) {
            if (y == x) continue;
            size_t yw, yh, yc, yp;
            spans(layers[y], yw, yh, yc, yp);
            const hscale_layer &a = layers[x], &b = layers[y];
            const size_t yi = init_mode == kInitGiven ? yc : 0;
            auto hits_b = [&](const void *p, size_t n) {
                return overlaps(p, n, b.W, yw) || overlaps(p, n, b.h, yh) || overlaps(p, n, b.init_codes, yi) ||
                       overlaps(p, n, b.scale_codes, yc) || overlaps(p, n, b.packed_e2m1, yp);
            };
            if (hits_b(a.scale_codes, xc) || hits_b(a.packed_e2m1, xp)) return HSCALE_ERR_OVERLAP;
        }
    }
    BatchArgs a;
    a.down = down;
    a.up = up;
    a.count = 0;
    uint32_t blocks = 0;
    bool flat = true, launched = false;
    auto flush = [&]() {
        if (a.count == 0) return;
        launched = true;
        switch (init_mode) {
            case kInitMaxAbs: launch_layers<kInitMaxAbs>(a, blocks, flat, stream); break;
            case kInitFourOverSix: launch_layers<kInitFourOverSix>(a, blocks, flat, stream); break;
            default: launch_layers<kInitGiven>(a, blocks, flat, stream); break;
        }
        a.count = 0;
        blocks = 0;
        flat = true;
    };
    for (int32_t k = 0; k < count; ++k) {
        const hscale_layer &l = layers[k];
        if (l.out == 0 || l.in == 0) continue;
        const int64_t groups = l.out * (l.in / kGroup);
        BatchLayer &b = a.layer[a.count++];
        b.W = static_cast<const u32x4 *>(l.W);
        b.h = reinterpret_cast<const float4 *>(l.h);
        b.init = l.init_codes;
        b.codes = l.scale_codes;
        b.packed = reinterpret_cast<uint2 *>(l.packed_e2m1);
        b.Gc = (uint32_t)(l.in / kGroup);
        b.groups = (uint32_t)groups;
        b.block0 = blocks;
        b.s_g = l.global_scale;
        blocks += (uint32_t)((groups + kSearchThreads - 1) / kSearchThreads);
        flat = flat && groups <= ((int64_t)1 << 27) && l.in <= ((int64_t)1 << 28);
        if (a.count == kMaxBatchLayers) flush();
    }
    flush();
    return launched ? launch_status() : HSCALE_OK;
}

}  // namespace

extern "C" {

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

int hscale_search_layers(const hscale_layer *layers, int32_t count, int32_t down, int32_t up, int32_t init_mode,
                         hipStream_t stream) {
    return search_layers(layers, count, down, up, init_mode, stream);
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
    hipLaunchKernelGGL(quantize_kernel, dim3(grid_for(groups, kSearchThreads)), dim3(kSearchThreads), 0, stream,
                       static_cast<const u32x4 *>(W), groups, global_scale, scale_codes,
                       reinterpret_cast<uint2 *>(packed_e2m1));
    return launch_status();
}

}  // extern "C"
