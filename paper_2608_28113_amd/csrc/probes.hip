// Measurement probes for the benchmark's roofline figures.  They are not part
// of the hscale C ABI and compute nothing of the method: each one measures what
// this chip sustains for one kind of work, so that a kernel's rate can be set
// beside what the hardware delivers for the same work, next to the published
// peaks.  Built into its own library (libhscale_probes.so).
//
//   hsprobe_stream_read  reads a device buffer once, block b taking a
//                        contiguous chunk, with 16-byte non-temporal loads and
//                        16 loads in flight per lane; lane i of block b writes
//                        the wrapping 32-bit sum of the words it read to
//                        lane_sums[256 b + i], so a caller can check that every
//                        byte of the chunks was read.  Returns the bytes read
//                        (the chunks, a multiple of 64 KiB each), or -1.
//   hsprobe_valu         runs a fixed instruction stream from registers (no
//                        memory access inside the loop) on `blocks` blocks of
//                        256 lanes; wave w records s_memtime and s_memrealtime
//                        before and after its loop in clocks[4 w .. 4 w + 3].
//                        Kinds:
//                          0  v_fma_f32, 8 independent chains (64 per iteration)
//                          1  FP4 pack conversion v_cvt_scalef32_pk_fp4_f32,
//                             8 independent destinations (64 per iteration)
//                          2  FP4 unpack conversion v_cvt_scalef32_pk_f32_fp4
//                             (64 per iteration)
//                          3  the scale search's instruction stream for two
//                             candidates of one 16-weight group: per candidate
//                             16 products w R and 8 pack conversions, 8 unpack
//                             conversions, 16 residual FMAs, 16 products h r,
//                             16 accumulating FMAs, 3 adds, then the
//                             first-minimum update (the plain walk)
//                          4  the same for the two members c and c + 8 of one
//                             residue class (the residue-class walk): the 16
//                             products once, converted at scale operands 1
//                             and 2
//                        sink[lane] receives a value that depends on the whole
//                        loop.  Returns 0, or -1 for a bad kind or size.
//   hsprobe_wall_clock_khz  frequency of s_memrealtime (device 0).

#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kReadInFlight = 16;

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const u32x4 *__restrict__ p, int64_t vecs_per_block,
                                                               uint32_t *__restrict__ lane_sums) {
    const u32x4 *q = p + (int64_t)blockIdx.x * vecs_per_block + threadIdx.x;
    uint32_t acc = 0;
    for (int64_t i = 0; i < vecs_per_block; i += kThreads * kReadInFlight) {
        u32x4 v[kReadInFlight];
#pragma unroll
        for (int u = 0; u < kReadInFlight; ++u) v[u] = __builtin_nontemporal_load(q + i + u * kThreads);
#pragma unroll
        for (int u = 0; u < kReadInFlight; ++u) acc += (v[u].x + v[u].y) + (v[u].z + v[u].w);
    }
    lane_sums[(int64_t)blockIdx.x * kThreads + threadIdx.x] = acc;
}

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

// One candidate of a 16-weight group: packed E2M1 codes of w R, then the
// h-weighted squared residual sum of w - v S in 4 chains.
template <int K>
__device__ __forceinline__ uint32_t pack_pair(const float (&w)[16], float R, uint32_t word) {
    return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(word, mul_e64(w[2 * K], R), mul_e64(w[2 * K + 1], R), 1.0f, K & 3);
}

__device__ __forceinline__ uint2 pack16(const float (&w)[16], float R, uint2 p) {
    p.x = pack_pair<0>(w, R, p.x);
    p.x = pack_pair<1>(w, R, p.x);
    p.x = pack_pair<2>(w, R, p.x);
    p.x = pack_pair<3>(w, R, p.x);
    p.y = pack_pair<4>(w, R, p.y);
    p.y = pack_pair<5>(w, R, p.y);
    p.y = pack_pair<6>(w, R, p.y);
    p.y = pack_pair<7>(w, R, p.y);
    return p;
}

// Two candidates of one residue class (codes c and c + 8, reciprocal scales R
// and R / 2) from one set of products: the conversion's power-of-two scale
// operand 2 halves each product before rounding.
template <int K>
__device__ __forceinline__ void pack_pair_class(const float (&w)[16], float R, uint32_t &word1, uint32_t &word2) {
    const float x0 = mul_e64(w[2 * K], R), x1 = mul_e64(w[2 * K + 1], R);
    word1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(word1, x0, x1, 1.0f, K & 3);
    word2 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(word2, x0, x1, 2.0f, K & 3);
}

__device__ __forceinline__ void pack16_class(const float (&w)[16], float R, uint2 &p, uint2 &q) {
    pack_pair_class<0>(w, R, p.x, q.x);
    pack_pair_class<1>(w, R, p.x, q.x);
    pack_pair_class<2>(w, R, p.x, q.x);
    pack_pair_class<3>(w, R, p.x, q.x);
    pack_pair_class<4>(w, R, p.y, q.y);
    pack_pair_class<5>(w, R, p.y, q.y);
    pack_pair_class<6>(w, R, p.y, q.y);
    pack_pair_class<7>(w, R, p.y, q.y);
}

template <int K>
__device__ __forceinline__ void error_pair(const float (&w)[16], const float (&h)[16], uint32_t word, float S,
                                           float (&e)[4]) {
    const f32x2 v = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(word, 1.0f, K & 3);
    const float r0 = fmaf(-v[0], S, w[2 * K]);
    const float r1 = fmaf(-v[1], S, w[2 * K + 1]);
    e[(2 * K) & 3] = fma_e64(mul_e64(h[2 * K], r0), r0, e[(2 * K) & 3]);
    e[(2 * K + 1) & 3] = fma_e64(mul_e64(h[2 * K + 1], r1), r1, e[(2 * K + 1) & 3]);
}

__device__ __forceinline__ float error16(const float (&w)[16], const float (&h)[16], uint2 p, float S) {
    float e[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    error_pair<0>(w, h, p.x, S, e);
    error_pair<1>(w, h, p.x, S, e);
    error_pair<2>(w, h, p.x, S, e);
    error_pair<3>(w, h, p.x, S, e);
    error_pair<4>(w, h, p.y, S, e);
    error_pair<5>(w, h, p.y, S, e);
    error_pair<6>(w, h, p.y, S, e);
    error_pair<7>(w, h, p.y, S, e);
    return add_e64(add_e64(e[0], e[1]), add_e64(e[2], e[3]));
}

// Kinds 0-2 issue 64 instructions per loop iteration (eight groups of eight
// independent ones).  A short loop that straddles a 256-byte boundary of the
// code runs markedly slower on this chip (measured: an 8-instruction loop,
// 1.4-1.9x), so the loops are made long enough that their placement does not
// matter.
#define FMA8                                                                                      \
    "v_fma_f32 %0, %0, %8, %9\n\tv_fma_f32 %1, %1, %8, %9\n\tv_fma_f32 %2, %2, %8, %9\n\t"           \
    "v_fma_f32 %3, %3, %8, %9\n\tv_fma_f32 %4, %4, %8, %9\n\tv_fma_f32 %5, %5, %8, %9\n\t"           \
    "v_fma_f32 %6, %6, %8, %9\n\tv_fma_f32 %7, %7, %8, %9\n\t"
#define PACK8                                                                                     \
    "v_cvt_scalef32_pk_fp4_f32 %0, %8, %9, 1.0\n\tv_cvt_scalef32_pk_fp4_f32 %1, %8, %9, 1.0\n\t"       \
    "v_cvt_scalef32_pk_fp4_f32 %2, %8, %9, 1.0\n\tv_cvt_scalef32_pk_fp4_f32 %3, %8, %9, 1.0\n\t"       \
    "v_cvt_scalef32_pk_fp4_f32 %4, %8, %9, 1.0\n\tv_cvt_scalef32_pk_fp4_f32 %5, %8, %9, 1.0\n\t"       \
    "v_cvt_scalef32_pk_fp4_f32 %6, %8, %9, 1.0\n\tv_cvt_scalef32_pk_fp4_f32 %7, %8, %9, 1.0\n\t"
#define UNPACK8                                                                                   \
    "v_cvt_scalef32_pk_f32_fp4 %0, %8, 1.0\n\tv_cvt_scalef32_pk_f32_fp4 %1, %9, 1.0\n\t"               \
    "v_cvt_scalef32_pk_f32_fp4 %2, %10, 1.0\n\tv_cvt_scalef32_pk_f32_fp4 %3, %11, 1.0\n\t"             \
    "v_cvt_scalef32_pk_f32_fp4 %4, %12, 1.0\n\tv_cvt_scalef32_pk_f32_fp4 %5, %13, 1.0\n\t"             \
    "v_cvt_scalef32_pk_f32_fp4 %6, %14, 1.0\n\tv_cvt_scalef32_pk_f32_fp4 %7, %15, 1.0\n\t"

template <int kKind>
__global__ __launch_bounds__(kThreads) void valu_kernel(int iters, float seed, float *__restrict__ sink,
                                                        uint64_t *__restrict__ clocks) {
    const int lane = threadIdx.x;
    float a[8];
    uint32_t pk[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = seed + (float)(lane + i);
        pk[i] = (uint32_t)(lane * 0x01010101u + i);
    }
    const float b = seed * 0.5f, c = seed * 0.25f;
    float w[16], h[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        w[j] = (float)(((lane + 5 * j) % 23) - 11) * 0.37f * seed;
        h[j] = 1.0f + (float)((lane * 3 + j) % 7);
    }
    float Ra = 0.9f, Rb = 1.1f, Sa = 1.0f / 0.9f, Sb = 1.0f / 1.1f;
    if constexpr (kKind == 4) Sb = 2.0f * Sa;  // the class member c + 8
    float best = INFINITY;
    int best_d = 0;
    uint2 pa = make_uint2(0u, 0u), pb = pa, bp = pa;
    // Materialise the set-up before the first clock read.
    if constexpr (kKind >= 3) {
#pragma unroll
        for (int j = 0; j < 16; ++j) asm volatile("" : "+v"(w[j]), "+v"(h[j]));
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) asm volatile("" : "+v"(a[i]), "+v"(pk[i]));

    const uint64_t t0 = __builtin_readcyclecounter();
    const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
    for (int it = 0; it < iters; ++it) {
        if constexpr (kKind == 0) {
            asm volatile(FMA8 FMA8 FMA8 FMA8 FMA8 FMA8 FMA8 FMA8
                         : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(a[4]), "+v"(a[5]), "+v"(a[6]),
                           "+v"(a[7])
                         : "v"(b), "v"(c));
        } else if constexpr (kKind == 1) {
            asm volatile(PACK8 PACK8 PACK8 PACK8 PACK8 PACK8 PACK8 PACK8
                         : "+v"(pk[0]), "+v"(pk[1]), "+v"(pk[2]), "+v"(pk[3]), "+v"(pk[4]), "+v"(pk[5]), "+v"(pk[6]),
                           "+v"(pk[7])
                         : "v"(b), "v"(c));
        } else if constexpr (kKind == 2) {
            f32x2 v[8];
            asm volatile(UNPACK8 UNPACK8 UNPACK8 UNPACK8 UNPACK8 UNPACK8 UNPACK8 UNPACK8
                         : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5]), "=&v"(v[6]),
                           "=&v"(v[7])
                         : "v"(pk[0]), "v"(pk[1]), "v"(pk[2]), "v"(pk[3]), "v"(pk[4]), "v"(pk[5]), "v"(pk[6]),
                           "v"(pk[7]));
#pragma unroll
            for (int i = 0; i < 8; ++i) asm volatile("" ::"v"(v[i]));
        } else {
            // The scales pass through an empty asm statement each iteration,
            // so no candidate's work can be hoisted out of the loop.
            asm volatile("" : "+v"(Ra), "+v"(Rb), "+v"(Sa), "+v"(Sb));
            if constexpr (kKind == 3) {
                pa = pack16(w, Ra, pa);
                pb = pack16(w, Rb, pb);
            } else {
                pack16_class(w, Ra, pa, pb);
            }
            const float ea = error16(w, h, pa, Sa);
            const float eb = error16(w, h, pb, Sb);
            if (ea < best) {
                best = ea;
                best_d = 2 * it;
                bp = pa;
            }
            if (eb < best) {
                best = eb;
                best_d = 2 * it + 1;
                bp = pb;
            }
        }
    }
    const uint64_t t1 = __builtin_readcyclecounter();
    const uint64_t r1 = __builtin_amdgcn_s_memrealtime();

    float s = best + (float)best_d + (float)(bp.x ^ bp.y);
#pragma unroll
    for (int i = 0; i < 8; ++i) s += a[i] + (float)pk[i];
    sink[(int64_t)blockIdx.x * kThreads + lane] = s;
    if ((lane & 63) == 0) {
        const int64_t wave = (int64_t)blockIdx.x * (kThreads / 64) + lane / 64;
        clocks[4 * wave + 0] = t0;
        clocks[4 * wave + 1] = t1;
        clocks[4 * wave + 2] = r0;
        clocks[4 * wave + 3] = r1;
    }
}

}  // namespace

extern "C" int64_t hsprobe_stream_read(const void *buf, int64_t bytes, int32_t blocks, uint32_t *lane_sums,
                                       hipStream_t stream) {
    constexpr int64_t step = (int64_t)kThreads * kReadInFlight;  // vectors per block per round
    if (!buf || !lane_sums || bytes <= 0 || blocks <= 0 || ((uintptr_t)buf & 15)) return -1;
    const int64_t vecs_per_block = bytes / 16 / blocks / step * step;
    if (vecs_per_block == 0) return -1;
    hipLaunchKernelGGL(stream_read_kernel, dim3(blocks), dim3(kThreads), 0, stream, (const u32x4 *)buf,
                       vecs_per_block, lane_sums);
    if (hipGetLastError() != hipSuccess) return -1;
    return vecs_per_block * 16 * blocks;
}

extern "C" int hsprobe_valu(int32_t kind, int32_t blocks, int32_t iters, float *sink, uint64_t *clocks,
                            hipStream_t stream) {
    if (!sink || !clocks || blocks <= 0 || iters <= 0) return -1;
    void (*k)(int, float, float *, uint64_t *) = nullptr;
    switch (kind) {
        case 0: k = valu_kernel<0>; break;
        case 1: k = valu_kernel<1>; break;
        case 2: k = valu_kernel<2>; break;
        case 3: k = valu_kernel<3>; break;
        case 4: k = valu_kernel<4>; break;
        default: return -1;
    }
    hipLaunchKernelGGL(k, dim3(blocks), dim3(kThreads), 0, stream, iters, 1.0f, sink, clocks);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

extern "C" int hsprobe_wall_clock_khz() {
    int khz = 0;
    if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, 0) != hipSuccess) return -1;
    return khz;
}
