// h = diag(X^T X) (Sec. 3.2, Eq. 4) behind the C ABI of include/hscale.h.
//
//   hdiag_partial  column sums of squares of bf16 X over one token slice.
//                  One wave covers 512 columns (16-byte loads, 8 columns per
//                  lane, a row segment of 1 KiB per wave); the four waves of
//                  a block interleave rows; 8 rows of loads are in flight per
//                  lane.  fp32 chains of at most 32 tokens fold into fp64; the
//                  block's four waves combine through LDS in a fixed order
//                  and one fp64 partial per (slice, column) goes to the
//                  caller's workspace.
//   hdiag_tree     fixed-order fp64 sum of the slice partials, one fp32 h per
//                  column (4, 16 or 64 lanes per column by slice count).  No atomics: results are bit-identical run to run.

#include "common.h"

#include <mutex>

// Device scratch of hscale_hdiag_noalloc (fp64 slice partials), sized for
// the largest problem it accepts: every hdiag plan with in <= 2^20 columns
// needs at most 8 MiB.
constexpr size_t kHdiagScratchBytes = (size_t)8 << 20;
static __device__ __align__(256) unsigned char scratch[kHdiagScratchBytes];

namespace {

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

__global__ __launch_bounds__(256) void hdiag_finalize_kernel(const double *__restrict__ h64, int64_t in,
                                                             float *__restrict__ h) {
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (j < in) h[j] = (float)h64[j];
}

// Checks of X and the output that need no workspace and no HIP call: HSCALE_OK
// when the arguments are valid (in == 0 included).
int hdiag_check_io(const void *X, int64_t tokens, int64_t in, const float *h, const double *h64) {
    if (tokens < 0 || in < 0 || in % kGroup != 0) return HSCALE_ERR_SHAPE;
    if (in > ((int64_t)1 << 40) || (in > 0 && tokens > ((int64_t)1 << 46) / in)) return HSCALE_ERR_SHAPE;
    if (in == 0) return HSCALE_OK;
    const bool accumulate = h64 != nullptr;
    if (!accumulate && !h) return HSCALE_ERR_NULL;
    if (!accumulate && !aligned(h, 4)) return HSCALE_ERR_ALIGN;
    if (accumulate && !aligned(h64, 8)) return HSCALE_ERR_ALIGN;
    if (tokens > 0) {
        if (!X) return HSCALE_ERR_NULL;
        if (!aligned(X, 16)) return HSCALE_ERR_ALIGN;
        const size_t nx = (size_t)tokens * (size_t)in * 2;
        const size_t nout = accumulate ? (size_t)in * 8 : (size_t)in * 4;
        const void *out = accumulate ? (const void *)h64 : (const void *)h;
        if (overlaps(out, nout, X, nx)) return HSCALE_ERR_OVERLAP;
    }
    return HSCALE_OK;
}

int hdiag_run(const void *X, int64_t tokens, int64_t in, float *h, double *h64, void *workspace,
              size_t workspace_bytes, hipStream_t stream) {
    const int status = hdiag_check_io(X, tokens, in, h, h64);
    if (status != HSCALE_OK || in == 0) return status;
    const bool accumulate = h64 != nullptr;
    const HdiagPlan p = hdiag_plan(tokens, in);
    const size_t need = hscale_hdiag_workspace_bytes(tokens, in);
    const size_t nout = accumulate ? (size_t)in * 8 : (size_t)in * 4;
    const void *out = accumulate ? (const void *)h64 : (const void *)h;
    if (tokens > 0) {
        if (workspace_bytes < need) return HSCALE_ERR_WORKSPACE;
        if (!workspace) return HSCALE_ERR_NULL;
        if (!aligned(workspace, 16)) return HSCALE_ERR_ALIGN;
        const size_t nx = (size_t)tokens * (size_t)in * 2;
        if (overlaps(workspace, need, X, nx) || overlaps(workspace, need, out, nout)) return HSCALE_ERR_OVERLAP;
        dim3 grid((unsigned)p.tiles, (unsigned)p.slices);
        hipLaunchKernelGGL(hdiag_partial, grid, dim3(kHdThreads), 0, stream, static_cast<const u32x4 *>(X),
                           tokens, in, p.slice_tokens, static_cast<double *>(workspace));
        if (launch_status() != HSCALE_OK) return HSCALE_ERR_HIP;
    } else if (accumulate) {
        return HSCALE_OK;  // nothing to add
    }
    if (accumulate)
        launch_tree<true>(static_cast<const double *>(workspace), p.slices, in, nullptr, h64, stream);
    else
        launch_tree<false>(static_cast<const double *>(workspace), p.slices, in, h, nullptr, stream);
    return launch_status();
}

// ---------------------------------------------------------------------------
// Static scratch for hscale_hdiag_noalloc: the slice partials live in a
// device array of the library instead of a caller workspace.  Each GPU holds
// its own copy at its own address, looked up once per device with that
// device current; host code uses only the looked-up address (the array's
// name is a host-side stand-in, not a device address).  The partials kernel
// writes every partial the tree reads, so nothing needs clearing between
// calls.
// ---------------------------------------------------------------------------

constexpr int kScratchDevices = 64;

struct ScratchSlot {
    std::once_flag once;
    void *ptr = nullptr;
    hipError_t err = hipSuccess;
};

ScratchSlot g_scratch_slot[kScratchDevices];

// The scratch address on the device `stream` runs on, which must be the
// current device (the lookup is made with it current).
int scratch_address(hipStream_t stream, void **out) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess || cur < 0 || cur >= kScratchDevices) return HSCALE_ERR_HIP;
    if (stream) {
        int dev = -1;
        if (hipStreamGetDevice(stream, &dev) != hipSuccess) return HSCALE_ERR_HIP;
        if (dev != cur) return HSCALE_ERR_DEVICE;
    }
    ScratchSlot &s = g_scratch_slot[cur];
    std::call_once(s.once, [&s] { s.err = hipGetSymbolAddress(&s.ptr, HIP_SYMBOL(scratch)); });
    if (s.err != hipSuccess || !s.ptr) return HSCALE_ERR_HIP;
    *out = s.ptr;
    return HSCALE_OK;
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
        case HSCALE_ERR_SCRATCH:
            return "HSCALE_ERR_SCRATCH: the problem needs more scratch than the library's static buffer holds";
        case HSCALE_ERR_DEVICE: return "HSCALE_ERR_DEVICE: the stream is not on the current device";
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

int hscale_hdiag_noalloc(const void *X, int64_t tokens, int64_t in, float *h, hipStream_t stream) {
    // Every host-side check comes before the first HIP call.
    const int status = hdiag_check_io(X, tokens, in, h, nullptr);
    if (status != HSCALE_OK || in == 0) return status;
    const size_t need = hscale_hdiag_workspace_bytes(tokens, in);
    if (need > kHdiagScratchBytes) return HSCALE_ERR_SCRATCH;
    void *ws = nullptr;
    if (need > 0) {
        const int st = scratch_address(stream, &ws);
        if (st != HSCALE_OK) return st;
    }
    return hdiag_run(X, tokens, in, h, nullptr, ws, need, stream);
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

}  // extern "C"
