/*
 * hscale.h - C ABI of the H-Scale hot path on AMD Instinct MI355X (gfx950).
 *
 * H-Scale (Hessian-guided scale refinement for NVFP4) picks, for every
 * 16-weight group of a linear layer, the E4M3 local scale that minimises the
 * h-weighted reconstruction error, where h = diag(X^T X) comes from
 * calibration activations X.  This library computes:
 *
 *   hscale_hdiag    h_j = sum_t X[t, j]^2                    (Sec. 3.2, Eq. 4)
 *   hscale_search   the windowed E4M3 scale search per group (Sec. 3.3,
 *                   Eq. 7 and 9-13, App. B Alg. HScaleGroupQuantize), emitting
 *                   NVFP4 scale bytes and packed E2M1 codes
 *   hscale_quantize the final re-quantization at given scale codes (Sec. 3.3,
 *                   "Final re-quantization"; Eq. 12 at a fixed scale)
 *
 * and the variants the paper's integration section and App. B use: the
 * search from baseline-provided initial scales (HScaleGroupQuantize takes
 * them as input), the 4over6 initialisation, a strided column-block form for
 * GPTQ-style blockwise use, and h accumulated over streamed calibration
 * batches.  Quality diagnostics of the appendix: the search with per-group
 * statistics (chosen shift, its error, the error at shift 0) and their
 * per-shift summary, and the layer-output error of Eq. 3 by which the
 * appendix scores a candidate window.
 *
 * Conventions shared by every entry point
 *   - All pointers are device pointers (hipMalloc'd or torch CUDA tensors)
 *     unless stated.  The caller allocates and owns every buffer; the library
 *     allocates nothing, never synchronises and is safe to call from several
 *     host threads on different streams.  Its only global state is the
 *     static scratch of hscale_hdiag_noalloc (see there).
 *   - Work is enqueued on `stream` (NULL = the default stream) and is
 *     complete only once the caller synchronises that stream.  Arguments are
 *     validated on the host before anything is enqueued; on any error
 *     nothing is launched.  Kernel faults surface at the caller's next sync.
 *   - bf16 tensors are passed as their 16-bit patterns, row-major.
 *   - Inputs must be finite (no NaN or Inf); outputs for non-finite inputs
 *     are unspecified.  Outputs must not overlap inputs.  h is formed from
 *     fp32 squares of bf16 activations, exact for 2^-63 <= |x| < 2^64; larger
 *     activations overflow h to +Inf.
 *   - Number formats: E4M3 is OCP E4M3FN.  Scale code byte c in 1..126 is
 *     the positive finite E4M3FN value l_c (2^-9 .. 448).  E2M1 magnitudes
 *     are {0, 0.5, 1, 1.5, 2, 3, 4, 6}; a 4-bit code is sign << 3 | index.
 *
 * Arithmetic (fixed so that results are reproducible bit for bit):
 *   S[c] = fp32(global_scale * l_c)             effective scale (Eq. 1)
 *   R[c] = fp32(1 / S[c])                       correctly rounded
 *   s_init = fp32(max_j |w_j| / 6)              correctly rounded (Eq. 7)
 *   t = fp32(s_init / global_scale)             correctly rounded
 *   c0 = clip(E4M3 round-to-nearest-even of t, saturating at 448, to 1..126)
 *   candidate codes c = clip(c0 + d, 1, 126), d = -window .. +window
 *   x_j = fp32(w_j * R[c]); code_j = E2M1 round-to-nearest-even of x_j
 *     (ties to the even index, |x| > 5 -> 6), sign copied from w_j
 *   score E(c) = sum_j h_j (w_j - v_j S[c])^2 evaluated in fp32; the first
 *     minimum in increasing d wins.  A score that overflows fp32 is +Inf
 *     and ties with every other +Inf score, so a group whose scores all
 *     overflow (finite but huge h) takes the smallest shift d = -down; its
 *     packed codes are still the quantization at the code it reports.
 */
#ifndef HSCALE_H
#define HSCALE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum hscale_status {
    HSCALE_OK = 0,
    HSCALE_ERR_NULL = -1,      /* a required pointer is NULL */
    HSCALE_ERR_SHAPE = -2,     /* negative size, in % 16 != 0, or too large */
    HSCALE_ERR_ALIGN = -3,     /* a pointer is not aligned as required */
    HSCALE_ERR_WINDOW = -4,    /* window outside 0..125 */
    HSCALE_ERR_SCALE = -5,     /* global_scale not finite, not > 0, or out of range */
    HSCALE_ERR_WORKSPACE = -6, /* workspace too small */
    HSCALE_ERR_HIP = -7,       /* the HIP runtime rejected a launch */
    HSCALE_ERR_OVERLAP = -8,   /* an output overlaps an input */
    HSCALE_ERR_SCRATCH = -9,   /* the problem needs more than the static scratch
                                  of hscale_hdiag_noalloc holds */
    HSCALE_ERR_DEVICE = -10    /* the stream is not on the current device */
} hscale_status;

/* How the search chooses each group's initial code c0 before the walk. */
typedef enum hscale_init_mode {
    HSCALE_INIT_MAXABS = 0,  /* Eq. 7: fp32(max|w| / 6), fp32(. / s_g), Q_fp8 */
    HSCALE_INIT_4OVER6 = 1,  /* App. B, 4over6 + H-Scale: anchors 4 and 6 as in
                                Eq. 7 (fp32(max|w| / anchor)), each scored by
                                the plain squared error sum_j (w_j - v_j S)^2
                                at its code; the smaller wins, anchor 4 on a
                                tie (scores in fp32, 4 chains of 4) */
    HSCALE_INIT_GIVEN = 2    /* caller-provided code bytes; values outside
                                1..126 are clipped into the ladder */
} hscale_init_mode;

/* Human-readable name of a status code (static string, never NULL). */
const char *hscale_status_string(int status);

/*
 * Workspace size in bytes that hscale_hdiag needs for `tokens` x `in`
 * activations: fp64 partial sums of each token slice, so that the cross-slice
 * reduction is a fixed-order tree (deterministic, no atomics).  Depends only
 * on (tokens, in).  Returns 0 when tokens == 0 or the sizes are invalid.
 */
size_t hscale_hdiag_workspace_bytes(int64_t tokens, int64_t in);

/*
 * The diagonal second-order proxy of Sec. 3.2, Eq. 4:
 *     h[j] = sum_{t < tokens} X[t, j]^2,   no normalisation.
 *
 * X          bf16 [tokens, in], row-major, 16-byte aligned.
 * tokens     >= 0.  tokens == 0 writes h = 0.
 * in         >= 0, in % 16 == 0 (h is aligned with the 16-weight groups).
 * h          fp32 [in], written.  4-byte aligned.
 * workspace  device scratch of at least hscale_hdiag_workspace_bytes(tokens,
 *            in) bytes, 16-byte aligned; may be NULL when that size is 0.
 *            Its contents on entry are ignored and on exit are unspecified.
 *
 * Squares of bf16 values are exact in fp32.  Each lane sums at most 32
 * tokens in fp32 before folding into fp64; slices combine in fp64 in a fixed
 * order; h is rounded to fp32 once.  The result is within a relative 2e-6 of
 * the exact sum and identical from run to run.
 */
int hscale_hdiag(const void *X, int64_t tokens, int64_t in, float *h,
                 void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * hscale_hdiag for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same h, bit for bit, with the slice partials held in a static device
 * array of the library (8 MiB per GPU, kept until the process ends) instead
 * of a caller workspace.  The call allocates nothing.
 *
 * X, tokens, in, h   as hscale_hdiag.
 * stream             must belong to the current device (HSCALE_ERR_DEVICE
 *                    otherwise); NULL is the current device's default stream.
 *
 * Limit: problems whose hscale_hdiag_workspace_bytes(tokens, in) exceeds
 * 8 MiB are rejected with HSCALE_ERR_SCRATCH before anything is enqueued;
 * every in <= 2^20 (any tokens) fits.  The first call on a device looks up
 * that device's copy of the array (hipGetSymbolAddress) and keeps its
 * address; a failed lookup returns HSCALE_ERR_HIP.  That lookup is a runtime
 * call: make the first call on each device outside stream capture (later
 * calls, captured or not, only enqueue kernels).
 *
 * All calls on one GPU share that GPU's array: calls that may run at the
 * same time on one GPU (different streams, or host threads that do not
 * order their streams) race on it and give undefined h.  Calls ordered on
 * one stream are safe: every partial a call reads is written earlier in the
 * same call, so the array needs no clearing and nothing is carried from one
 * call to the next.
 */
int hscale_hdiag_noalloc(const void *X, int64_t tokens, int64_t in, float *h,
                         hipStream_t stream);

/*
 * Streamed calibration (Eq. 4 over batches): h64[j] += sum_t X[t, j]^2 for
 * one batch, into a caller-owned fp64 accumulator [in] (8-byte aligned) that
 * the caller zeroes before the first batch.  Each batch's sum is formed
 * exactly as in hscale_hdiag and added in fp64, so splitting the tokens into
 * batches changes the result only at fp64 rounding level.  tokens == 0
 * leaves h64 unchanged.  Other arguments as hscale_hdiag.
 */
int hscale_hdiag_accumulate(const void *X, int64_t tokens, int64_t in,
                            double *h64, void *workspace,
                            size_t workspace_bytes, hipStream_t stream);

/* h[j] = fp32(h64[j]) (round to nearest even) for j < in; in % 16 == 0.
 * Accumulating from zero and finalizing gives the same h as hscale_hdiag. */
int hscale_hdiag_finalize(const double *h64, int64_t in, float *h,
                          hipStream_t stream);

/*
 * The per-group NVFP4 scale search of Sec. 3.3 (Eq. 7, 9-13) with the
 * symmetric shift set d = -window .. +window (K = 2 window + 1 candidates).
 * window == 0 is the plain max-abs (RTN) scale of Eq. 7; a single candidate
 * needs no score, so h is then not read (it must still be a valid pointer).
 *
 * W             bf16 [out, in], row-major, 16-byte aligned.  Group (r, i)
 *               is W[r, 16 i .. 16 i + 15].
 * out, in       out >= 0, in >= 0, in % 16 == 0, and fewer than 2^32
 *               groups (out * in / 16), which are indexed in 32 bits.
 * h             fp32 [in], the per-input-channel weights (diag of X^T X or
 *               of a GPTQ Hessian; any h >= 0), 16-byte aligned.  The
 *               choice is invariant to a positive scale of h.
 * window        0 .. 125; 125 reaches every code from any start.
 * global_scale  the FP32 tensor-level scale s_g, finite, with
 *               s_g * 2^-9 >= 2^-126 and s_g * 448 < 2^128.  A common
 *               choice is fp32(max|W| / 2688).
 * scale_codes   uint8 [out, in / 16]: the chosen E4M3FN code byte per group.
 * packed_e2m1   uint8 [out, in / 2], 8-byte aligned: the E2M1 codes at the
 *               chosen scale, element 2k in bits 3:0 of byte k, element
 *               2k + 1 in bits 7:4.
 */
int hscale_search(const void *W, int64_t out, int64_t in, const float *h,
                  int32_t window, float global_scale, uint8_t *scale_codes,
                  uint8_t *packed_e2m1, hipStream_t stream);

/*
 * The same search with the paper's asymmetric shift set (Eq. 9):
 * d = -down .. +up, K = down + up + 1 (the paper uses down = 9, up = 6).
 * hscale_search(..., window, ...) equals hscale_search_du(..., window,
 * window, ...).  0 <= down, up <= 125.  Other arguments as hscale_search.
 */
int hscale_search_du(const void *W, int64_t out, int64_t in, const float *h,
                     int32_t down, int32_t up, float global_scale,
                     uint8_t *scale_codes, uint8_t *packed_e2m1,
                     hipStream_t stream);

/*
 * The search with the 4over6 initial code (HSCALE_INIT_4OVER6); with
 * down = up = 0 it is the 4over6 quantizer alone.  Arguments as
 * hscale_search_du.
 */
int hscale_search_4over6(const void *W, int64_t out, int64_t in,
                         const float *h, int32_t down, int32_t up,
                         float global_scale, uint8_t *scale_codes,
                         uint8_t *packed_e2m1, hipStream_t stream);

/*
 * The search from baseline-provided initial codes (HSCALE_INIT_GIVEN), the
 * form of App. B's HScaleGroupQuantize: init_codes uint8 [out, in / 16], one
 * E4M3FN code byte per group.  init_codes may equal scale_codes (refinement
 * in place); any other overlap with an output is rejected.  Other arguments
 * as hscale_search_du.
 */
int hscale_search_from(const void *W, int64_t out, int64_t in,
                       const float *h, int32_t down, int32_t up,
                       float global_scale, const uint8_t *init_codes,
                       uint8_t *scale_codes, uint8_t *packed_e2m1,
                       hipStream_t stream);

/*
 * One layer of a batched search (hscale_search_layers).  Arrays contiguous
 * and aligned as for hscale_search; init_codes is read only when init_mode
 * is HSCALE_INIT_GIVEN (it may then equal scale_codes).
 */
typedef struct hscale_layer {
    const void *W;             /* bf16 [out, in] */
    int64_t out;
    int64_t in;                /* in % 16 == 0 */
    const float *h;            /* fp32 [in] */
    float global_scale;        /* s_g of this layer */
    const uint8_t *init_codes; /* uint8 [out, in / 16] or NULL */
    uint8_t *scale_codes;      /* uint8 [out, in / 16], written */
    uint8_t *packed_e2m1;      /* uint8 [out, in / 2], written */
} hscale_layer;

/*
 * The search of several layers (for example the seven linear layers of a
 * decoder block, each with its own W, h and s_g) in one launch per up to 32
 * layers, with one shift set d = -down .. +up and one initial-code rule for
 * all.  Each layer's result is bit for bit that of hscale_search_du /
 * _4over6 / _from on it alone; batching only fills the GPU better when some
 * layers are small and saves launches.
 *
 * layers     host array of `count` layers (count >= 0; NULL when 0).  It is
 *            read during the call only.  Layers with out == 0 or in == 0 are
 *            skipped.  Inputs may be shared between layers (one h for q, k
 *            and v); no layer's outputs may overlap any buffer of another
 *            layer (HSCALE_ERR_OVERLAP).
 * init_mode  HSCALE_INIT_MAXABS, HSCALE_INIT_4OVER6 or HSCALE_INIT_GIVEN.
 * Every layer is checked as hscale_search_du checks its arguments; the
 * first failing layer's status is returned and nothing is launched.
 */
int hscale_search_layers(const hscale_layer *layers, int32_t count,
                         int32_t down, int32_t up, int32_t init_mode,
                         hipStream_t stream);

/*
 * The general strided form, for a column block of a larger matrix (App. B,
 * the GPTQ combination searches W[:, i : i + B] with h[i : i + B] and the
 * layer's fixed s_g).  W points at the block's first element; group (r, k)
 * of the block is W[r * ldw + 16 k .. + 15].  h points at the block's h
 * slice ([cols]).  Codes go to scale_codes[r * ldc + k], packed bytes to
 * packed_e2m1[r * ldp + 8 k .. + 7]; init_codes[r * ldi + k] is read for
 * HSCALE_INIT_GIVEN (may be NULL otherwise).
 *
 * cols % 16 == 0; ldw >= cols and ldw % 8 == 0 (16-byte rows); ldc >=
 * cols / 16; ldp >= cols / 2 and ldp % 8 == 0; ldi >= cols / 16 when read.
 * Alignment, window and global_scale rules as hscale_search.  Every other
 * search entry point is this call with contiguous strides.
 */
int hscale_search_block(const void *W, int64_t ldw, int64_t out,
                        int64_t cols, const float *h, int32_t down,
                        int32_t up, float global_scale, int32_t init_mode,
                        const uint8_t *init_codes, int64_t ldi,
                        uint8_t *scale_codes, int64_t ldc,
                        uint8_t *packed_e2m1, int64_t ldp,
                        hipStream_t stream);

/*
 * The search with per-group statistics, for the selected-shift analysis of
 * the paper's appendix (which shift each group chose and how much of the
 * initial error it removed).  Writes scale_codes and packed_e2m1 exactly as
 * hscale_search_block with contiguous strides and the same init_mode /
 * init_codes ([out, in / 16] when HSCALE_INIT_GIVEN), and, for group
 * g = r * (in / 16) + k:
 *
 * shift      int8 [out, in / 16]: the chosen shift d* in -down .. up (the
 *            first minimum; code = clip(c0 + d*, 1, 126))
 * err_best   fp32 [out, in / 16]: the score E at d*, as the search computed it
 * err_init   fp32 [out, in / 16]: the score E at d = 0 (the initial code)
 *
 * All three are required (4-byte aligned errors) and must not overlap any
 * other buffer.  The kernel is the search kernel with these three extra
 * stores; the plain entry points do not pay for them.
 */
int hscale_search_stats(const void *W, int64_t out, int64_t in, const float *h,
                        int32_t down, int32_t up, float global_scale,
                        int32_t init_mode, const uint8_t *init_codes,
                        uint8_t *scale_codes, uint8_t *packed_e2m1,
                        int8_t *shift, float *err_best, float *err_init,
                        hipStream_t stream);

/* Workspace bytes hscale_shift_summary needs (0 when groups <= 0). */
size_t hscale_shift_summary_workspace_bytes(int64_t groups, int32_t down,
                                            int32_t up);

/*
 * Per-shift summary of hscale_search_stats' outputs (the appendix's
 * selected-shift figure): for bin k = d + down, d = -down .. up,
 *   count[k]     uint64: groups whose shift is d
 *   sum_init[k]  fp64: sum of their err_init
 *   sum_best[k]  fp64: sum of their err_best
 *   sum_rel[k]   fp64: sum of (err_init - err_best) / err_init (0 when
 *                err_init = 0); the bin's mean reduction is sum_rel / count
 * The fraction of the initial error removed over all groups is
 * 1 - sum(sum_best) / sum(sum_init).  Sums are formed in fp64 in a fixed
 * order (bitwise reproducible).  Groups whose shift lies outside
 * -down .. up are not counted.
 *
 * shift, err_best, err_init  [groups] as written by hscale_search_stats
 *                            (needed only when groups > 0)
 * count, sum_init, sum_best, sum_rel  [down + up + 1] each, 8-byte aligned,
 *                            always written (all zero when groups = 0)
 * workspace      >= hscale_shift_summary_workspace_bytes(groups, down, up)
 *                bytes, 8-byte aligned, scratch owned by the caller
 */
int hscale_shift_summary(const int8_t *shift, const float *err_best,
                         const float *err_init, int64_t groups, int32_t down,
                         int32_t up, uint64_t *count, double *sum_init,
                         double *sum_best, double *sum_rel, void *workspace,
                         size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes hscale_output_error needs (0 when any size is 0). */
size_t hscale_output_error_workspace_bytes(int64_t tokens, int64_t in,
                                           int64_t out);

/*
 * Layer-output error of a stored NVFP4 tensor on calibration activations
 * (Sec. 3.2, Eq. 3; the L_full by which the appendix's window sweep scores
 * chosen scales), split by output row:
 *
 *   row_err[r] += sum_t ( sum_j X[t, j] * dW[r, j] )^2,
 *   dW[r, j] = W[r, j] - v[r, j] * S[c]
 *
 * where c is the group's scale code, v the signed E2M1 value of its nibble
 * and S[c] = fp32(global_scale * l_c) (S[0] = 0).  The layer's
 * ||X dW^T||_F^2 = Tr(dW X^T X dW^T) is the sum of row_err.  row_err is
 * accumulated into, so calibration batches streamed through successive
 * calls add up; zero it first.
 *
 * Arithmetic: dW is formed in fp32 with one rounding and split into two bf16
 * parts hi + lo (within 2^-18 |dW|); X dW^T is computed on the matrix cores
 * as bf16 products accumulated in fp32; squares and sums are fp64 in a fixed
 * order (bitwise reproducible for a given problem).
 *
 * X            bf16 [tokens, in], 16-byte aligned
 * W            bf16 [out, in], 16-byte aligned
 * scale_codes  uint8 [out, in / 16], E4M3FN codes 0..126 (other bytes give
 *              unspecified results)
 * packed_e2m1  uint8 [out, in / 2], 8-byte aligned, element 2k in the low
 *              nibble of byte k
 * row_err      fp64 [out], 8-byte aligned, in/out
 * workspace    >= hscale_output_error_workspace_bytes(tokens, in, out)
 *              bytes, 256-byte aligned, scratch owned by the caller (it holds
 *              the two dW planes and per-tile partial sums)
 * in % 16 == 0 and in <= 2^21 (HSCALE_ERR_SHAPE beyond: the kernel
 * addresses a tile of X and of dW with 32-bit offsets); global_scale as
 * hscale_search.  tokens, in or out = 0 adds nothing.
 */
int hscale_output_error(const void *X, int64_t tokens, int64_t in,
                        const void *W, int64_t out, float global_scale,
                        const uint8_t *scale_codes, const uint8_t *packed_e2m1,
                        double *row_err, void *workspace,
                        size_t workspace_bytes, hipStream_t stream);

/*
 * Final re-quantization at given scale codes (Sec. 3.3; Eq. 12 at a fixed
 * effective scale S = s_g * l_c): packs the E2M1 codes of every group at its
 * code byte.  Produces the same packed bytes hscale_search writes when given
 * the codes it chose.
 *
 * W, out, in, global_scale, packed_e2m1   as hscale_search.
 * scale_codes   uint8 [out, in / 16], input, normally each in 1..126.  The
 *               byte's unsigned value is clipped into 1..126 (0 reads as 1,
 *               127..255 as 126), the clip the search applies to given
 *               initial codes, so the result equals the window-0 search from
 *               those codes (hscale_search_from with down = up = 0).
 */
int hscale_quantize(const void *W, int64_t out, int64_t in, float global_scale,
                    const uint8_t *scale_codes, uint8_t *packed_e2m1,
                    hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HSCALE_H */
