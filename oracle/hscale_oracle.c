/*
 * Reference oracle for the H-Scale hot path (diagonal proxy h and the
 * per-group NVFP4 scale search).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check of the
 * package entry module and the CPU-baseline leg of the benchmark may load
 * this library.  The product path (the HIP library) never calls it, and the
 * two share no source, header, table or helper.
 *
 * This is a deliberately plain, slow implementation written from the paper:
 *   - scoring in fp64;
 *   - the fp32 rounding points that the method fixes (effective scale
 *     s = s_g * l, its reciprocal, the max-abs initial scale and the scaled
 *     weight w / s) are emulated exactly: an fp64 product of two fp32 (or
 *     bf16) operands is exact, and rounding an fp64 quotient of two fp32
 *     values to fp32 equals the correctly rounded fp32 quotient because
 *     53 >= 2*24 + 2;
 *   - rounding to a format grid is done by brute force: the nearest grid
 *     value, ties to the even code.
 *
 * Paper sections followed (H-Scale, Hessian-guided scale refinement for
 * NVFP4):
 *   Sec. 3.1, Eq. 1-2   effective scale s = s_g * l and the FP4 quantizer
 *   Sec. 3.2, Eq. 3     layer-output error ||X dW^T||^2 (quality diagnostics)
 *   Sec. 3.2, Eq. 4     h = diag(X^T X)
 *   Sec. 3.2, Eq. 6     per-group weighted objective ||(w - w^) . sqrt(h)||^2
 *   Sec. 3.3, Eq. 7     l_init = Q_fp8(s_init / s_g), s_init from the group max
 *   Sec. 3.3, Eq. 8-11  E4M3 ladder, shift set, clipped walk, candidates
 *   Sec. 3.3, Eq. 12-13 FP4 quantization per candidate and the argmin
 *   Sec. 3.3 "Final re-quantization"
 *   App. B, Alg. HScaleGroupQuantize (the same steps as pseudocode)
 *   App. "Selected Scale Shifts" and "Candidate-Window Width" (statistics
 *                       of the chosen shift; L_full of a window)
 *
 * Readings where the paper is silent (each stated where it is used):
 *   E4M3 is OCP E4M3FN (max 448, 126 positive finite codes); Q_fp8 rounds to
 *   nearest with ties to even and saturates at 448; E2M1 rounding ties go to
 *   the even index; a group whose initial code rounds to 0 starts at code 1
 *   (the clip of Eq. 10); the argmin keeps the first minimum in increasing
 *   shift order; the nibble copies the sign bit of w (so -0 is 0x8); element
 *   2k of a row goes in the low nibble of byte k.
 *
 * Parity: every function here is pinned by the CPU tests (paper worked
 * example, library E4M3 decode and rounding, closed forms, invariants and
 * brute force).  Near-tie classification is a reporting aid, not a pin.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_M 126 /* positive finite E4M3FN codes 1..126 */

/* bf16 bit pattern -> its exact value. */
static double bf16_value(uint16_t bits) {
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static int bf16_signbit(uint16_t bits) { return (bits >> 15) & 1; }

/* Round an exact real (held in fp64) to fp32, round-to-nearest-even. */
static double rn32(double x) { return (double)(float)x; }

/* ------------------------------------------------------------------------
 * Formats (Sec. 3.1 and Eq. 8)
 * ---------------------------------------------------------------------- */

/* Value of a non-negative OCP E4M3FN code byte c in 0..126: 4 exponent bits
 * (bias 7), 3 mantissa bits; exponent field 0 is subnormal (m/8 * 2^-6). */
double oracle_e4m3_value(int c) {
    int e = c >> 3;
    int m = c & 7;
    if (e == 0) return (double)m / 8.0 * ldexp(1.0, -6);
    return (1.0 + (double)m / 8.0) * ldexp(1.0, e - 7);
}

/* Q_fp8 of Eq. 7 on a non-negative value: the code of the nearest value on
 * {0} u ladder, ties to the even code byte (the even mantissa), values past
 * 448 saturating to 448 (code 126). */
int oracle_e4m3_round(double t) {
    /* 448 is on the ladder and is the nearest value to anything beyond it;
     * clamping first keeps every distance below exact in fp64. */
    if (t > 448.0) t = 448.0;
    int best = 0;
    double best_d = fabs(t);
    for (int c = 1; c <= ORACLE_M; ++c) {
        double d = fabs(t - oracle_e4m3_value(c));
        if (d < best_d || (d == best_d && (c % 2) == 0)) {
            best = c;
            best_d = d;
        }
    }
    return best;
}

/* E2M1 magnitudes v_0..v_7 (Sec. 3.1: the FP4 grid, clipped to [-6, 6]). */
static const double kE2M1[8] = {0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0};

double oracle_e2m1_value(int i) { return kE2M1[i & 7]; }

/* Round(.) then Clip(.) of Eq. 2 on a magnitude: index of the nearest grid
 * value, ties to the even index; anything beyond 6 lands on 6. */
int oracle_e2m1_index(double x) {
    /* The Clip of Eq. 2: 6 is on the grid and is the nearest value to
     * anything beyond it; clamping first keeps the distances exact. */
    if (x > 6.0) x = 6.0;
    int best = 0;
    double best_d = fabs(x - kE2M1[0]);
    for (int i = 1; i < 8; ++i) {
        double d = fabs(x - kE2M1[i]);
        if (d < best_d || (d == best_d && (i % 2) == 0)) {
            best = i;
            best_d = d;
        }
    }
    return best;
}

/* Effective-scale candidates of Eq. 11 for every ladder code: S[c] is the
 * fp32 product s_g * l_c that a dequantizer forms (Eq. 1), R[c] the fp32
 * reciprocal used to form w / s.  Index 0 is unused and set to 0. */
void oracle_scale_tables(float s_g, float *S, float *R) {
    S[0] = 0.0f;
    R[0] = 0.0f;
    for (int c = 1; c <= ORACLE_M; ++c) {
        S[c] = (float)((double)s_g * oracle_e4m3_value(c));
        R[c] = (float)(1.0 / (double)S[c]);
    }
}

/* ------------------------------------------------------------------------
 * One group (Eq. 7, 10-13 and the final re-quantization)
 * ---------------------------------------------------------------------- */

/* Initial ladder index of Eq. 7: s_init = max|w| / 6 in fp32, then
 * Q_fp8(s_init / s_g) in fp32, then the clip of Eq. 10 to [1, M] (an
 * all-zero or underflowing group starts at code 1). */
int oracle_init_code_f(const double *w, int g, float s_g) {
    double amax = 0.0;
    for (int j = 0; j < g; ++j)
        if (fabs(w[j]) > amax) amax = fabs(w[j]);
    double s_init = rn32(amax / 6.0);
    double t = rn32(s_init / (double)s_g);
    int c = oracle_e4m3_round(t);
    if (c < 1) c = 1;
    if (c > ORACLE_M) c = ORACLE_M;
    return c;
}

/* Quantize a group at effective scale S (with fp32 reciprocal R), Eq. 12:
 * x_j = fp32(|w_j| * R), i_j = Round/Clip of x_j, w^_j = sign(w_j) v_i S.
 * Writes the 4-bit codes (sign << 3 | i) to nib and returns the weighted
 * squared error of Eq. 13 in fp64 (h == NULL means h = 1). */
double oracle_quantize_group(const double *w, const int *neg, const double *h,
                             int g, float S, float R, uint8_t *nib) {
    double err = 0.0;
    for (int j = 0; j < g; ++j) {
        double x = rn32(fabs(w[j]) * (double)R);
        int i = oracle_e2m1_index(x);
        double q = kE2M1[i] * (double)S;
        if (neg[j]) q = -q;
        double d = w[j] - q;
        double hj = h ? h[j] : 1.0;
        err += hj * d * d;
        if (nib) nib[j] = (uint8_t)((neg[j] << 3) | i);
    }
    return err;
}

int oracle_walk_group_d(const double *w, const int *neg, const double *h,
                        int g, int c0, int down, int up, const float *S,
                        const float *R, uint8_t *nib_out, double *e_best,
                        double *e_second, int *cand_codes, double *cand_err,
                        int *shift_out, double *e_init);

/* The walk of Eq. 9-13 from a given initial ladder index c0 (Alg.
 * HScaleGroupQuantize takes the baseline's initial scale as an input).
 * Candidate codes are clip(c0 + d, 1, M) for d = -down..up in increasing d;
 * each is scored with Eq. 13; the first minimum wins.  Outputs: chosen code,
 * its nibbles, its error, and the smallest error over candidate codes other
 * than the chosen one (INFINITY when every candidate is the chosen code).
 * cand_codes / cand_err, when non-NULL, receive all down+up+1 candidates. */
int oracle_walk_group(const double *w, const int *neg, const double *h, int g,
                      int c0, int down, int up, const float *S,
                      const float *R, uint8_t *nib_out, double *e_best,
                      double *e_second, int *cand_codes, double *cand_err) {
    return oracle_walk_group_d(w, neg, h, g, c0, down, up, S, R, nib_out,
                               e_best, e_second, cand_codes, cand_err, NULL,
                               NULL);
}

/* The walk, also reporting the chosen shift d* (the first minimum, as in
 * the paper's selected-shift statistics) and the error at d = 0, the
 * initial code's error. */
int oracle_walk_group_d(const double *w, const int *neg, const double *h,
                        int g, int c0, int down, int up, const float *S,
                        const float *R, uint8_t *nib_out, double *e_best,
                        double *e_second, int *cand_codes, double *cand_err,
                        int *shift_out, double *e_init) {
    int best_c = 0, best_d = -down;
    double best_e = 0.0;
    int k = 0;
    for (int d = -down; d <= up; ++d, ++k) {
        int c = c0 + d;
        if (c < 1) c = 1;
        if (c > ORACLE_M) c = ORACLE_M;
        double e = oracle_quantize_group(w, neg, h, g, S[c], R[c], NULL);
        if (cand_codes) cand_codes[k] = c;
        if (cand_err) cand_err[k] = e;
        if (d == 0 && e_init) *e_init = e;
        if (d == -down || e < best_e) {
            best_e = e;
            best_c = c;
            best_d = d;
        }
    }
    if (shift_out) *shift_out = best_d;
    double second = INFINITY;
    for (int d = -down; d <= up; ++d) {
        int c = c0 + d;
        if (c < 1) c = 1;
        if (c > ORACLE_M) c = ORACLE_M;
        if (c == best_c) continue;
        double e = oracle_quantize_group(w, neg, h, g, S[c], R[c], NULL);
        if (e < second) second = e;
    }
    /* Final re-quantization with the chosen scale. */
    oracle_quantize_group(w, neg, h, g, S[best_c], R[best_c], nib_out);
    if (e_best) *e_best = best_e;
    if (e_second) *e_second = second;
    return best_c;
}

/* Windowed search for one group from the max-abs (RTN) initial code. */
int oracle_search_group(const double *w, const int *neg, const double *h,
                        int g, float s_g, int down, int up, const float *S,
                        const float *R, uint8_t *nib_out, double *e_best,
                        double *e_second, int *c0_out, int *cand_codes,
                        double *cand_err) {
    int c0 = oracle_init_code_f(w, g, s_g);
    if (c0_out) *c0_out = c0;
    return oracle_walk_group(w, neg, h, g, c0, down, up, S, R, nib_out,
                             e_best, e_second, cand_codes, cand_err);
}

/* The 4over6 initialisation (App. B, Alg. combining 4over6 with H-Scale):
 * for each anchor a in (4, 6), s_a = max|w| / a in fp32, l_a = Q_fp8(s_a /
 * s_g) in fp32 (clipped to the ladder as in Eq. 10), quantize the group at
 * s_g l_a and score the plain squared error; the initial code is the anchor
 * with the smaller error, the first anchor (4) on a tie.  L4 / L6 and the
 * two anchor codes are returned for reporting. */
int oracle_init_code_4over6(const double *w, const int *neg, int g, float s_g,
                            const float *S, const float *R, double *L4,
                            double *L6, int *c4_out, int *c6_out) {
    static const double anchors[2] = {4.0, 6.0};
    double amax = 0.0;
    for (int j = 0; j < g; ++j)
        if (fabs(w[j]) > amax) amax = fabs(w[j]);
    int code[2];
    double loss[2];
    for (int a = 0; a < 2; ++a) {
        double s_a = rn32(amax / anchors[a]);
        double t = rn32(s_a / (double)s_g);
        int c = oracle_e4m3_round(t);
        if (c < 1) c = 1;
        if (c > ORACLE_M) c = ORACLE_M;
        code[a] = c;
        loss[a] = oracle_quantize_group(w, neg, NULL, g, S[c], R[c], NULL);
    }
    if (L4) *L4 = loss[0];
    if (L6) *L6 = loss[1];
    if (c4_out) *c4_out = code[0];
    if (c6_out) *c6_out = code[1];
    return loss[0] <= loss[1] ? code[0] : code[1];
}

/* ------------------------------------------------------------------------
 * Matrix-level entry points (bf16 inputs, row-major)
 * ---------------------------------------------------------------------- */

/* Eq. 4: h_j = sum_t X[t, j]^2, in fp64, no normalisation. */
void oracle_hdiag(const uint16_t *X, int64_t tokens, int64_t n, double *h) {
    for (int64_t j = 0; j < n; ++j) h[j] = 0.0;
    for (int64_t t = 0; t < tokens; ++t) {
        const uint16_t *row = X + t * n;
        for (int64_t j = 0; j < n; ++j) {
            double x = bf16_value(row[j]);
            h[j] += x * x;
        }
    }
}

/* Streamed calibration: h[j] += sum_t X[t, j]^2 into an fp64 accumulator
 * (Eq. 4 over the concatenation of every batch passed in). */
void oracle_hdiag_accumulate(const uint16_t *X, int64_t tokens, int64_t n,
                             double *h) {
    for (int64_t t = 0; t < tokens; ++t) {
        const uint16_t *row = X + t * n;
        for (int64_t j = 0; j < n; ++j) {
            double x = bf16_value(row[j]);
            h[j] += x * x;
        }
    }
}

/* Loads group (r, i) of a row-major bf16 matrix with n columns. */
static void load_group(const uint16_t *W, int64_t n, int64_t r, int64_t i,
                       double *w, int *neg) {
    const uint16_t *src = W + r * n + i * 16;
    for (int j = 0; j < 16; ++j) {
        w[j] = bf16_value(src[j]);
        neg[j] = bf16_signbit(src[j]);
    }
}

static void store_nibbles(uint8_t *packed, int64_t n, int64_t r, int64_t i,
                          const uint8_t *nib) {
    uint8_t *dst = packed + r * (n / 2) + i * 8;
    for (int k = 0; k < 8; ++k)
        dst[k] = (uint8_t)(nib[2 * k] | (nib[2 * k + 1] << 4));
}

int oracle_search_stats(const uint16_t *W, int64_t m, int64_t n, const float *h,
                        int down, int up, float s_g, int init_mode,
                        const uint8_t *init_codes, uint8_t *codes,
                        uint8_t *packed, double *e_best, double *e_second,
                        uint8_t *c0, double *l4, double *l6, int8_t *shift,
                        double *e_init);

/* Initial-code rules for the matrix-level search. */
#define ORACLE_INIT_RTN 0      /* max-abs scale, Eq. 7 */
#define ORACLE_INIT_4OVER6 1   /* the better of max/4 and max/6 (plain MSE) */
#define ORACLE_INIT_GIVEN 2    /* caller-provided code per group */

/* The search over a whole m x n matrix (n % 16 == 0) with shift set
 * {-down..up} and the given initial-code rule.  codes: [m, n/16] E4M3
 * bytes; packed: [m, n/2] bytes.  init_codes ([m, n/16]) is read for
 * ORACLE_INIT_GIVEN.  e_best / e_second / c0 / l4 / l6 (optional,
 * [m, n/16]) support near-tie reports; l4 / l6 are only written for
 * ORACLE_INIT_4OVER6.  Returns 0, or -1 on a bad argument. */
int oracle_search_init(const uint16_t *W, int64_t m, int64_t n, const float *h,
                       int down, int up, float s_g, int init_mode,
                       const uint8_t *init_codes, uint8_t *codes,
                       uint8_t *packed, double *e_best, double *e_second,
                       uint8_t *c0, double *l4, double *l6) {
    return oracle_search_stats(W, m, n, h, down, up, s_g, init_mode, init_codes,
                               codes, packed, e_best, e_second, c0, l4, l6,
                               NULL, NULL);
}

/* oracle_search_init plus the chosen shift per group (int8 [m, n/16]) and
 * the initial code's error (fp64 [m, n/16]), both optional. */
int oracle_search_stats(const uint16_t *W, int64_t m, int64_t n, const float *h,
                        int down, int up, float s_g, int init_mode,
                        const uint8_t *init_codes, uint8_t *codes,
                        uint8_t *packed, double *e_best, double *e_second,
                        uint8_t *c0, double *l4, double *l6, int8_t *shift,
                        double *e_init) {
    if (n % 16 != 0 || down < 0 || up < 0 || !(s_g > 0.0f)) return -1;
    if (init_mode < 0 || init_mode > 2) return -1;
    if (init_mode == ORACLE_INIT_GIVEN && !init_codes) return -1;
    float S[ORACLE_M + 1], R[ORACLE_M + 1];
    oracle_scale_tables(s_g, S, R);
    int64_t G = n / 16;
    double w[16], hh[16];
    int neg[16];
    uint8_t nib[16];
    for (int64_t r = 0; r < m; ++r) {
        for (int64_t i = 0; i < G; ++i) {
            load_group(W, n, r, i, w, neg);
            for (int j = 0; j < 16; ++j) hh[j] = (double)h[i * 16 + j];
            int c0v;
            double L4 = 0.0, L6 = 0.0;
            if (init_mode == ORACLE_INIT_RTN) {
                c0v = oracle_init_code_f(w, 16, s_g);
            } else if (init_mode == ORACLE_INIT_4OVER6) {
                c0v = oracle_init_code_4over6(w, neg, 16, s_g, S, R, &L4, &L6,
                                              NULL, NULL);
            } else {
                c0v = init_codes[r * G + i];
                if (c0v < 1) c0v = 1;
                if (c0v > ORACLE_M) c0v = ORACLE_M;
            }
            double eb, es, ei = 0.0;
            int dstar = 0;
            int c = oracle_walk_group_d(w, neg, hh, 16, c0v, down, up, S, R, nib,
                                        &eb, &es, NULL, NULL, &dstar, &ei);
            if (shift) shift[r * G + i] = (int8_t)dstar;
            if (e_init) e_init[r * G + i] = ei;
            codes[r * G + i] = (uint8_t)c;
            store_nibbles(packed, n, r, i, nib);
            if (e_best) e_best[r * G + i] = eb;
            if (e_second) e_second[r * G + i] = es;
            if (c0) c0[r * G + i] = (uint8_t)c0v;
            if (l4 && init_mode == ORACLE_INIT_4OVER6) l4[r * G + i] = L4;
            if (l6 && init_mode == ORACLE_INIT_4OVER6) l6[r * G + i] = L6;
        }
    }
    return 0;
}

/* The search from the max-abs initial code (Eq. 7). */
int oracle_search(const uint16_t *W, int64_t m, int64_t n, const float *h,
                  int down, int up, float s_g, uint8_t *codes,
                  uint8_t *packed, double *e_best, double *e_second,
                  uint8_t *c0) {
    return oracle_search_init(W, m, n, h, down, up, s_g, ORACLE_INIT_RTN, NULL,
                              codes, packed, e_best, e_second, c0, NULL, NULL);
}

/* Initial code of every group for a general anchor a (Eq. 7 has a = 6; the
 * 4over6 initialisation compares a = 4 and a = 6):
 * clip(Q_fp8(fp32(fp32(max|w| / a) / s_g)), 1, M).  out: [m, n/16]. */
int oracle_anchor_codes(const uint16_t *W, int64_t m, int64_t n, float s_g,
                        double anchor, uint8_t *out) {
    if (n % 16 != 0 || !(s_g > 0.0f) || !(anchor > 0.0)) return -1;
    int64_t G = n / 16;
    double w[16];
    int neg[16];
    for (int64_t r = 0; r < m; ++r) {
        for (int64_t i = 0; i < G; ++i) {
            load_group(W, n, r, i, w, neg);
            double amax = 0.0;
            for (int j = 0; j < 16; ++j)
                if (fabs(w[j]) > amax) amax = fabs(w[j]);
            int c = oracle_e4m3_round(rn32(rn32(amax / anchor) / (double)s_g));
            if (c < 1) c = 1;
            if (c > ORACLE_M) c = ORACLE_M;
            out[r * G + i] = (uint8_t)c;
        }
    }
    return 0;
}

/* Quantize every group at a given scale code (the final re-quantization
 * step on its own).  err (optional) receives each group's Eq. 13 error
 * under h (h == NULL means h = 1). */
int oracle_quantize(const uint16_t *W, int64_t m, int64_t n, float s_g,
                    const uint8_t *codes, const float *h, uint8_t *packed,
                    double *err) {
    if (n % 16 != 0 || !(s_g > 0.0f)) return -1;
    float S[ORACLE_M + 1], R[ORACLE_M + 1];
    oracle_scale_tables(s_g, S, R);
    int64_t G = n / 16;
    double w[16], hh[16];
    int neg[16];
    uint8_t nib[16];
    for (int64_t r = 0; r < m; ++r) {
        for (int64_t i = 0; i < G; ++i) {
            int c = codes[r * G + i];
            if (c < 1 || c > ORACLE_M) return -1;
            load_group(W, n, r, i, w, neg);
            if (h)
                for (int j = 0; j < 16; ++j) hh[j] = (double)h[i * 16 + j];
            double e = oracle_quantize_group(w, neg, h ? hh : NULL, 16, S[c],
                                             R[c], nib);
            store_nibbles(packed, n, r, i, nib);
            if (err) err[r * G + i] = e;
        }
    }
    return 0;
}

/* Eq. 13's error of every group at every ladder code c = 1..M, for brute
 * force over the whole E4M3 ladder on small inputs.  err: [m, n/16, M]. */
int oracle_all_code_errors(const uint16_t *W, int64_t m, int64_t n,
                           const float *h, float s_g, double *err) {
    if (n % 16 != 0 || !(s_g > 0.0f)) return -1;
    float S[ORACLE_M + 1], R[ORACLE_M + 1];
    oracle_scale_tables(s_g, S, R);
    int64_t G = n / 16;
    double w[16], hh[16];
    int neg[16];
    for (int64_t r = 0; r < m; ++r) {
        for (int64_t i = 0; i < G; ++i) {
            load_group(W, n, r, i, w, neg);
            for (int j = 0; j < 16; ++j) hh[j] = (double)h[i * 16 + j];
            for (int c = 1; c <= ORACLE_M; ++c)
                err[(r * G + i) * ORACLE_M + (c - 1)] =
                    oracle_quantize_group(w, neg, hh, 16, S[c], R[c], NULL);
        }
    }
    return 0;
}

/* Single group on plain fp64 weights (any length g <= 64), for worked
 * examples that are not bf16: quantize at an explicit fp32 scale. */
double oracle_group_at_scale(const double *w, const double *h, int g,
                             float S, uint8_t *nib, double *what) {
    if (g < 0 || g > 64) return -1.0;
    int neg[64] = {0};
    for (int j = 0; j < g; ++j) neg[j] = signbit(w[j]) ? 1 : 0;
    float R = (float)(1.0 / (double)S);
    uint8_t tmp[64];
    double e = oracle_quantize_group(w, neg, h, g, S, R, tmp);
    for (int j = 0; j < g; ++j) {
        if (nib) nib[j] = tmp[j];
        if (what) {
            double q = kE2M1[tmp[j] & 7] * (double)S;
            what[j] = (tmp[j] & 8) ? -q : q;
        }
    }
    return e;
}

/* Single group on plain fp64 weights: the windowed search, exposing every
 * candidate (codes and errors, down+up+1 entries each). */
int oracle_group_search(const double *w, const double *h, int g, float s_g,
                        int down, int up, uint8_t *nib, int *cand_codes,
                        double *cand_err, int *c0) {
    if (g < 0 || g > 64 || down < 0 || up < 0 || !(s_g > 0.0f)) return -1;
    float S[ORACLE_M + 1], R[ORACLE_M + 1];
    oracle_scale_tables(s_g, S, R);
    int neg[64] = {0};
    for (int j = 0; j < g; ++j) neg[j] = signbit(w[j]) ? 1 : 0;
    uint8_t tmp[64];
    int c = oracle_search_group(w, neg, h, g, s_g, down, up, S, R, tmp, NULL,
                                NULL, c0, cand_codes, cand_err);
    if (nib)
        for (int j = 0; j < g; ++j) nib[j] = tmp[j];
    return c;
}

/* ------------------------------------------------------------------------
 * Quality diagnostics (Sec. 3.2 Eq. 3; App. "Selected Scale Shifts" and
 * "Candidate-Window Width")
 * ---------------------------------------------------------------------- */

/* The rounding error Delta W = W - W^ of a stored NVFP4 tensor, in fp64:
 * element (r, j) of group i = j / 16 is w - v * S[c] with c the group's
 * scale code, v the signed E2M1 value of its nibble and S[c] the fp32
 * effective scale of Eq. 1 (S[0] = 0).  The fp64 value is exact: v has two
 * significant bits and S 24, and |w| / S stays below 2^21 for codes >= 1.
 * codes [m, n/16] in 0..M, packed [m, n/2] (element 2k in the low nibble),
 * delta [m, n] row-major. */
int oracle_delta(const uint16_t *W, int64_t m, int64_t n, float s_g,
                 const uint8_t *codes, const uint8_t *packed, double *delta) {
    if (n % 16 != 0 || !(s_g > 0.0f)) return -1;
    float S[ORACLE_M + 1], R[ORACLE_M + 1];
    oracle_scale_tables(s_g, S, R);
    int64_t G = n / 16;
    for (int64_t r = 0; r < m; ++r) {
        for (int64_t j = 0; j < n; ++j) {
            int c = codes[r * G + j / 16];
            if (c > ORACLE_M) return -1;
            uint8_t byte = packed[r * (n / 2) + j / 2];
            int nib = (j % 2 == 0) ? (byte & 15) : (byte >> 4);
            double v = kE2M1[nib & 7];
            if (nib & 8) v = -v;
            uint32_t bits = (uint32_t)W[r * n + j] << 16;
            float wf;
            memcpy(&wf, &bits, sizeof wf);
            delta[r * n + j] = (double)wf - v * (double)S[c];
        }
    }
    return 0;
}

/* Eq. 3, the layer-output error of Delta W on calibration activations X,
 * split by output row: row_err[r] += sum_t (sum_j x_tj * Delta_rj)^2.  The
 * total over r is ||X Delta W^T||_F^2 = Tr(Delta W X^T X Delta W^T), the
 * L_full the paper uses to score a window.  X bf16 [T, n] row-major; delta
 * fp64 [m, n]; plain fp64 loops in t, then j. */
int oracle_output_error(const uint16_t *X, int64_t T, int64_t n,
                        const double *delta, int64_t m, double *row_err) {
    if (T < 0 || n < 0 || m < 0) return -1;
    double *x = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    if (!x) return -1;
    for (int64_t t = 0; t < T; ++t) {
        for (int64_t j = 0; j < n; ++j) {
            uint32_t bits = (uint32_t)X[t * n + j] << 16;
            float xf;
            memcpy(&xf, &bits, sizeof xf);
            x[j] = (double)xf;
        }
        for (int64_t r = 0; r < m; ++r) {
            double y = 0.0;
            for (int64_t j = 0; j < n; ++j) y += x[j] * delta[r * n + j];
            row_err[r] += y * y;
        }
    }
    free(x);
    return 0;
}

/* The selected-shift statistics: for every shift d = -down..up (bin
 * d + down), the number of groups that chose it, the sums of their errors
 * at d = 0 and at the chosen shift, and the sum of their relative
 * reductions (e_init - e_best) / e_init (0 for a group whose initial error
 * is 0).  The mean reduction of a bin is sum_rel / count; the fraction of
 * the initial error removed is 1 - sum(sum_best) / sum(sum_init). */
int oracle_shift_summary(const int8_t *shift, const double *e_best,
                         const double *e_init, int64_t groups, int down,
                         int up, int64_t *count, double *sum_init,
                         double *sum_best, double *sum_rel) {
    if (groups < 0 || down < 0 || up < 0) return -1;
    for (int k = 0; k <= down + up; ++k) {
        count[k] = 0;
        sum_init[k] = sum_best[k] = sum_rel[k] = 0.0;
    }
    for (int64_t g = 0; g < groups; ++g) {
        int d = shift[g];
        if (d < -down || d > up) return -1;
        int k = d + down;
        count[k] += 1;
        sum_init[k] += e_init[g];
        sum_best[k] += e_best[g];
        if (e_init[g] > 0.0) sum_rel[k] += (e_init[g] - e_best[g]) / e_init[g];
    }
    return 0;
}
