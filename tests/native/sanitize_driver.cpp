// Host-side memory and undefined-behaviour check of the oracle and of the
// library's argument validation, built with -fsanitize=address,undefined for
// the host only.  Every library call here fails validation or is empty, so
// nothing reaches the GPU; the oracle runs a small problem end to end.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "hscale.h"

extern "C" {
int oracle_search_init(const uint16_t *W, int64_t m, int64_t n, const float *h, int down, int up, float s_g,
                       int init_mode, const uint8_t *init_codes, uint8_t *codes, uint8_t *packed, double *e_best,
                       double *e_second, uint8_t *c0, double *l4, double *l6);
void oracle_hdiag(const uint16_t *X, int64_t tokens, int64_t n, double *h);
int oracle_quantize(const uint16_t *W, int64_t m, int64_t n, float s_g, const uint8_t *codes, const float *h,
                    uint8_t *packed, double *err);
int oracle_all_code_errors(const uint16_t *W, int64_t m, int64_t n, const float *h, float s_g, double *err);
int oracle_search_stats(const uint16_t *W, int64_t m, int64_t n, const float *h, int down, int up, float s_g,
                        int init_mode, const uint8_t *init_codes, uint8_t *codes, uint8_t *packed, double *e_best,
                        double *e_second, uint8_t *c0, double *l4, double *l6, int8_t *shift, double *e_init);
int oracle_delta(const uint16_t *W, int64_t m, int64_t n, float s_g, const uint8_t *codes, const uint8_t *packed,
                 double *delta);
int oracle_output_error(const uint16_t *X, int64_t T, int64_t n, const double *delta, int64_t m, double *row_err);
int oracle_shift_summary(const int8_t *shift, const double *e_best, const double *e_init, int64_t groups, int down,
                         int up, int64_t *count, double *sum_init, double *sum_best, double *sum_rel);
}

static uint16_t bf16(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

int main() {
    int bad = 0;
    // Oracle: a small problem through every entry point.
    const int m = 8, n = 64, T = 32;
    std::vector<uint16_t> W(m * n), X(T * n);
    for (int i = 0; i < m * n; ++i) W[i] = bf16(std::sin(0.37f * i) * 0.05f);
    for (int i = 0; i < T * n; ++i) X[i] = bf16(std::cos(0.11f * i));
    std::vector<double> h64(n);
    oracle_hdiag(X.data(), T, n, h64.data());
    std::vector<float> h(n);
    for (int j = 0; j < n; ++j) h[j] = (float)h64[j];
    const int G = n / 16;
    std::vector<uint8_t> codes(m * G), packed(m * n / 2), c0(m * G), init(m * G, 200);
    std::vector<double> eb(m * G), es(m * G), l4(m * G), l6(m * G), err(m * G), all(m * G * 126);
    for (int mode = 0; mode < 3; ++mode)
        bad |= oracle_search_init(W.data(), m, n, h.data(), 9, 6, 1e-4f, mode, init.data(), codes.data(),
                                  packed.data(), eb.data(), es.data(), c0.data(), l4.data(), l6.data()) != 0;
    bad |= oracle_quantize(W.data(), m, n, 1e-4f, codes.data(), h.data(), packed.data(), err.data()) != 0;
    bad |= oracle_all_code_errors(W.data(), m, n, h.data(), 1e-4f, all.data()) != 0;
    bad |= oracle_search_init(W.data(), m, 15, h.data(), 4, 4, 1e-4f, 0, nullptr, codes.data(), packed.data(),
                              nullptr, nullptr, nullptr, nullptr, nullptr) != -1;
    std::vector<int8_t> shift(m * G);
    std::vector<double> ei(m * G), delta(m * n), row(m, 0.0), si(16), sb(16), sr(16);
    std::vector<int64_t> cnt(16);
    bad |= oracle_search_stats(W.data(), m, n, h.data(), 9, 6, 1e-4f, 0, nullptr, codes.data(), packed.data(),
                               eb.data(), es.data(), c0.data(), l4.data(), l6.data(), shift.data(), ei.data()) != 0;
    bad |= oracle_delta(W.data(), m, n, 1e-4f, codes.data(), packed.data(), delta.data()) != 0;
    bad |= oracle_output_error(X.data(), T, n, delta.data(), m, row.data()) != 0;
    bad |= oracle_shift_summary(shift.data(), eb.data(), ei.data(), m * G, 9, 6, cnt.data(), si.data(), sb.data(),
                                sr.data()) != 0;

    // Library validation: fake, aligned addresses; every call must be rejected
    // (or be empty) before any launch.
    char *A = reinterpret_cast<char *>(uintptr_t(1) << 20);
    const size_t ws = hscale_hdiag_workspace_bytes(64, 32);
    bad |= hscale_hdiag(A, 64, 33, (float *)(A + 4096), A + 8192, ws, nullptr) != HSCALE_ERR_SHAPE;
    bad |= hscale_hdiag(A, 64, 32, (float *)(A + 64), A + 8192, ws, nullptr) != HSCALE_ERR_OVERLAP;
    bad |= hscale_hdiag(A, 64, 32, (float *)(A + 4096), A + 8192, ws - 1, nullptr) != HSCALE_ERR_WORKSPACE;
    bad |= hscale_search(A, 4, 64, (float *)(A + 4096), 126, 1e-3f, (uint8_t *)(A + 8192),
                         (uint8_t *)(A + 12288), nullptr) != HSCALE_ERR_WINDOW;
    bad |= hscale_search(A, 4, 64, (float *)(A + 4096), 4, NAN, (uint8_t *)(A + 8192), (uint8_t *)(A + 12288),
                         nullptr) != HSCALE_ERR_SCALE;
    bad |= hscale_search_block(A, 68, 4, 64, (float *)(A + 4096), 4, 4, 1e-3f, 0, nullptr, 0,
                               (uint8_t *)(A + 8192), 4, (uint8_t *)(A + 12288), 32, nullptr) != HSCALE_ERR_ALIGN;
    bad |= hscale_search_from(A, 4, 64, (float *)(A + 4096), 4, 4, 1e-3f, nullptr, (uint8_t *)(A + 8192),
                              (uint8_t *)(A + 12288), nullptr) != HSCALE_ERR_NULL;
    bad |= hscale_quantize(A, 0, 64, 1e-3f, nullptr, nullptr, nullptr) != HSCALE_OK;
    bad |= hscale_hdiag_finalize(nullptr, 0, nullptr, nullptr) != HSCALE_OK;
    bad |= hscale_search_stats(A, 4, 64, (float *)(A + 4096), 4, 4, 1e-3f, 0, nullptr, (uint8_t *)(A + 8192),
                               (uint8_t *)(A + 12288), (int8_t *)(A + 16384), (float *)(A + 16386),
                               (float *)(A + 20480), nullptr) != HSCALE_ERR_ALIGN;
    bad |= hscale_shift_summary_workspace_bytes(5000, 9, 6) == 0;
    bad |= hscale_shift_summary((int8_t *)A, (float *)(A + 4096), (float *)(A + 8192), 1000, 9, 6,
                                (uint64_t *)(A + 12288), (double *)(A + 12296), (double *)(A + 16384),
                                (double *)(A + 20480), A + 24576, 1 << 20, nullptr) != HSCALE_ERR_OVERLAP;
    {
        hscale_layer L[3] = {};
        for (int k = 0; k < 3; ++k) {
            char *b = A + (k + 1) * (1 << 16);
            L[k] = hscale_layer{b, 4, 64, (const float *)(b + 4096), 1e-3f, nullptr, (uint8_t *)(b + 8192),
                                (uint8_t *)(b + 12288)};
        }
        bad |= hscale_search_layers(nullptr, 0, 4, 4, 0, nullptr) != HSCALE_OK;
        bad |= hscale_search_layers(L, 3, 126, 4, 0, nullptr) != HSCALE_ERR_WINDOW;
        bad |= hscale_search_layers(L, 3, 4, 4, 2, nullptr) != HSCALE_ERR_NULL;
        hscale_layer over[2] = {L[0], L[1]};
        over[1].scale_codes = (uint8_t *)L[0].W;
        bad |= hscale_search_layers(over, 2, 4, 4, 0, nullptr) != HSCALE_ERR_OVERLAP;
        hscale_layer empty[2] = {L[0], L[1]};
        empty[0].out = 0;
        empty[1].in = 0;
        bad |= hscale_search_layers(empty, 2, 4, 4, 0, nullptr) != HSCALE_OK;
    }
    for (int s = -9; s <= 1; ++s) bad |= hscale_status_string(s) == nullptr;
    std::printf(bad ? "sanitize driver: FAILED\n" : "sanitize driver: ok\n");
    return bad;
}
