/* Host sanitizer driver for the oracle (built with -fsanitize=address,undefined
 * by tests/test_sanitizers_cpu.py): every entry point on small inputs,
 * including the option paths and edge channels (zero, one element, equal
 * magnitudes).  Exits nonzero on a wrong status; the sanitizers abort on any
 * memory or undefined-behaviour error. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_levels(int bits);
int oracle_fit_ex(const float *W, int64_t C, int64_t d, int bits, int P, const float *grid, int G,
                  double tol, const float *X, int64_t N, int calib, double eps, int relative,
                  int refit, int clipG, double eta, int gate, float *offsets, int8_t *codes,
                  float *scales, int32_t *counts, double *err, double *xerr, int n_threads);
int oracle_verify_ex(const float *W, int64_t C, int64_t d, int bits, int P, const float *grid,
                     int G, double tol, const float *X, int64_t N, int calib, double eps,
                     int relative, int refit, int clipG, double eta, int gate,
                     const float *offsets, const int8_t *codes, const float *scales,
                     const int32_t *counts, const float *err, const float *xerr,
                     const int64_t *chan, int64_t n_chan, int32_t *status, int32_t *cand_ties,
                     int32_t *code_ties, int32_t *stop_ties, double *err_relmax, int n_threads);
int oracle_output_error_ex(const float *W, const float *offsets, const int8_t *codes,
                           const float *scales, const int32_t *counts, int64_t C, int64_t d, int P,
                           const float *X, int64_t N, const int64_t *chan, int64_t n_chan,
                           double *err, double *ref, int n_threads);
void oracle_reconstruct_ex(const float *offsets, const int8_t *codes, const float *scales,
                           const int32_t *counts, int64_t C, int64_t d, int P, float *W_hat);
int64_t oracle_integer_scales(const float *scales, const int32_t *counts, int64_t C, int P, int p,
                              int32_t *A);
int oracle_integer_forward(const int8_t *codes, const int32_t *A, const int32_t *counts, int64_t C,
                           int64_t d, int P, const int8_t *X, int64_t N, int p, int64_t *Y);

static uint64_t rng = 88172645463325252ull;
static double urand(void)
{
    rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
    return (double)(rng >> 11) / 9007199254740992.0;
}

int main(void)
{
    const int64_t C = 6, d = 13, N = 9;
    const int bits = 3, P = 4, G = 16;
    float W[6 * 13], X[13 * 9];
    for (int i = 0; i < C * d; ++i) W[i] = (float)(urand() * 2.0 - 1.0);
    for (int i = 0; i < d * N; ++i) X[i] = (float)(urand() * 2.0 - 1.0);
    memset(W, 0, sizeof(float) * d);                 /* a zero channel */
    for (int j = 0; j < d; ++j) W[d + j] = (j % 2) ? 0.5f : -0.5f;   /* equal magnitudes */
    int8_t codes[6 * 4 * 13];
    float scales[6 * 4], offsets[6], W_hat[6 * 13];
    int32_t counts[6], status[6], ct[6], qt[6], st[6];
    double err[6 * 4], xerr[6 * 4], relmax[6], e[6], r[6];
    float err32[6 * 4], xerr32[6 * 4];
    int64_t chan[6] = {0, 1, 2, 3, 4, 5};
    int bad = 0;
    /* option sets: plain, calib (relative / absolute), refit, clip, paper grid, asym, gate */
    const int opts[][8] = {
        /* calib relative refit clipG gate asym paper(1/0) */
        {0, 0, 0, 0, 0, 0, 0, 0}, {1, 1, 0, 0, 0, 0, 0, 0}, {1, 0, 0, 0, 0, 0, 0, 0},
        {0, 0, 1, 0, 0, 0, 0, 0}, {0, 0, 0, 5, 0, 0, 0, 0}, {1, 1, 0, 5, 0, 0, 0, 0},
        {0, 0, 0, 0, 0, 0, 1, 0}, {0, 0, 0, 0, 0, 1, 0, 0}, {1, 1, 0, 0, 1, 0, 0, 0},
        {0, 0, 0, 0, 1, 1, 0, 0}, {1, 0, 1, 0, 1, 0, 0, 0}};
    for (size_t o = 0; o < sizeof opts / sizeof opts[0]; ++o) {
        const int calib = opts[o][0], rel = opts[o][1], refit = opts[o][2], clipG = opts[o][3];
        const int gate = opts[o][4], asym = opts[o][5];
        const double eta = opts[o][6] ? 1.0 / 64.0 : 0.0;
        const double tol = 1e-2, eps = rel ? 1e-2 : 1e-3;
        if (oracle_fit_ex(W, C, d, bits, P, NULL, G, tol, X, N, calib, eps, rel, refit, clipG, eta,
                          gate, asym ? offsets : NULL, codes, scales, counts, err, xerr, 2) != 0) {
            printf("fit failed (option set %zu)\n", o);
            return 1;
        }
        for (int i = 0; i < C * P; ++i) { err32[i] = (float)err[i]; xerr32[i] = (float)xerr[i]; }
        if (oracle_verify_ex(W, C, d, bits, P, NULL, G, tol, X, N, calib, eps, rel, refit, clipG, eta,
                             gate, asym ? offsets : NULL, codes, scales, counts, err32,
                             calib ? xerr32 : NULL, chan, C, status, ct, qt, st, relmax, 2) != 0) {
            printf("verify failed (option set %zu)\n", o);
            return 1;
        }
        for (int k = 0; k < C; ++k)
            if (status[k] != 0) { printf("option set %zu channel %d status %d\n", o, k, status[k]); bad = 1; }
        if (oracle_output_error_ex(W, asym ? offsets : NULL, codes, scales, counts, C, d, P, X, N, NULL,
                                   0, e, r, 2) != 0) return 1;
        oracle_reconstruct_ex(asym ? offsets : NULL, codes, scales, counts, C, d, P, W_hat);
    }
    int32_t A[6 * 4];
    int8_t Xi[9 * 13];
    int64_t Y[6 * 9];
    for (int i = 0; i < N * d; ++i) Xi[i] = (int8_t)((int)(urand() * 255.0) - 127);
    (void)oracle_integer_scales(scales, counts, C, P, 16, A);
    if (oracle_integer_forward(codes, A, counts, C, d, P, Xi, N, 16, Y) != 0) bad = 1;
    if (oracle_levels(bits) != 3) bad = 1;
    printf(bad ? "sanitized oracle: wrong results\n" : "sanitized oracle: ok\n");
    return bad;
}
