// Host sanitizer driver for the library's C ABI (built with host-side
// -fsanitize=address,undefined by tests/test_sanitizers_cpu.py): every entry
// point with arguments its checks reject, which return before any HIP call,
// and the workspace cap, which fails the output error's allocation before it
// reaches the device.  No GPU is needed.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "mpq.h"

static int fails = 0;
static void expect(int got, int want, const char *what)
{
    if (got != want) {
        printf("%s: got %d, want %d (%s)\n", what, got, want, mpq_last_error());
        ++fails;
    }
}

int main()
{
    float *W = (float *)16, *S = (float *)32, *E = (float *)48, *Xf = (float *)64;
    int8_t *Q = (int8_t *)80;
    int32_t *N = (int32_t *)96;
    const int I = MPQ_ERR_INVALID_ARG;
    expect(mpq_fit_layer(W, -1, 4, 4, 2, nullptr, 8, 1e-3f, Q, S, N, nullptr, nullptr), I, "c_out < 0");
    expect(mpq_fit_layer(W, 4, 0, 4, 2, nullptr, 8, 1e-3f, Q, S, N, nullptr, nullptr), I, "d < 1");
    expect(mpq_fit_layer(W, 4, 4, 9, 2, nullptr, 8, 1e-3f, Q, S, N, nullptr, nullptr), I, "bits");
    float grid[3] = {0.5f, 0.25f, 1.0f};
    expect(mpq_fit_layer(W, 4, 4, 4, 2, grid, 3, 1e-3f, Q, S, N, nullptr, nullptr), I, "grid order");
    expect(mpq_fit_layer_dense(W, 4, 4, 4, 0, nullptr, 8, 1e-3f, Q, S, N, nullptr, nullptr), I,
           "max_points");
    expect(mpq_output_error(W, Q, S, N, 4, 4, 2, Xf, 0, E, nullptr, nullptr), I, "n < 1");
    expect(mpq_output_error_noalloc(W, Q, S, N, 4, 4, 2, nullptr, 8, E, nullptr, nullptr), I, "X NULL");
    expect(mpq_reconstruct(Q, S, N, 4, 4, 65, W, nullptr), I, "max_points > 64");
    mpq_layer L[2];
    memset(L, 0, sizeof L);
    L[0].W = W; L[0].c_out = 4; L[0].d = 4; L[0].codes = Q; L[0].scales = S; L[0].counts = N;
    L[1] = L[0];
    L[1].d = -3;
    expect(mpq_fit_layers(L, 2, 4, 4, nullptr, 8, 1e-3f, nullptr), I, "layer d");
    expect(mpq_quantize_layers(L, 2, 4, 4, nullptr, 8, -1.0f, nullptr), I, "tol < 0");
    expect(mpq_fit_layers_calib(L, 2, 4, 4, nullptr, 8, -1.0f, 1, nullptr), I, "eps < 0");
    mpq_fit_options o;
    memset(&o, 0, sizeof o);
    o.gate = 1;
    o.clip_grid = 20;
    L[1].d = 4;
    expect(mpq_fit_layers_ex(L, 2, 4, 4, nullptr, 8, 1e-3f, &o, nullptr), I, "gate with clip");
    expect(mpq_integer_scales(S, N, 4, 4, 63, nullptr, nullptr, nullptr), I, "p > 62");
    expect(mpq_integer_forward(Q, N, N, 4, 0, 4, Q, 4, 8, nullptr, nullptr), I, "d < 1");
    expect(mpq_fit_max_dim(0), I, "n_grid 0");
    char name[8];
    expect(mpq_fit_kernel_of(0, 4, 8, 1, name, 8), I, "kernel_of d");
    expect(mpq_timing_only("0123456789012345678901234567890123456789012345678901234567890123456789"),
           I, "timing name");
    // the workspace cap: the output error's scratch request fails before any HIP call
    setenv("MPQ_WORKSPACE_LIMIT", "64", 1);
    expect(mpq_output_error(W, Q, S, N, 4, 16, 2, Xf, 8, E, nullptr, nullptr), MPQ_ERR_NOMEM,
           "workspace cap");
    if (!strstr(mpq_last_error(), "scratch")) {
        printf("workspace cap: unexpected error text '%s'\n", mpq_last_error());
        ++fails;
    }
    unsetenv("MPQ_WORKSPACE_LIMIT");
    printf(fails ? "sanitized ABI checks: %d failures\n" : "sanitized ABI checks: ok\n", fails);
    return fails ? 1 : 0;
}
