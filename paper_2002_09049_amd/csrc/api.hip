// C ABI of the library (declared in include/mpq.h): argument checks, device
// limits, scratch allocation and kernel launches.  Argument checks run before
// any HIP call, so an invalid call never touches the device.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <string>

#include "internal.hpp"
#include "mpq.h"

namespace {

thread_local std::string g_last_error;

int fail(int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

int hip_fail(hipError_t e, const char *what)
{
    return fail(MPQ_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

// Largest dynamic LDS a workgroup may use on the current device.
int device_lds_limit(size_t *bytes)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    int v = 0;
    e = hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute(MaxSharedMemoryPerBlock)");
    // the fit kernel also holds ~1 KiB of static LDS
    *bytes = v > 2048 ? (size_t)v - 2048 : 0;
    return MPQ_OK;
}

int check_fit_args(const float *W, int64_t c_out, int64_t d, int bits, int max_points,
                   const float *grid_host, int n_grid, float tol, const int8_t *codes,
                   const float *scales, const int32_t *counts)
{
    if (c_out < 0) return fail(MPQ_ERR_INVALID_ARG, "c_out must be >= 0 (got %lld)", (long long)c_out);
    if (d < 1) return fail(MPQ_ERR_INVALID_ARG, "d must be >= 1 (got %lld)", (long long)d);
    if (bits < 2 || bits > MPQ_MAX_BITS)
        return fail(MPQ_ERR_INVALID_ARG, "bits must be in [2, %d] (got %d)", MPQ_MAX_BITS, bits);
    if (max_points < 1 || max_points > MPQ_MAX_POINTS)
        return fail(MPQ_ERR_INVALID_ARG, "max_points must be in [1, %d] (got %d)", MPQ_MAX_POINTS,
                    max_points);
    if (n_grid < 1 || n_grid > MPQ_MAX_GRID)
        return fail(MPQ_ERR_INVALID_ARG, "n_grid must be in [1, %d] (got %d)", MPQ_MAX_GRID, n_grid);
    if (!(tol >= 0.0f) || !isfinite(tol))
        return fail(MPQ_ERR_INVALID_ARG, "tol must be finite and >= 0");
    if (grid_host) {
        for (int g = 0; g < n_grid; ++g) {
            const float c = grid_host[g];
            if (!(c > 0.0f && c <= 1.0f))
                return fail(MPQ_ERR_INVALID_ARG, "grid[%d] = %g is outside (0, 1]", g, (double)c);
            if (g > 0 && !(c > grid_host[g - 1]))
                return fail(MPQ_ERR_INVALID_ARG, "grid must be strictly ascending (grid[%d])", g);
        }
    }
    if (c_out > 0 && (!W || !codes || !scales || !counts))
        return fail(MPQ_ERR_INVALID_ARG, "W, codes, scales and counts must not be NULL");
    if (c_out > 0x7fffffffLL)
        return fail(MPQ_ERR_INVALID_ARG, "c_out too large (%lld)", (long long)c_out);
    return MPQ_OK;
}

}  // namespace

namespace mpq {

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_pool_mu;
hipMemPool_t g_pool[kMaxDevices];
}  // namespace

hipError_t scratch_alloc(void **p, size_t bytes, hipStream_t s)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    hipMemPool_t pool;
    {
        std::lock_guard<std::mutex> lk(g_pool_mu);
        if (!g_pool[dev]) {
            hipMemPoolProps props = {};
            props.allocType = hipMemAllocationTypePinned;
            props.location.type = hipMemLocationTypeDevice;
            props.location.id = dev;
            e = hipMemPoolCreate(&g_pool[dev], &props);
            if (e != hipSuccess) return e;
            uint64_t keep = ~(uint64_t)0;
            e = hipMemPoolSetAttribute(g_pool[dev], hipMemPoolAttrReleaseThreshold, &keep);
            if (e != hipSuccess) return e;
        }
        pool = g_pool[dev];
    }
    return hipMallocFromPoolAsync(p, bytes == 0 ? 256 : bytes, pool, s);
}

hipError_t scratch_free(void *p, hipStream_t s) { return hipFreeAsync(p, s); }

}  // namespace mpq

extern "C" {

const char *mpq_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"

namespace {

int64_t dense_max_dim(int n_grid, size_t lim)
{
    // bisect the largest d whose dense layout fits
    int64_t lo = 0, hi = 1 << 22;
    while (lo < hi) {
        const int64_t mid = (lo + hi + 1) / 2;
        if (mpq::fit_layout(mid, n_grid).lds <= lim) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

enum class Search { kAuto, kDense };

int fit_layer_impl(Search mode, const float *W, int64_t c_out, int64_t d, int bits, int max_points,
                   const float *grid_host, int n_grid, float tol, int8_t *codes, float *scales,
                   int32_t *counts, float *err_opt, void *stream)
{
    int rc = check_fit_args(W, c_out, d, bits, max_points, grid_host, n_grid, tol, codes, scales,
                            counts);
    if (rc != MPQ_OK) return rc;
    if (c_out == 0) return MPQ_OK;
    size_t lim = 0;
    rc = device_lds_limit(&lim);
    if (rc != MPQ_OK) return rc;
    const bool hist = mode == Search::kAuto && mpq::fit_hist_supports(d) &&
                      mpq::fit_hist_lds(n_grid) <= lim;
    const mpq::FitLayout L = mpq::fit_layout(d, n_grid);
    if (!hist && L.lds > lim)
        return fail(MPQ_ERR_SHAPE, "d = %lld with n_grid = %d needs %zu bytes of LDS (limit %zu)",
                    (long long)d, n_grid, L.lds, lim);
    hipStream_t s = (hipStream_t)stream;
    float *dgrid = nullptr;
    if (grid_host) {
        hipError_t e = mpq::scratch_alloc((void **)&dgrid, sizeof(float) * (size_t)n_grid, s);
        if (e != hipSuccess) return fail(MPQ_ERR_NOMEM, "grid upload: %s", hipGetErrorString(e));
        e = hipMemcpyAsync(dgrid, grid_host, sizeof(float) * (size_t)n_grid, hipMemcpyHostToDevice, s);
        if (e != hipSuccess) {
            (void)mpq::scratch_free(dgrid, s);
            return hip_fail(e, "hipMemcpyAsync(grid)");
        }
    }
    mpq::FitParams p;
    p.W = W;
    p.C = c_out;
    p.d = d;
    p.M = (1 << (bits - 1)) - 1;
    p.P = max_points;
    p.grid = dgrid;
    p.G = n_grid;
    p.tol = (double)tol;
    p.codes = codes;
    p.scales = scales;
    p.counts = counts;
    p.err = err_opt;
    hipError_t e = hist ? mpq::launch_fit_hist(p, s) : mpq::launch_fit(p, L, s);
    if (dgrid) (void)mpq::scratch_free(dgrid, s);
    if (e != hipSuccess) return hip_fail(e, "fit kernel launch");
    return MPQ_OK;
}

}  // namespace

extern "C" {

int64_t mpq_fit_max_dim(int n_grid)
{
    if (n_grid < 1 || n_grid > MPQ_MAX_GRID)
        return fail(MPQ_ERR_INVALID_ARG, "n_grid must be in [1, %d] (got %d)", MPQ_MAX_GRID, n_grid);
    size_t lim = 0;
    int rc = device_lds_limit(&lim);
    if (rc != MPQ_OK) return rc;
    int64_t dmax = dense_max_dim(n_grid, lim);
    if (mpq::fit_hist_lds(n_grid) <= lim && mpq::kHistMaxDim > dmax) dmax = mpq::kHistMaxDim;
    return dmax;
}

int mpq_fit_layer(const float *W, int64_t c_out, int64_t d, int bits, int max_points,
                  const float *grid_host, int n_grid, float tol, int8_t *codes, float *scales,
                  int32_t *counts, float *err_opt, void *stream)
{
    return fit_layer_impl(Search::kAuto, W, c_out, d, bits, max_points, grid_host, n_grid, tol,
                          codes, scales, counts, err_opt, stream);
}

int mpq_fit_layer_dense(const float *W, int64_t c_out, int64_t d, int bits, int max_points,
                        const float *grid_host, int n_grid, float tol, int8_t *codes,
                        float *scales, int32_t *counts, float *err_opt, void *stream)
{
    return fit_layer_impl(Search::kDense, W, c_out, d, bits, max_points, grid_host, n_grid, tol,
                          codes, scales, counts, err_opt, stream);
}

int mpq_output_error(const float *W, const int8_t *codes, const float *scales,
                     const int32_t *counts, int64_t c_out, int64_t d, int max_points,
                     const float *X, int64_t n, float *err, float *ref_opt, void *stream)
{
    if (c_out < 0) return fail(MPQ_ERR_INVALID_ARG, "c_out must be >= 0 (got %lld)", (long long)c_out);
    if (d < 1) return fail(MPQ_ERR_INVALID_ARG, "d must be >= 1 (got %lld)", (long long)d);
    if (n < 1) return fail(MPQ_ERR_INVALID_ARG, "n must be >= 1 (got %lld)", (long long)n);
    if (max_points < 1 || max_points > MPQ_MAX_POINTS)
        return fail(MPQ_ERR_INVALID_ARG, "max_points must be in [1, %d] (got %d)", MPQ_MAX_POINTS,
                    max_points);
    if (c_out > 0 && (!W || !codes || !scales || !counts || !X || !err))
        return fail(MPQ_ERR_INVALID_ARG, "W, codes, scales, counts, X and err must not be NULL");
    if ((c_out + 127) / 128 > 65535)
        return fail(MPQ_ERR_INVALID_ARG, "c_out too large (%lld)", (long long)c_out);
    if ((n + 127) / 128 > 0x7fffffffLL)
        return fail(MPQ_ERR_INVALID_ARG, "n too large (%lld)", (long long)n);
    if (c_out == 0) return MPQ_OK;
    hipStream_t s = (hipStream_t)stream;
    void *scratch = nullptr;
    const size_t bytes = mpq::err_scratch_bytes(c_out, d, n);
    hipError_t e = mpq::scratch_alloc(&scratch, bytes, s);
    if (e != hipSuccess) return fail(MPQ_ERR_NOMEM, "scratch of %zu bytes: %s", bytes, hipGetErrorString(e));
    e = mpq::launch_output_error(W, codes, scales, counts, c_out, d, max_points, X, n, err, ref_opt,
                                 scratch, s);
    (void)mpq::scratch_free(scratch, s);
    if (e != hipSuccess) return hip_fail(e, "output error kernel launch");
    return MPQ_OK;
}

int mpq_reconstruct(const int8_t *codes, const float *scales, const int32_t *counts, int64_t c_out,
                    int64_t d, int max_points, float *W_hat, void *stream)
{
    if (c_out < 0) return fail(MPQ_ERR_INVALID_ARG, "c_out must be >= 0 (got %lld)", (long long)c_out);
    if (d < 1) return fail(MPQ_ERR_INVALID_ARG, "d must be >= 1 (got %lld)", (long long)d);
    if (max_points < 1 || max_points > MPQ_MAX_POINTS)
        return fail(MPQ_ERR_INVALID_ARG, "max_points must be in [1, %d] (got %d)", MPQ_MAX_POINTS,
                    max_points);
    if (c_out > 0 && (!codes || !scales || !counts || !W_hat))
        return fail(MPQ_ERR_INVALID_ARG, "codes, scales, counts and W_hat must not be NULL");
    if (c_out == 0) return MPQ_OK;
    hipError_t e = mpq::launch_reconstruct(codes, scales, counts, c_out, d, max_points, W_hat,
                                           (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "reconstruct kernel launch");
    return MPQ_OK;
}

}  // extern "C"
