// C ABI of the library (declared in include/mpq.h): argument checks, device
// limits, scratch allocation and kernel launches.  Argument checks run before
// any HIP call, so an invalid call never touches the device.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

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

// Largest dynamic LDS a workgroup may use on the current device (queried
// once per device).
constexpr int kMaxDevices = 64;
std::mutex g_lds_mu;
size_t g_lds_limit[kMaxDevices];

int device_lds_limit(size_t *bytes)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(MPQ_ERR_HIP, "device index %d out of range", dev);
    std::lock_guard<std::mutex> lk(g_lds_mu);
    if (g_lds_limit[dev] == 0) {
        int v = 0;
        e = hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
        if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute(MaxSharedMemoryPerBlock)");
        // the fit kernels also hold ~1 KiB of static LDS
        g_lds_limit[dev] = v > 2048 ? (size_t)v - 2048 : 1;
    }
    *bytes = g_lds_limit[dev];
    return MPQ_OK;
}

int check_fit_layer(const float *W, int64_t c_out, int64_t d, const int8_t *codes,
                    const float *scales, const int32_t *counts)
{
    if (c_out < 0) return fail(MPQ_ERR_INVALID_ARG, "c_out must be >= 0 (got %lld)", (long long)c_out);
    if (d < 1) return fail(MPQ_ERR_INVALID_ARG, "d must be >= 1 (got %lld)", (long long)d);
    if (c_out > 0 && (!W || !codes || !scales || !counts))
        return fail(MPQ_ERR_INVALID_ARG, "W, codes, scales and counts must not be NULL");
    if (c_out > 0x7fffffffLL)
        return fail(MPQ_ERR_INVALID_ARG, "c_out too large (%lld)", (long long)c_out);
    return MPQ_OK;
}

int check_fit_args(int bits, int max_points, const float *grid_host, int n_grid, float tol)
{
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
    return MPQ_OK;
}

}  // namespace

namespace mpq {

namespace {
std::mutex g_pool_mu;
hipMemPool_t g_pool[kMaxDevices];
}  // namespace

// MPQ_WORKSPACE_LIMIT (bytes, decimal): a cap on each stream-ordered scratch
// allocation, checked before any HIP call; a request above it fails as an
// allocation would (the calls then return MPQ_ERR_NOMEM).  Unset: no cap.
static bool over_workspace_limit(size_t bytes)
{
    const char *v = getenv("MPQ_WORKSPACE_LIMIT");
    if (!v || !*v) return false;
    char *end = nullptr;
    const unsigned long long lim = strtoull(v, &end, 10);
    return end && *end == '\0' && (unsigned long long)bytes > lim;
}

hipError_t scratch_alloc(void **p, size_t bytes, hipStream_t s)
{
    if (over_workspace_limit(bytes)) return hipErrorOutOfMemory;
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

namespace {

// Library-owned streams (default priority) on which the independent launches
// of one call run side by side: forked from the caller's stream by an event
// and joined back to it by one event per stream, so the call stays ordered on
// the caller's stream.  One set per device; its mutex serializes the enqueue
// of concurrent callers.  Each call re-records the events; a wait that is
// already enqueued keeps the record it saw.
constexpr int kForkStreams = 3;   // besides the caller's stream

struct ForkPool {
    std::mutex mu;
    bool ready = false;
    hipStream_t st[kForkStreams];
    hipEvent_t fork;
    hipEvent_t join[kForkStreams];
};
ForkPool g_fork[kMaxDevices];

// Creates the pool's streams and events on first use (mu held).
hipError_t fork_pool_init(ForkPool &F)
{
    if (F.ready) return hipSuccess;
    hipError_t e = hipEventCreateWithFlags(&F.fork, hipEventDisableTiming);
    for (int i = 0; i < kForkStreams && e == hipSuccess; ++i) {
        e = hipStreamCreateWithFlags(&F.st[i], hipStreamNonBlocking);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&F.join[i], hipEventDisableTiming);
    }
    F.ready = e == hipSuccess;
    return e;
}

// Runs launch(j, stream) for the jobs 0..n-1, longest work first, each on the
// least loaded of the caller's stream and up to kForkStreams pool streams.
// Falls back to the caller's stream alone when the pool cannot be created.
template <class Launch>
hipError_t run_concurrently(hipStream_t s, const std::vector<double> &work, Launch launch)
{
    const int n = (int)work.size();
    std::vector<int> order(n);
    for (int j = 0; j < n; ++j) order[j] = j;
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return work[a] > work[b]; });
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    ForkPool *F = (n > 1 && dev >= 0 && dev < kMaxDevices) ? &g_fork[dev] : nullptr;
    std::unique_lock<std::mutex> lk;
    if (F) {
        lk = std::unique_lock<std::mutex>(F->mu);
        if (fork_pool_init(*F) != hipSuccess) F = nullptr;
    }
    if (!F) {
        for (int j = 0; j < n && e == hipSuccess; ++j) e = launch(order[j], s);
        return e;
    }
    const int lanes = std::min(n, kForkStreams + 1);
    e = hipEventRecord(F->fork, s);
    for (int i = 1; i < lanes && e == hipSuccess; ++i) e = hipStreamWaitEvent(F->st[i - 1], F->fork, 0);
    if (e != hipSuccess) return e;
    std::vector<double> load(lanes, 0.0);
    for (int jj = 0; jj < n && e == hipSuccess; ++jj) {
        const int j = order[jj];
        int best = 0;
        for (int i = 1; i < lanes; ++i)
            if (load[i] < load[best]) best = i;
        load[best] += work[j];
        e = launch(j, best == 0 ? s : F->st[best - 1]);
    }
    // join every lane even after a failed launch
    for (int i = 1; i < lanes; ++i) {
        hipError_t e2 = hipEventRecord(F->join[i - 1], F->st[i - 1]);
        if (e2 == hipSuccess) e2 = hipStreamWaitEvent(s, F->join[i - 1], 0);
        if (e == hipSuccess) e = e2;
    }
    return e;
}

}  // namespace

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

// One fit launch: a dense-search layer, or the histogram-search layers of one
// kernel variant (up to kMaxBatchLayers), with the indices of its layers.
struct FitJob {
    bool dense;
    int variant;
    int64_t channels;
    mpq::FitParams p;
    mpq::HistBatch b;
    std::vector<int> layers;
    double work;   // ~ sum of c_out * d (dense: times n_grid)
};

// The fit launches of a set of layers: one per dense-search layer, one per
// histogram variant and kMaxBatchLayers layers; a histogram layer with at
// least own_launch_weights weights gets a launch of its own (< 0: never).
// Batching does not change any channel's result.
std::vector<FitJob> build_fit_jobs(Search mode, bool hist_fits, const mpq_layer *layers, int n_layers,
                                   int M, int max_points, const float *dgrid, int n_grid, float tol,
                                   double own_launch_weights, int refit = 0)
{
    std::vector<FitJob> jobs;
    auto hist = [&](const mpq_layer &L) {
        return mode == Search::kAuto && hist_fits && mpq::fit_hist_supports(L.d);
    };
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        if (L.c_out == 0 || hist(L)) continue;
        FitJob j = {};
        j.dense = true;
        mpq::FitParams &p = j.p;
        p.W = L.W;
        p.C = L.c_out;
        p.d = L.d;
        p.M = M;
        p.P = max_points;
        p.grid = dgrid;
        p.G = n_grid;
        p.tol = (double)tol;
        p.codes = L.codes;
        p.scales = L.scales;
        p.counts = L.counts;
        p.err = L.fit_err;
        j.layers.push_back(l);
        // the dense search evaluates every candidate: weigh it by G
        j.work = (double)L.c_out * (double)L.d * (double)n_grid;
        jobs.push_back(j);
    }
    auto own = [&](const mpq_layer &L) {
        return own_launch_weights >= 0.0 && (double)L.c_out * (double)L.d >= own_launch_weights;
    };
    auto fresh = [&](int v) {
        FitJob j = {};
        j.variant = v;
        j.b.M = M;
        j.b.P = max_points;
        j.b.G = n_grid;
        j.b.grid = dgrid;
        j.b.tol = (double)tol;
        j.b.start = 0;   // a fresh fit (calibration steps and resumed fits set these)
        j.b.single = 0;
        j.b.refit = refit;
        return j;
    };
    auto add_layer = [&](FitJob &j, int l) {
        const mpq_layer &L = layers[l];
        mpq::HistLayer &H = j.b.L[j.b.n_layers++];
        H.W = L.W;
        H.codes = L.codes;
        H.scales = L.scales;
        H.counts = L.counts;
        H.err = L.fit_err;
        H.d = (int)L.d;
        H.c_begin = (int)j.channels;
        j.channels += L.c_out;
        // estimated time: a histogram-search channel costs ~ d + G per step
        // (its elements' levels, then the candidates); a short channel's
        // direct search ~ d G / 24 (both measured on MI355X)
        j.work += (double)L.c_out *
                  (L.d <= mpq::kSmallMaxDim ? (double)L.d * (double)n_grid / 24.0 : (double)(L.d + n_grid));
        j.layers.push_back(l);
    };
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        if (L.c_out == 0 || !hist(L) || !own(L)) continue;
        FitJob j = fresh(mpq::hist_variant(L.d));
        add_layer(j, l);
        jobs.push_back(j);
    }
    for (int v = 0; v < mpq::hist_variant_count(); ++v) {
        FitJob j = fresh(v);
        for (int l = 0; l <= n_layers; ++l) {
            const bool flush = l == n_layers || j.b.n_layers == mpq::kMaxBatchLayers ||
                               j.channels + (l < n_layers ? layers[l].c_out : 0) > 0x7fffffffLL;
            if (flush && j.b.n_layers > 0) {
                jobs.push_back(j);
                j = fresh(v);
            }
            if (l == n_layers) break;
            const mpq_layer &L = layers[l];
            if (L.c_out == 0 || !hist(L) || own(L) || mpq::hist_variant(L.d) != v) continue;
            add_layer(j, l);
        }
    }
    // a launch takes at least the serial steps of one channel (~15 us, as
    // long as ~4e5 units of the estimate above), however few its channels
    for (FitJob &j : jobs)
        if (!j.dense) j.work = std::max(j.work, 4e5);
    return jobs;
}

hipError_t launch_fit_job(const FitJob &j, int n_grid, hipStream_t st)
{
    return j.dense ? mpq::launch_fit(j.p, mpq::fit_layout(j.p.d, n_grid), st)
                   : mpq::launch_fit_hist(j.b, j.variant, j.channels, st);
}

int clip_checks(const mpq_layer *layers, int n_layers, int clip_grid);
int clip_first_points(const mpq_layer *layers, int n_layers, int M, int P, int Gc, bool with_xerr,
                      const std::vector<mpq::ErrLayerIn> &extra, hipStream_t s);

// Checks shared by the calls that fit: arguments, every layer's buffers, and
// that every layer fits a search kernel (*hist_fits: the histogram search's
// LDS fits the device).  *any: some layer has channels.
int fit_checks(Search mode, const mpq_layer *layers, int n_layers, int bits, int max_points,
               const float *grid_host, int n_grid, float tol, bool *any, bool *hist_fits)
{
    if (n_layers < 0 || (n_layers > 0 && !layers))
        return fail(MPQ_ERR_INVALID_ARG, "layers must hold n_layers >= 0 entries");
    int rc = check_fit_args(bits, max_points, grid_host, n_grid, tol);
    if (rc != MPQ_OK) return rc;
    *any = false;
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        rc = check_fit_layer(L.W, L.c_out, L.d, L.codes, L.scales, L.counts);
        if (rc != MPQ_OK) return n_layers > 1 ? fail(rc, "layer %d: %s", l, g_last_error.c_str()) : rc;
        *any = *any || L.c_out > 0;
    }
    if (!*any) return MPQ_OK;
    size_t lim = 0;
    rc = device_lds_limit(&lim);
    if (rc != MPQ_OK) return rc;
    // which layers take the histogram search (and which variant)
    *hist_fits = mpq::fit_hist_lds(n_grid) <= lim;
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        if (L.c_out == 0) continue;
        const bool hist = mode == Search::kAuto && *hist_fits && mpq::fit_hist_supports(L.d);
        if (!hist && mpq::fit_layout(L.d, n_grid).lds > lim)
            return fail(MPQ_ERR_SHAPE, "%sd = %lld with n_grid = %d needs %zu bytes of LDS (limit %zu)",
                        n_layers > 1 ? "a layer's " : "", (long long)L.d, n_grid,
                        mpq::fit_layout(L.d, n_grid).lds, lim);
    }
    return MPQ_OK;
}

// A caller's grid, copied to stream-ordered scratch (NULL: the default grid).
int upload_grid(const float *grid_host, int n_grid, hipStream_t s, float **dgrid)
{
    *dgrid = nullptr;
    if (!grid_host) return MPQ_OK;
    hipError_t e = mpq::scratch_alloc((void **)dgrid, sizeof(float) * (size_t)n_grid, s);
    if (e != hipSuccess) return fail(MPQ_ERR_NOMEM, "grid upload: %s", hipGetErrorString(e));
    e = hipMemcpyAsync(*dgrid, grid_host, sizeof(float) * (size_t)n_grid, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) {
        (void)mpq::scratch_free(*dgrid, s);
        *dgrid = nullptr;
        return hip_fail(e, "hipMemcpyAsync(grid)");
    }
    return MPQ_OK;
}

// Layers that need the histogram search (the refit and the calibration
// steps exist only there): MPQ_ERR_SHAPE for a layer it does not take.
int require_hist(const mpq_layer *layers, int n_layers, bool hist_fits, const char *what)
{
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        if (L.c_out > 0 && !(hist_fits && mpq::fit_hist_supports(L.d)))
            return fail(MPQ_ERR_SHAPE, "%sd = %lld: %s needs the histogram search "
                        "(d <= %lld, n_grid within its LDS)", n_layers > 1 ? "a layer's " : "",
                        (long long)L.d, what, (long long)mpq::kHistMaxDim);
    }
    return MPQ_OK;
}

int fit_layers_impl(Search mode, const mpq_layer *layers, int n_layers, int bits, int max_points,
                    const float *grid_host, int n_grid, float tol, void *stream, int refit = 0,
                    int clip_grid = 0, int asym = 0, int gate = 0)
{
    if (asym && n_layers > 0 && layers) {
        for (int l = 0; l < n_layers; ++l)
            if (layers[l].c_out > 0 && !layers[l].offsets)
                return fail(MPQ_ERR_INVALID_ARG, "%sasym needs offsets", n_layers > 1 ? "a layer: " : "");
    }
    if (clip_grid && n_layers > 0 && layers) {
        const int rc0 = clip_checks(layers, n_layers, clip_grid);
        if (rc0 != MPQ_OK) return rc0;
    }
    bool any = false, hist_fits = false;
    int rc = fit_checks(mode, layers, n_layers, bits, max_points, grid_host, n_grid, tol, &any,
                        &hist_fits);
    if (rc != MPQ_OK || !any) return rc;
    if (refit && (rc = require_hist(layers, n_layers, hist_fits, "the refit")) != MPQ_OK) return rc;
    if (clip_grid && (rc = require_hist(layers, n_layers, hist_fits, "the clipping")) != MPQ_OK)
        return rc;
    if (asym && (rc = require_hist(layers, n_layers, hist_fits, "asym")) != MPQ_OK) return rc;
    if (gate && (rc = require_hist(layers, n_layers, hist_fits, "the naive first point")) != MPQ_OK)
        return rc;
    hipStream_t s = (hipStream_t)stream;
    float *dgrid = nullptr;
    rc = upload_grid(grid_host, n_grid, s, &dgrid);
    if (rc != MPQ_OK) return rc;
    const int M = (1 << (bits - 1)) - 1;
    std::vector<FitJob> jobs = build_fit_jobs(mode, hist_fits, layers, n_layers, M, max_points,
                                              dgrid, n_grid, tol, -1.0, refit);
    for (FitJob &j : jobs) {
        j.b.gate = gate;
        if (asym)
            for (int i = 0; i < j.b.n_layers; ++i) j.b.L[i].offsets = layers[j.layers[i]].offsets;
    }
    if (clip_grid) {   // point 1 from the clipping, then the fit resumes from it
        rc = clip_first_points(layers, n_layers, M, max_points, clip_grid, false, {}, s);
        if (rc != MPQ_OK) {
            if (dgrid) (void)mpq::scratch_free(dgrid, s);
            return rc;
        }
        for (FitJob &j : jobs) j.b.start = 1;
    }
    std::vector<double> work;
    for (const FitJob &j : jobs) work.push_back(j.work);
    const hipError_t e = run_concurrently(s, work, [&](int i, hipStream_t st) {
        return launch_fit_job(jobs[i], n_grid, st);
    });
    if (dgrid) (void)mpq::scratch_free(dgrid, s);
    if (e != hipSuccess) return hip_fail(e, "fit kernel launch");
    return MPQ_OK;
}

int one_layer_fit(Search mode, const float *W, int64_t c_out, int64_t d, int bits, int max_points,
                  const float *grid_host, int n_grid, float tol, int8_t *codes, float *scales,
                  int32_t *counts, float *err_opt, void *stream)
{
    mpq_layer L = {};
    L.W = W;
    L.c_out = c_out;
    L.d = d;
    L.codes = codes;
    L.scales = scales;
    L.counts = counts;
    L.fit_err = err_opt;
    return fit_layers_impl(mode, &L, 1, bits, max_points, grid_host, n_grid, tol, stream);
}

int check_error_layer(const mpq_layer &L, int max_points, bool need_x)
{
    if (L.c_out < 0) return fail(MPQ_ERR_INVALID_ARG, "c_out must be >= 0 (got %lld)", (long long)L.c_out);
    if (L.d < 1) return fail(MPQ_ERR_INVALID_ARG, "d must be >= 1 (got %lld)", (long long)L.d);
    if (max_points < 1 || max_points > MPQ_MAX_POINTS)
        return fail(MPQ_ERR_INVALID_ARG, "max_points must be in [1, %d] (got %d)", MPQ_MAX_POINTS,
                    max_points);
    if (need_x) {
        if (L.n < 1) return fail(MPQ_ERR_INVALID_ARG, "n must be >= 1 (got %lld)", (long long)L.n);
        if (L.c_out > 0 && (!L.W || !L.codes || !L.scales || !L.counts || !L.X || !L.out_err))
            return fail(MPQ_ERR_INVALID_ARG, "W, codes, scales, counts, X and err must not be NULL");
        if (L.n > MPQ_MAX_ERR_DIM || L.c_out > MPQ_MAX_ERR_DIM)
            return fail(MPQ_ERR_INVALID_ARG, "c_out and n must be <= %d (got %lld, %lld)",
                        MPQ_MAX_ERR_DIM, (long long)L.c_out, (long long)L.n);
        if (L.d > MPQ_MAX_ERR_D)
            return fail(MPQ_ERR_INVALID_ARG, "d must be <= %d (got %lld)", MPQ_MAX_ERR_D, (long long)L.d);
    } else {
        if (L.c_out > 0 && (!L.codes || !L.scales || !L.counts || !L.W_hat))
            return fail(MPQ_ERR_INVALID_ARG, "codes, scales, counts and W_hat must not be NULL");
        if (L.c_out > 0x7fffffffLL || L.d > 0x7fffffffLL)
            return fail(MPQ_ERR_INVALID_ARG, "c_out or d too large");
    }
    return MPQ_OK;
}

// The independent launch groups of an output error, with one scratch block
// holding each group's part.
struct ErrJobs {
    std::vector<size_t> off;
    std::vector<double> work;
    char *scratch = nullptr;
    bool owned = true;   // allocated by err_jobs (else a caller-held block)
};

// fixed != nullptr: the groups' scratch is that caller-held block of
// fixed_bytes (nothing is allocated); a call that needs more fails with
// MPQ_ERR_SHAPE.
int err_jobs(const std::vector<mpq::ErrLayerIn> &in, hipStream_t s, ErrJobs *j,
             char *fixed = nullptr, size_t fixed_bytes = 0)
{
    const int ng = mpq::err_group_count(in.data(), (int)in.size());
    size_t total = 0;
    for (int g = 0; g < ng; ++g) {
        j->off.push_back(total);
        total += (mpq::err_group_scratch_bytes(in.data(), (int)in.size(), g) + 255) / 256 * 256;
        j->work.push_back(mpq::err_group_flop(in.data(), (int)in.size(), g));
    }
    if (fixed) {
        if (total > fixed_bytes)
            return fail(MPQ_ERR_SHAPE, "the output error needs %zu bytes of workspace; the fixed "
                        "workspace holds %zu", total, fixed_bytes);
        j->scratch = fixed;
        j->owned = false;
        return MPQ_OK;
    }
    const hipError_t e = mpq::scratch_alloc((void **)&j->scratch, total, s);
    if (e != hipSuccess) {
        j->scratch = nullptr;
        return fail(MPQ_ERR_NOMEM, "scratch of %zu bytes: %s", total, hipGetErrorString(e));
    }
    return MPQ_OK;
}

hipError_t launch_err_job(const std::vector<mpq::ErrLayerIn> &in, const ErrJobs &j, int g, int P,
                          hipStream_t st, int parts = mpq::kErrUpload | mpq::kErrKernels)
{
    return mpq::launch_output_error_group(in.data(), (int)in.size(), g, P, j.scratch + j.off[g], st, parts);
}

int output_error_impl(const mpq_layer *layers, int n_layers, int max_points, void *stream,
                      char *fixed = nullptr, size_t fixed_bytes = 0)
{
    if (n_layers < 0 || (n_layers > 0 && !layers))
        return fail(MPQ_ERR_INVALID_ARG, "layers must hold n_layers >= 0 entries");
    std::vector<mpq::ErrLayerIn> in;
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        int rc = check_error_layer(L, max_points, true);
        if (rc != MPQ_OK) return n_layers > 1 ? fail(rc, "layer %d: %s", l, g_last_error.c_str()) : rc;
        if (L.c_out == 0) continue;
        mpq::ErrLayerIn I = {L.W, L.codes, L.scales, L.counts, L.X, L.out_err, L.out_ref,
                             L.c_out, L.d, L.n};
        I.offsets = L.offsets;   // reading B2 (NULL: symmetric)
        in.push_back(I);
    }
    if (in.empty()) return MPQ_OK;
    hipStream_t s = (hipStream_t)stream;
    ErrJobs jobs;
    int rc = err_jobs(in, s, &jobs, fixed, fixed_bytes);
    if (rc != MPQ_OK) return rc;
    const hipError_t e = run_concurrently(s, jobs.work, [&](int i, hipStream_t st) {
        return launch_err_job(in, jobs, i, max_points, st);
    });
    if (jobs.scratch && jobs.owned) (void)mpq::scratch_free(jobs.scratch, s);
    if (e != hipSuccess) return hip_fail(e, "output error kernel launch");
    return MPQ_OK;
}

// The workspace of mpq_output_error_noalloc: one array per device, part of
// the library's code object, so it is in device memory from the moment the
// library's kernels load until the process ends and no call allocates it.
// Host code never passes its name to a kernel (on the host the name is a
// stand-in, not a device address): each device's address comes from
// hipGetSymbolAddress, once, with that device current.
static __device__ __align__(256) char scratch[MPQ_NOALLOC_BYTES];

std::mutex g_noalloc_mu;
char *g_noalloc_ptr[kMaxDevices];

int noalloc_workspace(char **ws)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(MPQ_ERR_HIP, "device index %d out of range", dev);
    std::lock_guard<std::mutex> lk(g_noalloc_mu);
    if (!g_noalloc_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(workspace)");
        if (!p) return fail(MPQ_ERR_HIP, "hipGetSymbolAddress(workspace) returned NULL");
        g_noalloc_ptr[dev] = (char *)p;
    }
    *ws = g_noalloc_ptr[dev];
    return MPQ_OK;
}

int reconstruct_impl(const mpq_layer *layers, int n_layers, int max_points, void *stream)
{
    if (n_layers < 0 || (n_layers > 0 && !layers))
        return fail(MPQ_ERR_INVALID_ARG, "layers must hold n_layers >= 0 entries");
    std::vector<mpq::RecLayer> in;
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        int rc = check_error_layer(L, max_points, false);
        if (rc != MPQ_OK) return n_layers > 1 ? fail(rc, "layer %d: %s", l, g_last_error.c_str()) : rc;
        if (L.c_out > 0)
            in.push_back(mpq::RecLayer{L.codes, L.scales, L.counts, L.W_hat, L.c_out, L.d, L.offsets});
    }
    if (in.empty()) return MPQ_OK;
    hipError_t e = mpq::launch_reconstruct(in.data(), (int)in.size(), max_points, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "reconstruct kernel launch");
    return MPQ_OK;
}

// The launches of one whole-path step (mpq_quantize_layers), planned from
// the layers: the fit jobs, the output error's items and launch groups, and
// the reconstruction.
struct QuantizeStep {
    std::vector<FitJob> jobs;
    std::vector<mpq::ErrLayerIn> err;
    std::vector<mpq::RecLayer> rec;                 // reconstructed beside the output error
    std::vector<std::vector<mpq::RecLayer>> rec_after;   // by fit job: right behind it
    std::vector<int> err_of;   // by layer: its err item, or -1
    ErrJobs ej;
    double rec_bytes = 0.0;
    int n_grid = 0, max_points = 0;
};

// The checks of mpq_quantize_layers, before any HIP call but the device
// queries of fit_checks.  any: a layer with channels.
int quantize_checks(const mpq_layer *layers, int n_layers, int bits, int max_points,
                    const float *grid_host, int n_grid, float tol, bool *any, bool *hist_fits)
{
    if (n_layers < 0 || (n_layers > 0 && !layers))
        return fail(MPQ_ERR_INVALID_ARG, "layers must hold n_layers >= 0 entries");
    // the output-error and reconstruction fields first: fit_checks ends with
    // a device query, and no check may follow a HIP call
    int rc = MPQ_OK;
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        if (L.out_err) rc = check_error_layer(L, max_points, true);
        if (rc == MPQ_OK && L.W_hat) rc = check_error_layer(L, max_points, false);
        if (rc != MPQ_OK) return n_layers > 1 ? fail(rc, "layer %d: %s", l, g_last_error.c_str()) : rc;
    }
    return fit_checks(Search::kAuto, layers, n_layers, bits, max_points, grid_host, n_grid, tol, any,
                      hist_fits);
}

// The step's launches (no HIP call): the fit jobs on the device grid dgrid
// (NULL: the default grid), the output error of every layer that asks for it
// (a group's GEMM fills the device only with many layers' tiles) and the
// reconstruction (both only read the fit's outputs).
void quantize_build(const mpq_layer *layers, int n_layers, int bits, int max_points, const float *dgrid,
                    int n_grid, float tol, bool hist_fits, QuantizeStep *q)
{
    const int M = (1 << (bits - 1)) - 1;
    q->n_grid = n_grid;
    q->max_points = max_points;
    q->jobs = build_fit_jobs(Search::kAuto, hist_fits, layers, n_layers, M, max_points, dgrid, n_grid,
                             tol, -1.0);
    q->err_of.assign(n_layers, -1);
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        if (L.c_out == 0 || !L.out_err) continue;
        q->err_of[l] = (int)q->err.size();
        q->err.push_back(mpq::ErrLayerIn{L.W, L.codes, L.scales, L.counts, L.X, L.out_err, L.out_ref,
                                         L.c_out, L.d, L.n});
    }
    // The reconstruction (bound by HBM) of a fit launch's layers runs right
    // behind that launch, beside the other fits (bound by VALU), when the
    // launch holds at least kRecBehind weights and is not the longest one;
    // the rest runs in one launch beside the output error (bound by MFMA).
    // Small launches stay in that one launch: a launch costs host time that
    // the shorter steps (MobileNetV2's) cannot hide.
    constexpr double kRecBehind = 2e6;
    int longest = -1;
    for (int i = 0; i < (int)q->jobs.size(); ++i)
        if (longest < 0 || q->jobs[i].work > q->jobs[longest].work) longest = i;
    q->rec_after.assign(q->jobs.size(), {});
    std::vector<int> job_of(n_layers, -1);
    for (int i = 0; i < (int)q->jobs.size(); ++i) {
        double w = 0.0;
        for (int l : q->jobs[i].layers) {
            job_of[l] = i;
            if (layers[l].W_hat) w += (double)layers[l].c_out * (double)layers[l].d;
        }
        if (i == longest || w < kRecBehind) continue;
        for (int l : q->jobs[i].layers) job_of[l] = -2 - i;   // behind job i
    }
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        if (L.c_out == 0 || !L.W_hat) continue;
        const mpq::RecLayer R{L.codes, L.scales, L.counts, L.W_hat, L.c_out, L.d, nullptr};
        if (job_of[l] <= -2) {
            q->rec_after[-2 - job_of[l]].push_back(R);
        } else {
            q->rec.push_back(R);
            q->rec_bytes += 5.0 * (double)L.c_out * (double)L.d;
        }
    }
}

// Once the output error's scratch is placed (q->ej): a fit that keeps its
// residual in registers writes its layers' rows of D for the output error,
// which then forms none for them.
void quantize_link_d(QuantizeStep *q)
{
    if (q->err.empty()) return;
    std::vector<int64_t> d_off(q->err.size());
    std::vector<int> d_grp(q->err.size());
    mpq::err_item_d_offsets(q->err.data(), (int)q->err.size(), d_off.data(), d_grp.data());
    for (FitJob &j : q->jobs) {
        if (j.dense || !mpq::hist_variant_writes_d(j.variant)) continue;
        for (int i = 0; i < j.b.n_layers; ++i) {
            const int e = q->err_of[j.layers[i]];
            if (e < 0 || d_off[e] < 0) continue;
            j.b.L[i].dres = (float *)(q->ej.scratch + q->ej.off[d_grp[e]] + d_off[e]);
            q->err[e].d_ready = 1;
        }
    }
}

// Enqueues the step on s: (1) every fit, side by side (as mpq_fit_layers),
// each followed on its stream by the reconstruction of its layers when it
// has one (rec_after), and beside them the upload of the output error's
// descriptor tables, which reads nothing the fits write (so the GEMM starts
// as soon as the last fit ends); (2) the output error's launch groups and,
// beside them, one reconstruction of the remaining layers (it reads only
// the fit's outputs and is bound by HBM, the GEMM by MFMA).
hipError_t quantize_enqueue(QuantizeStep &q, hipStream_t s)
{
    std::vector<double> work;
    for (const FitJob &j : q.jobs) work.push_back(j.work);
    const int n_fit_jobs = (int)work.size();
    const int n_groups = (int)q.ej.work.size();
    if (n_groups > 0) work.push_back(0.0);
    hipError_t e = run_concurrently(s, work, [&](int i, hipStream_t st) {
        if (i < n_fit_jobs) {
            hipError_t e0 = launch_fit_job(q.jobs[i], q.n_grid, st);
            const std::vector<mpq::RecLayer> &r = q.rec_after[i];
            if (e0 == hipSuccess && !r.empty())
                e0 = mpq::launch_reconstruct(r.data(), (int)r.size(), q.max_points, st);
            return e0;
        }
        hipError_t e1 = hipSuccess;
        for (int g = 0; g < n_groups && e1 == hipSuccess; ++g)
            e1 = launch_err_job(q.err, q.ej, g, q.max_points, st, mpq::kErrUpload);
        return e1;
    });
    if (e != hipSuccess) return e;
    // work in GEMM FLOP and, for the reconstruction, bytes (at ~2 TB/s
    // against ~100 TFLOP/s: x 50)
    std::vector<double> w2 = q.ej.work;
    const int n_err_jobs = (int)w2.size();
    if (!q.rec.empty()) w2.push_back(q.rec_bytes * 50.0);
    return run_concurrently(s, w2, [&](int i, hipStream_t st) {
        return i < n_err_jobs ? launch_err_job(q.err, q.ej, i, q.max_points, st, mpq::kErrKernels)
                              : mpq::launch_reconstruct(q.rec.data(), (int)q.rec.size(), q.max_points, st);
    });
}

int quantize_impl(const mpq_layer *layers, int n_layers, int bits, int max_points,
                  const float *grid_host, int n_grid, float tol, void *stream)
{
    bool any = false, hist_fits = false;
    int rc = quantize_checks(layers, n_layers, bits, max_points, grid_host, n_grid, tol, &any, &hist_fits);
    if (rc != MPQ_OK || !any) return rc;
    hipStream_t s = (hipStream_t)stream;
    float *dgrid = nullptr;
    rc = upload_grid(grid_host, n_grid, s, &dgrid);
    if (rc != MPQ_OK) return rc;
    QuantizeStep q;
    quantize_build(layers, n_layers, bits, max_points, dgrid, n_grid, tol, hist_fits, &q);
    if (!q.err.empty()) {
        rc = err_jobs(q.err, s, &q.ej);
        if (rc != MPQ_OK) {
            if (dgrid) (void)mpq::scratch_free(dgrid, s);
            return rc;
        }
    }
    quantize_link_d(&q);
    const hipError_t e = quantize_enqueue(q, s);
    if (dgrid) (void)mpq::scratch_free(dgrid, s);
    if (q.ej.scratch) (void)mpq::scratch_free(q.ej.scratch, s);
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    return MPQ_OK;
}

// Checks of a clipped fit (reading C1): every layer needs its batch.
int clip_checks(const mpq_layer *layers, int n_layers, int clip_grid)
{
    if (clip_grid < 1 || clip_grid > MPQ_MAX_GRID)
        return fail(MPQ_ERR_INVALID_ARG, "clip_grid must be in [1, %d] (got %d)", MPQ_MAX_GRID, clip_grid);
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        int rc = MPQ_OK;
        if (L.c_out > 0) {
            if (!L.X) rc = fail(MPQ_ERR_INVALID_ARG, "the clipping needs X");
            else if (L.n < 1 || L.n > MPQ_MAX_ERR_DIM)
                rc = fail(MPQ_ERR_INVALID_ARG, "n must be in [1, %d] (got %lld)", MPQ_MAX_ERR_DIM,
                          (long long)L.n);
            else if ((double)L.c_out * clip_grid > MPQ_MAX_ERR_DIM)
                rc = fail(MPQ_ERR_INVALID_ARG, "c_out * clip_grid must be <= %d", MPQ_MAX_ERR_DIM);
        }
        if (rc != MPQ_OK) return n_layers > 1 ? fail(rc, "layer %d: %s", l, g_last_error.c_str()) : rc;
    }
    return MPQ_OK;
}

// Reading C1 for every layer: the clipping candidates of each channel, their
// output errors on X (one batched output-error pass, together with `extra`
// items such as the relative threshold's reference errors), then point 1 of
// every channel.  with_xerr: point 1's output error goes to fit_xerr.
int clip_first_points(const mpq_layer *layers, int n_layers, int M, int P, int Gc, bool with_xerr,
                      const std::vector<mpq::ErrLayerIn> &extra, hipStream_t s)
{
    std::vector<size_t> off(n_layers);
    size_t total = 0;
    for (int l = 0; l < n_layers; ++l) {
        off[l] = total;
        total += (size_t)std::max<int64_t>(layers[l].c_out, 0) * (size_t)Gc;
    }
    float *buf = nullptr;   // cand [total], then ecand [total]
    hipError_t e = mpq::scratch_alloc((void **)&buf, 2 * sizeof(float) * total, s);
    if (e != hipSuccess) return fail(MPQ_ERR_NOMEM, "scratch: %s", hipGetErrorString(e));
    float *cand = buf, *ecand = buf + total;
    // the launches of the candidate and choice kernels
    std::vector<std::pair<mpq::ClipBatch, int64_t>> batches;
    {
        mpq::ClipBatch b = {};
        b.M = M;
        b.P = P;
        b.Gc = Gc;
        int64_t ch = 0;
        for (int l = 0; l <= n_layers; ++l) {
            if ((l == n_layers || b.n_layers == mpq::kMaxClipLayers ||
                 (l < n_layers && ch + layers[l].c_out > 0x7fffffffLL)) && b.n_layers > 0) {
                batches.push_back({b, ch});
                b.n_layers = 0;
                ch = 0;
            }
            if (l == n_layers) break;
            const mpq_layer &L = layers[l];
            if (L.c_out == 0) continue;
            mpq::ClipLayer &C = b.L[b.n_layers++];
            C = mpq::ClipLayer{L.W, cand + off[l], ecand + off[l], L.codes, L.scales, L.counts,
                               L.fit_err, with_xerr ? L.fit_xerr : nullptr, (int)L.d, (int)ch};
            ch += L.c_out;
        }
    }
    std::vector<mpq::ErrLayerIn> in;
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        if (L.c_out == 0) continue;
        mpq::ErrLayerIn I = {};
        I.W = L.W;
        I.codes = L.codes;
        I.scales = L.scales;
        I.counts = L.counts;
        I.X = L.X;
        I.err = ecand + off[l];
        I.C = L.c_out;
        I.d = L.d;
        I.n = L.n;
        I.cand = cand + off[l];
        I.Gc = Gc;
        I.M = M;
        in.push_back(I);
    }
    in.insert(in.end(), extra.begin(), extra.end());
    ErrJobs ej;
    int rc = err_jobs(in, s, &ej);
    if (rc != MPQ_OK) {
        (void)mpq::scratch_free(buf, s);
        return rc;
    }
    for (size_t i = 0; i < batches.size() && e == hipSuccess; ++i)
        e = mpq::launch_clip(batches[i].first, batches[i].second, false, s);
    if (e == hipSuccess)
        e = run_concurrently(s, ej.work, [&](int i, hipStream_t st) { return launch_err_job(in, ej, i, P, st); });
    for (size_t i = 0; i < batches.size() && e == hipSuccess; ++i)
        e = mpq::launch_clip(batches[i].first, batches[i].second, true, s);
    if (ej.scratch) (void)mpq::scratch_free(ej.scratch, s);
    (void)mpq::scratch_free(buf, s);
    if (e != hipSuccess) return hip_fail(e, "clipping kernel launch");
    return MPQ_OK;
}

// Algorithm 2's stopping rule on a calibration batch, for every layer.  Per
// step s = 0 .. max_points - 1: the fit launches take point s + 1 of every
// channel that has not stopped (a channel stops once the output error of its
// points is at most the threshold) and list those channels; then the
// output-error pass scores the listed channels of every layer.  The relative
// threshold's output error of W runs beside the first fit step.
int calib_impl(const mpq_layer *layers, int n_layers, int bits, int max_points,
               const float *grid_host, int n_grid, float eps, int relative, void *stream,
               int refit = 0, int clip_grid = 0, int asym = 0, int gate = 0)
{
    if (asym && n_layers > 0 && layers) {
        for (int l = 0; l < n_layers; ++l)
            if (layers[l].c_out > 0 && !layers[l].offsets)
                return fail(MPQ_ERR_INVALID_ARG, "%sasym needs offsets", n_layers > 1 ? "a layer: " : "");
    }
    if (n_layers < 0 || (n_layers > 0 && !layers))
        return fail(MPQ_ERR_INVALID_ARG, "layers must hold n_layers >= 0 entries");
    if (!(eps >= 0.0f) || !isfinite(eps))
        return fail(MPQ_ERR_INVALID_ARG, "eps must be finite and >= 0");
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        int rc = MPQ_OK;
        if (L.c_out > 0) {
            if (!L.X || !L.fit_xerr) rc = fail(MPQ_ERR_INVALID_ARG, "X and xerr must not be NULL");
            else if (L.n < 1) rc = fail(MPQ_ERR_INVALID_ARG, "n must be >= 1 (got %lld)", (long long)L.n);
            else if (L.n > MPQ_MAX_ERR_DIM || L.c_out > MPQ_MAX_ERR_DIM)
                rc = fail(MPQ_ERR_INVALID_ARG, "c_out and n must be <= %d (got %lld, %lld)",
                          MPQ_MAX_ERR_DIM, (long long)L.c_out, (long long)L.n);
        }
        if (rc != MPQ_OK) return n_layers > 1 ? fail(rc, "layer %d: %s", l, g_last_error.c_str()) : rc;
    }
    if (clip_grid) {
        const int rc0 = clip_checks(layers, n_layers, clip_grid);
        if (rc0 != MPQ_OK) return rc0;
    }
    bool any = false, hist_fits = false;
    int rc = fit_checks(Search::kAuto, layers, n_layers, bits, max_points, grid_host, n_grid, 0.0f,
                        &any, &hist_fits);
    if (rc != MPQ_OK || !any) return rc;
    if ((rc = require_hist(layers, n_layers, hist_fits, "the calibration fit")) != MPQ_OK) return rc;
    hipStream_t s = (hipStream_t)stream;
    const int P = max_points;

    // state: every layer's per-step list lengths [P] (contiguous, zeroed
    // together), then per layer its channel list [C] and W's output error [C]
    std::vector<size_t> off_list(n_layers), off_ref(n_layers);
    size_t bytes = (sizeof(int32_t) * (size_t)P * (size_t)n_layers + 255) / 256 * 256;
    for (int l = 0; l < n_layers; ++l) {
        const size_t C = (size_t)std::max<int64_t>(layers[l].c_out, 0);
        off_list[l] = bytes;
        bytes += (sizeof(int32_t) * C + 255) / 256 * 256;
        off_ref[l] = bytes;
        if (relative) bytes += (sizeof(float) * C + 255) / 256 * 256;
    }
    float *dgrid = nullptr;
    rc = upload_grid(grid_host, n_grid, s, &dgrid);
    if (rc != MPQ_OK) return rc;
    char *state = nullptr;
    hipError_t e = mpq::scratch_alloc((void **)&state, bytes, s);
    if (e != hipSuccess) {
        if (dgrid) (void)mpq::scratch_free(dgrid, s);
        return fail(MPQ_ERR_NOMEM, "scratch of %zu bytes: %s", bytes, hipGetErrorString(e));
    }
    auto nlist = [&](int l) { return (int32_t *)state + (size_t)l * P; };
    auto list = [&](int l) { return (int32_t *)(state + off_list[l]); };
    auto ref = [&](int l) { return relative ? (float *)(state + off_ref[l]) : nullptr; };

    const int M = (1 << (bits - 1)) - 1;
    std::vector<FitJob> jobs = build_fit_jobs(Search::kAuto, true, layers, n_layers, M, P, dgrid,
                                              n_grid, 0.0f, -1.0, refit);
    for (FitJob &j : jobs) {
        j.b.eps = (double)eps;
        j.b.gate = gate;   // read at step 0 only
        for (int i = 0; i < j.b.n_layers; ++i) {
            const int l = j.layers[i];
            mpq::HistLayer &H = j.b.L[i];
            H.xerr = layers[l].fit_xerr;
            H.ref = ref(l);
            H.list = list(l);
            H.nlist = nlist(l);
            H.offsets = asym ? layers[l].offsets : nullptr;
        }
    }
    // the output-error items of one step (the same groups every step), and
    // the reference items of the relative threshold
    std::vector<mpq::ErrLayerIn> in, in_ref;
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        if (L.c_out == 0) continue;
        mpq::ErrLayerIn I = {L.W, L.codes, L.scales, L.counts, L.X, L.fit_xerr, nullptr,
                             L.c_out, L.d, L.n, list(l), nlist(l), P};
        I.offsets = asym ? L.offsets : nullptr;
        in.push_back(I);
        if (relative)
            in_ref.push_back(mpq::ErrLayerIn{L.W, L.codes, L.scales, L.counts, L.X, nullptr, ref(l),
                                             L.c_out, L.d, L.n, nullptr, nullptr, 0});
    }
    ErrJobs ej, ej_ref;
    rc = err_jobs(in, s, &ej);
    if (rc == MPQ_OK && relative) rc = err_jobs(in_ref, s, &ej_ref);
    auto release = [&]() {
        if (ej_ref.scratch) (void)mpq::scratch_free(ej_ref.scratch, s);
        if (ej.scratch) (void)mpq::scratch_free(ej.scratch, s);
        (void)mpq::scratch_free(state, s);
        if (dgrid) (void)mpq::scratch_free(dgrid, s);
    };
    if (rc != MPQ_OK) {
        release();
        return rc;
    }
    e = mpq::launch_zero_i32((int32_t *)state, (int64_t)P * n_layers, s);
    std::vector<double> fit_work;
    for (const FitJob &j : jobs) fit_work.push_back(j.work);
    int first = 0;
    // point 1 from the clipping, or (gate, reading F1) the naive point: the
    // one clipping candidate c = 1, so fl32(max|w|) / M; its output error is
    // e_1.  The reference errors of the relative threshold ride in the same
    // pass.  A clipped fit continues from point 1; a gated one decides at
    // step 0 whether the naive point stays or the fit restarts from w.
    const bool pre = clip_grid || gate;
    if (pre && e == hipSuccess) {
        rc = clip_first_points(layers, n_layers, M, P, clip_grid ? clip_grid : 1, true, in_ref, s);
        if (rc != MPQ_OK) {
            release();
            return rc;
        }
        first = clip_grid ? 1 : 0;
    }
    for (int step = first; step < P && e == hipSuccess; ++step) {
        for (FitJob &j : jobs) {
            j.b.start = step;
            j.b.single = 1;
        }
        // the fit step; at step 0 beside it the output error of W (ref)
        std::vector<double> w = fit_work;
        const int n_fit = (int)w.size();
        if (step == 0 && !pre) w.insert(w.end(), ej_ref.work.begin(), ej_ref.work.end());
        e = run_concurrently(s, w, [&](int i, hipStream_t st) {
            return i < n_fit ? launch_fit_job(jobs[i], n_grid, st)
                             : launch_err_job(in_ref, ej_ref, i - n_fit, P, st);
        });
        if (e != hipSuccess) break;
        // the output error of the channels that took point step + 1
        std::vector<mpq::ErrLayerIn> in_s = in;
        {
            int i = 0;
            for (int l = 0; l < n_layers; ++l) {
                if (layers[l].c_out == 0) continue;
                in_s[i].err = layers[l].fit_xerr + step;
                in_s[i].nrows = nlist(l) + step;
                ++i;
            }
        }
        e = run_concurrently(s, ej.work, [&](int i, hipStream_t st) {
            return launch_err_job(in_s, ej, i, P, st);
        });
    }
    release();
    if (e != hipSuccess) return hip_fail(e, "calibration fit launch");
    return MPQ_OK;
}

// Sec. 3.4: integer forward of a list of layers, in launches of up to
// kMaxIntLayers layers (all checks first).
int int_forward_impl(const mpq_int_layer *layers, int n_layers, int max_points, int p, void *stream)
{
    if (n_layers < 0 || (n_layers > 0 && !layers))
        return fail(MPQ_ERR_INVALID_ARG, "layers must hold n_layers >= 0 entries");
    if (max_points < 1 || max_points > MPQ_MAX_POINTS)
        return fail(MPQ_ERR_INVALID_ARG, "max_points must be in [1, %d] (got %d)", MPQ_MAX_POINTS,
                    max_points);
    if (p < 0 || p > 62) return fail(MPQ_ERR_INVALID_ARG, "p must be in [0, 62] (got %d)", p);
    for (int l = 0; l < n_layers; ++l) {
        const mpq_int_layer &L = layers[l];
        int rc = MPQ_OK;
        if (L.c_out < 0 || L.d < 1 || L.n < 0)
            rc = fail(MPQ_ERR_INVALID_ARG, "need c_out >= 0, d >= 1, n >= 0 (got %lld, %lld, %lld)",
                      (long long)L.c_out, (long long)L.d, (long long)L.n);
        else if (L.d > MPQ_MAX_INT_DIM)
            rc = fail(MPQ_ERR_INVALID_ARG, "d must be <= %d (got %lld)", MPQ_MAX_INT_DIM, (long long)L.d);
        else if (L.c_out > 0 && L.n > 0 && (!L.codes || !L.A || !L.counts || !L.X || !L.Y))
            rc = fail(MPQ_ERR_INVALID_ARG, "codes, A, counts, X and Y must not be NULL");
        else if ((double)L.c_out * max_points * (double)L.d >= 2147483648.0 ||
                 (double)L.n * (double)L.d >= 2147483648.0)
            rc = fail(MPQ_ERR_INVALID_ARG, "codes and X must each be below 2^31 bytes");
        if (rc != MPQ_OK) return n_layers > 1 ? fail(rc, "layer %d: %s", l, g_last_error.c_str()) : rc;
    }
    // launches of up to kMaxIntLayers layers of one load mode, side by side
    std::vector<mpq::IntGroup> groups;
    std::vector<int> modes;
    std::vector<double> work;
    for (int mode = 0; mode < mpq::kIntModes; ++mode) {
        mpq::IntGroup g;
        g.P = max_points;
        g.p = p;
        g.n_layers = 0;
        double w = 0.0;
        for (int l = 0; l <= n_layers; ++l) {
            if ((l == n_layers || g.n_layers == mpq::kMaxIntLayers) && g.n_layers > 0) {
                groups.push_back(g);
                modes.push_back(mode);
                work.push_back(w);
                g.n_layers = 0;
                w = 0.0;
            }
            if (l == n_layers) break;
            const mpq_int_layer &L = layers[l];
            if (L.c_out == 0 || L.n == 0) continue;
            mpq::IntLayer I = {};
            I.codes = L.codes;
            I.A = L.A;
            I.counts = L.counts;
            I.X = L.X;
            I.Y = L.Y;
            I.C = L.c_out;
            I.d = L.d;
            I.N = L.n;
            if (mpq::int_forward_mode(I) != mode) continue;
            g.L[g.n_layers++] = I;
            w += (double)L.c_out * (double)L.d * (double)L.n;
        }
    }
    if (groups.empty()) return MPQ_OK;
    const hipError_t e = run_concurrently((hipStream_t)stream, work, [&](int i, hipStream_t st) {
        return mpq::launch_int_forward(groups[i], modes[i], st);
    });
    if (e != hipSuccess) return hip_fail(e, "integer forward kernel launch");
    return MPQ_OK;
}

// The fit on the paper's own grid (Eq. (11), readings D1 and G3), with the
// isotropic stopping rule: one launch per kernel variant (up to
// kMaxBatchLayers layers), side by side.
int paper_impl(const mpq_layer *layers, int n_layers, int bits, int max_points, float tol, float eta,
               void *stream)
{
    if (n_layers < 0 || (n_layers > 0 && !layers))
        return fail(MPQ_ERR_INVALID_ARG, "layers must hold n_layers >= 0 entries");
    int rc = check_fit_args(bits, max_points, nullptr, 1, tol);
    if (rc != MPQ_OK) return rc;
    if (!(eta > 0.0f) || !isfinite(eta)) return fail(MPQ_ERR_INVALID_ARG, "paper_eta must be finite and > 0");
    bool any = false;
    int64_t dmax = 0;
    for (int l = 0; l < n_layers; ++l) {
        const mpq_layer &L = layers[l];
        rc = check_fit_layer(L.W, L.c_out, L.d, L.codes, L.scales, L.counts);
        if (rc != MPQ_OK) return n_layers > 1 ? fail(rc, "layer %d: %s", l, g_last_error.c_str()) : rc;
        if (L.c_out > 0) {
            any = true;
            dmax = std::max(dmax, L.d);
        }
    }
    if (!any) return MPQ_OK;
    if (dmax > mpq::kPaperBigMaxDim)
        return fail(MPQ_ERR_SHAPE, "the paper's grid takes d <= %lld (got %lld)",
                    (long long)mpq::kPaperBigMaxDim, (long long)dmax);
    // the LDS variants take d <= kPaperMaxDim; longer channels keep their
    // sorted magnitudes in a global scratch
    const int64_t dmax_lds = [&]() {
        int64_t m = 0;
        for (int l = 0; l < n_layers; ++l)
            if (layers[l].c_out > 0 && layers[l].d <= mpq::kPaperMaxDim) m = std::max(m, layers[l].d);
        return m;
    }();
    size_t lim = 0;
    rc = device_lds_limit(&lim);
    if (rc != MPQ_OK) return rc;
    if (dmax_lds > 0 && mpq::paper_lds(dmax_lds) > lim)
        return fail(MPQ_ERR_SHAPE, "d = %lld needs %zu bytes of LDS (limit %zu)", (long long)dmax_lds,
                    mpq::paper_lds(dmax_lds), lim);
    struct Job {
        mpq::PaperBatch b;
        int variant;
        int64_t channels, dmax;
        double work;
    };
    std::vector<Job> jobs;
    const int M = (1 << (bits - 1)) - 1;
    for (int v = 0; v <= mpq::kPaperBigVariant; ++v) {
        Job j = {};
        auto fresh = [&]() {
            j = Job{};
            j.b.M = M;
            j.b.P = max_points;
            j.b.tol = (double)tol;
            j.b.eta = (double)eta;
            j.variant = v;
        };
        fresh();
        for (int l = 0; l <= n_layers; ++l) {
            const bool flush = l == n_layers || j.b.n_layers == mpq::kMaxBatchLayers ||
                               j.channels + (l < n_layers ? layers[l].c_out : 0) > 0x7fffffffLL;
            if (flush && j.b.n_layers > 0) {
                jobs.push_back(j);
                fresh();
            }
            if (l == n_layers) break;
            const mpq_layer &L = layers[l];
            if (L.c_out == 0 || mpq::paper_variant(L.d) != v) continue;
            mpq::HistLayer &H = j.b.L[j.b.n_layers++];
            H.W = L.W;
            H.codes = L.codes;
            H.scales = L.scales;
            H.counts = L.counts;
            H.err = L.fit_err;
            H.d = (int)L.d;
            H.c_begin = (int)j.channels;
            j.channels += L.c_out;
            j.dmax = std::max(j.dmax, L.d);
            j.work += (double)L.c_out * (double)L.d * (double)L.d;
        }
    }
    // scratch of the long-channel launches (sorted magnitudes and prefix sums
    // of one channel per workgroup)
    hipStream_t s = (hipStream_t)stream;
    std::vector<size_t> big_off(jobs.size(), 0);
    size_t big_bytes = 0;
    for (size_t i = 0; i < jobs.size(); ++i) {
        if (jobs[i].variant != mpq::kPaperBigVariant) continue;
        big_off[i] = big_bytes;
        big_bytes += (sizeof(double) * mpq::paper_big_slice(jobs[i].dmax) *
                          (size_t)mpq::paper_big_grid(jobs[i].channels) + 255) / 256 * 256;
    }
    char *big = nullptr;
    if (big_bytes > 0) {
        const hipError_t ea = mpq::scratch_alloc((void **)&big, big_bytes, s);
        if (ea != hipSuccess) return fail(MPQ_ERR_NOMEM, "scratch of %zu bytes: %s", big_bytes,
                                          hipGetErrorString(ea));
    }
    std::vector<double> work;
    for (const Job &j : jobs) work.push_back(j.work);
    const hipError_t e = run_concurrently(s, work, [&](int i, hipStream_t st) {
        if (jobs[i].variant == mpq::kPaperBigVariant)
            return mpq::launch_fit_paper_big(jobs[i].b, jobs[i].channels, jobs[i].dmax,
                                             (double *)(big + big_off[i]), st);
        return mpq::launch_fit_paper(jobs[i].b, jobs[i].variant, jobs[i].channels, jobs[i].dmax, st);
    });
    if (big) (void)mpq::scratch_free(big, s);
    if (e != hipSuccess) return hip_fail(e, "paper-grid fit kernel launch");
    return MPQ_OK;
}

}  // namespace

extern "C" {

int mpq_integer_scales(const float *scales, const int32_t *counts, int64_t c_out, int max_points, int p,
                       int32_t *A, unsigned long long *n_clamped_opt, void *stream)
{
    if (c_out < 0) return fail(MPQ_ERR_INVALID_ARG, "c_out must be >= 0 (got %lld)", (long long)c_out);
    if (max_points < 1 || max_points > MPQ_MAX_POINTS)
        return fail(MPQ_ERR_INVALID_ARG, "max_points must be in [1, %d] (got %d)", MPQ_MAX_POINTS,
                    max_points);
    if (p < 0 || p > 62) return fail(MPQ_ERR_INVALID_ARG, "p must be in [0, 62] (got %d)", p);
    if (c_out > 0 && (!scales || !counts || !A))
        return fail(MPQ_ERR_INVALID_ARG, "scales, counts and A must not be NULL");
    const hipError_t e = mpq::launch_integer_scales(scales, counts, c_out, max_points, p, A, n_clamped_opt,
                                                    (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "integer scales kernel launch");
    return MPQ_OK;
}

int mpq_integer_forward(const int8_t *codes, const int32_t *A, const int32_t *counts, int64_t c_out,
                        int64_t d, int max_points, const int8_t *X, int64_t n, int p, int64_t *Y,
                        void *stream)
{
    mpq_int_layer L = {codes, A, counts, c_out, d, X, n, Y};
    return int_forward_impl(&L, 1, max_points, p, stream);
}

int mpq_integer_forward_layers(const mpq_int_layer *layers, int n_layers, int max_points, int p,
                               void *stream)
{
    return int_forward_impl(layers, n_layers, max_points, p, stream);
}

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

int mpq_fit_kernel_of(int64_t d, int bits, int n_grid, int default_grid, char *name, int cap)
{
    if (d < 1 || bits < 2 || bits > MPQ_MAX_BITS || n_grid < 1 || n_grid > MPQ_MAX_GRID || cap < 1 || !name)
        return fail(MPQ_ERR_INVALID_ARG, "mpq_fit_kernel_of: invalid argument");
    size_t lim = 0;
    const int rc = device_lds_limit(&lim);
    if (rc != MPQ_OK) return rc;
    const int M = (1 << (bits - 1)) - 1;
    std::string k;
    if (mpq::fit_hist_lds(n_grid) <= lim && mpq::fit_hist_supports(d))
        k = mpq::hist_kernel_name(d, M, n_grid, default_grid != 0);
    else
        k = "fit_dense_kernel";
    snprintf(name, (size_t)cap, "%s", k.c_str());
    return MPQ_OK;
}

int mpq_fit_layer(const float *W, int64_t c_out, int64_t d, int bits, int max_points,
                  const float *grid_host, int n_grid, float tol, int8_t *codes, float *scales,
                  int32_t *counts, float *err_opt, void *stream)
{
    return one_layer_fit(Search::kAuto, W, c_out, d, bits, max_points, grid_host, n_grid, tol,
                         codes, scales, counts, err_opt, stream);
}

int mpq_fit_layer_dense(const float *W, int64_t c_out, int64_t d, int bits, int max_points,
                        const float *grid_host, int n_grid, float tol, int8_t *codes,
                        float *scales, int32_t *counts, float *err_opt, void *stream)
{
    return one_layer_fit(Search::kDense, W, c_out, d, bits, max_points, grid_host, n_grid, tol,
                         codes, scales, counts, err_opt, stream);
}

int mpq_fit_layers(const mpq_layer *layers, int n_layers, int bits, int max_points,
                   const float *grid_host, int n_grid, float tol, void *stream)
{
    return fit_layers_impl(Search::kAuto, layers, n_layers, bits, max_points, grid_host, n_grid,
                           tol, stream);
}

int mpq_quantize_layers(const mpq_layer *layers, int n_layers, int bits, int max_points,
                        const float *grid_host, int n_grid, float tol, void *stream)
{
    return quantize_impl(layers, n_layers, bits, max_points, grid_host, n_grid, tol, stream);
}

int mpq_fit_layer_calib(const float *W, int64_t c_out, int64_t d, int bits, int max_points,
                        const float *grid_host, int n_grid, const float *X, int64_t n, float eps,
                        int relative, int8_t *codes, float *scales, int32_t *counts, float *err_opt,
                        float *xerr, void *stream)
{
    mpq_layer L = {};
    L.W = W;
    L.c_out = c_out;
    L.d = d;
    L.codes = codes;
    L.scales = scales;
    L.counts = counts;
    L.fit_err = err_opt;
    L.X = X;
    L.n = n;
    L.fit_xerr = xerr;
    return calib_impl(&L, 1, bits, max_points, grid_host, n_grid, eps, relative, stream);
}

int mpq_fit_layers_calib(const mpq_layer *layers, int n_layers, int bits, int max_points,
                         const float *grid_host, int n_grid, float eps, int relative, void *stream)
{
    return calib_impl(layers, n_layers, bits, max_points, grid_host, n_grid, eps, relative, stream);
}

int mpq_fit_layers_ex(const mpq_layer *layers, int n_layers, int bits, int max_points,
                      const float *grid_host, int n_grid, float tol, const mpq_fit_options *opt,
                      void *stream)
{
    if (opt && opt->paper_eta != 0.0f) {
        if (opt->calib || opt->refit || opt->clip_grid || opt->asym || opt->gate)
            return fail(MPQ_ERR_INVALID_ARG,
                        "paper_eta cannot be combined with calib, refit, clip_grid, asym or gate");
        return paper_impl(layers, n_layers, bits, max_points, tol, opt->paper_eta, stream);
    }
    if (!opt) return fit_layers_impl(Search::kAuto, layers, n_layers, bits, max_points, grid_host,
                                     n_grid, tol, stream);
    if (opt->clip_grid && opt->refit)
        return fail(MPQ_ERR_INVALID_ARG, "refit and clip_grid cannot be combined");
    if (opt->asym && opt->clip_grid)
        return fail(MPQ_ERR_INVALID_ARG, "asym and clip_grid cannot be combined");
    if (opt->clip_grid < 0) return fail(MPQ_ERR_INVALID_ARG, "clip_grid must be >= 0");
    if (opt->gate && opt->clip_grid)
        return fail(MPQ_ERR_INVALID_ARG, "gate and clip_grid cannot be combined");
    if (opt->gate && opt->calib && opt->asym)
        return fail(MPQ_ERR_INVALID_ARG, "gate and asym cannot be combined with calib");
    if (opt->calib)
        return calib_impl(layers, n_layers, bits, max_points, grid_host, n_grid, opt->eps,
                          opt->relative, stream, opt->refit != 0, opt->clip_grid, opt->asym != 0,
                          opt->gate != 0);
    return fit_layers_impl(Search::kAuto, layers, n_layers, bits, max_points, grid_host, n_grid, tol,
                           stream, opt->refit != 0, opt->clip_grid, opt->asym != 0, opt->gate != 0);
}

int mpq_output_error(const float *W, const int8_t *codes, const float *scales,
                     const int32_t *counts, int64_t c_out, int64_t d, int max_points,
                     const float *X, int64_t n, float *err, float *ref_opt, void *stream)
{
    mpq_layer L = {};
    L.W = W;
    L.c_out = c_out;
    L.d = d;
    L.codes = (int8_t *)codes;
    L.scales = (float *)scales;
    L.counts = (int32_t *)counts;
    L.X = X;
    L.n = n;
    L.out_err = err;
    L.out_ref = ref_opt;
    return output_error_impl(&L, 1, max_points, stream);
}

int mpq_output_error_layers(const mpq_layer *layers, int n_layers, int max_points, void *stream)
{
    return output_error_impl(layers, n_layers, max_points, stream);
}

int mpq_output_error_noalloc(const float *W, const int8_t *codes, const float *scales,
                             const int32_t *counts, int64_t c_out, int64_t d, int max_points,
                             const float *X, int64_t n, float *err, float *ref_opt, void *stream)
{
    mpq_layer L = {};
    L.W = W;
    L.c_out = c_out;
    L.d = d;
    L.codes = (int8_t *)codes;
    L.scales = (float *)scales;
    L.counts = (int32_t *)counts;
    L.X = X;
    L.n = n;
    L.out_err = err;
    L.out_ref = ref_opt;
    // the argument checks come first: the workspace lookup is a HIP call
    int rc = check_error_layer(L, max_points, true);
    if (rc != MPQ_OK || c_out == 0) return rc;
    char *ws = nullptr;
    rc = noalloc_workspace(&ws);
    if (rc != MPQ_OK) return rc;
    return output_error_impl(&L, 1, max_points, stream, ws, (size_t)MPQ_NOALLOC_BYTES);
}

int mpq_reconstruct(const int8_t *codes, const float *scales, const int32_t *counts, int64_t c_out,
                    int64_t d, int max_points, float *W_hat, void *stream)
{
    mpq_layer L = {};
    L.c_out = c_out;
    L.d = d;
    L.codes = (int8_t *)codes;
    L.scales = (float *)scales;
    L.counts = (int32_t *)counts;
    L.W_hat = W_hat;
    return reconstruct_impl(&L, 1, max_points, stream);
}

int mpq_reconstruct_layers(const mpq_layer *layers, int n_layers, int max_points, void *stream)
{
    return reconstruct_impl(layers, n_layers, max_points, stream);
}

}  // extern "C"
