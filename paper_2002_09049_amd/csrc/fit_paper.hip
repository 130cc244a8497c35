// Greedy multipoint fit on the paper's own grid (Eq. (11), Def. 1): at each
// step the candidate scales are a_g = g * gamma, g = 1 .. floor(2 M ||r|| /
// gamma), gamma = min(Delta_r / M, eta), Delta_r half the smallest positive
// difference of the |r_j| (no gap: gamma = eta).  The chosen scale is stored
// as fl32(a_g); the codes (Eq. (10)) and the residual (Eq. (7)) use that
// stored value.  Stopping rule as for the other fits (||r||^2 <= tol ||w||^2,
// cap, zero residual, no nonzero scale).
//
// The grid can hold far more points than can be enumerated (10^8 and more).
// The codes are constant between consecutive breakpoints b = |r_j| / (k+1/2),
// where E(a) = ||r||^2 - 2 a A + a^2 B is a convex quadratic, so the argmin
// over the grid is one of the three grid points around some breakpoint, or
// one of the two next to the vertex A / B of a piece that holds such a point.
// With the magnitudes sorted (descending) and their prefix sums S,
//   c_k(a) = #{ j : |r_j| > a (k + 1/2) }   (binary search; a magnitude
//            exactly on the boundary counts when k is odd, ties to even),
//   A(a) = sum_k S[c_k],  B(a) = sum_k (2k + 1) c_k,
// so each candidate costs O(M log d).  The d M breakpoints are spread over
// the threads; the smallest error wins, ties to the smallest g.  A piece
// whose quadratic minimum R - A^2 / B exceeds the best error a thread has
// found cannot hold the argmin, so its vertex candidates are skipped.
//
// One workgroup of 256 threads per channel; the fp64 residual stays in
// registers (EPT elements per thread); the sorted magnitudes and their
// prefix sums occupy 2 dpad doubles of LDS (dpad = d rounded up to a power
// of two, at most kPaperMaxDim).
#include <math.h>

#include <algorithm>
#include <stdio.h>

#include "internal.hpp"
#include "mpq.h"
#include "reduce.hpp"

namespace mpq {

namespace {

constexpr int kPT = 256;   // threads per workgroup

struct Best {
    double e;
    long long g;
};

__device__ __forceinline__ Best better(Best x, Best y)
{
    return (y.e < x.e || (y.e == x.e && y.g < x.g)) ? y : x;
}

template <int kT>
__device__ __forceinline__ Best block_best_n(Best v, double *se, long long *sg)
{
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        Best o{__shfl_xor(v.e, off), __shfl_xor(v.g, off)};
        v = better(v, o);
    }
    const int wid = threadIdx.x / kWave;
    if ((threadIdx.x % kWave) == 0) {
        se[wid] = v.e;
        sg[wid] = v.g;
    }
    __syncthreads();
    Best r{se[0], sg[0]};
#pragma unroll
    for (int i = 1; i < kT / kWave; ++i) r = better(r, Best{se[i], sg[i]});
    __syncthreads();
    return r;
}

__device__ __forceinline__ Best block_best(Best v, double *se, long long *sg)
{
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        Best o{__shfl_xor(v.e, off), __shfl_xor(v.g, off)};
        v = better(v, o);
    }
    const int wid = threadIdx.x / kWave;
    if ((threadIdx.x % kWave) == 0) {
        se[wid] = v.e;
        sg[wid] = v.g;
    }
    __syncthreads();
    Best r{se[0], sg[0]};
#pragma unroll
    for (int i = 1; i < kPT / kWave; ++i) r = better(r, Best{se[i], sg[i]});
    __syncthreads();
    return r;
}

// number of sorted (descending) magnitudes s[0 .. d) greater than x, or with
// or_equal, greater than or equal to x
__device__ __forceinline__ int count_above(const double *s, int d, double x, bool or_equal)
{
    int lo = 0, hi = d;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (s[mid] > x || (or_equal && s[mid] == x)) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// E(a) from the sorted magnitudes s and their prefix sums S; also A, B.  A
// magnitude exactly at a (k + 1/2) has the code of the even neighbour (Eq.
// (2)'s ties to even): past level k when k + 1 is even.
__device__ __forceinline__ double paper_error(const double *s, const double *S, int d, int M, double R,
                                              double a, double &A, double &B)
{
    double sa = 0.0, sb = 0.0;
    for (int k = 0; k < M; ++k) {
        const int c = count_above(s, d, a * ((double)k + 0.5), (k & 1) != 0);
        sa += S[c];
        sb += (double)(2 * k + 1) * (double)c;
    }
    A = sa;
    B = sb;
    return (R - 2.0 * a * sa) + a * a * sb;
}

template <int EPT>
__global__ void __launch_bounds__(kPT) fit_paper_kernel(const PaperBatch B)
{
    extern __shared__ __align__(16) double psmem[];
    __shared__ float s_redf[kPT / kWave];
    __shared__ double s_redd[kPT / kWave];
    __shared__ long long s_redg[kPT / kWave];

    const int li = last_at_most(B.n_layers, (int)blockIdx.x, [&](int i) { return B.L[i].c_begin; });
    const HistLayer &Ly = B.L[li];
    const int64_t k = (int64_t)blockIdx.x - Ly.c_begin;
    const int t = threadIdx.x, d = Ly.d, P = B.P, M = B.M;
    const double Md = (double)M;
    int dpad = 1;
    while (dpad < d) dpad <<= 1;
    double *s = psmem;          // [dpad] magnitudes, sorted descending (pads -1)
    double *S = psmem + dpad;   // [d + 1] prefix sums of s
    int8_t *qk = Ly.codes + k * (int64_t)P * d;
    const float *wk = Ly.W + k * (int64_t)d;

    double r[EPT];
#pragma unroll
    for (int u = 0; u < EPT; ++u) {
        const int j = t + kPT * u;
        r[u] = j < d ? (double)wk[j] : 0.0;
    }
    double Ew = 0.0;
    float apend = 0.0f;
    int n = 0;
    for (int i = 0;; ++i) {
        // ---- apply the pending point (codes of Eq. (10) at the stored scale)
        float lmax = 0.0f;
        double lsum = 0.0;
        if (i >= 1) {
            const double ap = (double)apend, ia = 1.0 / ap;
            int8_t *qrow = qk + (int64_t)(i - 1) * d;
#pragma unroll
            for (int u = 0; u < EPT; ++u) {
                const int j = t + kPT * u;
                if (j < d) {
                    const double y = r[u] * ia;
                    double c = rint(y);
                    if (fabs(fabs(y - c) - 0.5) < 0x1p-40) c = rint(r[u] / ap);
                    c = fmin(fmax(c, -Md), Md);
                    qrow[j] = (int8_t)(int)c;
                    r[u] = fma(-ap, c, r[u]);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < EPT; ++u) {
            lmax = fmaxf(lmax, fabsf((float)r[u]));
            lsum = fma(r[u], r[u], lsum);
        }
        block_max_sum<kPT>(lmax, lsum, s_redf, s_redd);
        const double Er = lsum;
        if (i == 0) Ew = Er;
        else if (Ly.err && t == 0) Ly.err[k * P + (i - 1)] = (float)Er;
        if (i >= P || Er == 0.0 || (i >= 1 && Er <= B.tol * Ew)) {
            n = i;
            break;
        }

        // ---- sorted magnitudes (bitonic, descending; pads -1 sort last)
        for (int j = t; j < dpad; j += kPT) s[j] = -1.0;
        __syncthreads();
#pragma unroll
        for (int u = 0; u < EPT; ++u) {
            const int j = t + kPT * u;
            if (j < d) s[j] = fabs(r[u]);
        }
        __syncthreads();
        for (int kk = 2; kk <= dpad; kk <<= 1) {
            for (int jj = kk >> 1; jj > 0; jj >>= 1) {
                for (int x = t; x < dpad; x += kPT) {
                    const int y = x ^ jj;
                    if (y > x) {
                        const double a = s[x], b = s[y];
                        const bool desc = (x & kk) == 0;
                        if (desc ? (a < b) : (a > b)) {
                            s[x] = b;
                            s[y] = a;
                        }
                    }
                }
                __syncthreads();
            }
        }
        // ---- minimal gap (Def. 1), gamma and the grid size (Eq. (11))
        double lgap = INFINITY;
        for (int j = t; j + 1 < d; j += kPT) {
            const double diff = s[j] - s[j + 1];
            if (diff > 0.0) lgap = fmin(lgap, diff);
        }
        lgap = block_reduce<kPT>(lgap, MinOp(), s_redd);
        double gamma = lgap == INFINITY ? B.eta : fmin(lgap / 2.0 / Md, B.eta);
        // (grid indices stay far below 2^63: clamped at 4e18)
        const long long count = (long long)fmin(floor(2.0 * Md * sqrt(Er) / gamma), 4e18);
        // ---- prefix sums S[0..d] of the sorted magnitudes (fixed order)
        {
            const int per = (d + kPT - 1) / kPT, j0 = min(t * per, d), j1 = min(j0 + per, d);
            double loc = 0.0;
            for (int j = j0; j < j1; ++j) loc += s[j];
            // exclusive scan of the per-thread sums over the workgroup
            double v = loc;
#pragma unroll
            for (int off = 1; off < kWave; off <<= 1) {
                const double o = __shfl_up(v, off);
                if ((t % kWave) >= off) v += o;
            }
            if ((t % kWave) == kWave - 1) s_redd[t / kWave] = v;
            __syncthreads();
            double base = 0.0;
            for (int w = 0; w < t / kWave; ++w) base += s_redd[w];
            double run = base + v - loc;
            for (int j = j0; j < j1; ++j) {
                S[j] = run;
                run += s[j];
            }
            if (t == kPT - 1) S[d] = run;
            __syncthreads();
        }
        // ---- candidates around every breakpoint and at the pieces' vertices
        Best best{INFINITY, 0x7fffffffffffffffLL};
        auto try_g = [&](long long g) {
            if (g < 1 || g > count) return;
            double A, Bq;
            const double E = paper_error(s, S, d, M, Er, (double)g * gamma, A, Bq);
            best = better(best, Best{E, g});
        };
        for (int e = t; e < d * M; e += kPT) {
            const int j = e / M, kl = e - j * M;
            const double b = s[j] / ((double)kl + 0.5);
            if (!(b > 0.0)) continue;
            const long long g0 = (long long)fmin(floor(b / gamma), 4e18);
            for (long long g = g0 - 1; g <= g0 + 1; ++g) {
                if (g < 1 || g > count) continue;
                double A, Bq;
                const double E = paper_error(s, S, d, M, Er, (double)g * gamma, A, Bq);
                best = better(best, Best{E, g});
                // the piece's quadratic has its minimum R - A^2 / B at the
                // vertex, a lower bound for every grid point of the piece:
                // skip the vertex candidates when it already exceeds the best
                // error found (with a margin for rounding)
                if (Bq > 0.0 && Er - A * A / Bq <= best.e + 1e-12 * Er) {
                    const long long gv = (long long)fmin(floor((A / Bq) / gamma), 4e18);
                    try_g(gv);
                    try_g(gv + 1);
                }
            }
        }
        best = block_best(best, s_redd, s_redg);
        const float af = best.e == INFINITY ? 0.0f : (float)((double)best.g * gamma);
        if (af == 0.0f) {   // no candidate with a nonzero scale
            n = i;
            break;
        }
        apend = af;
        if (t == 0) Ly.scales[k * P + i] = af;
        __syncthreads();   // s and S are rewritten by the next step
    }

    if (t == 0) Ly.counts[k] = n;
    for (int q = n + t; q < P; q += kPT) {
        Ly.scales[k * P + q] = 0.0f;
        if (Ly.err) Ly.err[k * P + q] = 0.0f;
    }
    for (int q = n; q < P; ++q)
        for (int j = t; j < d; j += kPT) qk[(int64_t)q * d + j] = 0;
}

// ---- channels longer than kPaperMaxDim: the same steps, with the sorted
// magnitudes s and their prefix sums S of a channel in a global scratch (2 d
// doubles do not fit a workgroup's LDS), and the residual rebuilt at each
// step from W and the stored points (the fp64 operations of the register
// version, in point order, so bitwise the same residual).  The sort is the
// bitonic network of the LDS version, its stages with partner distance below
// kPaperChunk run on kPaperChunk-element chunks staged in LDS, the others as
// passes over the global array.  Workgroups take channels in turn (a
// grid-stride loop), so the scratch is one slice per workgroup.
constexpr int kPBT = 512;            // threads per workgroup
constexpr int kPaperChunk = 4096;    // elements of an LDS chunk of the sort

// compare-exchange of the bitonic network's stage (kk, jj) on x and x ^ jj
// (descending where x & kk == 0); v holds the array
template <class Arr>
__device__ __forceinline__ void bitonic_cx(Arr &v, int x, int y, int kk, int gx)
{
    const double a = v[x], b = v[y];
    const bool desc = (gx & kk) == 0;
    if (desc ? (a < b) : (a > b)) {
        v[x] = b;
        v[y] = a;
    }
}

// stages (kk, jj) for jj from jstart down to 1 on the chunk of s at base,
// staged in LDS (the chunk's global index gives each pair's direction);
// kk_lo..kk_hi: every kk from kk_lo (with jj from kk / 2) to kk_hi, except
// that the first kk starts at jstart
__device__ __forceinline__ void chunk_stages(double *s, double *lds, int base, int kk_lo, int kk_hi,
                                             int jstart)
{
    const int t = threadIdx.x;
    for (int x = t; x < kPaperChunk; x += kPBT) lds[x] = s[base + x];
    __syncthreads();
    for (int kk = kk_lo; kk <= kk_hi; kk <<= 1) {
        for (int jj = kk == kk_lo ? jstart : kk >> 1; jj > 0; jj >>= 1) {
            for (int x = t; x < kPaperChunk; x += kPBT) {
                const int y = x ^ jj;
                if (y > x) bitonic_cx(lds, x, y, kk, base + x);
            }
            __syncthreads();
        }
    }
    for (int x = t; x < kPaperChunk; x += kPBT) s[base + x] = lds[x];
    __syncthreads();
}

__global__ void __launch_bounds__(kPBT) fit_paper_big_kernel(const PaperBatch B, int64_t channels,
                                                             double *scratch, int64_t slice)
{
    __shared__ __align__(16) double lds[kPaperChunk];
    __shared__ float s_redf[kPBT / kWave];
    __shared__ double s_redd[kPBT / kWave];
    __shared__ long long s_redg[kPBT / kWave];
    __shared__ float s_scale[MPQ_MAX_POINTS];
    const int t = threadIdx.x, P = B.P, M = B.M;
    const double Md = (double)M;
    double *s = scratch + (int64_t)blockIdx.x * slice;   // [dpad] sorted magnitudes
    for (int64_t ch = blockIdx.x; ch < channels; ch += gridDim.x) {
        const int li = last_at_most(B.n_layers, (int)ch, [&](int i) { return B.L[i].c_begin; });
        const HistLayer &Ly = B.L[li];
        const int64_t k = ch - Ly.c_begin;
        const int d = Ly.d;
        int dpad = kPaperChunk;
        while (dpad < d) dpad <<= 1;
        double *S = s + dpad;   // [d + 1] prefix sums
        int8_t *qk = Ly.codes + k * (int64_t)P * d;
        const float *wk = Ly.W + k * (int64_t)d;
        auto rebuild = [&](int j, int np) {
            double v = (double)wk[j];
            for (int p = 0; p < np; ++p) v = fma(-(double)s_scale[p], (double)qk[(int64_t)p * d + j], v);
            return v;
        };
        double Ew = 0.0;
        float apend = 0.0f;
        int n = 0;
        for (int i = 0;; ++i) {
            // ---- apply the pending point; |r| of the new residual into s
            float lmax = 0.0f;
            double lsum = 0.0;
            const double ap = (double)apend, ia = 1.0 / ap;
            int8_t *qrow = qk + (int64_t)(i - 1) * d;
            for (int j = t; j < dpad; j += kPBT) {
                double r = -1.0;   // pads sort last
                if (j < d) {
                    r = rebuild(j, i >= 1 ? i - 1 : 0);
                    if (i >= 1) {
                        const double y = r * ia;
                        double c = rint(y);
                        if (fabs(fabs(y - c) - 0.5) < 0x1p-40) c = rint(r / ap);
                        c = fmin(fmax(c, -Md), Md);
                        qrow[j] = (int8_t)(int)c;
                        r = fma(-ap, c, r);
                    }
                    lmax = fmaxf(lmax, fabsf((float)r));
                    lsum = fma(r, r, lsum);
                    r = fabs(r);
                }
                s[j] = r;
            }
            block_max_sum<kPBT>(lmax, lsum, s_redf, s_redd);
            const double Er = lsum;
            if (i == 0) Ew = Er;
            else if (Ly.err && t == 0) Ly.err[k * P + (i - 1)] = (float)Er;
            if (i >= P || Er == 0.0 || (i >= 1 && Er <= B.tol * Ew)) {
                n = i;
                break;
            }
            __syncthreads();   // every |r| is in s
            // ---- sorted magnitudes (descending): each chunk sorted in LDS
            // in its direction, then the stages across chunks
            for (int base = 0; base < dpad; base += kPaperChunk) chunk_stages(s, lds, base, 2, kPaperChunk, 1);
            for (int kk = 2 * kPaperChunk; kk <= dpad; kk <<= 1) {
                for (int jj = kk >> 1; jj >= kPaperChunk; jj >>= 1) {
                    for (int x = t; x < dpad; x += kPBT) {
                        const int y = x ^ jj;
                        if (y > x) bitonic_cx(s, x, y, kk, x);
                    }
                    __syncthreads();
                }
                for (int base = 0; base < dpad; base += kPaperChunk)
                    chunk_stages(s, lds, base, kk, kk, kPaperChunk >> 1);
            }
            // ---- minimal gap (Def. 1), gamma and the grid size (Eq. (11))
            double lgap = INFINITY;
            for (int j = t; j + 1 < d; j += kPBT) {
                const double diff = s[j] - s[j + 1];
                if (diff > 0.0) lgap = fmin(lgap, diff);
            }
            lgap = block_reduce<kPBT>(lgap, MinOp(), s_redd);
            const double gamma = lgap == INFINITY ? B.eta : fmin(lgap / 2.0 / Md, B.eta);
            const long long count = (long long)fmin(floor(2.0 * Md * sqrt(Er) / gamma), 4e18);
            // ---- prefix sums S[0..d] (fixed order: per-thread chunks, then
            // the threads' totals in order)
            {
                const int per = (d + kPBT - 1) / kPBT, j0 = min(t * per, d), j1 = min(j0 + per, d);
                double loc = 0.0;
                for (int j = j0; j < j1; ++j) loc += s[j];
                double v = loc;
#pragma unroll
                for (int off = 1; off < kWave; off <<= 1) {
                    const double o = __shfl_up(v, off);
                    if ((t % kWave) >= off) v += o;
                }
                if ((t % kWave) == kWave - 1) s_redd[t / kWave] = v;
                __syncthreads();
                double base = 0.0;
                for (int w = 0; w < t / kWave; ++w) base += s_redd[w];
                double run = base + v - loc;
                for (int j = j0; j < j1; ++j) {
                    S[j] = run;
                    run += s[j];
                }
                if (t == kPBT - 1) S[d] = run;
                __syncthreads();
            }
            // ---- candidates around every breakpoint and at the pieces' vertices
            Best best{INFINITY, 0x7fffffffffffffffLL};
            auto try_g = [&](long long g) {
                if (g < 1 || g > count) return;
                double A, Bq;
                const double E = paper_error(s, S, d, M, Er, (double)g * gamma, A, Bq);
                best = better(best, Best{E, g});
            };
            for (int e = t; e < d * M; e += kPBT) {
                const int j = e / M, kl = e - j * M;
                const double b = s[j] / ((double)kl + 0.5);
                if (!(b > 0.0)) continue;
                const long long g0 = (long long)fmin(floor(b / gamma), 4e18);
                for (long long g = g0 - 1; g <= g0 + 1; ++g) {
                    if (g < 1 || g > count) continue;
                    double A, Bq;
                    const double E = paper_error(s, S, d, M, Er, (double)g * gamma, A, Bq);
                    best = better(best, Best{E, g});
                    if (Bq > 0.0 && Er - A * A / Bq <= best.e + 1e-12 * Er) {
                        const long long gv = (long long)fmin(floor((A / Bq) / gamma), 4e18);
                        try_g(gv);
                        try_g(gv + 1);
                    }
                }
            }
            best = block_best_n<kPBT>(best, s_redd, s_redg);
            const float af = best.e == INFINITY ? 0.0f : (float)((double)best.g * gamma);
            if (af == 0.0f) {   // no candidate with a nonzero scale
                n = i;
                break;
            }
            apend = af;
            if (t == 0) {
                Ly.scales[k * P + i] = af;
                s_scale[i] = af;
            }
            __syncthreads();   // s, S and s_scale are read by the next step
        }

        if (t == 0) Ly.counts[k] = n;
        for (int q = n + t; q < P; q += kPBT) {
            Ly.scales[k * P + q] = 0.0f;
            if (Ly.err) Ly.err[k * P + q] = 0.0f;
        }
        for (int q = n; q < P; ++q)
            for (int j = t; j < d; j += kPBT) qk[(int64_t)q * d + j] = 0;
        __syncthreads();   // the next channel rewrites s and s_scale
    }
}

template <int EPT>
hipError_t launch_paper_t(const PaperBatch &b, int64_t channels, size_t lds, hipStream_t s)
{
    auto kern = fit_paper_kernel<EPT>;
    if (lds > 65536) {
        hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)lds);
        if (e != hipSuccess) return e;
    }
    char name[48];
    snprintf(name, sizeof name, "fit_paper_kernel<%d>", EPT);
    LaunchTimer timer(s, name);
    hipLaunchKernelGGL(kern, dim3((unsigned)channels), dim3(kPT), lds, s, b);
    return hipGetLastError();
}

}  // namespace

int paper_variant(int64_t d)
{
    return d <= 2 * kPT ? 0 : d <= 4 * kPT ? 1 : d <= 8 * kPT ? 2 : d <= 16 * kPT ? 3 :
           d <= kPaperMaxDim ? 4 : kPaperBigVariant;
}

int paper_big_grid(int64_t channels)
{
    return (int)std::min<int64_t>(channels, kPaperBigGrid);
}

size_t paper_big_slice(int64_t dmax)
{
    int64_t dpad = kPaperChunk;
    while (dpad < dmax) dpad <<= 1;
    return (size_t)(dpad + dmax + 1);   // doubles
}

hipError_t launch_fit_paper_big(const PaperBatch &b, int64_t channels, int64_t dmax, double *scratch,
                                hipStream_t s)
{
    if (channels <= 0) return hipSuccess;
    if (channels > 0x7fffffffLL || dmax > kPaperBigMaxDim) return hipErrorInvalidValue;
    LaunchTimer timer(s, "fit_paper_big_kernel");
    hipLaunchKernelGGL(fit_paper_big_kernel, dim3((unsigned)paper_big_grid(channels)), dim3(kPBT), 0, s, b,
                       channels, scratch, (int64_t)paper_big_slice(dmax));
    return hipGetLastError();
}

size_t paper_lds(int64_t dmax)
{
    int64_t dpad = 1;
    while (dpad < dmax) dpad <<= 1;
    return (size_t)(2 * dpad + 1) * sizeof(double);
}

hipError_t launch_fit_paper(const PaperBatch &b, int variant, int64_t channels, int64_t dmax, hipStream_t s)
{
    if (channels <= 0) return hipSuccess;
    if (channels > 0x7fffffffLL || dmax > kPaperMaxDim) return hipErrorInvalidValue;
    const size_t lds = paper_lds(dmax);
    switch (variant) {
    case 0: return launch_paper_t<2>(b, channels, lds, s);
    case 1: return launch_paper_t<4>(b, channels, lds, s);
    case 2: return launch_paper_t<8>(b, channels, lds, s);
    case 3: return launch_paper_t<16>(b, channels, lds, s);
    case 4: return launch_paper_t<32>(b, channels, lds, s);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace mpq
