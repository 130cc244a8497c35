// Greedy multipoint fit (Algorithm 1, Sec. 3.2, with the stopping rule of
// Algorithm 2, Sec. 3.3) with an exact O(d*M + G) evaluation of the
// candidate errors of Eq. (9).
//
// For a candidate scale a and x = |r_j|, the code magnitude of element j is
// the number of levels k in [0, M) whose boundary (k + 1/2) a lies below x
// (Eq. (2); an exact half-way point gives the same error either way, so the
// boundary may be taken as strict).  The candidates are sorted
// (a_g = fl32(m c_g / M) with c_g ascending), so for each (j, k) the
// candidates that lift element j past level k are a prefix g < n_jk with
//     n_jk = #{ g : (k + 1/2) a_g < x_j }       ((k+1/2) a_g is exact in fp64).
// With A(g) = sum_j x_j |q_j(g)| and B(g) = sum_j q_j(g)^2,
//     E(g) = ||r||^2 - 2 a_g A(g) + a_g^2 B(g),
// and A, B are suffix sums of histograms that receive, per (j, k) with
// n_jk > 0, x_j (in 64-bit fixed point) and 2k + 1 at bin n_jk - 1.  Integer
// LDS atomics make the histograms exact and order independent.  Every E(g)
// carries an error bound; the candidates whose interval reaches the minimum
// are re-evaluated directly (fp64, like Eq. (9) written out) and the smallest
// error wins, ties to the smallest g.
//
// Lattice mode (default grid, (2M-1) G + 1 buckets fit): with u = m / (2 G M)
// every boundary (k + 1/2) a_g lies within relative 2^-23 of the lattice
// point L = (2k+1)(g+1) times u.  An element whose x / u is farther than
// N 2^-21 from its nearest integer N crosses exactly the boundaries with
// L <= floor(x / u), so it goes to that one bucket (fixed-point x and a count
// packed in one 64-bit word); A(g) and B(g) are then sums over k of suffix
// sums at L = (2k+1)(g+1).  An element that near N goes to bucket N - 1, and
// each boundary at L = N is decided exactly and, when crossed, added to a
// per-candidate correction.  This replaces M atomics per element with one
// and gives the same integer sums.
//
// One workgroup per channel.  The fp64 residual stays in registers for the
// whole fit (EPT elements per thread, element j = t + T * u), so each step
// reads nothing from HBM: it writes the codes of the point chosen by the
// previous step (Eq. (10), fp64 quotient) and updates the residual (Eq. (7)).
#include <math.h>
#include <stdio.h>

#include "internal.hpp"
#include "mpq.h"
#include "point_code.hpp"
#include "reduce.hpp"

namespace mpq {

namespace {

constexpr int kMaxFinalists = 8;

// lattice buckets: fixed-point x in the low kLatShift bits, count above
constexpr int kLatShift = 49;
constexpr unsigned long long kLatOne = 1ull << kLatShift;
constexpr unsigned long long kLatMask = kLatOne - 1;
constexpr int kLatMaxBuckets = 4096;

struct HistShared {
    // ha and hb hold a candidate's histogram sums until its error is formed;
    // the same slots then hold that error (fp64 bits) and its bound (fp32
    // bits, rounded up, in units of 2^be with be the exponent of ||r||^2, so
    // that the ratio lies far inside fp32's range)
    long long *ha;   // [G] fixed-point sum of x per bin (lattice mode: per-candidate corrections)
    int *hb;         // [G] sum of (2k + 1) per bin (lattice mode: corrections)
    float *af;       // [G + 2]: af[0] = 0, af[g + 1] = a_g, af[G + 1] = +inf
    unsigned long long *lat;   // [nlat] lattice buckets (lattice mode only)

    // the bound in fp32 above b 2^-be: that value is at least 2^-51 (b holds
    // 8 2^-53 ||r||^2), so fl32 is normal and within relative 2^-24, and the
    // product by 1 + 2^-22, rounded, lies above it
    __device__ void put_err(int g, double e, double b, int be) const
    {
        ha[g] = __double_as_longlong(e);
        hb[g] = __float_as_int((float)ldexp(b, -be) * 0x1.000004p0f);
    }
    __device__ double err(int g) const { return __longlong_as_double(ha[g]); }
    __device__ double bnd(int g, int be) const { return ldexp((double)__int_as_float(hb[g]), be); }
};

// n = #{ g : h * a_g < x } over the non-decreasing candidates, by binary
// search (general grids).  af is the sentinel table of HistShared (a_g is an
// fp32 value, so its fp64 widening is exact).
__device__ __forceinline__ int count_bsearch(const float *af, int G, double h, double x)
{
    int lo = 0, hi = G;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (fma(h, (double)af[mid + 1], -x) < 0.0) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// The same count for the default grid a_g = fl32(m fl32((g+1)/G) / M), from
// est = fl32 of x G M / (h m), computed as fl32(fl32(fl32(x) fl32(G M / m))
// rcp(h)): within relative 6 2^-24 of E = x G M / (h m) (five roundings and
// the reciprocal's one ulp), so within 0.0015 of E while est <= G + 1.  The
// boundary test (k + 1/2) a_g < x reads (g + 1)(1 + delta) < E with |delta|
// <= 2^-23 (the roundings of c_g and a_g), within 0.0005 of (g + 1) < E for
// G <= 4096.  So unless an integer N in [1, G] lies within 0.003 of est, the
// count is min(floor(est), G) with no table read; otherwise only candidate
// N - 1 is undecided and one exact comparison settles it (h a is exact in
// fp64 and the fma rounds once, so its sign is exact; af[N] = a_{N-1}).
__device__ __forceinline__ int count_linear(const float *af, int G, double h, double x, float est)
{
    const float Nf = rintf(est);
    const int N = (int)Nf;
    int n = min((int)est, G);
    if (fabsf(est - Nf) <= 0.003f && N >= 1 && N <= G)
        n = N - 1 + (fma(h, (double)af[N], -x) < 0.0 ? 1 : 0);
    return n;
}

// Histogram of the level boundaries of this thread's elements.  Level-major:
// for each level, the counts of a chunk of elements are found first
// (independent LDS reads in flight together), then binned.  A boundary that
// every candidate passes (n = G: most elements at the low levels) would send
// most lanes to bin G-1 at once; those are summed in fullA / fullB and added
// by the caller with one atomic per wavefront.
template <int T, int EPT, bool kLinear>
__device__ __forceinline__ void bin_levels(const double (&r)[EPT], const HistShared &S, int G, int M,
                                           float m, int sh, unsigned long long &fullA, int &fullB)
{
    const float gm = (float)G * (float)M / m;
    // per element and step: fixed-point |r| and the scaled estimate base
    constexpr bool kKeep = EPT <= 16 && T <= 256;
    unsigned long long Xk[kKeep ? EPT : 1];
    float Bk[kKeep ? EPT : 1];
    if constexpr (kKeep) {
#pragma unroll
        for (int u = 0; u < EPT; ++u) {
            Xk[u] = (unsigned long long)rint(ldexp(fabs(r[u]), sh));
            Bk[u] = (float)fabs(r[u]) * gm;
        }
    }
    constexpr int kChunk = EPT < 4 ? EPT : 4;
    for (int kk = 0; kk < M; ++kk) {
        const double h = (double)kk + 0.5;
        const float rh = __builtin_amdgcn_rcpf((float)h);
        const int inc = 2 * kk + 1;
#pragma unroll
        for (int u0 = 0; u0 < EPT; u0 += kChunk) {
            int nb[kChunk];
#pragma unroll
            for (int v = 0; v < kChunk; ++v) {
                const int u = u0 + v;
                if (u >= EPT) break;   // last chunk of an EPT that kChunk does not divide
                const double x = fabs(r[u]);
                if constexpr (kLinear) {
                    const float base = kKeep ? Bk[kKeep ? u : 0] : (float)x * gm;
                    nb[v] = count_linear(S.af, G, h, x, base * rh);
                } else {
                    nb[v] = count_bsearch(S.af, G, h, x);
                }
            }
#pragma unroll
            for (int v = 0; v < kChunk; ++v) {
                const int u = u0 + v;
                if (u >= EPT) break;
                const unsigned long long X =
                    kKeep ? Xk[kKeep ? u : 0] : (unsigned long long)rint(ldexp(fabs(r[u]), sh));
                const bool full = nb[v] == G;
                fullA += full ? X : 0ull;
                fullB += full ? inc : 0;
                if (nb[v] > 0 && !full) {
                    atomicAdd((unsigned long long *)&S.ha[nb[v] - 1], X);
                    atomicAdd(&S.hb[nb[v] - 1], inc);
                }
            }
        }
    }
}

// The per-level histogram of bin_levels, element-major: for the variant that
// rebuilds each residual element from memory, so that an element is rebuilt
// once per step rather than once per level.
// One element x = |r_j| of the per-level histogram, level by level until no
// candidate lifts it (gm = G M / m).
template <bool kLinear>
__device__ __forceinline__ void bin_levels_elem(double x, const HistShared &S, int G, int M, float gm,
                                                int sh, unsigned long long &fullA, int &fullB)
{
    const unsigned long long X = (unsigned long long)rint(ldexp(x, sh));
    const float base = (float)x * gm;
    for (int kk = 0; kk < M; ++kk) {
        const double h = (double)kk + 0.5;
        int nb;
        if constexpr (kLinear) nb = count_linear(S.af, G, h, x, base * __builtin_amdgcn_rcpf((float)h));
        else nb = count_bsearch(S.af, G, h, x);
        if (nb == 0) break;   // higher levels have higher boundaries
        const int inc = 2 * kk + 1;
        if (nb == G) {
            fullA += X;
            fullB += inc;
        } else {
            atomicAdd((unsigned long long *)&S.ha[nb - 1], X);
            atomicAdd(&S.hb[nb - 1], inc);
        }
    }
}

// The same histogram over this thread's slots of four consecutive elements
// (the variant that rebuilds its residual; r4(v, o) fills slot v).
template <int T, int kSlots, bool kLinear, class Res4>
__device__ __forceinline__ void bin_levels_slots(Res4 r4, const HistShared &S, int G, int M, int d,
                                                 float m, int sh, unsigned long long &fullA, int &fullB)
{
    const float gm = (float)G * (float)M / m;
    for (int v = 0; v < kSlots; ++v) {
        if (4 * T * v >= d) break;
        double o[4];
        r4(v, o);
#pragma unroll
        for (int c = 0; c < 4; ++c) bin_levels_elem<kLinear>(fabs(o[c]), S, G, M, gm, sh, fullA, fullB);
    }
}

// Lattice-mode binning of this thread's elements (see the header).  inv =
// 1 / u in fp64; Lmax = nlat - 1 is the largest lattice point of a boundary;
// scale = 2^sh.
//
// z = x inv is x / u within relative 2^-51, and N = rint(z).  The boundaries
// at lattice point N lie within N 2^-23 of N (in units of u; a_g carries one
// fp32 rounding of m c_g / M, relative 2^-23 with c_g's), the others at least
// 1 - 4096 2^-23 from x / u.  So |z - N| > N 2^-22 (a 2x margin) puts x / u
// on N's side of every boundary at N, and the element crosses exactly the
// boundaries at L <= floor(z); otherwise it crosses every boundary below N
// (bucket N - 1) and those at N are decided one by one.  The tolerance grows
// with N, so the small residuals, most of a channel, are rarely near.  The
// bucket word is formed by one fma: x 2^sh + 2^52 + 2^kLatShift rounds
// x 2^sh to the nearest integer (ties to even, as rint) and its low 52 bits
// are that integer plus the count bit.
__device__ __forceinline__ void bin_lattice_elem(double x, const HistShared &S, int G, int M, int Lmax,
                                                 double inv, double scale)
{
    constexpr double kBias = 0x1p52 + (double)kLatOne;
    {
        const double z = x * inv;
        const double Nd = rint(z);
        const int Ni = (int)Nd;
        const bool near = Ni >= 1 && fabs(z - Nd) <= Nd * 0x1p-22;
        const int b = near ? Ni - 1 : (z >= Nd ? Ni : Ni - 1);
        const unsigned long long word =
            (unsigned long long)__double_as_longlong(fma(x, scale, kBias)) & ((1ull << 52) - 1);
        if (b >= 1) atomicAdd(&S.lat[min(b, Lmax)], word);
        if (near && Ni >= 1) {
            // boundaries at lattice point N: (2k+1) divides N, g + 1 = N / (2k+1) <= G
            const unsigned long long X = word - kLatOne;
            for (int kk = 0; kk < M; ++kk) {
                const int o = 2 * kk + 1;
                // N / o rounded from fp32 (N < 2^12, o < 2^8): exact when o
                // divides N, and q o == N tells whether it does
                const int q = (int)rintf((float)Ni * __builtin_amdgcn_rcpf((float)o));
                if (q < 1) break;
                if (q * o != Ni || q > G) continue;
                const int g = q - 1;
                if (fma((double)kk + 0.5, (double)S.af[g + 1], -x) < 0.0) {
                    atomicAdd((unsigned long long *)&S.ha[g], X);
                    atomicAdd(&S.hb[g], o);
                }
            }
        }
    }
}

template <int T, int EPT, int kUnroll, class Res>
__device__ __forceinline__ void bin_lattice(Res r, const HistShared &S, int G, int M, int d, int Lmax,
                                            double inv, double scale)
{
#pragma unroll kUnroll
    for (int u = 0; u < EPT; ++u) {
        if (T * u >= d) continue;   // a slot past the channel end in every thread
        bin_lattice_elem(fabs(r(u)), S, G, M, Lmax, inv, scale);
    }
}

// The same over this thread's slots of four consecutive elements (the
// variant that rebuilds its residual; r4(v, o) fills slot v).
template <int T, int kSlots, class Res4>
__device__ __forceinline__ void bin_lattice_slots(Res4 r4, const HistShared &S, int G, int M, int d,
                                                  int Lmax, double inv, double scale)
{
    for (int v = 0; v < kSlots; ++v) {
        if (4 * T * v >= d) break;
        double o[4];
        r4(v, o);
#pragma unroll
        for (int c = 0; c < 4; ++c) bin_lattice_elem(fabs(o[c]), S, G, M, Lmax, inv, scale);
    }
}

// In-place inclusive suffix sums of h[0, n) by the whole workgroup: thread t
// owns the t-th chunk from the top, so a prefix over threads is a suffix over
// buckets.  An odd chunk length keeps the lanes of a wavefront on distinct
// LDS banks.  scan holds one value per wavefront.  Ends with a barrier.
template <int T>
__device__ __forceinline__ void block_suffix_sums(unsigned long long *h, int n,
                                                  unsigned long long *scan)
{
    constexpr int kWaves = T / kWave;
    constexpr int kPerMax = ((kLatMaxBuckets + T - 1) / T) | 1;
    const int t = threadIdx.x;
    const int per = ((n + T - 1) / T) | 1;  // n <= kLatMaxBuckets
    const int top = n - t * per;            // exclusive upper end of the chunk
    const int bot = max(top - per, 0);
    unsigned long long v = 0;
#pragma unroll 4
    for (int z = 0; z < kPerMax; ++z) {
        const int i = top - 1 - z;
        v += i >= bot ? h[max(i, 0)] : 0ull;
    }
    const unsigned long long incl = wave_prefix_sum(v);
    const int wid = t / kWave;
    if ((t % kWave) == kWave - 1) scan[wid] = incl;
    __syncthreads();
    unsigned long long run = incl - v;
#pragma unroll
    for (int w = 0; w < kWaves - 1; ++w) run += w < wid ? scan[w] : 0ull;
#pragma unroll 4
    for (int z = 0; z < kPerMax; ++z) {
        const int i = top - 1 - z;
        if (i >= bot) {
            run += h[i];
            h[i] = run;
        }
    }
    __syncthreads();
}

// Wavefronts per SIMD the register budget aims at.  The search is VALU
// bound, so more wavefronts hide its LDS and barrier waits: seven (72 VGPRs)
// for two elements per thread or fewer and six (80) for four, in the
// per-level modes; five (96) for the 256-thread lattice variants of up to
// eight elements; four (128) for the others, unless the residual alone
// needs more (EPT = 32: two); a workgroup of 1024 threads needs four per
// SIMD.
template <int T, int EPT, bool kLat, bool kGlobal>
constexpr int hist_waves_per_simd()
{
    if (EPT >= 32 && !kGlobal && T <= 512) return 2;
    if (kLat && !kGlobal && T <= 256 && EPT <= 8) return 5;
    if (kLat || kGlobal || EPT > 4) return 4;
    return EPT == 4 ? 6 : 7;
}

// kGlobal: the residual is not held in registers; each phase rebuilds
// element j as fl64 w_j - sum_{p<i} a_p q_pj from the weights, the codes this
// workgroup already wrote and the scales kept in LDS, with the same fp64
// operations in the same order as the register variants (so bitwise the same
// value), for channels longer than the registers of a workgroup hold.
template <int T, int EPT, bool kLinear, bool kLat, bool kGlobal>
__global__ void __launch_bounds__(T)
__attribute__((amdgpu_waves_per_eu(hist_waves_per_simd<T, EPT, kLat, kGlobal>())))
fit_hist_kernel(const HistBatch B)
{
    constexpr int kWaves = T / kWave;
    constexpr int kUnroll = kGlobal ? 1 : EPT;   // the rebuilt residual is not an array
    extern __shared__ __align__(16) double hsmem[];
    __shared__ float s_redf[kWaves];
    __shared__ double s_redd[kWaves];
    __shared__ double s_redd2[kWaves];
    __shared__ int s_fin[kMaxFinalists];
    __shared__ int s_nfin;
    __shared__ int s_gbest;
    __shared__ int s_other;   // lattice mode: a candidate besides the best may be a finalist
    __shared__ unsigned long long s_scan[kWaves];
    __shared__ ArgMin s_arg[kWaves];
    __shared__ float s_scale[MPQ_MAX_POINTS];

    // layer of this workgroup (uniform: the descriptors are kernel arguments)
    const int li = last_at_most(B.n_layers, (int)blockIdx.x, [&](int i) { return B.L[i].c_begin; });
    const HistLayer &Ly = B.L[li];

    const int G = B.G;
    HistShared S;
    S.ha = (long long *)hsmem;
    S.lat = (unsigned long long *)(S.ha + G);
    const int nlat = kLat ? B.nlat : 0;
    S.af = (float *)(S.lat + nlat);
    S.hb = (int *)(S.af + G + 2);

    const int64_t k = (int64_t)blockIdx.x - Ly.c_begin;
    const int t = threadIdx.x;
    const int d = Ly.d;              // <= kHistMaxDim; per-channel offsets fit 32 bits
    const int P = B.P;
    const int M = B.M;
    const double Md = (double)M;
    int8_t *qk = Ly.codes + k * (int64_t)P * d;
    const float *wk = Ly.W + k * (int64_t)d;

    // resume a channel that holds s0 points and has not stopped (its count
    // is s0) from its stored points; in a calibration step take at most one
    const bool stepping = B.single != 0;
    const int s0 = B.start;
    if (s0 >= 1 && Ly.counts[k] != s0) return;   // uniform: one value per workgroup
    if (s0 >= 1) {
        for (int p = t; p < s0; p += T) s_scale[p] = Ly.scales[k * P + p];
        __syncthreads();
    }

    // asymmetric codes (reading B2): the points fit w - beta, beta the fp32
    // midpoint of the channel's range; the stopping rule keeps ||w||^2
    double beta = 0.0;
    double Ew = 0.0;
    const bool asym = Ly.offsets != nullptr;
    if (asym) {
        float mx = -INFINITY, mn = INFINITY;
        for (int j = t; j < d; j += T) {
            mx = fmaxf(mx, wk[j]);
            mn = fminf(mn, wk[j]);
        }
        mx = block_reduce<T>(mx, MaxOp(), s_redf);
        mn = block_reduce<T>(mn, MinOp(), s_redf);
        const float b = (float)(((double)mx + (double)mn) / 2.0);
        beta = (double)b;
        if (t == 0) Ly.offsets[k] = b;
    }
    if (asym || (s0 >= 1 && !stepping)) {   // ||w||^2 when the first residual is not w
        double sw = 0.0;
        for (int j = t; j < d; j += T) sw = fma((double)wk[j], (double)wk[j], sw);
        Ew = block_reduce<T>(sw, SumOp(), s_redd);
    }

    // residual element u of this thread after np points (0 past the channel)
    auto rebuild = [&](int u, int np) {
        const int j = t + T * u;
        if (j >= d) return 0.0;
        double v = (double)wk[j] - beta;
        for (int p = 0; p < np; ++p) v = fma(-(double)s_scale[p], (double)qk[(int64_t)p * d + j], v);
        return v;
    };
    // kGlobal: thread t owns slots of four consecutive elements, slot v
    // holding j = 4 (t + T v) + c (c < 4), so that a slot's weights load as
    // one float4 and each stored point's codes as one 32-bit word (rows of a
    // multiple of 4 bytes; otherwise one element at a time).  Each element is
    // rebuilt with the fp64 operations of rebuild, in point order.
    constexpr int kSlots = kGlobal ? (EPT + 3) / 4 : 1;
    const bool vec4 = kGlobal && d % 4 == 0 && (uintptr_t)wk % 16 == 0 && (uintptr_t)qk % 4 == 0;
    auto rebuild4 = [&](int v, int np, double (&o)[4]) {
        const int j0 = 4 * (t + T * v);
        if (vec4 && j0 + 4 <= d) {
            const float4 w4 = *(const float4 *)(wk + j0);
            o[0] = (double)w4.x - beta;
            o[1] = (double)w4.y - beta;
            o[2] = (double)w4.z - beta;
            o[3] = (double)w4.w - beta;
            for (int p = 0; p < np; ++p) {
                const uint32_t q = *(const uint32_t *)(qk + (int64_t)p * d + j0);
                const double a = -(double)s_scale[p];
#pragma unroll
                for (int c = 0; c < 4; ++c) o[c] = fma(a, (double)(int)(int8_t)(uint8_t)(q >> (8 * c)), o[c]);
            }
        } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int j = j0 + c;
                double v = 0.0;
                if (j < d) {
                    v = (double)wk[j] - beta;
                    for (int p = 0; p < np; ++p) v = fma(-(double)s_scale[p], (double)qk[(int64_t)p * d + j], v);
                }
                o[c] = v;
            }
        }
    };
    // stores the four codes of slot v (bytes past d are not stored)
    auto store4 = [&](int8_t *row, int v, uint32_t q) {
        const int j0 = 4 * (t + T * v);
        if (vec4 && j0 + 4 <= d) {
            *(uint32_t *)(row + j0) = q;
        } else {
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if (j0 + c < d) row[j0 + c] = (int8_t)(uint8_t)(q >> (8 * c));
        }
    };
    double r[kGlobal ? 1 : EPT];
    // The channel's row of the output error's D, outside calibration steps:
    // the residual after the points so far in fp32 (the same fp64 steps, in
    // the same order, as forming it from the stored points; zero past d, up
    // to nkb * 32 <= T * EPT).  D holds tiles of 128 rows by 32 k, row-major
    // inside: element j of row k is float ((k / 128) nkb + j / 32) 4096 +
    // (k % 128) 32 + j % 32.  Element j = t + T u lies in 32-k chunk
    // t / 32 + u T / 32 at place t % 32; a lane stores only while that chunk
    // is one of the row's nkb, so every store stays inside the row (the
    // chunk's elements past d store the zero residual of j >= d).  The
    // buffer resource spans the row as a second guard.
    static_assert(T % 32 == 0, "a thread's elements keep their place in a 32-k chunk");
    const int nkb = (d + 31) / 32;
    const bool has_d = !kGlobal && Ly.dres && !stepping;
    const __amdgpu_buffer_rsrc_t rs_d = __builtin_amdgcn_make_buffer_rsrc(
        has_d ? (void *)(Ly.dres + (k / 128) * nkb * 4096 + (k % 128) * 32) : nullptr, (short)0,
        has_d ? (nkb * 4096 - (int)(k % 128) * 32) * 4 : 0, 0x00020000);
    const int d_chunk = t / 32;                          // chunk of element t (u = 0)
    const int d_voff = (d_chunk * 4096 + t % 32) * 4;   // element t; + u (T / 32) 4096 floats
    if constexpr (!kGlobal) {
#pragma unroll
        for (int u = 0; u < EPT; ++u) r[u] = rebuild(u, s0);
    }

    // the grid multiplier c_g: the caller's, or the default fl32((g + 1) / G),
    // the correctly rounded fp32 quotient of the two integers (which equals
    // fl32 of the fp64 one for every g < G <= 4096, checked exhaustively on
    // the host); for G = 2^k that is (g + 1) 2^-k exactly
    const bool pow2 = (G & (G - 1)) == 0;
    const float invG = __fdiv_rn(1.0f, (float)G);
    auto mult = [&](int g) {
        return B.grid ? B.grid[g] : pow2 ? (float)(g + 1) * invG : __fdiv_rn((float)(g + 1), (float)G);
    };

    float apend = 0.0f;
    int n = 0;
    bool more = false;   // calibration step: the channel took its point and goes on
    // Algorithm 2's naive point (reading F1).  Calibration fit, first step:
    // the point is stored with its output error; the channel keeps it (and
    // takes no other) when that error meets the threshold.  Fresh fit:
    // gstate 1 takes the naive point at step 0, gstate 2 decides at step 1,
    // after it is applied, whether it stays or the fit restarts from w.
    bool kept = false;
    if (B.gate && stepping && s0 == 0) {
        const double thr = Ly.ref ? B.eps * (double)Ly.ref[k] : B.eps;
        kept = Ly.counts[k] == 1 && (double)Ly.xerr[k * P] <= thr;   // uniform
        if (kept) n = 1;
    }
    int gstate = (B.gate && !stepping && s0 == 0) ? 1 : 0;
    for (int i = s0; !kept; ++i) {
        // ---- apply the pending point: codes of Eq. (10), residual of Eq. (7)
        float lmax = 0.0f;
        double lsum = 0.0;
        int8_t *qrow = qk + (int64_t)(i - 1) * d;
        // code of Eq. (10) at the searched scale (fp32 first, fp64 near a
        // half-integer)
        const PointCode code_of(apend, M);
        const double ap = code_of.ap;
        // the scale the residual update uses: the searched one, or (refit)
        // the least-squares scale of the codes, fl32(<r, q> / <q, q>)
        double aupd = ap;
        if (B.refit && i > s0 && gstate != 2) {   // the naive point keeps its scale
            double rq = 0.0, qq = 0.0;
            if constexpr (kGlobal) {
                for (int v = 0; v < kSlots; ++v) {
                    if (4 * T * v >= d) break;
                    const int j0 = 4 * (t + T * v);
                    double o[4];
                    rebuild4(v, i - 1, o);
                    uint32_t qw = 0;
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        if (j0 + c < d) {
                            const double cd = code_of(o[c]);
                            qw |= (uint32_t)(uint8_t)(int8_t)(int)cd << (8 * c);
                            rq = fma(o[c], cd, rq);
                            qq = fma(cd, cd, qq);
                        }
                    }
                    store4(qrow, v, qw);
                }
            } else {
#pragma unroll
                for (int u = 0; u < EPT; ++u) {
                    const int j = t + T * u;
                    if (j < d) {
                        const double ru = r[u];
                        const double c = code_of(ru);
                        qrow[j] = (int8_t)(int)c;
                        rq = fma(ru, c, rq);
                        qq = fma(c, c, qq);
                    }
                }
            }
            block_sum2<T>(rq, qq, s_redd, s_redd2);
            const float afit = (float)(rq / qq);
            if (t == 0) {
                Ly.scales[k * P + (i - 1)] = afit;
                s_scale[i - 1] = afit;   // read only after the next barrier
            }
            aupd = (double)afit;
        }
        if constexpr (kGlobal) {
            const bool codes_here = i > s0 && (!B.refit || gstate == 2);
            for (int v = 0; v < kSlots; ++v) {
                if (4 * T * v >= d) break;
                const int j0 = 4 * (t + T * v);
                double o[4];
                rebuild4(v, i > s0 ? i - 1 : i, o);
                uint32_t qw = 0;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    double ru = o[c];
                    if (i > s0 && j0 + c < d) {
                        const double cd = code_of(ru);
                        qw |= (uint32_t)(uint8_t)(int8_t)(int)cd << (8 * c);
                        ru = fma(-aupd, cd, ru);
                    }
                    lmax = fmaxf(lmax, fabsf((float)ru));
                    lsum = fma(ru, ru, lsum);
                }
                if (codes_here) store4(qrow, v, qw);
            }
        } else {
#pragma unroll
            for (int u = 0; u < EPT; ++u) {
                const int j = t + T * u;
                double ru = r[u];
                if (i > s0 && j < d) {
                    const double c = code_of(ru);
                    if (!B.refit || gstate == 2) qrow[j] = (int8_t)(int)c;
                    ru = fma(-aupd, c, ru);
                }
                r[u] = ru;
                // rewritten each step: the last write holds the n points
                if (has_d && d_chunk + u * (T / 32) < nkb)
                    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint((float)ru), rs_d,
                                                          d_voff + u * (T / 32) * 4096 * 4, 0, 0);
                lmax = fmaxf(lmax, fabsf((float)ru));
                lsum = fma(ru, ru, lsum);
            }
        }
        // no trailing barrier: the scratch is next written after the setup
        // barrier below
        block_max_sum<T, false>(lmax, lsum, s_redf, s_redd);
        const float m = lmax;
        const double Er = lsum;

        // ---- stop / point count
        if (i == 0 && !asym) Ew = Er;
        else if (i > s0 && Ly.err && t == 0) Ly.err[k * P + (i - 1)] = (float)Er;
        if (stepping && i > s0) {   // one point per calibration step
            n = i;
            more = true;
            break;
        }
        bool stop = (i >= P) || (Er == 0.0);
        if (!stop && i >= 1) {
            if (stepping) {
                // output error of the i points on the batch (the error pass
                // of the previous step) against the threshold
                const double thr = Ly.ref ? B.eps * (double)Ly.ref[k] : B.eps;
                stop = (double)Ly.xerr[k * P + (i - 1)] <= thr;
            } else {
                stop = Er <= B.tol * Ew;
            }
        }
        if (gstate == 2) {   // step 1 of a gated fit: the naive point is applied
            gstate = 0;
            if (Er <= B.tol * Ew) {   // Algorithm 2's test: the only point
                n = 1;
                break;
            }
            // discarded: restart from w (its codes, scale and err are
            // rewritten by the point that replaces it)
            if constexpr (!kGlobal) {
#pragma unroll
                for (int u = 0; u < EPT; ++u) r[u] = rebuild(u, 0);
            }
            i = -1;
            __syncthreads();   // the next step's reduction rewrites s_redf, s_redd
            continue;
        }
        if (stop) {
            n = i;
            break;
        }
        if (gstate == 1) {   // step 0 of a gated fit: the naive point first
            gstate = 0;
            const float aN = (float)((double)m / Md);   // the candidate c = 1
            if (aN != 0.0f) {
                gstate = 2;
                apend = aN;
                if (t == 0) {
                    Ly.scales[k * P] = aN;
                    s_scale[0] = aN;
                }
                __syncthreads();   // s_scale (rebuilt residual); s_redf, s_redd
                continue;
            }
        }

        // ---- candidates, cleared histograms
        for (int g = t; g < G; g += T) {
            const float a = (float)((double)m * (double)mult(g) / Md);
            S.af[g + 1] = a;
            S.ha[g] = 0;
            S.hb[g] = 0;
        }
        // lattice mode needs normal candidates (relative error 2^-23)
        const bool lat = kLat && m >= 0x1p-100f;
        if (lat)
            for (int b = t; b < nlat; b += T) S.lat[b] = 0;
        if (t == 0) {
            s_other = 0;
            S.af[0] = 0.0f;
            S.af[G + 1] = INFINITY;
        }
        // fixed-point shift: every x < 2^(ex+1); sums of up to M*d values
        // < 2^62, or in lattice mode sums of d values < 2^kLatShift
        int ex = 0;
        (void)frexpf(m, &ex);
        const long long span = lat ? (long long)d : (long long)M * d;   // >= 1
        const int lg = span <= 1 ? 0 : 64 - __clzll(span - 1);          // ceil(log2(span))
        const int sh = (lat ? kLatShift : 61) - (ex + 1) - lg;
        __syncthreads();

        const double q2 = ldexp(1.0, -sh);
        const double slack = Md * (double)d * q2;   // fixed-point error of A, per unit a
        int be = 0;                                  // ||r||^2 < 2^be: the unit of stored bounds
        (void)frexp(Er, &be);
        ArgMin best{INFINITY, 0x7fffffff};
        if (lat) {
            // ---- lattice buckets, their suffix sums, then every candidate
            const double inv = (double)(2 * G * M) / (double)m;
            // residual after the i points so far (kGlobal: rebuilt)
            if constexpr (kGlobal) {
                auto res4 = [&](int v, double (&o)[4]) { rebuild4(v, i, o); };
                bin_lattice_slots<T, kSlots>(res4, S, G, M, d, nlat - 1, inv, ldexp(1.0, sh));
            } else {
                auto res = [&](int u) { return r[kGlobal ? 0 : u]; };
                bin_lattice<T, EPT, kUnroll>(res, S, G, M, d, nlat - 1, inv, ldexp(1.0, sh));
            }
            __syncthreads();
            block_suffix_sums<T>(S.lat, nlat, s_scan);
            for (int g = t; g < G; g += T) {
                unsigned long long A = (unsigned long long)S.ha[g];
                uint32_t Bc = (uint32_t)S.hb[g];
                for (int k0 = 0; k0 < M; k0 += 8) {
                    // eight independent reads in flight; lanes past M read
                    // bucket 0 and drop it
                    unsigned long long v[8];
#pragma unroll
                    for (int z = 0; z < 8; ++z) {
                        const int kk = k0 + z;
                        v[z] = S.lat[kk < M ? (2 * kk + 1) * (g + 1) : 0];
                    }
#pragma unroll
                    for (int z = 0; z < 8; ++z) {
                        const int kk = k0 + z;
                        if (kk < M) {
                            A += v[z] & kLatMask;
                            Bc += (uint32_t)(2 * kk + 1) * (uint32_t)(v[z] >> kLatShift);
                        }
                    }
                }
                const double a = (double)S.af[g + 1];
                double e = INFINITY, b = 0.0;
                if (a != 0.0) {
                    const double Ad = ldexp((double)A, -sh);
                    const double t2 = 2.0 * a * Ad, t3 = a * a * (double)Bc;
                    e = (Er - t2) + t3;
                    b = a * slack + 8.0 * 0x1p-53 * (Er + t2 + t3);
                }
                S.put_err(g, e, b, be);
                if (e < best.e || (e == best.e && g < best.g)) best = ArgMin{e, g};
            }
            // its barrier publishes the errors and bounds; s_arg is next written a step later
            best = block_argmin<T, false>(best, s_arg);
            // another candidate whose interval reaches the best one's (rare)
            // is flagged by its own thread, so that in the common case no
            // wavefront scans the candidates again
            const double thr0 = best.e == INFINITY ? INFINITY : best.e + S.bnd(best.g, be);
            bool other = false;
            for (int g = t; g < G; g += T)
                other = other || (g != best.g && S.err(g) != INFINITY && S.err(g) - S.bnd(g, be) <= thr0);
            if (other) s_other = 1;
            __syncthreads();
        } else {
            // ---- histograms of the level boundaries (bin_levels)
            unsigned long long fullA = 0;
            int fullB = 0;
            // the closed-form counts need normal candidates and a finite
            // estimate (in a lattice-mode kernel this branch only runs when
            // they do not)
            if constexpr (kGlobal) {
                auto res4 = [&](int v, double (&o)[4]) { rebuild4(v, i, o); };
                if (kLinear && !kLat && m >= 0x1p-100f)
                    bin_levels_slots<T, kSlots, true>(res4, S, G, M, d, m, sh, fullA, fullB);
                else
                    bin_levels_slots<T, kSlots, false>(res4, S, G, M, d, m, sh, fullA, fullB);
            } else if (kLinear && !kLat && m >= 0x1p-100f) {
                bin_levels<T, EPT, true>(r, S, G, M, m, sh, fullA, fullB);
            } else {
                bin_levels<T, EPT, false>(r, S, G, M, m, sh, fullA, fullB);
            }
#pragma unroll
            for (int off = 1; off < kWave; off <<= 1) {
                fullA += (unsigned long long)__shfl_xor((long long)fullA, off);
                fullB += __shfl_xor(fullB, off);
            }
            if ((t % kWave) == 0) {
                atomicAdd((unsigned long long *)&S.ha[G - 1], fullA);
                atomicAdd(&S.hb[G - 1], fullB);
            }
            __syncthreads();
        }

        // ---- wavefront 0: (histogram mode) suffix sums, candidate errors and
        // bounds, argmin; then the finalists (lattice mode: only when flagged)
        const bool pick = !lat || s_other != 0;   // uniform
        if (pick && t < kWave) {
            // lane l owns the l-th chunk from the top, so a prefix over lanes
            // is a suffix over candidates
            const int per = (G + kWave - 1) / kWave;
            const int g0 = (kWave - 1 - t) * per, g1 = min(g0 + per, G);
            if (!lat) {
            unsigned long long la = 0;
            uint32_t lb = 0;
            for (int g = g0; g < g1; ++g) {
                la += (unsigned long long)S.ha[g];
                lb += (uint32_t)S.hb[g];
            }
            long long A = (long long)(wave_prefix_sum(la) - la);   // exclusive
            int B = (int)(wave_prefix_sum(lb) - lb);
            for (int g = g1 - 1; g >= g0; --g) {
                A += S.ha[g];
                B += S.hb[g];
                const double a = (double)S.af[g + 1];
                double e = INFINITY, b = 0.0;
                if (a != 0.0) {
                    const double Ad = ldexp((double)A, -sh);
                    const double t2 = 2.0 * a * Ad, t3 = a * a * (double)B;
                    e = (Er - t2) + t3;
                    b = a * slack + 8.0 * 0x1p-53 * (Er + t2 + t3);
                }
                S.put_err(g, e, b, be);
                if (e < best.e || (e == best.e && g < best.g)) best = ArgMin{e, g};
            }
            best = wave_argmin(best);
            }
            // finalists: candidates whose interval reaches the best one's
            const double thr = best.e == INFINITY ? INFINITY : best.e + S.bnd(best.g, be);
            int cnt = 0;
            for (int g = g0; g < g1; ++g)
                if (S.err(g) != INFINITY && S.err(g) - S.bnd(g, be) <= thr) ++cnt;
            cnt = wave_reduce(cnt, SumOp());
            if (t == 0) {
                s_gbest = best.e == INFINITY ? -1 : best.g;
                s_nfin = cnt;
            }
            if (cnt > 1) {
                // up to kMaxFinalists, smallest (E, g) first
                int nf = 0;
                double last_e = -INFINITY;
                int last_g = -1;
                for (; nf < kMaxFinalists && nf < cnt; ++nf) {
                    ArgMin c{INFINITY, 0x7fffffff};
                    for (int g = g0; g < g1; ++g) {
                        const double e = S.err(g);
                        if (e == INFINITY || e - S.bnd(g, be) > thr) continue;
                        const bool after = e > last_e || (e == last_e && g > last_g);
                        if (after && (e < c.e || (e == c.e && g < c.g))) c = ArgMin{e, g};
                    }
                    c = wave_argmin(c);
                    if (t == 0) s_fin[nf] = c.g;
                    last_e = c.e;
                    last_g = c.g;
                }
                if (t == 0) s_nfin = nf;
            }
        }
        if (pick) __syncthreads();

        int gstar = pick ? s_gbest : (best.e == INFINITY ? -1 : best.g);
        const int nfin = pick ? s_nfin : 1;
        if (gstar >= 0 && nfin > 1) {
            // direct fp64 evaluation of the finalists (Eq. (9) written out)
            ArgMin best{INFINITY, 0x7fffffff};
            for (int f = 0; f < nfin; ++f) {
                const int g = s_fin[f];
                const double a = (double)S.af[g + 1];
                double le = 0.0;
                // signed form: (r - a q)^2 with q = clip(rne(r / a)) equals
                // (|r| - a |q|)^2, and keeps |r| from being hoisted per element
                auto err_of = [&](double ru) {
                    const double c = fmin(fmax(rint(ru / a), -Md), Md);
                    const double e = ru - a * c;
                    le = fma(e, e, le);
                };
                if constexpr (kGlobal) {
                    for (int v = 0; v < kSlots; ++v) {
                        if (4 * T * v >= d) break;
                        double o[4];
                        rebuild4(v, i, o);
#pragma unroll
                        for (int c = 0; c < 4; ++c) err_of(o[c]);   // 0 past d adds 0
                    }
                } else {
#pragma unroll
                    for (int u = 0; u < EPT; ++u) err_of(r[kGlobal ? 0 : u]);
                }
                const double E = block_reduce<T>(le, SumOp(), s_redd);
                if (E < best.e || (E == best.e && g < best.g)) best = ArgMin{E, g};
            }
            gstar = best.g;
        }
        if (gstar < 0) {   // every candidate scale is zero
            n = i;
            break;
        }
        apend = S.af[gstar + 1];
        if (t == 0) {
            Ly.scales[k * P + i] = apend;
            s_scale[i] = apend;
        }
        // the next step rewrites S.af only after its first barrier; this one
        // is needed when the finalists' reductions used s_redd, which the next
        // step's first reduction writes, or when the rebuilt residual reads
        // s_scale[i]
        if (kGlobal || nfin > 1) __syncthreads();
    }

    if constexpr (kGlobal) {
        // the channel's row of the output error's D, outside calibration
        // steps: the residual after its n points in fp32 (rebuild4's fp64
        // steps in point order, as forming it from the stored points does),
        // zero past d; the slots cover the row's nkb 32-k chunks, four
        // consecutive k each (one float4 of a chunk; each thread reads back
        // only the codes it wrote)
        if (Ly.dres && !stepping) {
            float *drow = Ly.dres + (k / 128) * nkb * 4096 + (k % 128) * 32;
            for (int v = 0; v < kSlots; ++v) {
                if (4 * T * v >= d) break;
                const int j0 = 4 * (t + T * v);
                if (j0 >= nkb * 32) continue;
                double o[4];
                rebuild4(v, n, o);
                *(float4 *)(drow + (j0 / 32) * 4096 + j0 % 32) =
                    make_float4((float)o[0], (float)o[1], (float)o[2], (float)o[3]);
            }
        }
    }
    if (t == 0) Ly.counts[k] = n;
    if (more) {
        if (t == 0) Ly.list[atomicAdd(Ly.nlist + s0, 1)] = (int32_t)k;
        return;
    }
    for (int q = n + t; q < P; q += T) {
        Ly.scales[k * P + q] = 0.0f;
        if (Ly.err) Ly.err[k * P + q] = 0.0f;
        if (Ly.xerr) Ly.xerr[k * P + q] = 0.0f;
    }
    // code rows n .. P - 1: one contiguous byte range, in 16-byte stores
    // between its unaligned head and tail
    int8_t *z0 = qk + (int64_t)n * d, *z1 = qk + (int64_t)P * d;
    int8_t *a0 = (int8_t *)(((uintptr_t)z0 + 15) & ~(uintptr_t)15);
    int8_t *a1 = (int8_t *)((uintptr_t)z1 & ~(uintptr_t)15);
    if (a0 >= a1) {
        for (int8_t *p = z0 + t; p < z1; p += T) *p = 0;
    } else {
        if (z0 + t < a0) z0[t] = 0;   // head < 16 <= T bytes
        if (a1 + t < z1) a1[t] = 0;   // tail < 16 bytes
        for (int64_t v = t; v < (a1 - a0) / 16; v += T) ((uint4 *)a0)[v] = make_uint4(0, 0, 0, 0);
    }
}

template <int T, int EPT, bool kGlobal = false>
hipError_t launch_hist_t(const HistBatch &b, int64_t channels, size_t lds, hipStream_t s)
{
    // the default grid (grid == nullptr) has the closed-form boundary counts
    // and, when its buckets fit, the lattice mode
    auto kern = b.grid ? fit_hist_kernel<T, EPT, false, false, kGlobal>
                : b.nlat ? fit_hist_kernel<T, EPT, true, true, kGlobal>
                         : fit_hist_kernel<T, EPT, true, false, kGlobal>;
    if (lds > 65536) {
        hipError_t e = hipFuncSetAttribute((const void *)kern,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    char name[64];
    snprintf(name, sizeof name, "fit_hist_kernel<%d,%d,%s%s>", T, EPT,
             b.grid ? "grid" : b.nlat ? "lattice" : "linear", kGlobal ? ",rebuilt" : "");
    LaunchTimer timer(s, name);
    hipLaunchKernelGGL(kern, dim3((unsigned)channels), dim3(T), lds, s, b);
    return hipGetLastError();
}

// (threads, elements per thread) of each variant; variant v takes the
// channels longer than the capacity T * EPT of variant v - 1, up to its own.
// 256-thread variants let four channels share a CU (128 VGPRs, under 40 KB of
// LDS each), so one channel's barriers and serial phases overlap another's
// arithmetic (256 x 9 takes d = 2304, the 3 x 3 kernels over 256 input
// channels, which a 512-thread workgroup would run half idle, two per CU);
// the 512- and 1024-thread variants cover lengths whose residual
// would not fit 128 VGPRs at 256 threads without spilling to scratch (at
// 256 x 18 the spills moved ~7x the channel's algorithmic bytes through HBM).
// The last variant (1024 x 32, up to 32768) holds no residual copy: it
// rebuilds each element from the weights and the codes (kGlobal).
struct Variant {
    int threads, ept;
    bool rebuilt;
};
constexpr Variant kVariants[] = {{64, 1, false},   {64, 2, false},   {64, 4, false},
                                 {256, 2, false},  {256, 4, false},  {256, 8, false},
                                 {256, 9, false},  {512, 9, false},  {1024, 8, false},
                                 {512, 32, false}, {1024, 32, true}};
constexpr int kNumVariants = sizeof(kVariants) / sizeof(kVariants[0]);
static_assert(kVariants[kNumVariants - 1].threads * kVariants[kNumVariants - 1].ept == kHistMaxDim,
              "the last variant covers the longest channels");
// variants whose capacity reaches this length use the lattice mode (at 4
// bits and 256 candidates on ResNet-50's layers it beat the per-level
// histograms on lengths 576-1024, 165 against 197 us, and lost on 512 and
// below: its O((2M - 1) G) bucket pass per step outweighs M atomics per
// element there)
constexpr int kLatMinDim = 1024;

}  // namespace

size_t fit_hist_lds(int G)
{
    return (size_t)G * (sizeof(long long) + 2 * sizeof(float)) + 2 * sizeof(float);
}

bool fit_hist_supports(int64_t d) { return d >= 1 && d <= kHistMaxDim; }

// the short-channel variants (fit_small.hip), one per length 1 ..
// kSmallMaxDim, follow the histogram ones
constexpr int kSmallVariant = kNumVariants;

bool hist_variant_writes_d(int v)
{
    return (v >= kSmallVariant && v < kSmallVariant + kSmallMaxDim) || (v >= 0 && v < kNumVariants);
}

int hist_variant_count() { return kNumVariants + (int)kSmallMaxDim; }

int hist_variant(int64_t d)
{
    if (d >= 1 && d <= kSmallMaxDim) return kSmallVariant + (int)d - 1;
    int v = 0;
    while (v + 1 < kNumVariants && d > (int64_t)kVariants[v].threads * kVariants[v].ept) ++v;
    return v;
}

namespace {

// lattice mode: default grid, longer channels (the bucket pass costs O(nlat)
// per step), buckets within kLatMaxBuckets and 64 KiB of LDS
int lattice_buckets(int variant, int M, int G, bool default_grid)
{
    const int64_t nlat = (int64_t)(2 * M - 1) * G + 1;
    return (default_grid && kVariants[variant].threads * kVariants[variant].ept >= kLatMinDim &&
            nlat <= kLatMaxBuckets &&
            fit_hist_lds(G) + (size_t)nlat * sizeof(unsigned long long) <= 65536)
               ? (int)nlat
               : 0;
}

}  // namespace

std::string hist_kernel_name(int64_t d, int M, int G, bool default_grid)
{
    const int v = hist_variant(d);
    if (v >= kSmallVariant) return fit_small_name((int)d);
    char name[64];
    snprintf(name, sizeof name, "fit_hist_kernel<%d,%d,%s%s>", kVariants[v].threads, kVariants[v].ept,
             !default_grid ? "grid" : lattice_buckets(v, M, G, true) ? "lattice" : "linear",
             kVariants[v].rebuilt ? ",rebuilt" : "");
    return name;
}

namespace {
__global__ void zero_i32_kernel(int32_t *p, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}
}  // namespace

hipError_t launch_zero_i32(int32_t *p, int64_t n, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    if (n > (int64_t)256 * 0x7fffffff) return hipErrorInvalidValue;
    LaunchTimer timer(s, "zero_i32_kernel");
    hipLaunchKernelGGL(zero_i32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, n);
    return hipGetLastError();
}

hipError_t launch_fit_hist(const HistBatch &batch, int variant, int64_t channels, hipStream_t s)
{
    HistBatch b = batch;
    if (variant >= kSmallVariant && variant < kSmallVariant + kSmallMaxDim)
        return launch_fit_small(b, variant - kSmallVariant + 1, channels, s);
    if (variant < 0 || variant >= kNumVariants) return hipErrorInvalidValue;
    b.nlat = lattice_buckets(variant, b.M, b.G, !b.grid);
    const size_t lds = fit_hist_lds(b.G) + (size_t)b.nlat * sizeof(unsigned long long);
    switch (variant) {
    case 0: return launch_hist_t<64, 1>(b, channels, lds, s);
    case 1: return launch_hist_t<64, 2>(b, channels, lds, s);
    case 2: return launch_hist_t<64, 4>(b, channels, lds, s);
    case 3: return launch_hist_t<256, 2>(b, channels, lds, s);
    case 4: return launch_hist_t<256, 4>(b, channels, lds, s);
    case 5: return launch_hist_t<256, 8>(b, channels, lds, s);
    case 6: return launch_hist_t<256, 9>(b, channels, lds, s);
    case 7: return launch_hist_t<512, 9>(b, channels, lds, s);
    case 8: return launch_hist_t<1024, 8>(b, channels, lds, s);
    // 512 threads leave 256 VGPRs per thread for the register-resident residual
    case 9: return launch_hist_t<512, 32>(b, channels, lds, s);
    case 10: return launch_hist_t<1024, 32, true>(b, channels, lds, s);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace mpq
