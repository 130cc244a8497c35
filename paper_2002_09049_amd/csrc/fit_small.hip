// Greedy multipoint fit (Algorithm 1, Sec. 3.2, with the stopping rule of
// Algorithm 2, Sec. 3.3) for short channels, d <= kSmallMaxDim (the 3 x 3
// depthwise filters have d = 9): one wavefront per channel, its lanes over
// the candidates, several channels per workgroup.
//
// Every lane holds the channel's whole fp64 residual (the same d values in
// each lane), so the point's codes (Eq. (10)), the residual update (Eq. (7)),
// max|r| and ||r||^2 need no exchange between lanes.  Lane l evaluates the
// candidates g = l, l + 64, ... directly (Eq. (9)):
//     E(g) = sum_j (|r_j| - a_g n_j)^2,  n_j = min(M, rint(|r_j| / a_g)),
// the value of (r_j - a_g clip(rint(r_j / a_g)))^2 term by term (rint is odd),
// summed in fp64 over j in order, and a DPP argmin over the wavefront takes
// the smallest (E, g).  After the workgroup's first barrier a wavefront
// synchronizes with nothing, and apart from the grid multipliers it holds
// no LDS, so a CU keeps many channels in flight (the histogram search's
// per-channel LDS would allow a handful).
//
// The codes n_j of the search come from fp32 first: y32 = fl32(|r_j|) v with
// v = rcp(fl32 a) (v_rcp_f32, within 1 ulp of 1 / a for 2^-100 <= a <=
// 2^100), so y32 is within |y| (2^-24 + 2^-23 + 2^-24)(1 + 2^-22) < |y|
// 2^-21.99 of y = |r_j| / a.  Below y = M + 1 that is under
// delta = (M + 2) 2^-21, so a y32 farther than delta from every half-integer
// rounds as y does; above, both clip to M.  A candidate with an element
// nearer than delta (or a scale outside that range) is evaluated again with
// the fp64 quotient's codes, as the point's codes are formed.
#include <math.h>
#include <stdio.h>

#include "internal.hpp"
#include "mpq.h"
#include "point_code.hpp"
#include "reduce.hpp"

namespace mpq {

namespace {

constexpr int kSmallWaves = 4;   // channels (wavefronts) per workgroup

// A value every lane of the wavefront holds alike, moved to scalar registers
// (the residual: VALU instructions read it as their one scalar operand, so
// it takes no vector registers).
__device__ __forceinline__ double uniform(double v)
{
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)u);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(u >> 32));
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

__device__ __forceinline__ float uniform(float v)
{
    return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}

// The best (E, g) of lane's candidates g = lane, lane + 64, ... for the
// residual r of kN elements (x32 = fl32|r|), by Eq. (9) written out.
template <int kN, int kD>
__device__ __forceinline__ ArgMin lane_candidates(const double (&r)[kD], const float (&x32)[kD],
                                                  const float *s_c, int G, int lane, double mdd, int M)
{
    const double Md = (double)M;
    const float Mf = (float)M;
    const float lim = 0.5f - (Mf + 2.0f) * 0x1p-21f;
    ArgMin best{INFINITY, 0x7fffffff};
    for (int g = lane; g < G; g += kWave) {
        const float a = (float)(mdd * (double)s_c[g] / Md);
        if (a == 0.0f) continue;
        const double ad = (double)a;
        double E = 0.0;
        bool near = !(a >= 0x1p-100f && a <= 0x1p100f);
        if (!near) {
            const float v = __builtin_amdgcn_rcpf(a);
#pragma unroll
            for (int j = 0; j < kN; ++j) {
                const float y = x32[j] * v;
                const float c = rintf(y);
                near |= fabsf(y - c) >= lim;
                const double e = fma(-ad, (double)fminf(c, Mf), fabs(r[j]));
                E = fma(e, e, E);
            }
        }
        if (near) {   // the codes from the fp64 quotient
            const double ia = 1.0 / ad;
            E = 0.0;
#pragma unroll
            for (int j = 0; j < kN; ++j) {
                const double x = fabs(r[j]);
                const double y = x * ia;
                double c = rint(y);
                if (fabs(fabs(y - c) - 0.5) < 0x1p-40) c = rint(x / ad);
                const double e = fma(-ad, fmin(c, Md), x);
                E = fma(e, e, E);
            }
        }
        if (E < best.e || (E == best.e && g < best.g)) best = ArgMin{E, g};
    }
    return best;
}

template <int kD>
__global__ void __launch_bounds__(kSmallWaves * kWave) fit_small_kernel(const HistBatch B, int channels)
{
    extern __shared__ float s_c[];   // [G] grid multipliers c_g
    const int G = B.G;
    // the default multipliers fl32((g + 1) / G), as in the histogram search
    for (int g = threadIdx.x; g < G; g += kSmallWaves * kWave)
        s_c[g] = B.grid ? B.grid[g] : __fdiv_rn((float)(g + 1), (float)G);
    __syncthreads();

    const int lane = threadIdx.x % kWave;
    // the wavefront's channel (uniform: kept in a scalar register)
    const int ch = __builtin_amdgcn_readfirstlane(blockIdx.x * kSmallWaves + threadIdx.x / kWave);
    if (ch >= channels) return;
    const int li = last_at_most(B.n_layers, ch, [&](int i) { return B.L[i].c_begin; });
    const HistLayer &Ly = B.L[li];
    const int64_t k = (int64_t)ch - Ly.c_begin;
    constexpr int d = kD;   // every layer of the launch has channels of kD weights
    const int P = B.P;
    const int M = B.M;
    const double Md = (double)M;
    int8_t *qk = Ly.codes + k * (int64_t)P * d;
    const float *wk = Ly.W + k * (int64_t)d;

    // resume a channel that holds s0 points and has not stopped (count s0);
    // a calibration step takes at most one point
    const bool stepping = B.single != 0;
    const int s0 = B.start;
    if (s0 >= 1 && Ly.counts[k] != s0) return;

    // asymmetric codes (reading B2): the points fit w - beta, beta the fp32
    // midpoint of the range; the stopping rule keeps ||w||^2
    double beta = 0.0;
    double Ew = 0.0;
    const bool asym = Ly.offsets != nullptr;
    if (asym) {
        float mx = -INFINITY, mn = INFINITY;
#pragma unroll
        for (int j = 0; j < kD; ++j) {
            if (j < d) {
                mx = fmaxf(mx, wk[j]);
                mn = fminf(mn, wk[j]);
            }
        }
        const float b = (float)(((double)mx + (double)mn) / 2.0);
        beta = (double)b;
        if (lane == 0) Ly.offsets[k] = b;
    }
    if (asym || (s0 >= 1 && !stepping)) {   // ||w||^2 when the first residual is not w
        double sw = 0.0;
#pragma unroll
        for (int j = 0; j < kD; ++j)
            if (j < d) sw = fma((double)wk[j], (double)wk[j], sw);
        Ew = sw;
    }

    // residual after the first np stored points (0 past d)
    double r[kD];
    auto rebuild = [&](int np) {
#pragma unroll
        for (int j = 0; j < kD; ++j) {
            double v = 0.0;
            if (j < d) {
                v = (double)wk[j] - beta;
                for (int p = 0; p < np; ++p)
                    v = fma(-(double)Ly.scales[k * P + p], (double)qk[(int64_t)p * d + j], v);
            }
            r[j] = v;
        }
    };
    rebuild(s0);

    float apend = 0.0f;
    int n = 0;
    bool more = false;   // calibration step: the channel took its point and goes on
    // Algorithm 2's naive point (reading F1), as in the histogram search:
    // a calibration fit's first step keeps a stored naive point whose output
    // error meets the threshold; a fresh fit applies it at step 0 (gstate 1)
    // and decides at step 1 (gstate 2) whether it stays or the fit restarts
    bool kept = false;
    if (B.gate && stepping && s0 == 0) {
        const double thr = Ly.ref ? B.eps * (double)Ly.ref[k] : B.eps;
        kept = Ly.counts[k] == 1 && (double)Ly.xerr[k * P] <= thr;
        if (kept) n = 1;
    }
    int gstate = (B.gate && !stepping && s0 == 0) ? 1 : 0;
    for (int i = s0; !kept; ++i) {
        // ---- apply the pending point: codes of Eq. (10), residual of Eq. (7)
        if (i > s0) {
            const PointCode code_of(apend, M);
            int8_t *qrow = qk + (int64_t)(i - 1) * d;
            double aupd = code_of.ap;
            if (B.refit && gstate != 2) {   // reading A2; the naive point keeps its scale
                double rq = 0.0, qq = 0.0;
                int mine = 0;
#pragma unroll
                for (int j = 0; j < kD; ++j) {
                    if (j < d) {
                        const double c = code_of(r[j]);
                        if (lane == j) mine = (int)c;
                        rq = fma(r[j], c, rq);
                        qq = fma(c, c, qq);
                    }
                }
                if (lane < d) qrow[lane] = (int8_t)mine;
                const float afit = (float)(rq / qq);
                if (lane == 0) Ly.scales[k * P + (i - 1)] = afit;
                aupd = (double)afit;
            }
            int mine = 0;
#pragma unroll
            for (int j = 0; j < kD; ++j) {
                if (j < d) {
                    const double c = code_of(r[j]);
                    if (lane == j) mine = (int)c;
                    r[j] = fma(-aupd, c, r[j]);
                }
            }
            if ((!B.refit || gstate == 2) && lane < d) qrow[lane] = (int8_t)mine;
        }
        float m = 0.0f;
        double Er = 0.0;
#pragma unroll
        for (int j = 0; j < kD; ++j) {
            m = fmaxf(m, fabsf((float)r[j]));
            Er = fma(r[j], r[j], Er);
        }
        m = uniform(m);
        Er = uniform(Er);

        // ---- stop / point count
        if (i == 0 && !asym) Ew = Er;
        else if (i > s0 && Ly.err && lane == 0) Ly.err[k * P + (i - 1)] = (float)Er;
        if (stepping && i > s0) {   // one point per calibration step
            n = i;
            more = true;
            break;
        }
        bool stop = (i >= P) || (Er == 0.0);
        if (!stop && i >= 1) {
            if (stepping) {
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
            rebuild(0);   // discarded: restart from w
            i = -1;
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
                if (lane == 0) Ly.scales[k * P] = aN;
                continue;
            }
        }

        // ---- candidate errors, lanes over candidates
        float x32[kD];
#pragma unroll
        for (int j = 0; j < kD; ++j) x32[j] = (float)fabs(r[j]);
        const double mdd = (double)m;
        ArgMin best{INFINITY, 0x7fffffff};
        best = lane_candidates<kD, kD>(r, x32, s_c, G, lane, mdd, M);
        best = wave_argmin(best);
        if (best.e == INFINITY) {   // every candidate scale is zero
            n = i;
            break;
        }
        apend = (float)(mdd * (double)s_c[best.g] / Md);
        if (lane == 0) Ly.scales[k * P + i] = apend;
    }

    if (lane == 0) Ly.counts[k] = n;
    if (more) {
        if (lane == 0) Ly.list[atomicAdd(Ly.nlist + s0, 1)] = (int32_t)k;
        return;
    }
    // the row of the output error's D (tiles of 128 rows by 32 k; one
    // 32-k chunk holds the whole channel): the final residual in fp32
    if (Ly.dres && !stepping) {
        float v = 0.0f;
#pragma unroll
        for (int j = 0; j < kD; ++j)
            if (lane == j) v = (float)r[j];   // 0 past d
        if (lane < 32) Ly.dres[(k / 128) * 4096 + (k % 128) * 32 + lane] = v;
    }
    for (int q = n + lane; q < P; q += kWave) {
        Ly.scales[k * P + q] = 0.0f;
        if (Ly.err) Ly.err[k * P + q] = 0.0f;
        if (Ly.xerr) Ly.xerr[k * P + q] = 0.0f;
    }
    for (int64_t b = (int64_t)n * d + lane; b < (int64_t)P * d; b += kWave) qk[b] = 0;
}

}  // namespace

std::string fit_small_name(int d)
{
    char name[32];
    snprintf(name, sizeof name, "fit_small_kernel<%d>", d);
    return name;
}

namespace {

template <int kD>
hipError_t launch_small_t(const HistBatch &b, int64_t channels, hipStream_t s)
{
    for (int l = 0; l < b.n_layers; ++l)
        if (b.L[l].d != kD) return hipErrorInvalidValue;   // one length per launch
    LaunchTimer timer(s, fit_small_name(kD).c_str());
    const unsigned groups = (unsigned)((channels + kSmallWaves - 1) / kSmallWaves);
    hipLaunchKernelGGL(fit_small_kernel<kD>, dim3(groups), dim3(kSmallWaves * kWave),
                       (size_t)b.G * sizeof(float), s, b, (int)channels);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_fit_small(const HistBatch &b, int d, int64_t channels, hipStream_t s)
{
    if (channels <= 0) return hipSuccess;
    if (channels > 0x7fffffffLL - kSmallWaves) return hipErrorInvalidValue;
    static_assert(kSmallMaxDim == 16, "one instantiation per length below");
    switch (d) {
    case 1: return launch_small_t<1>(b, channels, s);
    case 2: return launch_small_t<2>(b, channels, s);
    case 3: return launch_small_t<3>(b, channels, s);
    case 4: return launch_small_t<4>(b, channels, s);
    case 5: return launch_small_t<5>(b, channels, s);
    case 6: return launch_small_t<6>(b, channels, s);
    case 7: return launch_small_t<7>(b, channels, s);
    case 8: return launch_small_t<8>(b, channels, s);
    case 9: return launch_small_t<9>(b, channels, s);
    case 10: return launch_small_t<10>(b, channels, s);
    case 11: return launch_small_t<11>(b, channels, s);
    case 12: return launch_small_t<12>(b, channels, s);
    case 13: return launch_small_t<13>(b, channels, s);
    case 14: return launch_small_t<14>(b, channels, s);
    case 15: return launch_small_t<15>(b, channels, s);
    case 16: return launch_small_t<16>(b, channels, s);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace mpq
