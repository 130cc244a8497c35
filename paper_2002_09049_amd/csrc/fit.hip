// Greedy multipoint fit of a layer: one workgroup per output channel runs
// every step of Algorithm 1 (Sec. 3.2) with the stopping rule of Algorithm 2
// (Sec. 3.3) for its channel.
//
// Per step, inside the workgroup:
//   1. residual pass (HBM-bound): rebuild r = w - sum_{p<i} a_p q_p in fp64
//      from the weights and the codes this channel already wrote, emit the
//      codes of the point chosen in the previous step (Eq. (10)) and apply it
//      (Eq. (7)); stage fl32(r) in LDS; reduce max|r| and ||r||^2.
//      The codes are the state: no residual workspace exists.
//   2. stop / point count (Alg. 2, Eq. (12) under an isotropic batch).
//   3. candidate scales a_g = fl32(fl32(max|r|) c_g / M), g = 1..G.
//   4. dense candidate search (Eq. (8)-(9)), VALU-bound, on r and a scaled
//      by the same power of two (exact; the argmin is unchanged): every thread holds
//      kCandPerThread candidates in registers and sweeps an LDS slice of the
//      residual with broadcast reads; per (element, candidate):
//      q = rne(clamp(r * 1/a, -M, M)), e = r - a q, E += e^2 in fp32 blocks of
//      16 elements, blocks summed in fp64.  Slices are summed in fp64 in LDS.
//   5. argmin over candidates (ties: smallest g) with DPP/ds_swizzle wave
//      reductions.
// The codes are emitted in fp64 (q = rne(r / a), IEEE quotient) so they are
// exactly the rounding of Eq. (10) on the exact residual.
#include <math.h>

#include "internal.hpp"
#include "mpq.h"
#include "reduce.hpp"

namespace mpq {

namespace {

__device__ __forceinline__ float eval_candidate(float x, float a, float inv, float Mf, float acc)
{
    float t = __builtin_amdgcn_fmed3f(x * inv, -Mf, Mf);
    float q = __builtin_rintf(t);
    float e = __builtin_fmaf(-a, q, x);
    return __builtin_fmaf(e, e, acc);
}

template <int kCt>
__global__ void __launch_bounds__(kFitThreads) fit_dense_kernel(FitParams p, FitLayout L)
{
    extern __shared__ __align__(16) float smem[];
    __shared__ float s_scale[MPQ_MAX_POINTS];
    __shared__ float s_redf[kFitThreads / kWave];
    __shared__ double s_redd[kFitThreads / kWave];
    __shared__ ArgMin s_arg[kFitThreads / kWave];

    const int G = p.G;
    const int gpad = L.passes * L.chunk;
    // dpad is a multiple of 16 and gpad of 128, so every region below starts
    // 16-byte aligned (float4 reads of sR, fp64 in sE / sPart).
    float *sR = smem;                                    // [dpad]
    float *sA = sR + L.dpad;                             // [gpad]
    float *sAs = sA + gpad;                              // [gpad]
    float *sInv = sAs + gpad;                            // [gpad]
    double *sE = (double *)(sInv + gpad);                // [G]
    double *sPart = sE + G;                              // [slices * chunk]

    const int64_t k = blockIdx.x;
    const int t = threadIdx.x;
    const int64_t d = p.d;
    const int P = p.P;
    const double Md = (double)p.M;
    const float Mf = (float)p.M;
    const float *w = p.W + k * d;
    int8_t *qk = p.codes + k * (int64_t)P * d;

    for (int64_t j = d + t; j < L.dpad; j += kFitThreads) sR[j] = 0.0f;

    double Ew = 0.0;
    int n = 0;
    for (int i = 0;; ++i) {
        // ---- 1. residual pass
        float lmax = 0.0f;
        double lsum = 0.0;
        const double apend = i >= 1 ? (double)s_scale[i - 1] : 0.0;
        for (int64_t j = t; j < d; j += kFitThreads) {
            double r = (double)w[j];
            for (int q = 0; q + 1 < i; ++q)
                r = fma(-(double)s_scale[q], (double)qk[(int64_t)q * d + j], r);
            if (i >= 1) {
                double c = rint(r / apend);
                c = fmin(fmax(c, -Md), Md);
                qk[(int64_t)(i - 1) * d + j] = (int8_t)(int)c;
                r = fma(-apend, c, r);
            }
            const float rf = (float)r;
            lmax = fmaxf(lmax, fabsf(rf));
            lsum = fma(r, r, lsum);
            sR[j] = rf;
        }
        const float m = block_reduce<kFitThreads>(lmax, MaxOp(), s_redf);
        const double Er = block_reduce<kFitThreads>(lsum, SumOp(), s_redd);

        // ---- 2. stop / point count
        if (i == 0) Ew = Er;
        else if (p.err && t == 0) p.err[k * P + (i - 1)] = (float)Er;
        bool stop = (i >= P) || (Er == 0.0) || (i >= 1 && Er <= p.tol * Ew);
        if (!stop) {
            // ---- 3. candidate scales.  The search works on r and a scaled by
            // 2^-ex (max|r| = f 2^ex, f in [0.5, 1)): exact, argmin-preserving,
            // and it keeps the fp32 squared errors clear of overflow/underflow.
            int ex = 0;
            (void)frexpf(m, &ex);
            for (int64_t j = t; j < d; j += kFitThreads) sR[j] = ldexpf(sR[j], -ex);
            for (int g = t; g < gpad; g += kFitThreads) {
                float a = 1.0f, as = 1.0f, inv = 1.0f;
                if (g < G) {
                    const float c = p.grid ? p.grid[g] : (float)((double)(g + 1) / (double)G);
                    a = (float)((double)m * (double)c / Md);
                    as = ldexpf(a, -ex);
                    inv = as != 0.0f ? 1.0f / as : 0.0f;
                }
                sA[g] = a;       // the candidate itself (stored as the scale)
                sAs[g] = as;     // scaled, used by the search
                sInv[g] = inv;
            }
            __syncthreads();

            // ---- 4. dense search
            const int s = t / L.lanes, l = t % L.lanes;
            const int64_t dslice = L.dpad / L.slices;
            const float *xs = sR + s * dslice;
            for (int pass = 0; pass < L.passes; ++pass) {
                float a[kCt], inv[kCt];
                double acc[kCt];
#pragma unroll
                for (int c = 0; c < kCt; ++c) {
                    const int g = pass * L.chunk + l + c * L.lanes;
                    a[c] = sAs[g];
                    inv[c] = sInv[g];
                    acc[c] = 0.0;
                }
                for (int64_t j = 0; j < dslice; j += 16) {
                    float blk[kCt];
#pragma unroll
                    for (int c = 0; c < kCt; ++c) blk[c] = 0.0f;
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const float4 x4 = *(const float4 *)(xs + j + 4 * u);
#pragma unroll
                        for (int c = 0; c < kCt; ++c) {
                            blk[c] = eval_candidate(x4.x, a[c], inv[c], Mf, blk[c]);
                            blk[c] = eval_candidate(x4.y, a[c], inv[c], Mf, blk[c]);
                            blk[c] = eval_candidate(x4.z, a[c], inv[c], Mf, blk[c]);
                            blk[c] = eval_candidate(x4.w, a[c], inv[c], Mf, blk[c]);
                        }
                    }
#pragma unroll
                    for (int c = 0; c < kCt; ++c) acc[c] += (double)blk[c];
                }
#pragma unroll
                for (int c = 0; c < kCt; ++c) sPart[s * L.chunk + l + c * L.lanes] = acc[c];
                __syncthreads();
                for (int idx = t; idx < L.chunk; idx += kFitThreads) {
                    const int g = pass * L.chunk + idx;
                    if (g < G) {
                        double tot = 0.0;
                        for (int s2 = 0; s2 < L.slices; ++s2) tot += sPart[s2 * L.chunk + idx];
                        sE[g] = sA[g] == 0.0f ? INFINITY : tot;
                    }
                }
                __syncthreads();
            }

            // ---- 5. argmin over candidates (ties: smallest g)
            ArgMin best{INFINITY, 0x7fffffff};
            for (int g = t; g < G; g += kFitThreads)
                if (sE[g] < best.e) best = ArgMin{sE[g], g};
            best = block_argmin<kFitThreads>(best, s_arg);
            if (best.e == INFINITY) {
                stop = true;  // every candidate scale is zero
            } else {
                if (t == 0) {
                    s_scale[i] = sA[best.g];
                    p.scales[k * P + i] = sA[best.g];
                }
                __syncthreads();
            }
        }
        if (stop) {
            n = i;
            break;
        }
    }

    // counts and zero fill of the unused slots
    if (t == 0) p.counts[k] = n;
    for (int q = n + t; q < P; q += kFitThreads) {
        p.scales[k * P + q] = 0.0f;
        if (p.err) p.err[k * P + q] = 0.0f;
    }
    for (int q = n; q < P; ++q)
        for (int64_t j = t; j < d; j += kFitThreads) qk[(int64_t)q * d + j] = 0;
}

}  // namespace

FitLayout fit_layout(int64_t d, int G)
{
    FitLayout L;
    int need = (G + kCandPerThread - 1) / kCandPerThread;
    int lanes = kWave;
    while (lanes < need && lanes < kFitThreads) lanes *= 2;
    L.lanes = lanes;
    L.slices = kFitThreads / lanes;
    L.chunk = lanes * kCandPerThread;
    L.passes = (G + L.chunk - 1) / L.chunk;
    const int64_t q = 16 * (int64_t)L.slices;
    L.dpad = (d + q - 1) / q * q;
    const int gpad = L.passes * L.chunk;
    L.lds = sizeof(float) * ((size_t)L.dpad + 3 * (size_t)gpad) +
            sizeof(double) * ((size_t)G + (size_t)L.slices * L.chunk);
    return L;
}

hipError_t launch_fit(const FitParams &p, const FitLayout &L, hipStream_t s)
{
    static_assert(kCandPerThread == 2, "layout assumes two candidates per thread");
    auto kern = fit_dense_kernel<kCandPerThread>;
    if (L.lds > 65536) {
        hipError_t e = hipFuncSetAttribute((const void *)kern,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)L.lds);
        if (e != hipSuccess) return e;
    }
    LaunchTimer timer(s, "fit_dense_kernel");
    hipLaunchKernelGGL(kern, dim3((unsigned)p.C), dim3(kFitThreads), L.lds, s, p, L);
    return hipGetLastError();
}

}  // namespace mpq
