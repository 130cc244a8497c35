// Clipping of Eq. (13), per channel, as the first point of the fit (a
// variant the paper applies before the points are added).
//
// clip_cand_kernel: the Gc clipping candidates of a channel, the scales
//   a_j = fl32(fl32(max|w|) c_j / M), c_j = fl32(j / Gc), j = 1..Gc (the
//   factors K = c_j max|w| of the grid [1/Gc : 1/Gc : 1] folded into the
//   code step K / M; products and quotient in fp64).
// The output error of each candidate's naive quantization on the
// calibration batch runs through the output-error kernels (candidate rows).
// clip_choose_kernel: the candidate with the smallest output error (ties: the
//   smallest j; zero scales skipped) becomes point 1: its codes (Eq. (10)),
//   scale, ||w - a q||^2 and count 1; a channel with no nonzero candidate
//   (an all-zero channel) gets count 0 and zeroed slots.
#include <math.h>

#include "internal.hpp"
#include "mpq.h"
#include "reduce.hpp"

namespace mpq {

namespace {

constexpr int kClipThreads = 256;

__device__ __forceinline__ int layer_of(const ClipBatch &B)
{
    return last_at_most(B.n_layers, (int)blockIdx.x, [&](int i) { return B.L[i].c_begin; });
}

__global__ void __launch_bounds__(kClipThreads) clip_cand_kernel(const ClipBatch B)
{
    __shared__ float s_max[kClipThreads / kWave];
    const ClipLayer &L = B.L[layer_of(B)];
    const int64_t k = (int64_t)blockIdx.x - L.c_begin;
    const float *w = L.W + k * L.d;
    float m = 0.0f;
    for (int j = threadIdx.x; j < L.d; j += kClipThreads) m = fmaxf(m, fabsf(w[j]));
    m = block_reduce<kClipThreads>(m, MaxOp(), s_max);
    for (int j = threadIdx.x; j < B.Gc; j += kClipThreads) {
        const float c = (float)((double)(j + 1) / (double)B.Gc);
        L.cand[k * B.Gc + j] = (float)((double)m * (double)c / (double)B.M);
    }
}

__global__ void __launch_bounds__(kClipThreads) clip_choose_kernel(const ClipBatch B)
{
    __shared__ double s_red[kClipThreads / kWave];
    __shared__ int s_best;
    const ClipLayer &L = B.L[layer_of(B)];
    const int64_t k = (int64_t)blockIdx.x - L.c_begin;
    const int P = B.P, d = L.d;
    const double Md = (double)B.M;
    if (threadIdx.x == 0) {
        int best = -1;
        for (int j = 0; j < B.Gc; ++j) {
            if (L.cand[k * B.Gc + j] == 0.0f) continue;
            if (best < 0 || L.ecand[k * B.Gc + j] < L.ecand[k * B.Gc + best]) best = j;
        }
        s_best = best;
    }
    __syncthreads();
    const int best = s_best;
    int8_t *q = L.codes + k * (int64_t)P * d;
    if (best < 0) {   // every candidate scale is zero: no point
        if (threadIdx.x == 0) L.counts[k] = 0;
        for (int i = threadIdx.x; i < P; i += kClipThreads) {
            L.scales[k * P + i] = 0.0f;
            if (L.err) L.err[k * P + i] = 0.0f;
            if (L.xerr) L.xerr[k * P + i] = 0.0f;
        }
        for (int64_t j = threadIdx.x; j < (int64_t)P * d; j += kClipThreads) q[j] = 0;
        return;
    }
    const float a = L.cand[k * B.Gc + best];
    const double ap = (double)a, ia = 1.0 / ap;
    const float *w = L.W + k * (int64_t)d;
    double sr = 0.0;
    for (int j = threadIdx.x; j < d; j += kClipThreads) {
        // Eq. (10): the fp64 quotient's rounding, formed only near a half-integer
        const double wj = (double)w[j], y = wj * ia;
        double c = rint(y);
        if (fabs(fabs(y - c) - 0.5) < 0x1p-40) c = rint(wj / ap);
        c = fmin(fmax(c, -Md), Md);
        q[j] = (int8_t)(int)c;
        const double r = fma(-ap, c, wj);
        sr = fma(r, r, sr);
    }
    sr = block_reduce<kClipThreads>(sr, SumOp(), s_red);
    if (threadIdx.x == 0) {
        L.scales[k * P] = a;
        L.counts[k] = 1;
        if (L.err) L.err[k * P] = (float)sr;
        if (L.xerr) L.xerr[k * P] = L.ecand[k * B.Gc + best];
    }
}

}  // namespace

hipError_t launch_clip(const ClipBatch &b, int64_t channels, bool choose, hipStream_t s)
{
    if (channels <= 0) return hipSuccess;
    if (channels > 0x7fffffffLL) return hipErrorInvalidValue;
    LaunchTimer timer(s, choose ? "clip_choose_kernel" : "clip_cand_kernel");
    hipLaunchKernelGGL(choose ? clip_choose_kernel : clip_cand_kernel, dim3((unsigned)channels),
                       dim3(kClipThreads), 0, s, b);
    return hipGetLastError();
}

}  // namespace mpq
