// Quantized weights of Eq. (4): W_hat[k][j] = fl32(sum_{i<n_k} a_i q_i[j]),
// summed in fp64 in point order (with asymmetric codes, reading B2, the sum
// starts at the channel's offset).  Elementwise and HBM-bound: it reads the
// n_k code rows of each channel and writes its fp32 row once.
//
// Up to kMaxRecLayers layers share one launch (descriptors by value in the
// kernel arguments).  A workgroup takes a group of whole rows of one layer
// (about kRowElems elements), so a row's count and scales are uniform loads:
//  - a layer with d % 4 == 0 and aligned buffers: the group's rows form one
//    flat range of 4-element chunks (one 32-bit word of codes per point, one
//    float4 store per chunk);
//  - other rows of fewer than 256 elements (depthwise kernels, d = 9): the
//    group's elements are spread over the threads as one flat range;
//  - other rows: the workgroup sweeps each row in turn.
#include <algorithm>

#include "internal.hpp"
#include "reduce.hpp"

namespace mpq {

namespace {

constexpr int kRecThreads = 256;
constexpr int kRowElems = 4096;

struct RecDesc {
    const int8_t *codes;
    const float *scales;
    const int32_t *counts;
    float *W_hat;
    int C, d;
    int rows;          // rows per workgroup
    int block_begin;   // first workgroup of this layer
    int vec;           // d % 4 == 0, codes 4-byte and W_hat 16-byte aligned
    const float *offsets;   // reading B2: each row's sum starts at its offset, or nullptr
};

struct RecGroup {
    int n_layers;
    int P;
    RecDesc L[kMaxRecLayers];
};
static_assert(sizeof(RecGroup) <= 4096, "kernel arguments");

__global__ void __launch_bounds__(kRecThreads) reconstruct_kernel(const RecGroup g)
{
    const int li = last_at_most(g.n_layers, (int)blockIdx.x, [&](int i) { return g.L[i].block_begin; });
    const RecDesc &L = g.L[li];
    const int P = g.P;
    const int d = L.d;
    const int k0 = ((int)blockIdx.x - L.block_begin) * L.rows;
    const int k1 = min(k0 + L.rows, L.C);
    const int t = threadIdx.x;

    if (L.vec) {
        // the group's rows as one flat range of 4-element chunks; per chunk
        // the code words and scales of up to four points are loaded before
        // any is used (points past the fourth follow in order)
        const int q4 = d / 4;
        const int total = (k1 - k0) * q4;
        for (int e = t; e < total; e += kRecThreads) {
            const int kr = e / q4, j = (e - kr * q4) * 4;
            const int64_t k = k0 + kr;
            const int n = min(max(L.counts[k], 0), P);   // clamp: counts is caller data
            const int8_t *crow = L.codes + k * (int64_t)P * d + j;
            const float *a = L.scales + k * (int64_t)P;
            uint32_t w[4];
            float ai[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                w[i] = i < n ? *(const uint32_t *)(crow + (int64_t)i * d) : 0u;
                ai[i] = i < n ? a[i] : 0.0f;
            }
            const double beta = L.offsets ? (double)L.offsets[k] : 0.0;
            double s[4] = {beta, beta, beta, beta};
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (i < n) {
#pragma unroll
                    for (int u = 0; u < 4; ++u)
                        s[u] = fma((double)ai[i], (double)(int)(int8_t)(uint8_t)(w[i] >> (8 * u)), s[u]);
                }
            for (int i = 4; i < n; ++i) {
                const uint32_t wi = *(const uint32_t *)(crow + (int64_t)i * d);
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    s[u] = fma((double)a[i], (double)(int)(int8_t)(uint8_t)(wi >> (8 * u)), s[u]);
            }
            *(float4 *)(L.W_hat + k * d + j) = make_float4((float)s[0], (float)s[1], (float)s[2], (float)s[3]);
        }
        return;
    }
    if (d < kRecThreads) {
        // flat range of short rows
        const int total = (k1 - k0) * d;
        for (int e = t; e < total; e += kRecThreads) {
            const int kr = e / d, j = e - kr * d;
            const int64_t k = k0 + kr;
            const int n = min(max(L.counts[k], 0), P);   // clamp: counts is caller data
            const int8_t *q = L.codes + k * (int64_t)P * d + j;
            const float *a = L.scales + k * (int64_t)P;
            double s = L.offsets ? (double)L.offsets[k] : 0.0;
            for (int i = 0; i < n; ++i) s = fma((double)a[i], (double)q[(int64_t)i * d], s);
            L.W_hat[k * d + j] = (float)s;
        }
        return;
    }
    for (int64_t k = k0; k < k1; ++k) {
        const int n = min(max(L.counts[k], 0), P);
        const int8_t *crow = L.codes + k * (int64_t)P * d;
        const float *a = L.scales + k * (int64_t)P;
        float *out = L.W_hat + k * d;
        const double beta = L.offsets ? (double)L.offsets[k] : 0.0;
        for (int j = t; j < d; j += kRecThreads) {
            double s = beta;
            for (int i = 0; i < n; ++i) s = fma((double)a[i], (double)crow[(int64_t)i * d + j], s);
            out[j] = (float)s;
        }
    }
}

}  // namespace

hipError_t launch_reconstruct(const RecLayer *in, int n_in, int P, hipStream_t s)
{
    for (int base = 0; base < n_in; base += kMaxRecLayers) {
        RecGroup g;
        g.n_layers = std::min(kMaxRecLayers, n_in - base);
        g.P = P;
        int64_t blocks = 0;
        for (int i = 0; i < g.n_layers; ++i) {
            const RecLayer &I = in[base + i];
            RecDesc &L = g.L[i];
            L.codes = I.codes;
            L.scales = I.scales;
            L.counts = I.counts;
            L.W_hat = I.W_hat;
            L.C = (int)I.C;
            L.d = (int)I.d;
            L.rows = (int)std::max<int64_t>(1, kRowElems / I.d);
            L.block_begin = (int)blocks;
            blocks += (I.C + L.rows - 1) / L.rows;
            L.vec = I.d % 4 == 0 && ((uintptr_t)I.codes) % 4 == 0 && ((uintptr_t)I.W_hat) % 16 == 0;
            L.offsets = I.offsets;
        }
        if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
        LaunchTimer timer(s, "reconstruct_kernel");
        hipLaunchKernelGGL(reconstruct_kernel, dim3((unsigned)blocks), dim3(kRecThreads), 0, s, g);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace mpq
