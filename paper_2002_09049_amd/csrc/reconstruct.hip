// Quantized weights of Eq. (4): W_hat[k][j] = fl32(sum_{i<n_k} a_i q_i[j]),
// summed in fp64 in point order.  Elementwise and HBM-bound: consecutive
// threads on consecutive j.  Up to kMaxRecLayers layers share one launch
// (blockIdx.y = layer; descriptors by value in the kernel arguments).
#include <algorithm>

#include "internal.hpp"

namespace mpq {

namespace {

struct RecGroup {
    int n_layers;
    int P;
    RecLayer L[kMaxRecLayers];
};

__global__ void __launch_bounds__(256) reconstruct_kernel(const RecGroup g)
{
    const RecLayer &L = g.L[blockIdx.y];
    const int P = g.P;
    const int64_t total = L.C * L.d;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t k = e / L.d, j = e - k * L.d;
        const int n = min(max(L.counts[k], 0), P);  // clamp: counts is caller data
        const int8_t *q = L.codes + k * (int64_t)P * L.d + j;
        const float *a = L.scales + k * (int64_t)P;
        double s = 0.0;
        for (int i = 0; i < n; ++i) s = fma((double)a[i], (double)q[(int64_t)i * L.d], s);
        L.W_hat[e] = (float)s;
    }
}

}  // namespace

hipError_t launch_reconstruct(const RecLayer *in, int n_in, int P, hipStream_t s)
{
    for (int base = 0; base < n_in; base += kMaxRecLayers) {
        RecGroup g;
        g.n_layers = std::min(kMaxRecLayers, n_in - base);
        g.P = P;
        int64_t most = 0;
        for (int i = 0; i < g.n_layers; ++i) {
            g.L[i] = in[base + i];
            most = std::max<int64_t>(most, g.L[i].C * g.L[i].d);
        }
        const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((most + 255) / 256, 4096));
        hipLaunchKernelGGL(reconstruct_kernel, dim3((unsigned)blocks, (unsigned)g.n_layers), dim3(256),
                           0, s, g);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace mpq
