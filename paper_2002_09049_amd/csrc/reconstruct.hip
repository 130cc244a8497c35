// Quantized weights of Eq. (4): W_hat[k][j] = fl32(sum_{i<n_k} a_i q_i[j]),
// summed in fp64 in point order.  Elementwise and HBM-bound: one thread per
// element, consecutive threads on consecutive j.
#include "internal.hpp"

namespace mpq {

namespace {

__global__ void __launch_bounds__(256)
reconstruct_kernel(const int8_t *__restrict__ codes, const float *__restrict__ scales,
                   const int32_t *__restrict__ counts, int64_t C, int64_t d, int P,
                   float *__restrict__ out)
{
    const int64_t total = C * d;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t k = e / d, j = e - k * d;
        const int n = min(max(counts[k], 0), P);  // clamp: counts is caller data
        const int8_t *q = codes + k * (int64_t)P * d + j;
        const float *a = scales + k * (int64_t)P;
        double s = 0.0;
        for (int i = 0; i < n; ++i) s = fma((double)a[i], (double)q[(int64_t)i * d], s);
        out[e] = (float)s;
    }
}

}  // namespace

hipError_t launch_reconstruct(const int8_t *codes, const float *scales, const int32_t *counts,
                              int64_t C, int64_t d, int P, float *W_hat, hipStream_t s)
{
    const int64_t total = C * d;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(reconstruct_kernel, dim3((unsigned)blocks), dim3(256), 0, s, codes, scales,
                       counts, C, d, P, W_hat);
    return hipGetLastError();
}

}  // namespace mpq
