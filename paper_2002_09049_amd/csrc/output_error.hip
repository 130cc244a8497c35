// Output error of a quantized layer on a calibration batch (Sec. 3.3,
// Eq. (12)): err[k] = (1/n) sum_t ((w_k - w~_k) . x_t)^2 and optionally
// ref[k] = (1/n) sum_t (w_k . x_t)^2.
//
// This is the path's one dense contraction, so it runs on MFMA:
// v_mfma_f32_32x32x2f32 (fp32 in, fp32 accumulate).  A workgroup of four
// wavefronts owns a 128 x 128 tile of Y = D X (rows: channels, columns:
// batch); each wavefront owns 64 x 64 as 2 x 2 MFMA blocks.  The A tile is the
// residual D = w - sum_i a_i q_i, formed in fp64 from W, the codes and the
// scales while staging it into LDS (it is never written to HBM) and rounded
// to fp32.  The epilogue squares Y, sums each row over the tile's columns
// (fp64 cross-lane sums with DPP / ds_swizzle) and writes one partial per
// (column tile, row); a second kernel sums the partials in a fixed order.
#include "internal.hpp"
#include "mpq.h"
#include "reduce.hpp"

namespace mpq {

namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kBM = 128, kBN = 128, kBK = 16;
constexpr int kThreads = 256;
constexpr int kPadA = 4;  // LDS row padding (floats)

template <bool kRef>
__global__ void __launch_bounds__(kThreads)
err_gemm_kernel(const float *__restrict__ W, const int8_t *__restrict__ codes,
                const float *__restrict__ scales, const int32_t *__restrict__ counts,
                int64_t C, int64_t d, int P, const float *__restrict__ X, int64_t n,
                double *__restrict__ partial)
{
    __shared__ __align__(16) float sD[kBK][kBM + kPadA];
    __shared__ __align__(16) float sW[kRef ? kBK : 1][kBM + kPadA];
    __shared__ __align__(16) float sX[kBK][kBN + kPadA];
    __shared__ double sRow[kRef ? 2 : 1][kBM];

    const int t = threadIdx.x;
    const int lane = t % kWave, wid = t / kWave;
    const int wm = wid / 2, wn = wid % 2;  // wave position in the 2 x 2 grid
    const int64_t row0 = (int64_t)blockIdx.y * kBM;
    const int64_t col0 = (int64_t)blockIdx.x * kBN;

    // staging roles: A tile = 128 rows x 16 k, each thread 8 consecutive k of one row
    const int arow = t / 2, ak0 = (t % 2) * 8;
    const int64_t grow = row0 + arow;
    const bool row_ok = grow < C;
    const int nk = row_ok ? min(max(counts[grow], 0), P) : 0;  // clamp: counts is caller data
    const float *wrow = W + (row_ok ? grow : 0) * d;
    const int8_t *qrow = codes + (row_ok ? grow : 0) * (int64_t)P * d;
    const float *srow = scales + (row_ok ? grow : 0) * (int64_t)P;

    floatx16 acc[2][2], accw[kRef ? 2 : 1][kRef ? 2 : 1];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.0f;
    if constexpr (kRef) {
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int v = 0; v < 16; ++v) accw[a][b][v] = 0.0f;
    }

    for (int64_t k0 = 0; k0 < d; k0 += kBK) {
        // ---- stage D (and W) : fp64 residual rounded to fp32
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int64_t j = k0 + ak0 + u;
            float dv = 0.0f, wv = 0.0f;
            if (row_ok && j < d) {
                const float w = wrow[j];
                double r = (double)w;
                for (int i = 0; i < nk; ++i)
                    r = fma(-(double)srow[i], (double)qrow[(int64_t)i * d + j], r);
                dv = (float)r;
                wv = w;
            }
            sD[ak0 + u][arow] = dv;
            if constexpr (kRef) sW[ak0 + u][arow] = wv;
        }
        // ---- stage X: 16 rows x 128 columns, each thread 8 values of one row
        {
            const int xk = t / 16, xc0 = (t % 16) * 8;
            const int64_t j = k0 + xk;
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int64_t c = col0 + xc0 + u;
                sX[xk][xc0 + u] = (j < d && c < n) ? X[j * n + c] : 0.0f;
            }
        }
        __syncthreads();
        // ---- MFMA over the 16-deep slab, 2 k per instruction
#pragma unroll
        for (int kk = 0; kk < kBK; kk += 2) {
            const int kr = kk + lane / 32;
            float af[2], bf[2], wf[2];
#pragma unroll
            for (int a = 0; a < 2; ++a) {
                af[a] = sD[kr][wm * 64 + a * 32 + lane % 32];
                if constexpr (kRef) wf[a] = sW[kr][wm * 64 + a * 32 + lane % 32];
            }
#pragma unroll
            for (int b = 0; b < 2; ++b) bf[b] = sX[kr][wn * 64 + b * 32 + lane % 32];
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[a], bf[b], acc[a][b], 0, 0, 0);
                    if constexpr (kRef)
                        accw[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(wf[a], bf[b], accw[a][b], 0, 0, 0);
                }
        }
        __syncthreads();
    }

    // ---- epilogue: per row, sum of squares over this tile's 128 columns.
    // Output layout of a 32 x 32 MFMA block: lane holds column lane % 32 and,
    // in register v, row 8 * (v / 4) + 4 * (lane / 32) + (v % 4).
    for (int pass = 0; pass < 2; ++pass) {
        if (wn == pass) {
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    double s = (double)(acc[a][0][v] * acc[a][0][v]) +
                               (double)(acc[a][1][v] * acc[a][1][v]);
                    s = half_wave_reduce(s, SumOp());
                    double sw = 0.0;
                    if constexpr (kRef) {
                        sw = (double)(accw[a][0][v] * accw[a][0][v]) +
                             (double)(accw[a][1][v] * accw[a][1][v]);
                        sw = half_wave_reduce(sw, SumOp());
                    }
                    if (lane % 32 == 0) {
                        const int r = wm * 64 + a * 32 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
                        sRow[0][r] = pass == 0 ? s : sRow[0][r] + s;
                        if constexpr (kRef) sRow[1][r] = pass == 0 ? sw : sRow[1][r] + sw;
                    }
                }
        }
        __syncthreads();
    }
    for (int r = t; r < kBM; r += kThreads) {
        const int64_t gr = row0 + r;
        if (gr < C) {
            partial[(int64_t)blockIdx.x * C + gr] = sRow[0][r];
            if constexpr (kRef)
                partial[((int64_t)gridDim.x + blockIdx.x) * C + gr] = sRow[1][r];
        }
    }
}

__global__ void err_finish_kernel(const double *__restrict__ partial, int64_t C, int ntiles,
                                  int64_t n, float *__restrict__ err, float *__restrict__ ref)
{
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= C) return;
    double s = 0.0;
    for (int i = 0; i < ntiles; ++i) s += partial[(int64_t)i * C + k];
    err[k] = (float)(s / (double)n);
    if (ref) {
        double sr = 0.0;
        for (int i = 0; i < ntiles; ++i) sr += partial[((int64_t)ntiles + i) * C + k];
        ref[k] = (float)(sr / (double)n);
    }
}

}  // namespace

size_t err_partial_bytes(int64_t C, int64_t n, bool with_ref)
{
    const int64_t ntiles = (n + kBN - 1) / kBN;
    return sizeof(double) * (size_t)(ntiles * C * (with_ref ? 2 : 1));
}

hipError_t launch_output_error(const float *W, const int8_t *codes, const float *scales,
                               const int32_t *counts, int64_t C, int64_t d, int P,
                               const float *X, int64_t n, float *err, float *ref,
                               double *partial, hipStream_t s)
{
    const int64_t ntiles = (n + kBN - 1) / kBN;
    dim3 grid((unsigned)ntiles, (unsigned)((C + kBM - 1) / kBM));
    if (ref)
        hipLaunchKernelGGL(err_gemm_kernel<true>, grid, dim3(kThreads), 0, s, W, codes, scales,
                           counts, C, d, P, X, n, partial);
    else
        hipLaunchKernelGGL(err_gemm_kernel<false>, grid, dim3(kThreads), 0, s, W, codes, scales,
                           counts, C, d, P, X, n, partial);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(err_finish_kernel, dim3((unsigned)((C + 255) / 256)), dim3(256), 0, s,
                       partial, C, (int)ntiles, n, err, ref);
    return hipGetLastError();
}

}  // namespace mpq
