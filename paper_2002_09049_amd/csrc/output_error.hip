// Output error of a quantized layer on a calibration batch (Sec. 3.3,
// Eq. (12)): err[k] = (1/n) sum_t ((w_k - w~_k) . x_t)^2 and optionally
// ref[k] = (1/n) sum_t (w_k . x_t)^2.
//
// Three kernels:
//  1. form_rows: A[k][j] = fl32(w_kj - sum_i a_i q_ij) (fp64 sum in point
//     order) into a scratch matrix whose rows are padded to a multiple of 16
//     with zeros (aligned float4 rows, no K tail).  HBM-bound, coalesced.
//     With use_points = 0 it writes a padded copy of W (for ref).
//  2. gemm: Y = A X on MFMA (v_mfma_f32_32x32x2f32, fp32 in and accumulate),
//     the path's one dense contraction.  A workgroup of four wavefronts owns
//     a 128 x 128 tile of Y and one K range; each wavefront owns 64 x 64 as
//     2 x 2 MFMA blocks.  The K loop stages 16-deep slabs of A and X through
//     double-buffered LDS, loading the next slab into registers while the
//     MFMAs consume the current one.  When the layer has too few tiles to fill
//     the chip, K is split across workgroups (splits).
//       splits == 1: the epilogue squares Y and sums each row over the tile's
//         columns (fp64 cross-lane sums with DPP / ds_swizzle) -> one partial
//         per (column tile, row).
//       splits  > 1: the epilogue stores the fp32 Y tile of its K range.
//  3. finish: splits == 1: sum the row partials in tile order; splits > 1:
//     per row, sum the K-range tiles of every column, square, and sum over the
//     columns (fp64), in a fixed order.  Divide by n.
#include "internal.hpp"
#include "mpq.h"
#include "reduce.hpp"

namespace mpq {

namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kBM = 128, kBN = 128, kBK = 16;
constexpr int kThreads = 256;
constexpr int kPad = 4;  // LDS row padding (floats)

__global__ void __launch_bounds__(256)
form_rows_kernel(const float *__restrict__ W, const int8_t *__restrict__ codes,
                 const float *__restrict__ scales, const int32_t *__restrict__ counts,
                 int64_t C, int64_t d, int64_t ld, int P, int use_points, float *__restrict__ A)
{
    const int64_t total = C * ld;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t k = e / ld, j = e - k * ld;
        float v = 0.0f;
        if (j < d) {
            double r = (double)W[k * d + j];
            if (use_points) {
                const int nk = min(max(counts[k], 0), P);  // clamp: counts is caller data
                const int8_t *q = codes + k * (int64_t)P * d + j;
                const float *a = scales + k * (int64_t)P;
                for (int i = 0; i < nk; ++i) r = fma(-(double)a[i], (double)q[(int64_t)i * d], r);
            }
            v = (float)r;
        }
        A[e] = v;
    }
}

// One K range [kbeg, kend) of a 128 x 128 tile; kbeg, kend multiples of 16.
// A: [C][lda] (lda multiple of 16, zero padded), X: [d][n].
template <bool kSquare, bool kVecX>
__global__ void __launch_bounds__(kThreads)
gemm_kernel(const float *__restrict__ A, int64_t lda, int64_t C, const float *__restrict__ X,
            int64_t d, int64_t n, int64_t kchunk, double *__restrict__ rowpart,
            float *__restrict__ ypart)
{
    __shared__ __align__(16) float sA[2][kBK][kBM + kPad];
    __shared__ __align__(16) float sX[2][kBK][kBN + kPad];
    __shared__ double sRow[kBM];

    const int t = threadIdx.x;
    const int lane = t % kWave, wid = t / kWave;
    const int wm = wid / 2, wn = wid % 2;
    const int64_t row0 = (int64_t)blockIdx.y * kBM;
    const int64_t col0 = (int64_t)blockIdx.x * kBN;
    const int split = blockIdx.z;
    const int64_t kbeg = (int64_t)split * kchunk;
    const int64_t kend = min(kbeg + kchunk, lda);

    // staging roles
    const int arow = t / 2, ak0 = (t % 2) * 8;     // A: 8 consecutive k of one row
    const int64_t agrow = row0 + arow;
    const bool arow_ok = agrow < C;
    const float *ap = A + (arow_ok ? agrow : 0) * lda;
    const int xk = t / 16, xc0 = (t % 16) * 8;     // X: 8 consecutive columns of one k

    float ra[8], rx[8];
    auto load = [&](int64_t k0) {
        if (arow_ok) {
            const float4 v0 = *(const float4 *)(ap + k0 + ak0);
            const float4 v1 = *(const float4 *)(ap + k0 + ak0 + 4);
            ra[0] = v0.x; ra[1] = v0.y; ra[2] = v0.z; ra[3] = v0.w;
            ra[4] = v1.x; ra[5] = v1.y; ra[6] = v1.z; ra[7] = v1.w;
        } else {
#pragma unroll
            for (int u = 0; u < 8; ++u) ra[u] = 0.0f;
        }
        const int64_t j = k0 + xk;
        const int64_t c = col0 + xc0;
        if (j < d) {
            const float *xp = X + j * n + c;
            if (kVecX && c + 8 <= n) {
                const float4 v0 = *(const float4 *)xp;
                const float4 v1 = *(const float4 *)(xp + 4);
                rx[0] = v0.x; rx[1] = v0.y; rx[2] = v0.z; rx[3] = v0.w;
                rx[4] = v1.x; rx[5] = v1.y; rx[6] = v1.z; rx[7] = v1.w;
            } else {
#pragma unroll
                for (int u = 0; u < 8; ++u) rx[u] = (c + u < n) ? xp[u] : 0.0f;
            }
        } else {
#pragma unroll
            for (int u = 0; u < 8; ++u) rx[u] = 0.0f;
        }
    };
    auto store = [&](int buf) {
#pragma unroll
        for (int u = 0; u < 8; ++u) sA[buf][ak0 + u][arow] = ra[u];
        *(float4 *)&sX[buf][xk][xc0] = make_float4(rx[0], rx[1], rx[2], rx[3]);
        *(float4 *)&sX[buf][xk][xc0 + 4] = make_float4(rx[4], rx[5], rx[6], rx[7]);
    };

    floatx16 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.0f;

    int buf = 0;
    if (kbeg < kend) {
        load(kbeg);
        store(0);
    }
    __syncthreads();
    for (int64_t k0 = kbeg; k0 < kend; k0 += kBK) {
        const bool more = k0 + kBK < kend;
        if (more) load(k0 + kBK);   // global loads in flight during the MFMAs
#pragma unroll
        for (int kk = 0; kk < kBK; kk += 2) {
            const int kr = kk + lane / 32;
            float af[2], bf[2];
#pragma unroll
            for (int a = 0; a < 2; ++a) af[a] = sA[buf][kr][wm * 64 + a * 32 + lane % 32];
#pragma unroll
            for (int b = 0; b < 2; ++b) bf[b] = sX[buf][kr][wn * 64 + b * 32 + lane % 32];
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b)
                    acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[a], bf[b], acc[a][b], 0, 0, 0);
        }
        if (more) store(buf ^ 1);
        __syncthreads();
        buf ^= 1;
    }

    // Output layout of a 32 x 32 MFMA block: lane holds column lane % 32 and,
    // in register v, row 8 * (v / 4) + 4 * (lane / 32) + (v % 4).
    if constexpr (kSquare) {
        for (int pass = 0; pass < 2; ++pass) {
            if (wn == pass) {
#pragma unroll
                for (int a = 0; a < 2; ++a)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        double s = (double)(acc[a][0][v] * acc[a][0][v]) +
                                   (double)(acc[a][1][v] * acc[a][1][v]);
                        s = half_wave_reduce(s, SumOp());
                        if (lane % 32 == 0) {
                            const int r = wm * 64 + a * 32 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
                            sRow[r] = pass == 0 ? s : sRow[r] + s;
                        }
                    }
            }
            __syncthreads();
        }
        for (int r = t; r < kBM; r += kThreads) {
            const int64_t gr = row0 + r;
            if (gr < C) rowpart[(int64_t)blockIdx.x * C + gr] = sRow[r];
        }
    } else {
        // Y tile of this K range: ypart[split][row][col]
        float *yp = ypart + (int64_t)split * C * n;
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int64_t r = row0 + wm * 64 + a * 32 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
                    const int64_t c = col0 + wn * 64 + b * 32 + lane % 32;
                    if (r < C && c < n) yp[r * n + c] = acc[a][b][v];
                }
    }
}

__global__ void finish_rows_kernel(const double *__restrict__ rowpart, int64_t C, int ntiles,
                                   double inv_n, float *__restrict__ out)
{
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= C) return;
    double s = 0.0;
    for (int i = 0; i < ntiles; ++i) s += rowpart[(int64_t)i * C + k];
    out[k] = (float)(s * inv_n);
}

// one workgroup per row: sum the K-range tiles, square, sum over columns
__global__ void __launch_bounds__(256)
finish_split_kernel(const float *__restrict__ ypart, int64_t C, int64_t n, int splits,
                    double inv_n, float *__restrict__ out)
{
    __shared__ double red[256 / kWave];
    const int64_t k = blockIdx.x;
    double s = 0.0;
    for (int64_t c = threadIdx.x; c < n; c += 256) {
        float y = 0.0f;
        for (int sp = 0; sp < splits; ++sp) y += ypart[((int64_t)sp * C + k) * n + c];
        s += (double)y * (double)y;
    }
    s = block_reduce<256>(s, SumOp(), red);
    if (threadIdx.x == 0) out[k] = (float)(s * inv_n);
}

struct Plan {
    int64_t lda;       // padded row length of the scratch matrix
    int64_t ntiles_n;  // column tiles
    int64_t ntiles_m;  // row tiles
    int splits;
    int64_t kchunk;    // K per split (multiple of kBK)
};

Plan plan(int64_t C, int64_t d, int64_t n)
{
    Plan p;
    p.lda = (d + kBK - 1) / kBK * kBK;
    p.ntiles_n = (n + kBN - 1) / kBN;
    p.ntiles_m = (C + kBM - 1) / kBM;
    const int64_t tiles = p.ntiles_n * p.ntiles_m;
    const int64_t kslabs = p.lda / kBK;
    int64_t s = 1;
    // aim for >= 2 workgroups per CU (256 CUs) with >= 16 slabs of K each
    while (tiles * s < 512 && kslabs / (s * 2) >= 16) s *= 2;
    p.splits = (int)s;
    p.kchunk = (kslabs + s - 1) / s * kBK;
    return p;
}

}  // namespace

size_t err_scratch_bytes(int64_t C, int64_t d, int64_t n)
{
    const Plan p = plan(C, d, n);
    size_t a = sizeof(float) * (size_t)(C * p.lda);
    size_t part = p.splits == 1 ? sizeof(double) * (size_t)(p.ntiles_n * C)
                                : sizeof(float) * (size_t)(p.splits * C * n);
    return (a + 255) / 256 * 256 + part;
}

hipError_t launch_output_error(const float *W, const int8_t *codes, const float *scales,
                               const int32_t *counts, int64_t C, int64_t d, int P,
                               const float *X, int64_t n, float *err, float *ref,
                               void *scratch, hipStream_t s)
{
    const Plan p = plan(C, d, n);
    float *A = (float *)scratch;
    char *part = (char *)scratch + (sizeof(float) * (size_t)(C * p.lda) + 255) / 256 * 256;
    const bool vecx = (n % 4 == 0) && (((uintptr_t)X) % 16 == 0);
    const double inv_n = 1.0 / (double)n;
    for (int pass = 0; pass < (ref ? 2 : 1); ++pass) {
        const int use_points = pass == 0;
        float *out = pass == 0 ? err : ref;
        int64_t blocks = (C * p.lda + 255) / 256;
        if (blocks > 65536) blocks = 65536;
        hipLaunchKernelGGL(form_rows_kernel, dim3((unsigned)blocks), dim3(256), 0, s, W, codes,
                           scales, counts, C, d, p.lda, P, use_points, A);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        dim3 grid((unsigned)p.ntiles_n, (unsigned)p.ntiles_m, (unsigned)p.splits);
        if (p.splits == 1) {
            if (vecx)
                hipLaunchKernelGGL((gemm_kernel<true, true>), grid, dim3(kThreads), 0, s, A, p.lda, C,
                                   X, d, n, p.kchunk, (double *)part, (float *)nullptr);
            else
                hipLaunchKernelGGL((gemm_kernel<true, false>), grid, dim3(kThreads), 0, s, A, p.lda, C,
                                   X, d, n, p.kchunk, (double *)part, (float *)nullptr);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
            hipLaunchKernelGGL(finish_rows_kernel, dim3((unsigned)((C + 255) / 256)), dim3(256), 0, s,
                               (const double *)part, C, (int)p.ntiles_n, inv_n, out);
        } else {
            if (vecx)
                hipLaunchKernelGGL((gemm_kernel<false, true>), grid, dim3(kThreads), 0, s, A, p.lda, C,
                                   X, d, n, p.kchunk, (double *)nullptr, (float *)part);
            else
                hipLaunchKernelGGL((gemm_kernel<false, false>), grid, dim3(kThreads), 0, s, A, p.lda, C,
                                   X, d, n, p.kchunk, (double *)nullptr, (float *)part);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
            hipLaunchKernelGGL(finish_split_kernel, dim3((unsigned)C), dim3(256), 0, s,
                               (const float *)part, C, n, p.splits, inv_n, out);
        }
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace mpq
