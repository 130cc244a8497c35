// Deployment arithmetic of Sec. 3.4: integer scales (Eq. (14)) and the
// multipoint layer's integer dot products (Eq. (15), Steps 1-3).
//
// integer_scales_kernel: A_i = nearest integer to 2^p a_i, ties to even
// (2^p a_i is exact in fp64), clamped to [-(2^31 - 1), 2^31 - 1] (clamped
// values counted), zero after a channel's count.
//
// int_forward_kernel: for channel k and column t of the batch (X [N][d],
// one signed int8 vector of d per column),
//   Step 1  z_i = q_i . x_t            (int8 MFMA, 32-bit accumulators)
//   Step 2  s   = sum_{i<n_k} A_i z_i   (64-bit, in registers)
//   Step 3  y   = s >> p                (arithmetic shift: floor(s / 2^p))
// A workgroup of four wavefronts owns 128 channels x 128 columns; for each
// point index i up to the largest count among its channels it runs the K
// loop of Step 1 (v_mfma_i32_32x32x16_i8 on 64-deep K slabs staged through
// double-buffered LDS) and folds the block of z_i into the 64-bit sums with
// the channels' A_i (zero for channels with fewer points).  Codes [C][P][d]
// and X [N][d] are both k-contiguous, so both operands are staged alike, as
// rows of 64 bytes; buffer loads return zeros past the rows and past d.
#include <stdio.h>

#include "internal.hpp"
#include "mpq.h"
#include "reduce.hpp"

namespace mpq {

namespace {

typedef int int32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int kIM = 128, kIN = 128, kIK = 64;   // tile and K slab (bytes)
constexpr int kIPad = 16;                       // LDS row: 80 bytes
constexpr int kIRow = kIK + kIPad;
constexpr int kIThreads = 256;
constexpr uint32_t kIOob = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

__global__ void integer_scales_kernel(const float *scales, const int32_t *counts, int64_t C, int P, int p,
                                      int32_t *A, unsigned long long *clamped)
{
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= C * P) return;
    const int64_t k = e / P;
    const int i = (int)(e - k * P);
    double v = 0.0;
    if (i < counts[k]) {
        v = rint(ldexp((double)scales[e], p));
        const double lim = 2147483647.0;
        if (v > lim || v < -lim) {
            v = v > 0.0 ? lim : -lim;
            if (clamped) atomicAdd(clamped, 1ull);
        }
    }
    A[e] = (int32_t)v;
}

// Load mode of the operands: 16-byte chunks (d % 16 == 0, rows 16-byte
// aligned), 4-byte words (d % 4 == 0, 4-byte aligned) or bytes.
enum { kLoad16 = 0, kLoad4 = 1, kLoad1 = 2 };

// One operand slab: rows r0 .. r0+127 of an int8 matrix whose row r starts
// at byte base + r * stride, bytes k0 .. k0+63 of each row (zeros past `rows`
// and past d).  Thread t stages the 16-byte pieces t and t + 256 (row =
// piece / 4, bytes 16 * (piece % 4) of the slab).
template <int kMode>
__device__ __forceinline__ void load_slab(__amdgpu_buffer_rsrc_t rs, int64_t rows, int64_t stride, int64_t base,
                                          int64_t d, int64_t r0, int64_t k0, i32x4 (&v)[2])
{
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int piece = (int)threadIdx.x + h * kIThreads;
        const int64_t r = r0 + piece / 4;
        const int64_t k = k0 + 16 * (piece % 4);
        const bool row_ok = r < rows;
        const int64_t at = base + r * stride + k;
        if constexpr (kMode == kLoad16) {
            const uint32_t o = (row_ok && k < d) ? (uint32_t)at : kIOob;
            v[h] = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, o, 0, 0));
        } else if constexpr (kMode == kLoad4) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const uint32_t o = (row_ok && k + 4 * w < d) ? (uint32_t)(at + 4 * w) : kIOob;
                v[h][w] = (int)__builtin_amdgcn_raw_buffer_load_b32(rs, o, 0, 0);
            }
        } else {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                uint32_t word = 0;
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const int64_t kk = 4 * w + b;
                    const uint32_t o = (row_ok && k + kk < d) ? (uint32_t)(at + kk) : kIOob;
                    word |= (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(rs, o, 0, 0) << (8 * b);
                }
                v[h][w] = (int)word;
            }
        }
    }
}

__device__ __forceinline__ void store_slab(int8_t (*s)[kIRow], const i32x4 (&v)[2])
{
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int piece = (int)threadIdx.x + h * kIThreads;
        *(i32x4 *)&s[piece / 4][16 * (piece % 4)] = v[h];
    }
}

template <int kMode>
__global__ void __launch_bounds__(kIThreads) int_forward_kernel(const IntGroup g)
{
    __shared__ __align__(16) int8_t sA[2][kIM][kIRow];
    __shared__ __align__(16) int8_t sB[2][kIN][kIRow];
    __shared__ int32_t s_coef[kIM];
    __shared__ int s_nmax;

    int li = 0;
    while (li + 1 < g.n_layers && (int)blockIdx.x >= g.L[li + 1].block_begin) ++li;
    const IntLayer &L = g.L[li];
    int tn = (int)blockIdx.x - L.block_begin, tm = 0;
    while (tn >= L.ntn) {
        tn -= L.ntn;
        ++tm;
    }
    const int P = g.P;
    const int64_t C = L.C, d = L.d, N = L.N;
    const int64_t row0 = (int64_t)tm * kIM, col0 = (int64_t)tn * kIN;
    const int t = threadIdx.x;
    const int lane = t % kWave, wid = t / kWave;
    const int wm = wid / 2, wn = wid % 2;

    // the largest count among this tile's channels (caller data: clamped to [0, P])
    if (t == 0) s_nmax = 0;
    __syncthreads();
    if (t < kIM && row0 + t < C) atomicMax(&s_nmax, min(max(L.counts[row0 + t], 0), P));
    __syncthreads();
    const int nmax = s_nmax;

    // point i of channel k: bytes (k * P + i) * d .. + d of the codes; column
    // t of the batch: bytes t * d .. + d of X (both below 2^31, checked on the host)
    const __amdgpu_buffer_rsrc_t rsA = rsrc(L.codes, (uint32_t)(C * P * d));
    const __amdgpu_buffer_rsrc_t rsB = rsrc(L.X, (uint32_t)(N * d));

    long long S[2][2][16];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) S[a][b][v] = 0;

    for (int i = 0; i < nmax; ++i) {
        // A_i of each channel of the tile, zero where the channel has fewer points
        if (t < kIM) {
            const int64_t r = row0 + t;
            s_coef[t] = (r < C && i < L.counts[r]) ? L.A[r * P + i] : 0;
        }
        int32x16 acc[2][2];
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[a][b][v] = 0;

        // Step 1: z_i for the tile, K slab by K slab
        i32x4 ra[2], rb[2];
        auto load = [&](int64_t k0) {
            load_slab<kMode>(rsA, C, (int64_t)P * d, (int64_t)i * d, d, row0, k0, ra);
            load_slab<kMode>(rsB, N, d, 0, d, col0, k0, rb);
        };
        int buf = 0;
        load(0);
        store_slab(sA[0], ra);
        store_slab(sB[0], rb);
        __syncthreads();   // also publishes s_coef
        for (int64_t k0 = 0; k0 < d; k0 += kIK) {
            const bool more = k0 + kIK < d;
            if (more) load(k0 + kIK);   // global loads in flight during the MFMAs
#pragma unroll
            for (int ks = 0; ks < kIK; ks += 16) {
                const int kk = ks + 8 * (lane / 32);
                long long av[2], bv[2];
#pragma unroll
                for (int a = 0; a < 2; ++a) av[a] = *(const long long *)&sA[buf][wm * 64 + a * 32 + lane % 32][kk];
#pragma unroll
                for (int b = 0; b < 2; ++b) bv[b] = *(const long long *)&sB[buf][wn * 64 + b * 32 + lane % 32][kk];
#pragma unroll
                for (int a = 0; a < 2; ++a)
#pragma unroll
                    for (int b = 0; b < 2; ++b)
                        acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x16_i8(av[a], bv[b], acc[a][b], 0, 0, 0);
            }
            if (more) {
                store_slab(sA[buf ^ 1], ra);
                store_slab(sB[buf ^ 1], rb);
            }
            __syncthreads();
            buf ^= 1;
        }
        // Step 2 for this point.  Output layout of a 32 x 32 block: lane
        // holds column lane % 32 and, in register v, row
        // 8 * (v / 4) + 4 * (lane / 32) + (v % 4).
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int r = wm * 64 + a * 32 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
                const long long c = (long long)s_coef[r];
#pragma unroll
                for (int b = 0; b < 2; ++b) S[a][b][v] += c * (long long)acc[a][b][v];
            }
        __syncthreads();   // s_coef is rewritten for the next point
    }

    // Step 3 and the store of Y [C][N]
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t r = row0 + wm * 64 + a * 32 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
                const int64_t c = col0 + wn * 64 + b * 32 + lane % 32;
                if (r < C && c < N) L.Y[r * N + c] = S[a][b][v] >> g.p;
            }
}

}  // namespace

hipError_t launch_integer_scales(const float *scales, const int32_t *counts, int64_t C, int P, int p,
                                 int32_t *A, unsigned long long *clamped, hipStream_t s)
{
    const int64_t n = C * P;
    if (n <= 0) return hipSuccess;
    if ((n + 255) / 256 > 0x7fffffffLL) return hipErrorInvalidValue;
    LaunchTimer timer(s, "integer_scales_kernel");
    hipLaunchKernelGGL(integer_scales_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, scales,
                       counts, C, P, p, A, clamped);
    return hipGetLastError();
}

hipError_t launch_int_forward(IntGroup &g, hipStream_t s)
{
    int64_t blocks = 0;
    int mode = kLoad16;
    for (int l = 0; l < g.n_layers; ++l) {
        IntLayer &L = g.L[l];
        L.ntn = (int)((L.N + kIN - 1) / kIN);
        L.block_begin = (int)blocks;
        blocks += (L.C + kIM - 1) / kIM * L.ntn;
        const bool a16 = ((uintptr_t)L.codes % 16 == 0) && ((uintptr_t)L.X % 16 == 0);
        const bool a4 = ((uintptr_t)L.codes % 4 == 0) && ((uintptr_t)L.X % 4 == 0);
        const int m = (L.d % 16 == 0 && a16) ? kLoad16 : (L.d % 4 == 0 && a4) ? kLoad4 : kLoad1;
        mode = m > mode ? m : mode;
    }
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    auto kern = mode == kLoad16 ? int_forward_kernel<kLoad16>
              : mode == kLoad4 ? int_forward_kernel<kLoad4> : int_forward_kernel<kLoad1>;
    const char *name = mode == kLoad16 ? "int_forward_kernel<16>"
                     : mode == kLoad4 ? "int_forward_kernel<4>" : "int_forward_kernel<1>";
    LaunchTimer timer(s, name);
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kIThreads), 0, s, g);
    return hipGetLastError();
}

}  // namespace mpq
