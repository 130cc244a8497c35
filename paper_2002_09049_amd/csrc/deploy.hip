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
//   Step 2  s   = sum_{i<n_k} A_i z_i   (64 bits)
//   Step 3  y   = s >> p                (arithmetic shift: floor(s / 2^p))
// The GEMM's rows are (channel, point) pairs: row k * Pp + i is point i of
// channel k, with Pp = max_points rounded up to a power of two, so a tile of
// 128 rows holds 128 / Pp whole channels.  A row past the channel's count
// (or past max_points) loads as zeros and adds nothing.  A workgroup of four
// wavefronts computes a 128 x 128 tile of z (v_mfma_i32_32x32x32_i8, 64-deep
// K slabs through double-buffered LDS); the epilogue puts the int32 tile in
// LDS and each thread forms Step 2 and 3 for (channel, column) pairs and
// writes Y [C][N] row-contiguously.  Codes [C][P][d] and X [N][d] are both
// k-contiguous, so both operands are staged alike, as rows of 64 bytes;
// buffer loads return zeros past the rows and past d.
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

// Row r of the A operand starts at byte rowoff[r] of the codes, or is
// absent (rowoff < 0: zeros); row r of B at byte r * d of X.
template <int kMode>
__device__ __forceinline__ void load_rows(__amdgpu_buffer_rsrc_t rs, const int *rowoff, int64_t d, int64_t k0,
                                          i32x4 (&v)[2])
{
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int piece = (int)threadIdx.x + h * kIThreads;
        const int ro = rowoff[piece / 4];
        const int64_t k = k0 + 16 * (piece % 4);
        const bool ok = ro >= 0;
        const int64_t at = (int64_t)ro + k;
        if constexpr (kMode == kLoad16) {
            v[h] = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                 rs, (ok && k < d) ? (uint32_t)at : kIOob, 0, 0));
        } else if constexpr (kMode == kLoad4) {
#pragma unroll
            for (int w = 0; w < 4; ++w)
                v[h][w] = (int)__builtin_amdgcn_raw_buffer_load_b32(
                    rs, (ok && k + 4 * w < d) ? (uint32_t)(at + 4 * w) : kIOob, 0, 0);
        } else {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                uint32_t word = 0;
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const int64_t kk = 4 * w + b;
                    word |= (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(
                                rs, (ok && k + kk < d) ? (uint32_t)(at + kk) : kIOob, 0, 0)
                            << (8 * b);
                }
                v[h][w] = (int)word;
            }
        }
    }
}

__device__ __forceinline__ void store_slab(int8_t *s, const i32x4 (&v)[2])
{
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int piece = (int)threadIdx.x + h * kIThreads;
        *(i32x4 *)(s + (piece / 4) * kIRow + 16 * (piece % 4)) = v[h];
    }
}

constexpr int kSlabBytes = kIM * kIRow;          // one operand, one buffer
constexpr int kZRow = 72;                        // int32 row of the z tile (bank spread)
constexpr int kLdsBytes = 4 * kSlabBytes;        // 2 operands x 2 buffers
static_assert(kIM * kZRow * 4 <= kLdsBytes, "the z tile reuses the staging LDS");

template <int kMode>
__global__ void __launch_bounds__(kIThreads) int_forward_kernel(const IntGroup g)
{
    __shared__ __align__(16) int8_t lds[kLdsBytes];
    __shared__ int s_offA[kIM], s_offB[kIN];
    __shared__ int32_t s_coef[kIM];

    const int li = last_at_most(g.n_layers, (int)blockIdx.x, [&](int i) { return g.L[i].block_begin; });
    const IntLayer &L = g.L[li];
    int tn = (int)blockIdx.x - L.block_begin, tm = 0;
    while (tn >= L.ntn) {
        tn -= L.ntn;
        ++tm;
    }
    const int P = g.P, lp = g.log2_pp, Pp = 1 << lp;
    const int64_t C = L.C, d = L.d, N = L.N;
    const int64_t row0 = (int64_t)tm * kIM, col0 = (int64_t)tn * kIN;
    const int t = threadIdx.x;
    const int lane = t % kWave, wid = t / kWave;
    const int wm = wid / 2, wn = wid % 2;

    // rows of this tile: point i of channel k (or absent) and its A_i
    if (t < kIM) {
        const int64_t r = row0 + t, k = r >> lp;
        const int i = (int)(r & (Pp - 1));
        const bool ok = k < C && i < P && i < L.counts[k];
        s_offA[t] = ok ? (int)((k * P + i) * d) : -1;   // codes below 2^31 bytes (host check)
        s_coef[t] = ok ? L.A[k * P + i] : 0;
    } else {
        const int64_t c = col0 + (t - kIM);
        s_offB[t - kIM] = c < N ? (int)(c * d) : -1;    // X below 2^31 bytes (host check)
    }
    const __amdgpu_buffer_rsrc_t rsA = rsrc(L.codes, (uint32_t)(C * P * d));
    const __amdgpu_buffer_rsrc_t rsB = rsrc(L.X, (uint32_t)(N * d));
    __syncthreads();

    int32x16 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[a][b][v] = 0;

    // Step 1: the tile of z, K slab by K slab
    auto sA = [&](int b) { return lds + b * kSlabBytes; };
    auto sB = [&](int b) { return lds + (2 + b) * kSlabBytes; };
    i32x4 ra[2], rb[2];
    int buf = 0;
    load_rows<kMode>(rsA, s_offA, d, 0, ra);
    load_rows<kMode>(rsB, s_offB, d, 0, rb);
    store_slab(sA(0), ra);
    store_slab(sB(0), rb);
    __syncthreads();
    for (int64_t k0 = 0; k0 < d; k0 += kIK) {
        const bool more = k0 + kIK < d;
        if (more) {   // global loads in flight during the MFMAs
            load_rows<kMode>(rsA, s_offA, d, k0 + kIK, ra);
            load_rows<kMode>(rsB, s_offB, d, k0 + kIK, rb);
        }
        // v_mfma_i32_32x32x32_i8: lane l supplies row (or column) l % 32,
        // bytes 16 * (l / 32) .. +15 of the 32-deep K step
#pragma unroll
        for (int ks = 0; ks < kIK; ks += 32) {
            const int kk = ks + 16 * (lane / 32);
            i32x4 av[2], bv[2];
#pragma unroll
            for (int a = 0; a < 2; ++a)
                av[a] = *(const i32x4 *)(sA(buf) + (wm * 64 + a * 32 + lane % 32) * kIRow + kk);
#pragma unroll
            for (int b = 0; b < 2; ++b)
                bv[b] = *(const i32x4 *)(sB(buf) + (wn * 64 + b * 32 + lane % 32) * kIRow + kk);
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b)
                    acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(av[a], bv[b], acc[a][b], 0, 0, 0);
        }
        if (more) {
            store_slab(sA(buf ^ 1), ra);
            store_slab(sB(buf ^ 1), rb);
        }
        __syncthreads();
        buf ^= 1;
    }

    // Steps 2 and 3, one half of the columns at a time: the waves of that
    // half put their z blocks in LDS (lane holds column lane % 32 and, in
    // register v, row 8 * (v / 4) + 4 * (lane / 32) + (v % 4) of a 32 x 32
    // block), then every thread sums A_i z_i over the rows of a channel
    int32_t *Z = (int32_t *)lds;   // [kIM][kZRow], columns 0..63 of the half
    const int cpt = kIM >> lp;     // channels per tile
    for (int half = 0; half < 2; ++half) {
        if (wn == half) {
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int r = wm * 64 + a * 32 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
                        Z[r * kZRow + b * 32 + lane % 32] = acc[a][b][v];
                    }
        }
        __syncthreads();
        for (int e = t; e < cpt * 64; e += kIThreads) {
            const int kk = e / 64, c = e % 64;
            const int64_t k = (row0 >> lp) + kk, col = col0 + half * 64 + c;
            long long sum = 0;
            for (int i = 0; i < Pp; ++i) {
                const int r = kk * Pp + i;
                sum += (long long)s_coef[r] * (long long)Z[r * kZRow + c];
            }
            if (k < C && col < N) L.Y[k * N + col] = sum >> g.p;
        }
        __syncthreads();
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

int int_forward_mode(const IntLayer &L)
{
    const bool a16 = ((uintptr_t)L.codes % 16 == 0) && ((uintptr_t)L.X % 16 == 0);
    const bool a4 = ((uintptr_t)L.codes % 4 == 0) && ((uintptr_t)L.X % 4 == 0);
    return (L.d % 16 == 0 && a16) ? kLoad16 : (L.d % 4 == 0 && a4) ? kLoad4 : kLoad1;
}

hipError_t launch_int_forward(IntGroup &h, int mode, hipStream_t s)
{
    int lp = 0;
    while ((1 << lp) < h.P) ++lp;
    h.log2_pp = lp;
    int64_t blocks = 0;
    for (int l = 0; l < h.n_layers; ++l) {
        IntLayer &L = h.L[l];
        if (int_forward_mode(L) != mode) return hipErrorInvalidValue;
        L.ntn = (int)((L.N + kIN - 1) / kIN);
        L.block_begin = (int)blocks;
        blocks += ((L.C << lp) + kIM - 1) / kIM * L.ntn;
    }
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    auto kern = mode == kLoad16 ? int_forward_kernel<kLoad16>
              : mode == kLoad4 ? int_forward_kernel<kLoad4> : int_forward_kernel<kLoad1>;
    const char *name = mode == kLoad16 ? "int_forward_kernel<16>"
                     : mode == kLoad4 ? "int_forward_kernel<4>" : "int_forward_kernel<1>";
    LaunchTimer timer(s, name);
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kIThreads), 0, s, h);
    return hipGetLastError();
}

}  // namespace mpq
