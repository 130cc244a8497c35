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
// A workgroup of four wavefronts owns 32 channels by 128 columns.  The GEMM's
// rows are point-major: row block i (32 rows) holds point i of the 32
// channels, and the points run in chunks of kPts = 4 only up to the
// largest count among the tile's channels, so points
// that no channel of the tile has are neither loaded nor multiplied; a row
// past its channel's count loads as zeros and adds nothing.  Wavefront w
// multiplies every row block by its 32 columns (v_mfma_i32_32x32x32_i8,
// 128-byte K slabs through double-buffered LDS), so a lane holds, for one
// column, z of every point of the 16 channels it covers: Step 2 and 3 run
// in its registers (no exchange), and each store writes a column run of
// two channels' rows of Y [C][N].  Codes [C][P][d] and X [N][d] are both
// k-contiguous, so both operands are staged alike, as rows of 128 bytes;
// buffer loads return zeros past the rows and past d.
#include <stdio.h>

#include <algorithm>

#include "internal.hpp"
#include "mpq.h"
#include "reduce.hpp"

namespace mpq {

namespace {

typedef int int32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int kICh = 32, kIN = 128, kIK = 128; // channels and columns of a tile; K slab (bytes)
constexpr int kIPieces = kIK / 16;             // 16-byte pieces of a slab row
constexpr int kIPad = 16;                       // LDS row: 80 bytes
constexpr int kIRow = kIK + kIPad;
constexpr int kIThreads = 256;
constexpr uint32_t kIOob = 0x80000000u;
constexpr int kIXcds = 8;                       // MI355X: workgroups are dealt to 8 XCDs in turn

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
// aligned), 4-byte words (d % 4 == 0, 4-byte aligned) or bytes (aligned
// dwords shifted into place when the buffer's base is 4-byte aligned).
enum { kLoad16 = 0, kLoad4 = 1, kLoad1 = 2 };

// kRows rows of kIK bytes from K offset k0, kIPieces 16-byte pieces a row,
// kRows kIPieces / kIThreads pieces per thread.  Row r starts at byte rowoff[r] of the buffer, or
// is absent (rowoff < 0, or r >= live: zeros, nothing loaded).  words: in
// bytes mode, the bytes of the buffer that aligned dwords may serve (0 when
// its base is not 4-byte aligned; a dword that reaches past the buffer's
// end loads as zero, so the last bytes go one by one).
template <int kMode, int kRows>
__device__ __forceinline__ void load_rows(__amdgpu_buffer_rsrc_t rs, const int *rowoff, int live, int64_t d,
                                          int64_t k0, int64_t words, i32x4 (&v)[kRows * kIPieces / kIThreads])
{
#pragma unroll
    for (int h = 0; h < kRows * kIPieces / kIThreads; ++h) {
        const int piece = (int)threadIdx.x + h * kIThreads;
        const int row = piece / kIPieces;
        const int ro = row < live ? rowoff[row] : -1;
        const int64_t k = k0 + 16 * (piece % kIPieces);
        const bool ok = ro >= 0;
        const int64_t at = (int64_t)ro + k;
        if (!ok) {
            v[h] = i32x4{0, 0, 0, 0};
        } else if constexpr (kMode == kLoad16) {
            v[h] = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                 rs, k < d ? (uint32_t)at : kIOob, 0, 0));
        } else if constexpr (kMode == kLoad4) {
#pragma unroll
            for (int w = 0; w < 4; ++w)
                v[h][w] = (int)__builtin_amdgcn_raw_buffer_load_b32(
                    rs, k + 4 * w < d ? (uint32_t)(at + 4 * w) : kIOob, 0, 0);
        } else if ((at & ~(int64_t)3) + 20 <= words) {
            // the five aligned dwords around the 16 bytes (those wholly at
            // or past d not loaded), funnel-shifted into place; the bytes at
            // or past d zeroed
            const int sh = (int)(at & 3);
            const int64_t a0 = at - sh;
            uint32_t wd[5];
#pragma unroll
            for (int q = 0; q < 5; ++q)
                wd[q] = __builtin_amdgcn_raw_buffer_load_b32(
                    rs, k - sh + 4 * q < d ? (uint32_t)(a0 + 4 * q) : kIOob, 0, 0);
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                uint32_t word = __builtin_amdgcn_alignbyte(wd[w + 1], wd[w], (uint32_t)sh);
                const int64_t left = d - (k + 4 * w);   // bytes of the word before d
                if (left < 4) word = left <= 0 ? 0u : word & ((1u << (8 * (int)left)) - 1u);
                v[h][w] = (int)word;
            }
        } else {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                uint32_t word = 0;
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const int64_t kk = 4 * w + b;
                    word |= (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(
                                rs, k + kk < d ? (uint32_t)(at + kk) : kIOob, 0, 0)
                            << (8 * b);
                }
                v[h][w] = (int)word;
            }
        }
    }
}

template <int kRows>
__device__ __forceinline__ void store_slab(int8_t *s, const i32x4 (&v)[kRows * kIPieces / kIThreads])
{
#pragma unroll
    for (int h = 0; h < kRows * kIPieces / kIThreads; ++h) {
        const int piece = (int)threadIdx.x + h * kIThreads;
        *(i32x4 *)(s + (piece / kIPieces) * kIRow + 16 * (piece % kIPieces)) = v[h];
    }
}

// Step 1 for one chunk of kN live points (row blocks 0 .. kN - 1 of the A
// slab): z of the wavefront's 32 columns, K slab by K slab, into acc, and
// Step 2's terms added to the lane's 64-bit sums.  The point count is a
// template argument so that the LDS reads of a K step are issued ahead of
// its MFMAs.
template <int kMode, int kPts, int kN>
__device__ __forceinline__ void chunk_sums(__amdgpu_buffer_rsrc_t rsA, __amdgpu_buffer_rsrc_t rsB,
                                           int64_t wordsA, int64_t wordsB,
                                           const int *s_offA, const int *s_offB, const int32_t *s_coef,
                                           int8_t (*ldsA)[kPts * kICh * kIRow], int8_t (*ldsB)[kIN * kIRow],
                                           int64_t d, long long (&sum)[16])
{
    constexpr int kARows = kPts * kICh;
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    int32x16 acc[kN];
#pragma unroll
    for (int i = 0; i < kN; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][v] = 0;
    i32x4 ra[kARows * kIPieces / kIThreads], rb[kIN * kIPieces / kIThreads];
    int buf = 0;
    load_rows<kMode, kARows>(rsA, s_offA, kN * kICh, d, 0, wordsA, ra);
    load_rows<kMode, kIN>(rsB, s_offB, kIN, d, 0, wordsB, rb);
    store_slab<kARows>(ldsA[0], ra);
    store_slab<kIN>(ldsB[0], rb);
    __syncthreads();
    for (int64_t k0 = 0; k0 < d; k0 += kIK) {
        const bool more = k0 + kIK < d;
        if (more) {   // global loads in flight during the MFMAs
            load_rows<kMode, kARows>(rsA, s_offA, kN * kICh, d, k0 + kIK, wordsA, ra);
            load_rows<kMode, kIN>(rsB, s_offB, kIN, d, k0 + kIK, wordsB, rb);
        }
        // v_mfma_i32_32x32x32_i8: lane l supplies row (or column) l % 32,
        // bytes 16 * (l / 32) .. +15 of the 32-deep K step
#pragma unroll
        for (int ks = 0; ks < kIK; ks += 32) {
            const int kk = ks + 16 * (lane / 32);
            const i32x4 bv = *(const i32x4 *)(ldsB[buf] + (wid * 32 + lane % 32) * kIRow + kk);
            i32x4 av[kN];
#pragma unroll
            for (int i = 0; i < kN; ++i) av[i] = *(const i32x4 *)(ldsA[buf] + (i * kICh + lane % 32) * kIRow + kk);
#pragma unroll
            for (int i = 0; i < kN; ++i) acc[i] = __builtin_amdgcn_mfma_i32_32x32x32_i8(av[i], bv, acc[i], 0, 0, 0);
        }
        if (more) {
            store_slab<kARows>(ldsA[buf ^ 1], ra);
            store_slab<kIN>(ldsB[buf ^ 1], rb);
        }
        __syncthreads();
        buf ^= 1;
    }
    // Step 2 for the chunk's points, in the lane's registers
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const int ch = 8 * (v / 4) + 4 * (lane / 32) + v % 4;
#pragma unroll
        for (int i = 0; i < kN; ++i) sum[v] += (long long)s_coef[i * kICh + ch] * (long long)acc[i][v];
        // one channel's terms at a time (hoisting every coefficient read
        // ahead would hold them all in registers)
        __builtin_amdgcn_sched_barrier(0);
    }
}

template <int kMode, int kPts>
__global__ void __launch_bounds__(kIThreads) int_forward_kernel(const IntGroup g)
{
    constexpr int kARows = kPts * kICh;   // rows of a chunk's A slab
    __shared__ __align__(16) int8_t ldsA[2][kARows * kIRow];
    __shared__ __align__(16) int8_t ldsB[2][kIN * kIRow];
    __shared__ int s_offA[kARows], s_offB[kIN];
    __shared__ int32_t s_coef[kARows];
    __shared__ int s_imax;

    const int li = last_at_most(g.n_layers, (int)blockIdx.x, [&](int i) { return g.L[i].block_begin; });
    const IntLayer &L = g.L[li];
    // XCD-contiguous tiles: block_begin is a multiple of kIXcds, so b % kIXcds
    // is the XCD this block runs on.  Each XCD takes a contiguous run of the
    // layer's tiles, row tiles fastest, so the row tiles that read one
    // column tile of X run together under one L2.
    const int b = (int)blockIdx.x - L.block_begin;
    const int T = L.ntm * L.ntn;
    const int xcd = b % kIXcds, slot = b / kIXcds;
    const int q = T / kIXcds, rem = T % kIXcds;
    if (slot >= q + (xcd < rem ? 1 : 0)) return;   // padding block
    const int tile = xcd * q + (xcd < rem ? xcd : rem) + slot;
    const int tn = tile / L.ntm, tm = tile - tn * L.ntm;
    const int P = g.P;
    const int64_t C = L.C, d = L.d, N = L.N;
    const int64_t ch0 = (int64_t)tm * kICh, col0 = (int64_t)tn * kIN;
    const int t = threadIdx.x;
    const int lane = t % kWave, wid = t / kWave;   // wavefront wid: columns 32 wid ..

    // the columns of the tile, and the largest point count of its channels
    if (t < kIN) {
        const int64_t c = col0 + t;
        s_offB[t] = c < N ? (int)(c * d) : -1;    // X below 2^31 bytes (host check)
    }
    if (t < kWave) {
        const int64_t k = ch0 + t;
        int n = (t < kICh && k < C) ? L.counts[k] : 0;
        n = wave_reduce(n, MaxOp());
        if (t == 0) s_imax = n < P ? n : P;
    }
    const __amdgpu_buffer_rsrc_t rsA = rsrc(L.codes, (uint32_t)(C * P * d));
    const __amdgpu_buffer_rsrc_t rsB = rsrc(L.X, (uint32_t)(N * d));
    const int64_t wordsA = ((uintptr_t)L.codes & 3) == 0 ? C * P * d : 0;
    const int64_t wordsB = ((uintptr_t)L.X & 3) == 0 ? N * d : 0;
    __syncthreads();
    const int imax = s_imax;

    // lane: column col0 + 32 wid + lane % 32; in register v of a 32 x 32
    // block, row (channel of the tile) 8 (v / 4) + 4 (lane / 32) + v % 4
    long long sum[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) sum[v] = 0;
    for (int p0 = 0; p0 < imax; p0 += kPts) {
        // rows of the chunk: point p0 + r / 32 of channel ch0 + r % 32
        for (int r = t; r < kARows; r += kIThreads) {
            const int64_t k = ch0 + r % kICh;
            const int i = p0 + r / kICh;
            const bool ok = k < C && i < P && i < L.counts[k];
            s_offA[r] = ok ? (int)((k * P + i) * d) : -1;   // codes below 2^31 bytes (host check)
            s_coef[r] = ok ? L.A[k * P + i] : 0;
        }
        __syncthreads();
        const int npts = imax - p0 < kPts ? imax - p0 : kPts;   // uniform
        switch (npts) {
#define MPQ_CHUNK(n) \
    case n: if constexpr (n <= kPts) chunk_sums<kMode, kPts, n>(rsA, rsB, wordsA, wordsB, s_offA, s_offB, s_coef, ldsA, ldsB, d, sum); break;
            MPQ_CHUNK(1) MPQ_CHUNK(2) MPQ_CHUNK(3) MPQ_CHUNK(4)
            MPQ_CHUNK(5) MPQ_CHUNK(6) MPQ_CHUNK(7) MPQ_CHUNK(8)
#undef MPQ_CHUNK
        default: break;
        }
        __syncthreads();   // the next chunk rewrites s_offA and s_coef
    }

    // Step 3 and the stores: a store writes two 32-column runs of Y rows
    const int64_t col = col0 + wid * 32 + lane % 32;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const int64_t k = ch0 + 8 * (v / 4) + 4 * (lane / 32) + v % 4;
        if (k < C && col < N) L.Y[k * N + col] = sum[v] >> g.p;
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
    // longest K first: a long layer's tiles start before the short ones that
    // fill in beside them (the layers are independent)
    std::stable_sort(h.L, h.L + h.n_layers, [](const IntLayer &a, const IntLayer &b) { return a.d > b.d; });
    int64_t blocks = 0;
    for (int l = 0; l < h.n_layers; ++l) {
        IntLayer &L = h.L[l];
        if (int_forward_mode(L) != mode) return hipErrorInvalidValue;
        L.ntn = (int)((L.N + kIN - 1) / kIN);
        L.ntm = (int)((L.C + kICh - 1) / kICh);
        L.block_begin = (int)blocks;   // a multiple of kIXcds
        const int64_t tiles = (int64_t)L.ntm * L.ntn;
        if (tiles > 0x7fffffffLL) return hipErrorInvalidValue;
        blocks += (tiles + kIXcds - 1) / kIXcds * kIXcds;
    }
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    // chunks of four points (eight per chunk held a workgroup to one per CU,
    // 113 KB of LDS: ResNet-50's step took 0.81 ms against 0.60 ms)
    auto kern = mode == kLoad16 ? int_forward_kernel<kLoad16, 4>
              : mode == kLoad4  ? int_forward_kernel<kLoad4, 4> : int_forward_kernel<kLoad1, 4>;
    const char *name = mode == kLoad16 ? "int_forward_kernel<16>"
                     : mode == kLoad4 ? "int_forward_kernel<4>" : "int_forward_kernel<1>";
    LaunchTimer timer(s, name);
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kIThreads), 0, s, h);
    return hipGetLastError();
}

}  // namespace mpq
