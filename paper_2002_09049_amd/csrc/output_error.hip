// Output error of quantized layers on their calibration batches (Sec. 3.3,
// Eq. (12)): err[k] = (1/n) sum_t ((w_k - w~_k) . x_t)^2 and optionally
// ref[k] = (1/n) sum_t (w_k . x_t)^2.
//
// Up to kMaxErrLayers layers go through three launches together (their
// descriptors travel by value in the kernel arguments):
//  1. form: A[k][j] = fl32(w_kj - sum_i a_i q_ij) (fp64 sum in point order)
//     into a scratch matrix whose rows are padded to a multiple of 16 with
//     zeros (aligned float4 rows, no K tail).  HBM-bound, coalesced.  A ref
//     output is one more item of the group with A = W.
//  2. gemm: Y = A X on MFMA (v_mfma_f32_32x32x2f32, fp32 in and accumulate),
//     the path's one dense contraction.  A workgroup of four wavefronts owns a
//     128 x 128 tile of Y and one K range; each wavefront owns 64 x 64 as
//     2 x 2 MFMA blocks.  The K loop stages 16-deep slabs of A and X through
//     double-buffered LDS, loading the next slab into registers while the
//     MFMAs consume the current one.  The tiles of all layers form one grid,
//     longest first; a layer's K is split when it has too few tiles.
//       splits == 1: the epilogue squares Y and sums each row over the tile's
//         columns (fp64 cross-lane sums with DPP / ds_swizzle) -> one partial
//         per (column tile, row).
//       splits  > 1: the epilogue stores the fp32 Y tile of its K range.
//  3. finish: one workgroup per row: sum the row partials in tile order, or
//     sum the K-range tiles of every column, square, and sum over the columns
//     (fp64), in a fixed order.  Divide by n.
#include <algorithm>
#include <vector>

#include "internal.hpp"
#include "mpq.h"
#include "reduce.hpp"

namespace mpq {

namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kBM = 128, kBN = 128, kBK = 16;
constexpr int kThreads = 256;
constexpr int kPad = 4;  // LDS row padding (floats)
constexpr int kMaxErrLayers = 32;

struct ErrLayer {
    const float *W;
    const int8_t *codes;
    const float *scales;
    const int32_t *counts;
    const float *X;
    float *out;        // err or ref
    float *A;          // scratch [C][lda]
    void *part;        // scratch: double [ntn][C] (splits == 1) or float [splits][C][n]
    int C, d, n, lda;
    int ntm, ntn, splits, kchunk;
    int tile_begin;    // first gemm workgroup of this layer
    int row_begin;     // first finish workgroup of this layer
    int use_points;    // 1: A = residual (err), 0: A = W (ref)
};

struct ErrGroup {
    int n_layers;
    int P;
    int vecx;          // every X row start is 16-byte aligned and n % 4 == 0
    ErrLayer L[kMaxErrLayers];
};

__global__ void __launch_bounds__(256) form_rows_kernel(const ErrGroup g)
{
    const ErrLayer &L = g.L[blockIdx.y];
    const int64_t total = (int64_t)L.C * L.lda;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t k = e / L.lda, j = e - k * L.lda;
        float v = 0.0f;
        if (j < L.d) {
            double r = (double)L.W[k * L.d + j];
            if (L.use_points) {
                const int nk = min(max(L.counts[k], 0), g.P);  // clamp: counts is caller data
                const int8_t *q = L.codes + k * (int64_t)g.P * L.d + j;
                const float *a = L.scales + k * (int64_t)g.P;
                for (int i = 0; i < nk; ++i) r = fma(-(double)a[i], (double)q[(int64_t)i * L.d], r);
            }
            v = (float)r;
        }
        L.A[e] = v;
    }
}

template <bool kVecX>
__global__ void __launch_bounds__(kThreads) gemm_kernel(const ErrGroup g)
{
    __shared__ __align__(16) float sA[2][kBK][kBM + kPad];
    __shared__ __align__(16) float sX[2][kBK][kBN + kPad];
    __shared__ double sRow[kBM];

    int li = 0;
    while (li + 1 < g.n_layers && (int)blockIdx.x >= g.L[li + 1].tile_begin) ++li;
    const ErrLayer &L = g.L[li];
    const int local = (int)blockIdx.x - L.tile_begin;
    const int per_split = L.ntm * L.ntn;
    const int split = local / per_split;
    const int tm = (local % per_split) / L.ntn, tn = local % L.ntn;

    const int t = threadIdx.x;
    const int lane = t % kWave, wid = t / kWave;
    const int wm = wid / 2, wn = wid % 2;
    const int64_t C = L.C, n = L.n, d = L.d, lda = L.lda;
    const int64_t row0 = (int64_t)tm * kBM;
    const int64_t col0 = (int64_t)tn * kBN;
    const int64_t kbeg = (int64_t)split * L.kchunk;
    const int64_t kend = min(kbeg + (int64_t)L.kchunk, lda);
    const float *__restrict__ X = L.X;

    // staging roles
    const int arow = t / 2, ak0 = (t % 2) * 8;     // A: 8 consecutive k of one row
    const int64_t agrow = row0 + arow;
    const bool arow_ok = agrow < C;
    const float *ap = L.A + (arow_ok ? agrow : 0) * lda;
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
    if (L.splits == 1) {
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
        double *rowpart = (double *)L.part;
        for (int r = t; r < kBM; r += kThreads) {
            const int64_t gr = row0 + r;
            if (gr < C) rowpart[(int64_t)tn * C + gr] = sRow[r];
        }
    } else {
        // Y tile of this K range: ypart[split][row][col]
        float *yp = (float *)L.part + (int64_t)split * C * n;
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

// one workgroup per row of every layer
__global__ void __launch_bounds__(256) finish_kernel(const ErrGroup g)
{
    __shared__ double red[256 / kWave];
    int li = 0;
    while (li + 1 < g.n_layers && (int)blockIdx.x >= g.L[li + 1].row_begin) ++li;
    const ErrLayer &L = g.L[li];
    const int64_t k = (int64_t)blockIdx.x - L.row_begin;
    const int64_t C = L.C, n = L.n;
    double s = 0.0;
    if (L.splits == 1) {
        const double *rp = (const double *)L.part;
        if (threadIdx.x == 0)
            for (int i = 0; i < L.ntn; ++i) s += rp[(int64_t)i * C + k];
    } else {
        const float *yp = (const float *)L.part;
        for (int64_t c = threadIdx.x; c < n; c += 256) {
            float y = 0.0f;
            for (int sp = 0; sp < L.splits; ++sp) y += yp[((int64_t)sp * C + k) * n + c];
            s += (double)y * (double)y;
        }
    }
    s = block_reduce<256>(s, SumOp(), red);
    if (threadIdx.x == 0) L.out[k] = (float)(s / (double)n);
}

struct Item {
    const ErrLayerIn *in;
    int use_points;
};

struct Plan {
    int64_t lda, ntm, ntn, splits, kchunk;
    size_t a_bytes, part_bytes;
};

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

// err items for every layer, then ref items for the layers that want ref
std::vector<Item> items_of(const ErrLayerIn *in, int n_in)
{
    std::vector<Item> it;
    for (int i = 0; i < n_in; ++i)
        if (in[i].C > 0) it.push_back(Item{&in[i], 1});
    for (int i = 0; i < n_in; ++i)
        if (in[i].C > 0 && in[i].ref) it.push_back(Item{&in[i], 0});
    return it;
}

// K split of a layer: tiles of about work / 512 slabs (two per CU), at least
// 32 slabs.  It depends on the layer alone, so a layer's result does not
// depend on the other layers of the call.
std::vector<Plan> plan_group(const Item *it, int cnt)
{
    std::vector<Plan> p(cnt);
    for (int i = 0; i < cnt; ++i) {
        const ErrLayerIn &I = *it[i].in;
        Plan &q = p[i];
        q.lda = (I.d + kBK - 1) / kBK * kBK;
        q.ntm = (I.C + kBM - 1) / kBM;
        q.ntn = (I.n + kBN - 1) / kBN;
        const int64_t slabs = q.lda / kBK;
        const double work = (double)(q.ntm * q.ntn) * (double)slabs;
        const int64_t target = std::max<int64_t>(32, (int64_t)(work / 512.0 + 0.5));
        int64_t sp = (slabs + target / 2) / target;
        sp = std::max<int64_t>(1, std::min<int64_t>(sp, slabs));
        q.splits = sp;
        q.kchunk = (slabs + sp - 1) / sp * kBK;
        q.a_bytes = align256(sizeof(float) * (size_t)(I.C * q.lda));
        q.part_bytes = align256(sp == 1 ? sizeof(double) * (size_t)(q.ntn * I.C)
                                        : sizeof(float) * (size_t)(sp * I.C * I.n));
    }
    return p;
}

}  // namespace

size_t err_scratch_bytes(const ErrLayerIn *in, int n_in)
{
    const std::vector<Item> it = items_of(in, n_in);
    size_t total = 0;
    for (size_t base = 0; base < it.size(); base += kMaxErrLayers) {
        const int cnt = (int)std::min<size_t>(kMaxErrLayers, it.size() - base);
        std::vector<Plan> p = plan_group(it.data() + base, cnt);
        size_t b = 0;
        for (const Plan &q : p) b += q.a_bytes + q.part_bytes;
        total = std::max(total, b);
    }
    return total;
}

hipError_t launch_output_error(const ErrLayerIn *in, int n_in, int P, void *scratch, hipStream_t s)
{
    const std::vector<Item> it = items_of(in, n_in);
    for (size_t base = 0; base < it.size(); base += kMaxErrLayers) {
        const int cnt = (int)std::min<size_t>(kMaxErrLayers, it.size() - base);
        const Item *grp = it.data() + base;
        std::vector<Plan> p = plan_group(grp, cnt);
        // longest tiles first
        std::vector<int> order(cnt);
        for (int i = 0; i < cnt; ++i) order[i] = i;
        std::stable_sort(order.begin(), order.end(),
                         [&](int a, int b) { return p[a].kchunk > p[b].kchunk; });
        ErrGroup g;
        g.n_layers = cnt;
        g.P = P;
        g.vecx = 1;
        char *cur = (char *)scratch;
        int64_t tiles = 0, rows = 0, max_elems = 0;
        for (int o = 0; o < cnt; ++o) {
            const int i = order[o];
            const ErrLayerIn &I = *grp[i].in;
            const Plan &q = p[i];
            ErrLayer &L = g.L[o];
            L.W = I.W;
            L.codes = I.codes;
            L.scales = I.scales;
            L.counts = I.counts;
            L.X = I.X;
            L.out = grp[i].use_points ? I.err : I.ref;
            L.use_points = grp[i].use_points;
            L.A = (float *)cur;
            cur += q.a_bytes;
            L.part = cur;
            cur += q.part_bytes;
            L.C = (int)I.C;
            L.d = (int)I.d;
            L.n = (int)I.n;
            L.lda = (int)q.lda;
            L.ntm = (int)q.ntm;
            L.ntn = (int)q.ntn;
            L.splits = (int)q.splits;
            L.kchunk = (int)q.kchunk;
            L.tile_begin = (int)tiles;
            L.row_begin = (int)rows;
            tiles += q.ntm * q.ntn * q.splits;
            rows += I.C;
            max_elems = std::max<int64_t>(max_elems, I.C * q.lda);
            if (I.n % 4 != 0 || ((uintptr_t)I.X) % 16 != 0) g.vecx = 0;
        }
        const int64_t fblocks = std::min<int64_t>((max_elems + 255) / 256, 4096);
        hipLaunchKernelGGL(form_rows_kernel, dim3((unsigned)fblocks, (unsigned)cnt), dim3(256), 0, s, g);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        if (g.vecx)
            hipLaunchKernelGGL(gemm_kernel<true>, dim3((unsigned)tiles), dim3(kThreads), 0, s, g);
        else
            hipLaunchKernelGGL(gemm_kernel<false>, dim3((unsigned)tiles), dim3(kThreads), 0, s, g);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(finish_kernel, dim3((unsigned)rows), dim3(256), 0, s, g);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace mpq
