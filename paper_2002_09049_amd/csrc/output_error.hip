// Output error of quantized layers on their calibration batches (Sec. 3.3,
// Eq. (12)): err[k] = (1/n) sum_t ((w_k - w~_k) . x_t)^2 and optionally
// ref[k] = (1/n) sum_t (w_k . x_t)^2.
//
// All layers of a call (items: an err item per layer, a ref item per layer
// that asks for ref; up to kMaxErrItems) go through three launches together.
// Their descriptors sit in a table at the head of the call's scratch, filled
// by small upload kernels that carry kDescChunk descriptors each in their
// kernel arguments (stream-ordered, so no host buffer outlives the call);
// each workgroup finds its item by a binary search of the table:
//
//  1. form (HBM-bound): D[k][j] = fl32(w_kj - sum_{i<n_k} a_i q_ij), the fp64
//     sum in point order (D = W for a ref item), one float4 of a row per
//     thread.  D is stored as tiles of kBM rows by kBK k (row-major inside,
//     k past d zero), so a row is written in 128-byte pieces and a GEMM
//     slab of a row tile is one contiguous block.  Items whose rows the fit
//     already wrote (d_ready) are not formed.
//
//  2. gemm: Y = D X, the path's one dense contraction, in fp32 from bf16
//     matrix products: each fp32 operand is split into three bf16 pieces
//     (hi + mid + lo, exact) and six of the nine piece products are summed
//     by v_mfma_f32_32x32x16_bf16 with fp32 accumulation (the three left
//     out lie below one rounding of the fp32 product).  A workgroup owns a
//     128 x 128 tile of Y and one K range, with eight wavefronts: four
//     multiply (64 x 64 each, as 2 x 2 MFMA blocks) and four stage.  The
//     staging ones load a 16-k slab of D (a half of a tile block's rows) and
//     of X (16 rows of 128 samples) four slabs ahead into a ring of
//     registers, split it once into bf16 piece tiles (k contiguous per row
//     of D and per column of X) and store it to one of two LDS buffers
//     while the multiplying ones read the other: one barrier per slab
//     (buffer loads: offsets past a range read as zeros).  Two workgroups
//     per CU cover each other's start and end.  The epilogue squares Y
//     (fp64) and sums each row over the tile's columns into a partial per
//     (column tile, row); a layer whose K is split (to balance a grid of
//     long and short K ranges) stores its fp32 Y tiles per K range instead.
//
// An err item may be restricted to a device list of channels (rows of D =
// the listed channels, in list order; the list length is read by each
// kernel, and workgroups past it return at once), with the result of row m
// written to err[rows[m] * stride].  A row's result does not depend on its
// position, so the list order does not matter.
//
//  3. finish: per row, the partials summed in column-tile order, or the K
//     ranges of Y summed in range order, squared and summed over the columns;
//     divided by n.  Every order is fixed, so results are deterministic.  The
//     kernel boundary publishes the partials (no cross-workgroup handshake:
//     agent-scope fences would write back and invalidate the L2 the GEMM
//     relies on).
//
// The tiles of all layers form one grid, longest K range first.  Workgroups
// are dealt to the 8 XCDs in turn, so within a layer the tiles are
// renumbered to give each XCD a contiguous run (rows of D and columns of X
// reused by neighbouring tiles stay in one L2), and a layer's tiles % 8
// spare tiles go to the XCDs after those that took the previous layer's.
// Tile coordinates come from uniform subtraction loops, not divisions, so
// they and the buffer resources built from them stay in scalar registers.
#include <algorithm>
#include <vector>

#include "internal.hpp"
#include "mpq.h"
#include "reduce.hpp"

namespace mpq {

namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kBM = 128, kBN = 128, kBK = 32;
constexpr int kRangeK = 768;      // K of a split layer's K range, about
constexpr int kMinSlabs = 4;      // shortest K range (slabs) of a listed layer's live rows
constexpr int kThreads = 512;   // GEMM workgroup: four wavefronts multiply (64 x 64 of the tile each), four stage
constexpr int kStageT = 256;    // threads of the staging wavefronts
constexpr int kPieces = 3;      // bf16 pieces of an fp32 operand
constexpr int kSlabK = 16;      // k per staged slab (one 16-k MFMA step)
constexpr int kRowK = kSlabK + 8;   // LDS row of a piece: 16 bf16 and 16 bytes of padding (48 bytes)
constexpr int kRing = 4;        // staging register sets: loads run four slabs ahead
constexpr int kMaxErrItems = 1024;   // items (err and ref) per launch group
constexpr int kDescChunk = 20;       // descriptors per upload kernel
constexpr int kXcds = 8;         // MI355X: workgroups are dealt to 8 XCDs in turn
constexpr int kFormThreads = 256;
constexpr int kFinRows = 256 / kWave;   // finish: rows of a split layer per workgroup

// Raw buffer resource (gfx9 descriptor word 3: 32-bit dwords, no swizzle).
// Loads at offsets >= num_records return zeros; kOob is past every range.
constexpr uint32_t kOob = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t num_records)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)num_records,
                                             0x00020000);
}
__device__ __forceinline__ f32x4 load4(__amdgpu_buffer_rsrc_t r, uint32_t off)
{
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

struct ErrLayer {
    const float *W;
    const int8_t *codes;
    const float *scales;
    const int32_t *counts;
    const float *X;
    float *out;          // err or ref
    float *D;            // tiles [ntm][nkb][kBM][kBK] of the rows; k past d zero
    double *rowpart;     // [ntn][C]
    float *ypart;        // [splits][rows][n] (a split layer's K ranges of Y)
    const int32_t *rows; // nullptr, or the channels of rows 0 .. *nrows of D
    const int32_t *nrows;
    const float *cand;   // use_points == 2: [C / Gc][Gc] candidate scales (C counts rows of D)
    const float *offsets;   // use_points == 1: per-channel offsets (reading B2) or nullptr
    int64_t stride;      // out[channel * stride]
    int C, d, n, nkb;    // nkb = ceil(d / kBK)
    int ntm, ntn, splits, kchunk;
    int tiles;           // gemm workgroups: ntm * ntn * splits, more for a listed layer
    int block_begin;     // first gemm workgroup (a multiple of kXcds)
    int extra_begin;     // first of the workgroups past the plan's tiles (a multiple of kXcds)
    int xoff;            // XCD rank offset: the layer's spare tiles go to XCDs xoff, xoff + 1, ...
    int form_begin;      // first form workgroup
    int fin_begin;       // first finish workgroup
    int use_points;      // 1: D = residual (err), 0: D = W (ref), 2: D = clipping candidates
    int Gc, M;
    int vecw;            // d % 4 == 0, W 16-byte and codes 4-byte aligned
};

struct ErrGroup {
    int n_layers;
    int P;
    int extra_start;     // gemm workgroups past every layer's planned tiles start here
    int vecx;            // n % 4 == 0 and every X 16-byte aligned
};

// kDescChunk descriptors for the table (kernel arguments of one upload)
struct DescChunk {
    ErrLayer *dst;
    int count;
    ErrLayer L[kDescChunk];
};
static_assert(sizeof(DescChunk) <= 4096, "kernel arguments");
static_assert(sizeof(ErrLayer) % 4 == 0, "copied as 32-bit words");

__global__ void __launch_bounds__(64) desc_upload_kernel(const DescChunk c)
{
    constexpr int kWords = (int)(sizeof(ErrLayer) / 4);
    const uint32_t *src = (const uint32_t *)c.L;
    uint32_t *dst = (uint32_t *)c.dst;
    for (int i = threadIdx.x; i < c.count * kWords; i += 64) dst[i] = src[i];
}

// The K split of the live rows 0 .. nact of D.  A layer's full rows take the
// host's plan.  When a listed layer scores fewer rows (the later steps of the
// calibration rule), its workgroups take shorter K ranges (at least
// kMinSlabs slabs), so the few live rows still spread over the layer's
// workgroups.  The split depends on the layer and nact alone; the GEMM and
// the finish kernel derive it alike.
struct LiveSplit {
    int ntm, splits, kchunk;
};
__device__ __forceinline__ LiveSplit live_split(const ErrLayer &L, int64_t nact)
{
    const int ntm = (int)((nact + kBM - 1) / kBM);
    if (!L.rows || nact >= L.C) return LiveSplit{L.ntm, L.splits, L.kchunk};
    if (ntm == 0) return LiveSplit{0, 1, L.kchunk};
    const int slabs = (L.d + kBK - 1) / kBK;
    const int s = max(1, min(L.tiles / (ntm * L.ntn), slabs / kMinSlabs));
    const int kch = min((slabs + s - 1) / s * kBK, L.kchunk);   // never above the plan's
    return LiveSplit{ntm, (L.d + kch - 1) / kch, kch};
}

__device__ __forceinline__ double int8_of(uint32_t w, int u)
{
    return (double)(int)(int8_t)(uint8_t)(w >> (8 * u));
}

// Float index in D of row m, k (a multiple of 4 for a float4): tiles of
// kBM rows by kBK k, row-major inside, so a GEMM slab of a row tile is one
// contiguous block and a row's kBK consecutive k are 128 contiguous bytes.
__device__ __forceinline__ int64_t d_index(int64_t m, int64_t k, int nkb)
{
    return ((m / kBM) * nkb + k / kBK) * (kBM * kBK) + (m % kBM) * kBK + k % kBK;
}

// ---- 1. form: rows of D, four consecutive k (one float4) per thread, k
// past d written as zeros
__global__ void __launch_bounds__(kFormThreads) form_d_kernel(const ErrGroup g,
                                                              const ErrLayer *__restrict__ Ls)
{
    const int li = last_at_most(g.n_layers, (int)blockIdx.x, [&](int i) { return Ls[i].form_begin; });
    const ErrLayer &L = Ls[li];
    const int P = g.P;
    const int64_t d = L.d, C = L.C, q4 = (int64_t)L.nkb * (kBK / 4);
    const int64_t e = (int64_t)((int)blockIdx.x - L.form_begin) * kFormThreads + threadIdx.x;
    const int64_t m = e / q4, k = (e - m * q4) * 4;
    const int64_t nact = L.rows ? (int64_t)*L.nrows : C;
    if (m >= nact) return;   // rows past the list feed only output rows nobody reads
    double r[4] = {0.0, 0.0, 0.0, 0.0};
    if (L.use_points == 2) {
        // clipping candidate j of channel ch: w - a [w / a]_Q (Eq. (10)'s
        // rounding of the fp64 quotient, formed only near a half-integer)
        const int64_t ch = m / L.Gc;
        const double a = (double)L.cand[m];
        const double ia = 1.0 / a, Md = (double)L.M;
        const float *wr = L.W + ch * d;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            if (k + u < d) {
                const double wj = (double)wr[k + u];
                double c = 0.0;
                if (a != 0.0) {
                    const double y = wj * ia;
                    c = rint(y);
                    if (fabs(fabs(y - c) - 0.5) < 0x1p-40) c = rint(wj / a);
                    c = fmin(fmax(c, -Md), Md);
                }
                r[u] = fma(-a, c, wj);
            }
        }
    } else {
        const int64_t row = L.rows ? (int64_t)L.rows[m] : m;
        const int nk = L.use_points ? min(max(L.counts[row], 0), P) : 0;  // counts is caller data
        const double beta = (L.use_points && L.offsets) ? (double)L.offsets[row] : 0.0;
        const float *wr = L.W + row * d;
        const int8_t *cr = L.codes + row * (int64_t)P * d;
        const float *sr = L.scales + row * (int64_t)P;
        if (L.vecw && k < d) {   // d % 4 == 0: the four k lie inside the row
            const float4 w = *(const float4 *)(wr + k);
            r[0] = (double)w.x - beta; r[1] = (double)w.y - beta;
            r[2] = (double)w.z - beta; r[3] = (double)w.w - beta;
            for (int p = 0; p < nk; ++p) {
                const double a = (double)sr[p];
                const uint32_t q = *(const uint32_t *)(cr + (int64_t)p * d + k);
#pragma unroll
                for (int u = 0; u < 4; ++u) r[u] = fma(-a, int8_of(q, u), r[u]);
            }
        } else {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (k + u < d) {
                    double v = (double)wr[k + u] - beta;
                    for (int p = 0; p < nk; ++p)
                        v = fma(-(double)sr[p], (double)cr[(int64_t)p * d + k + u], v);
                    r[u] = v;
                }
            }
        }
    }
    *(float4 *)(L.D + d_index(m, k, L.nkb)) = make_float4((float)r[0], (float)r[1], (float)r[2], (float)r[3]);
}

// ---- 2. gemm: Y = D X, squared and summed per row

// The three bf16 pieces of fp32 values, in pairs: x = hi + mid + lo exactly
// for finite x below bf16's largest value.  Each piece is the remainder so
// far rounded to nearest (8 significant bits): x - hi is exact in fp32
// (at most 16 bits), and so is its remainder after mid, which has at most 8
// bits and is lo.
__device__ __forceinline__ void split_pair(float x0, float x1, bf16x2 &h, bf16x2 &m, bf16x2 &l)
{
    const f32x2 x = {x0, x1};
    h = __builtin_convertvector(x, bf16x2);
    const f32x2 r1 = x - __builtin_convertvector(h, f32x2);
    m = __builtin_convertvector(r1, bf16x2);
    const f32x2 r2 = r1 - __builtin_convertvector(m, f32x2);
    l = __builtin_convertvector(r2, bf16x2);
}

// Eight consecutive k of one row (D) or one column (X): the pieces, one
// 16-byte vector each, stored to a row of each piece tile.
__device__ __forceinline__ void split_store8(const float (&v)[8], __bf16 *h, __bf16 *m, __bf16 *l)
{
    bf16x8 vh, vm, vl;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        bf16x2 ph, pm, pl;
        split_pair(v[2 * i], v[2 * i + 1], ph, pm, pl);
        vh[2 * i] = ph[0]; vh[2 * i + 1] = ph[1];
        vm[2 * i] = pm[0]; vm[2 * i + 1] = pm[1];
        vl[2 * i] = pl[0]; vl[2 * i + 1] = pl[1];
    }
    *(bf16x8 *)h = vh;
    *(bf16x8 *)m = vm;
    *(bf16x8 *)l = vl;
}

// Y = D X in fp32 from bf16 matrix products (v_mfma_f32_32x32x16_bf16):
// with D = Dh + Dm + Dl and X = Xh + Xm + Xl (split_pair), each product
// D X is summed from the six piece products Dh Xh, Dh Xm, Dm Xh, Dh Xl,
// Dl Xh and Dm Xm (bf16 products are exact in fp32, accumulated in fp32).
// The three left out (Dm Xl, Dl Xm, Dl Xl) are below 2^-23 |D X| together,
// under one rounding of the fp32 product, so the sums carry the error of an
// fp32 accumulation.  Six bf16 products cost 6/16 of one fp32 product's
// matrix-core time.
template <bool kVecX>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4)))
gemm_err_kernel(const ErrGroup g, const ErrLayer *__restrict__ Ls)
{
    // double-buffered piece tiles of a 16-k slab: rows of D (channels) and
    // columns of X (samples); a 16-byte read of 16 rows covers the 64 banks once
    __shared__ __align__(16) __bf16 sD[2][kPieces][kBM][kRowK];
    __shared__ __align__(16) __bf16 sX[2][kPieces][kBN][kRowK];
    __shared__ double sPart[2][kBM];

    // a layer's workgroups: the planned tiles' from block_begin, and any
    // more (for the short K ranges of a listed layer's few live rows) from
    // extra_begin, after every layer's planned ones
    const bool extra = (int)blockIdx.x >= g.extra_start;
    const int li = extra ? last_at_most(g.n_layers, (int)blockIdx.x,
                                        [&](int i) { return Ls[i].extra_begin; })
                         : last_at_most(g.n_layers, (int)blockIdx.x,
                                        [&](int i) { return Ls[i].block_begin; });
    const ErrLayer &L = Ls[li];
    // the live tiles: (split, tm, tn) over the live row tiles, split-major
    const int64_t nact = L.rows ? (int64_t)*L.nrows : (int64_t)L.C;
    LiveSplit ls = live_split(L, nact);
    // uniform values: keep them in scalar registers
    ls.ntm = __builtin_amdgcn_readfirstlane(ls.ntm);
    ls.splits = __builtin_amdgcn_readfirstlane(ls.splits);
    ls.kchunk = __builtin_amdgcn_readfirstlane(ls.kchunk);
    const int per_split = ls.ntm * L.ntn;
    const int live = per_split * ls.splits;   // <= L.tiles
    // XCD-contiguous renumbering of the live tiles (block_begin and
    // extra_begin are multiples of kXcds, so b % kXcds is the XCD this block
    // runs on); an XCD's slots continue from the planned region into the extra one
    const int planned = (L.ntm * L.ntn * L.splits + kXcds - 1) / kXcds;   // slots per XCD
    const int b = (int)blockIdx.x - (extra ? L.extra_begin : L.block_begin);
    const int xcd = b % kXcds, slot = b / kXcds + (extra ? planned : 0);
    const int q = live / kXcds, rem = live % kXcds;
    const int xr = (xcd - L.xoff + kXcds) % kXcds;   // the XCD's rank for this layer
    if (slot >= q + (xr < rem ? 1 : 0)) return;   // padding block
    int tn = xr * q + min(xr, rem) + slot;
    int split = 0, tm = 0;
    while (tn >= per_split) {
        tn -= per_split;
        ++split;
    }
    while (tn >= L.ntn) {
        tn -= L.ntn;
        ++tm;
    }

    const int64_t row0 = (int64_t)tm * kBM;

    const int t = threadIdx.x;
    const int lane = t % kWave, wid = __builtin_amdgcn_readfirstlane(t / kWave);   // uniform per wavefront
    const bool stager = wid >= 4;           // wavefronts 4 .. 7 stage, 0 .. 3 multiply
    const int wm = (wid % 4) / 2, wn = wid % 2;   // rows wm * 64 + [0, 64), columns wn * 64 + [0, 64)
    const int64_t C = L.C, n = L.n;
    const int64_t col0 = (int64_t)tn * kBN;
    const int64_t kbeg = (int64_t)split * ls.kchunk;   // a multiple of kBK
    const int64_t kend = min(kbeg + (int64_t)ls.kchunk, (int64_t)L.d);
    const int nslab = (int)((kend - kbeg + kSlabK - 1) / kSlabK);

    // acc[cb][rb]: samples wn * 64 + cb * 32 + [0, 32) by rows wm * 64 + rb
    // * 32 + [0, 32).  The blocks hold Y transposed (X's pieces as the MFMA's
    // A operand, D's as its B), so a lane's registers run over samples of
    // one row.
    floatx16 acc[2][2];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[cb][rb][v] = 0.0f;

    // One barrier per slab for all eight wavefronts: the multiplying ones
    // read slab s from buffer s % 2 while the staging ones split slab s + 1
    // into the other buffer.
    if (stager) {
        // buffer resources: this row tile's 32-k chunks of D (one
        // contiguous block each; rows past C feed only output rows nobody
        // reads) and this K range's rows of X (below 2^31 bytes, see
        // plan_item; rows past kend read as zeros)
        const __amdgpu_buffer_rsrc_t rsD =
            make_rsrc(L.D + (int64_t)tm * L.nkb * (kBM * kBK), (uint32_t)L.nkb * (kBM * kBK * 4));
        const __amdgpu_buffer_rsrc_t rsX = make_rsrc(L.X + kbeg * n, (uint32_t)((kend - kbeg) * n * 4));
        // staging roles: D row dr, k dh * 8 .. + 7 of the slab (two float4
        // of the chunk's row); X column xc, k xh * 8 .. + 7 (eight floats,
        // one per row of X: a wavefront's load covers 64 consecutive columns)
        const int st = t - kStageT;
        const int dr = st / 2, dh = st % 2;
        const int xc = st % kBN, xh = st / kBN;
        const uint32_t offD = (uint32_t)((kbeg / kBK * (kBM * kBK) + dr * kBK + dh * 8) * 4);
        // a column past n reads at offset 2^32 - 1 (past every range, as a
        // bit mask: no carry); the others stay below 2^32, as kchunk n 4 < 2^31
        const uint32_t offX = (uint32_t)(((int64_t)xh * 8 * n + col0 + xc) * 4);
        const uint32_t oobX = col0 + xc < n ? 0u : 0xffffffffu;
        const uint32_t rowX = (uint32_t)(n * 4);
        // slab s: chunk s / 2 of the range, k (s % 2) 16 within it
        auto load = [&](float (&r)[16], int s) {
            const uint32_t o = offD + (uint32_t)(s / 2) * (kBM * kBK * 4) + (uint32_t)(s % 2) * (kSlabK * 4);
            const f32x4 a = load4(rsD, o), b = load4(rsD, o + 16);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                r[u] = a[u];
                r[4 + u] = b[u];
            }
#pragma unroll
            for (int u = 0; u < 8; ++u)
                r[8 + u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                    rsX, (offX + (uint32_t)(s * kSlabK + u) * rowX) | oobX, 0, 0));
        };
        auto store = [&](const float (&r)[16], int buf) {
            const float(&rd)[8] = *(const float(*)[8])&r[0];
            const float(&rx)[8] = *(const float(*)[8])&r[8];
            split_store8(rd, &sD[buf][0][dr][dh * 8], &sD[buf][1][dr][dh * 8], &sD[buf][2][dr][dh * 8]);
            split_store8(rx, &sX[buf][0][xc][xh * 8], &sX[buf][1][xc][xh * 8], &sX[buf][2][xc][xh * 8]);
        };
        float ring[kRing][16];
#pragma unroll
        for (int j = 0; j < kRing; ++j)
            if (j < nslab) load(ring[j], j);
        store(ring[0], 0);
        if (kRing < nslab) load(ring[0], kRing);
        __syncthreads();
        for (int s0 = 0; s0 < nslab; s0 += kRing) {
#pragma unroll
            for (int j = 0; j < kRing; ++j) {
                const int s = s0 + j;   // the multiplying wavefronts read slab s
                if (s >= nslab) break;
                if (s + 1 < nslab) store(ring[(j + 1) % kRing], (s + 1) % 2);
                if (s + 1 + kRing < nslab) load(ring[(j + 1) % kRing], s + 1 + kRing);
                __syncthreads();
            }
        }
    } else {
        // A wavefront with no live row of D (a layer of few channels, a few
        // listed rows) multiplies nothing: its products are of rows nobody
        // reads.  Slabs past d hold zeros.
        const bool rows_live = row0 + wm * 64 < nact;   // uniform per wavefront
        constexpr int kPx[6] = {1, 2, 0, 1, 0, 0}, kPd[6] = {1, 0, 2, 0, 1, 0};   // the small products first
        const int ko = 8 * (lane / 32);
        __syncthreads();
        for (int s = 0; s < nslab; ++s) {
            if (rows_live) {
                const int buf = s % 2;
                bf16x8 xp[2][kPieces], dp[2][kPieces];
#pragma unroll
                for (int p = 0; p < kPieces; ++p) {
#pragma unroll
                    for (int c = 0; c < 2; ++c) {
                        xp[c][p] = *(const bf16x8 *)&sX[buf][p][wn * 64 + c * 32 + lane % 32][ko];
                        dp[c][p] = *(const bf16x8 *)&sD[buf][p][wm * 64 + c * 32 + lane % 32][ko];
                    }
                }
#pragma unroll
                for (int z = 0; z < 6; ++z)
#pragma unroll
                    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                        for (int rb = 0; rb < 2; ++rb)
                            acc[cb][rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xp[cb][kPx[z]], dp[rb][kPd[z]],
                                                                                  acc[cb][rb], 0, 0, 0);
            }
            __syncthreads();
        }
    }

    // Output layout of a 32 x 32 MFMA block: lane holds block column
    // lane % 32 (here row rb * 32 + lane % 32 of the wavefront's 64) and, in
    // register v, block row 8 (v / 4) + 4 (lane / 32) + v % 4 (here a
    // sample: four consecutive ones per group v / 4)
    const int64_t row_w = row0 + wm * 64 + lane % 32;   // + rb * 32
    auto col_of = [&](int cb, int grp) { return col0 + wn * 64 + cb * 32 + 8 * grp + 4 * (lane / 32); };

    if (ls.splits > 1) {
        // this K range's Y tile (rows of stride nact); the finish kernel sums
        // the ranges
        if (stager) return;
        float *yp = L.ypart;
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
            const int64_t r = row_w + rb * 32;
            if (r >= nact) continue;
            float *yr = yp + ((int64_t)split * nact + r) * n;
#pragma unroll
            for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                for (int grp = 0; grp < 4; ++grp) {
                    const int64_t c = col_of(cb, grp);
                    const floatx16 &y = acc[cb][rb];
                    if (kVecX) {   // n % 4 == 0: the four samples lie inside the row or past it
                        if (c < n)
                            *(f32x4 *)(yr + c) = f32x4{y[4 * grp], y[4 * grp + 1], y[4 * grp + 2], y[4 * grp + 3]};
                    } else {
#pragma unroll
                        for (int u = 0; u < 4; ++u)
                            if (c + u < n) yr[c + u] = y[4 * grp + u];
                    }
                }
        }
        return;
    }

    // squares summed over the tile's columns, per row (fp64, fixed order):
    // a lane's 32 samples (block cb, then register order), then the other
    // half-wave's 32 (samples past n are zeros), then the two column halves
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
        double sq = 0.0;
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
            for (int v = 0; v < 16; ++v) sq = fma((double)acc[cb][rb][v], (double)acc[cb][rb][v], sq);
        const double o = __shfl_xor(sq, 32);
        if (!stager && lane < 32) sPart[wn][wm * 64 + rb * 32 + lane] = sq + o;
    }
    __syncthreads();
    if (t < kBM) {
        const int64_t gr = row0 + t;
        if (gr < C) L.rowpart[(int64_t)tn * C + gr] = sPart[0][t] + sPart[1][t];
    }
}

// ---- 3. finish: per row, the sum over column tiles of the row partials
// (256 rows per workgroup), or for a split layer the sum over K ranges of Y,
// squared and summed over the columns (one wavefront per row, four rows per
// workgroup); fixed order, fp64, divided by n
__global__ void __launch_bounds__(256) finish_err_kernel(const ErrGroup g,
                                                         const ErrLayer *__restrict__ Ls)
{
    const int li = last_at_most(g.n_layers, (int)blockIdx.x, [&](int i) { return Ls[i].fin_begin; });
    const ErrLayer &L = Ls[li];
    const int64_t C = L.C, n = L.n;
    const int b = (int)blockIdx.x - L.fin_begin;
    const int64_t nact = L.rows ? (int64_t)*L.nrows : C;
    const int splits = live_split(L, nact).splits;
    // output slot of row m of D
    auto slot = [&](int64_t m) { return (L.rows ? (int64_t)L.rows[m] : m) * L.stride; };
    if (splits == 1) {
        const int64_t k = (int64_t)b * 256 + threadIdx.x;
        if (k < nact) {
            double s = 0.0;
            for (int i = 0; i < L.ntn; ++i) s += L.rowpart[(int64_t)i * C + k];
            L.out[slot(k)] = (float)(s / (double)n);
        }
        return;
    }
    // a split layer: one wavefront per row, four rows per workgroup
    const int lane = (int)threadIdx.x % kWave;
    const int64_t k = (int64_t)b * kFinRows + (int64_t)threadIdx.x / kWave;
    if (k >= nact) return;   // uniform per wavefront
    double s = 0.0;
    if (g.vecx) {
        // n % 4 == 0: four columns per lane and pass, the K ranges' loads
        // of up to four ranges issued together
        for (int64_t c = 4 * lane; c < n; c += 4 * kWave) {
            f32x4 y = {0.0f, 0.0f, 0.0f, 0.0f};
            for (int sp0 = 0; sp0 < splits; sp0 += 4) {
                f32x4 v[4];
#pragma unroll
                for (int z = 0; z < 4; ++z)
                    if (sp0 + z < splits)
                        v[z] = *(const f32x4 *)(L.ypart + ((int64_t)(sp0 + z) * nact + k) * n + c);
#pragma unroll
                for (int z = 0; z < 4; ++z)
                    if (sp0 + z < splits) y += v[z];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) s = fma((double)y[u], (double)y[u], s);
        }
    } else {
        for (int64_t c = lane; c < n; c += kWave) {
            float y = 0.0f;
            for (int sp = 0; sp < splits; ++sp) y += L.ypart[((int64_t)sp * nact + k) * n + c];
            s = fma((double)y, (double)y, s);
        }
    }
    s = wave_reduce(s, SumOp());
    if (lane == 0) L.out[slot(k)] = (float)(s / (double)n);
}

struct Item {
    const ErrLayerIn *in;
    int use_points;
};

// rows of D of an item: the channels, or their clipping candidates
int64_t item_rows(const ErrLayerIn &I) { return I.cand ? I.C * I.Gc : I.C; }

// an item whose rows are the first *nrows channels of a list
bool listed(const ErrLayerIn &I, int use_points) { return use_points == 1 && I.rows; }

struct Plan {
    int64_t nkb, ntm, ntn, splits, kchunk;
    int64_t budget;   // splits of the workgroup budget (ntm * ntn * budget workgroups)
    size_t d_bytes, rowpart_bytes, ypart_bytes;
};

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

// err items for the layers that want err, then ref items for the layers that want ref
std::vector<Item> items_of(const ErrLayerIn *in, int n_in)
{
    std::vector<Item> it;
    for (int i = 0; i < n_in; ++i)
        if (in[i].C > 0 && in[i].err) it.push_back(Item{&in[i], in[i].cand ? 2 : 1});
    for (int i = 0; i < n_in; ++i)
        if (in[i].C > 0 && in[i].ref) it.push_back(Item{&in[i], 0});
    return it;
}

// K split of a layer: K ranges of at most kRangeK, or of work / 512 slabs (two
// tiles per CU) for a layer that alone fills the GPU, and K ranges whose rows
// of X stay below 2^31 bytes (a row tile of D does: d <= MPQ_MAX_ERR_D).  The ranges of a split layer make the
// GEMM store fp32 Y tiles that the finish kernel reads back, so a layer of
// short K stays whole: the other layers of a call fill the GPU.  The split
// depends on the layer alone, so a layer's result does not depend on the
// other layers of the call.  A listed layer gets workgroups for
// ceil(slabs / kMinSlabs / ntm) K ranges if that is more, and Y room for
// them, so live_split can spread a few live rows over shorter K ranges.
Plan plan_item(const ErrLayerIn &I, bool list)
{
    Plan q;
    const int64_t C = item_rows(I);
    q.nkb = (I.d + kBK - 1) / kBK;
    q.ntm = (C + kBM - 1) / kBM;
    q.ntn = (I.n + kBN - 1) / kBN;
    const int64_t slabs = (I.d + kBK - 1) / kBK;
    const double work = (double)(q.ntm * q.ntn) * (double)slabs;
    const int64_t target = std::max<int64_t>(kRangeK / kBK, (int64_t)(work / 512.0 + 0.5));
    // enough ranges that none exceeds the target (MobileNetV2's d = 960
    // layers, 30 slabs, took ~100 us as one range; 15-slab halves, 88 us)
    int64_t sp = (slabs + target - 1) / target;
    sp = std::max<int64_t>(1, std::min<int64_t>(sp, slabs));
    int64_t kchunk = (slabs + sp - 1) / sp * kBK;
    const int64_t max_chunk = ((1LL << 31) - 1) / (4 * I.n) / kBK * kBK;   // >= kBK (n < 2^24)
    kchunk = std::min(kchunk, max_chunk);
    q.kchunk = kchunk;
    q.splits = (I.d + kchunk - 1) / kchunk;   // no empty K range
    q.d_bytes = align256(sizeof(float) * (size_t)(q.ntm * q.nkb * kBM * kBK));
    q.rowpart_bytes = align256(sizeof(double) * (size_t)(q.ntn * C));
    q.budget = q.splits;
    if (list) {
        const int64_t want = (slabs / kMinSlabs + q.ntm - 1) / q.ntm;
        q.budget = std::max(q.splits, want);
        // live_split: splits * nact <= budget * ntm * kBM rows of Y
        q.ypart_bytes = align256(sizeof(float) * (size_t)(q.budget * q.ntm * kBM * I.n));
    } else {
        q.ypart_bytes = q.splits > 1 ? align256(sizeof(float) * (size_t)(q.splits * C * I.n)) : 0;
    }
    return q;
}

// A group's items in launch order (longest K ranges first) and the byte
// offset of each item's scratch (D, row partials, Y ranges) in the group's,
// after the descriptor table at its head.
struct GroupLayout {
    std::vector<Plan> p;
    std::vector<int> order;
    std::vector<size_t> off;   // by item
};
size_t table_bytes(int cnt) { return align256(sizeof(ErrLayer) * (size_t)cnt); }
GroupLayout group_layout(const Item *grp, int cnt)
{
    GroupLayout G;
    G.p.resize(cnt);
    for (int i = 0; i < cnt; ++i) G.p[i] = plan_item(*grp[i].in, listed(*grp[i].in, grp[i].use_points));
    G.order.resize(cnt);
    for (int i = 0; i < cnt; ++i) G.order[i] = i;
    std::stable_sort(G.order.begin(), G.order.end(),
                     [&](int a, int b) { return G.p[a].kchunk > G.p[b].kchunk; });
    G.off.assign(cnt, 0);
    size_t cur = table_bytes(cnt);
    for (int o = 0; o < cnt; ++o) {
        const int i = G.order[o];
        G.off[i] = cur;
        cur += G.p[i].d_bytes + G.p[i].rowpart_bytes + G.p[i].ypart_bytes;
    }
    return G;
}

size_t group_bytes(const Item *it, int cnt)
{
    size_t b = table_bytes(cnt);
    for (int i = 0; i < cnt; ++i) {
        const Plan q = plan_item(*it[i].in, listed(*it[i].in, it[i].use_points));
        b += q.d_bytes + q.rowpart_bytes + q.ypart_bytes;
    }
    return b;
}

}  // namespace

int err_group_count(const ErrLayerIn *in, int n_in)
{
    const size_t n = items_of(in, n_in).size();
    return (int)((n + kMaxErrItems - 1) / kMaxErrItems);
}

size_t err_group_scratch_bytes(const ErrLayerIn *in, int n_in, int group)
{
    const std::vector<Item> it = items_of(in, n_in);
    const size_t base = (size_t)group * kMaxErrItems;
    if (base >= it.size()) return 0;
    const int cnt = (int)std::min<size_t>(kMaxErrItems, it.size() - base);
    return group_bytes(it.data() + base, cnt);
}

void err_item_d_offsets(const ErrLayerIn *in, int n_in, int64_t *off, int *group)
{
    for (int i = 0; i < n_in; ++i) {
        off[i] = -1;
        group[i] = -1;
    }
    const std::vector<Item> it = items_of(in, n_in);
    // each group's layout once
    for (size_t base = 0; base < it.size(); base += kMaxErrItems) {
        const int cnt = (int)std::min<size_t>(kMaxErrItems, it.size() - base);
        const GroupLayout lay = group_layout(it.data() + base, cnt);
        for (int x = 0; x < cnt; ++x) {
            const Item &I = it[base + (size_t)x];
            if (I.use_points != 1) continue;
            const int i = (int)(I.in - in);
            off[i] = (int64_t)lay.off[x];
            group[i] = (int)(base / kMaxErrItems);
        }
    }
}

double err_group_flop(const ErrLayerIn *in, int n_in, int group)
{
    const std::vector<Item> it = items_of(in, n_in);
    double f = 0.0;
    for (size_t i = (size_t)group * kMaxErrItems; i < it.size() && i < (size_t)(group + 1) * kMaxErrItems; ++i)
        f += 2.0 * (double)item_rows(*it[i].in) * (double)it[i].in->d * (double)it[i].in->n;
    return f;
}

hipError_t launch_output_error_group(const ErrLayerIn *in, int n_in, int group, int P, void *scratch,
                                     hipStream_t s, int parts)
{
    const std::vector<Item> it = items_of(in, n_in);
    const size_t base = (size_t)group * kMaxErrItems;
    if (base >= it.size()) return hipSuccess;
    {
        const int cnt = (int)std::min<size_t>(kMaxErrItems, it.size() - base);
        const Item *grp = it.data() + base;
        const GroupLayout lay = group_layout(grp, cnt);   // longest K ranges first
        const std::vector<Plan> &p = lay.p;
        const std::vector<int> &order = lay.order;
        ErrGroup g;
        g.n_layers = cnt;
        g.P = P;
        g.vecx = 1;
        std::vector<ErrLayer> table(cnt);
        int64_t blocks = 0, fblocks = 0, nblocks = 0;
        int xoff = 0;
        for (int o = 0; o < cnt; ++o) {
            const int i = order[o];
            const ErrLayerIn &I = *grp[i].in;
            const Plan &q = p[i];
            ErrLayer &L = table[o];
            L.W = I.W;
            L.codes = I.codes;
            L.scales = I.scales;
            L.counts = I.counts;
            L.X = I.X;
            L.out = grp[i].use_points ? I.err : I.ref;
            L.use_points = grp[i].use_points;
            L.rows = grp[i].use_points == 1 ? I.rows : nullptr;
            L.nrows = grp[i].use_points == 1 ? I.nrows : nullptr;
            L.stride = grp[i].use_points == 1 && I.err_stride > 0 ? I.err_stride : 1;
            L.cand = grp[i].use_points == 2 ? I.cand : nullptr;
            L.offsets = grp[i].use_points == 1 ? I.offsets : nullptr;
            L.Gc = I.Gc;
            L.M = I.M;
            char *cur = (char *)scratch + lay.off[i];
            L.D = (float *)cur;
            cur += q.d_bytes;
            L.rowpart = (double *)cur;
            cur += q.rowpart_bytes;
            L.ypart = q.ypart_bytes ? (float *)cur : nullptr;
            L.C = (int)item_rows(I);
            L.d = (int)I.d;
            L.n = (int)I.n;
            L.nkb = (int)q.nkb;
            L.ntm = (int)q.ntm;
            L.ntn = (int)q.ntn;
            L.splits = (int)q.splits;
            L.kchunk = (int)q.kchunk;
            if (q.ntm * q.ntn * q.budget > 0x7fffffffLL) return hipErrorInvalidValue;
            L.tiles = (int)(q.ntm * q.ntn * q.budget);
            const int64_t planned = q.ntm * q.ntn * q.splits;
            L.block_begin = (int)blocks;
            blocks += (planned + kXcds - 1) / kXcds * kXcds;
            // the spare tiles (planned % kXcds) of successive layers go to
            // successive XCDs, so no XCD collects one from every layer
            L.xoff = xoff;
            xoff = (xoff + (int)(planned % kXcds)) % kXcds;
            L.form_begin = (int)fblocks;
            // rows the fit wrote need no forming
            const bool ready = grp[i].use_points == 1 && I.d_ready && !I.cand;
            if (!ready) fblocks += ((int64_t)L.C * L.nkb * (kBK / 4) + kFormThreads - 1) / kFormThreads;
            L.fin_begin = (int)nblocks;
            nblocks += q.ypart_bytes ? (L.C + kFinRows - 1) / kFinRows : (L.C + 255) / 256;
            L.vecw = I.d % 4 == 0 && ((uintptr_t)I.W) % 16 == 0 && ((uintptr_t)I.codes) % 4 == 0;
            if (I.n % 4 != 0 || ((uintptr_t)I.X) % 16 != 0) g.vecx = 0;
        }
        // the workgroup budget past the planned tiles, after every layer's
        // planned ones: per XCD, ceil(tiles / kXcds) slots in all
        if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
        g.extra_start = (int)blocks;
        for (int o = 0; o < cnt; ++o) {
            ErrLayer &L = table[o];
            const int64_t planned = (int64_t)L.ntm * L.ntn * L.splits;
            L.extra_begin = (int)blocks;
            blocks += ((int64_t)L.tiles + kXcds - 1) / kXcds * kXcds -
                      (planned + kXcds - 1) / kXcds * kXcds;
        }
        if (blocks > 0x7fffffffLL || fblocks > 0x7fffffffLL || nblocks > 0x7fffffffLL)
            return hipErrorInvalidValue;
        hipError_t e = hipSuccess;
        // the descriptor table at the head of the group's scratch
        ErrLayer *dtab = (ErrLayer *)scratch;
        for (int o = 0; (parts & kErrUpload) && o < cnt && e == hipSuccess; o += kDescChunk) {
            DescChunk c;
            c.dst = dtab + o;
            c.count = std::min(kDescChunk, cnt - o);
            for (int i = 0; i < c.count; ++i) c.L[i] = table[o + i];
            LaunchTimer timer(s, "desc_upload_kernel");
            hipLaunchKernelGGL(desc_upload_kernel, dim3(1), dim3(64), 0, s, c);
            e = hipGetLastError();
        }
        if (e != hipSuccess || !(parts & kErrKernels)) return e;
        if (fblocks > 0) {
            LaunchTimer timer(s, "form_d_kernel");
            hipLaunchKernelGGL(form_d_kernel, dim3((unsigned)fblocks), dim3(kFormThreads), 0, s, g,
                               (const ErrLayer *)dtab);
            e = hipGetLastError();
        }
        if (e != hipSuccess) return e;
        {
            LaunchTimer timer(s, "gemm_err_kernel");
            auto kern = g.vecx ? gemm_err_kernel<true> : gemm_err_kernel<false>;
            hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kThreads), 0, s, g,
                               (const ErrLayer *)dtab);
            e = hipGetLastError();
        }
        if (e != hipSuccess) return e;
        {
            LaunchTimer timer(s, "finish_err_kernel");
            hipLaunchKernelGGL(finish_err_kernel, dim3((unsigned)nblocks), dim3(256), 0, s, g,
                               (const ErrLayer *)dtab);
            e = hipGetLastError();
        }
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace mpq
