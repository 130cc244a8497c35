// Wavefront and workgroup reductions for gfx950 (wave64).
//
// Within a wavefront the exchange steps are, in order: DPP quad_perm
// [1,0,3,2] and [2,3,0,1], DPP row_half_mirror, DPP row_mirror (these
// combine lanes within a row of 16), ds_swizzle with xor mask 16 (combines
// the two rows of each half-wave) and finally a readlane of lanes 0 and 32.
// Every step combines a lane with a partner holding the other half of its
// group, so with a commutative, associative combine every lane of a group
// ends with the same value; the result is uniform across the wavefront.
// Across wavefronts the per-wave results go through LDS and every thread
// combines them in wave order, so the result is deterministic.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mpq {

constexpr int kWave = 64;

// The last index i in [0, n) with begin(i) <= b, for non-decreasing begins
// with begin(0) <= b: which of a launch's layers a workgroup b belongs to
// (layers with no workgroups share their begin with the next one and are
// never returned).  Binary search: ceil(log2 n) dependent reads of the
// descriptors instead of one per layer.
template <class Begin>
__device__ __forceinline__ int last_at_most(int n, int b, Begin begin)
{
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (begin(mid) <= b) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

template <int kCtrl>
__device__ __forceinline__ uint32_t dpp(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, kCtrl, 0xF, 0xF, true);
}

__device__ __forceinline__ uint32_t swizzle_xor16(uint32_t v)
{
    // bitmask mode: and_mask = 0x1f, or_mask = 0, xor_mask = 0x10
    return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x401F);
}

// exchange step s (0..4) of a 32-bit value
template <int kStep>
__device__ __forceinline__ uint32_t xstep(uint32_t v)
{
    if constexpr (kStep == 0) return dpp<0xB1>(v);   // quad_perm [1,0,3,2]
    else if constexpr (kStep == 1) return dpp<0x4E>(v);  // quad_perm [2,3,0,1]
    else if constexpr (kStep == 2) return dpp<0x141>(v); // row_half_mirror
    else if constexpr (kStep == 3) return dpp<0x140>(v); // row_mirror
    else return swizzle_xor16(v);
}

template <int kStep>
__device__ __forceinline__ float xstep(float v)
{
    return __uint_as_float(xstep<kStep>(__float_as_uint(v)));
}

template <int kStep>
__device__ __forceinline__ double xstep(double v)
{
    uint64_t u = (uint64_t)__double_as_longlong(v);
    uint32_t lo = xstep<kStep>((uint32_t)u), hi = xstep<kStep>((uint32_t)(u >> 32));
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

template <int kStep>
__device__ __forceinline__ int xstep(int v)
{
    return (int)xstep<kStep>((uint32_t)v);
}

__device__ __forceinline__ float readlane(float v, int l)
{
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

__device__ __forceinline__ double readlane(double v, int l)
{
    uint64_t u = (uint64_t)__double_as_longlong(v);
    uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
    uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

__device__ __forceinline__ int readlane(int v, int l)
{
    return __builtin_amdgcn_readlane(v, l);
}

struct MaxOp {
    template <typename T>
    __device__ __forceinline__ T operator()(T a, T b) const { return a > b ? a : b; }
};
struct MinOp {
    template <typename T>
    __device__ __forceinline__ T operator()(T a, T b) const { return a < b ? a : b; }
};
struct SumOp {
    template <typename T>
    __device__ __forceinline__ T operator()(T a, T b) const { return a + b; }
};

// Reduction over the 32 lanes of each half-wave: every lane ends with its
// half's result.
template <typename T, typename Op>
__device__ __forceinline__ T half_wave_reduce(T v, Op op)
{
    v = op(v, xstep<0>(v));
    v = op(v, xstep<1>(v));
    v = op(v, xstep<2>(v));
    v = op(v, xstep<3>(v));
    v = op(v, xstep<4>(v));
    return v;
}

// Reduction over the whole wavefront; the result is wave-uniform.
template <typename T, typename Op>
__device__ __forceinline__ T wave_reduce(T v, Op op)
{
    v = half_wave_reduce(v, op);
    return op(readlane(v, 0), readlane(v, 32));
}

// Lexicographic (value, index) minimum: the smaller value, then the smaller
// index.  Used for the candidate argmin (ties go to the smaller index).
struct ArgMin {
    double e;
    int g;
};

__device__ __forceinline__ ArgMin argmin_combine(ArgMin a, ArgMin b)
{
    return (b.e < a.e || (b.e == a.e && b.g < a.g)) ? b : a;
}

template <int kStep>
__device__ __forceinline__ ArgMin xstep(ArgMin v)
{
    return ArgMin{xstep<kStep>(v.e), xstep<kStep>(v.g)};
}

__device__ __forceinline__ ArgMin wave_argmin(ArgMin v)
{
    v = argmin_combine(v, xstep<0>(v));
    v = argmin_combine(v, xstep<1>(v));
    v = argmin_combine(v, xstep<2>(v));
    v = argmin_combine(v, xstep<3>(v));
    v = argmin_combine(v, xstep<4>(v));
    ArgMin lo{readlane(v.e, 0), readlane(v.g, 0)};
    ArgMin hi{readlane(v.e, 32), readlane(v.g, 32)};
    return argmin_combine(lo, hi);
}

// Inclusive prefix sum over the 64 lanes (lane 0 first), DPP only:
// row_shr 1, 2, 4, 8 with zero fill within each row of 16, then row_bcast15
// (rows 1 and 3 add lane 15 of the row before) and row_bcast31 (rows 2 and 3
// add lane 31).
template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint32_t dpp_zero(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kCtrl, kRowMask, 0xF, true);
}

template <int kCtrl, int kRowMask>
__device__ __forceinline__ unsigned long long dpp_zero64(unsigned long long v)
{
    const uint32_t lo = dpp_zero<kCtrl, kRowMask>((uint32_t)v);
    const uint32_t hi = dpp_zero<kCtrl, kRowMask>((uint32_t)(v >> 32));
    return ((unsigned long long)hi << 32) | lo;
}

__device__ __forceinline__ unsigned long long wave_prefix_sum(unsigned long long v)
{
    v += dpp_zero64<0x111, 0xF>(v);  // row_shr:1
    v += dpp_zero64<0x112, 0xF>(v);  // row_shr:2
    v += dpp_zero64<0x114, 0xF>(v);  // row_shr:4
    v += dpp_zero64<0x118, 0xF>(v);  // row_shr:8
    v += dpp_zero64<0x142, 0xA>(v);  // row_bcast:15
    v += dpp_zero64<0x143, 0xC>(v);  // row_bcast:31
    return v;
}

__device__ __forceinline__ uint32_t wave_prefix_sum(uint32_t v)
{
    v += dpp_zero<0x111, 0xF>(v);
    v += dpp_zero<0x112, 0xF>(v);
    v += dpp_zero<0x114, 0xF>(v);
    v += dpp_zero<0x118, 0xF>(v);
    v += dpp_zero<0x142, 0xA>(v);
    v += dpp_zero<0x143, 0xC>(v);
    return v;
}

// Workgroup reductions.  `scratch` must hold one T per wavefront and must
// not be in use by another reduction between the two barriers.
template <int kThreads, typename T, typename Op>
__device__ __forceinline__ T block_reduce(T v, Op op, T *scratch)
{
    constexpr int kWaves = kThreads / kWave;
    v = wave_reduce(v, op);
    const int wid = threadIdx.x / kWave;
    if ((threadIdx.x % kWave) == 0) scratch[wid] = v;
    __syncthreads();
    T r = scratch[0];
#pragma unroll
    for (int i = 1; i < kWaves; ++i) r = op(r, scratch[i]);
    __syncthreads();
    return r;
}

// max of a float and sum of a double over the workgroup, with one pair of
// barriers (kTrail = false: the first barrier only; the caller then passes
// another barrier before scratch_f / scratch_d are written again).
// scratch_f / scratch_d hold one value per wavefront.
template <int kThreads, bool kTrail = true>
__device__ __forceinline__ void block_max_sum(float &vmax, double &vsum, float *scratch_f,
                                              double *scratch_d)
{
    constexpr int kWaves = kThreads / kWave;
    vmax = half_wave_reduce(vmax, MaxOp());
    vsum = half_wave_reduce(vsum, SumOp());
    vmax = MaxOp()(readlane(vmax, 0), readlane(vmax, 32));
    vsum = SumOp()(readlane(vsum, 0), readlane(vsum, 32));
    if constexpr (kWaves > 1) {
        const int wid = threadIdx.x / kWave;
        if ((threadIdx.x % kWave) == 0) {
            scratch_f[wid] = vmax;
            scratch_d[wid] = vsum;
        }
        __syncthreads();
        float m = scratch_f[0];
        double sm = scratch_d[0];
#pragma unroll
        for (int i = 1; i < kWaves; ++i) {
            m = MaxOp()(m, scratch_f[i]);
            sm = SumOp()(sm, scratch_d[i]);
        }
        if constexpr (kTrail) __syncthreads();
        vmax = m;
        vsum = sm;
    }
}

// two sums of doubles over the workgroup, with one pair of barriers; fixed
// order.  scratch_a / scratch_b hold one value per wavefront.
template <int kThreads>
__device__ __forceinline__ void block_sum2(double &a, double &b, double *scratch_a, double *scratch_b)
{
    constexpr int kWaves = kThreads / kWave;
    a = wave_reduce(a, SumOp());
    b = wave_reduce(b, SumOp());
    if constexpr (kWaves > 1) {
        const int wid = threadIdx.x / kWave;
        if ((threadIdx.x % kWave) == 0) {
            scratch_a[wid] = a;
            scratch_b[wid] = b;
        }
        __syncthreads();
        double x = scratch_a[0], y = scratch_b[0];
#pragma unroll
        for (int i = 1; i < kWaves; ++i) {
            x += scratch_a[i];
            y += scratch_b[i];
        }
        __syncthreads();
        a = x;
        b = y;
    }
}

// kTrail = false: the first barrier only (as block_max_sum)
template <int kThreads, bool kTrail = true>
__device__ __forceinline__ ArgMin block_argmin(ArgMin v, ArgMin *scratch)
{
    constexpr int kWaves = kThreads / kWave;
    v = wave_argmin(v);
    const int wid = threadIdx.x / kWave;
    if ((threadIdx.x % kWave) == 0) scratch[wid] = v;
    __syncthreads();
    ArgMin r = scratch[0];
#pragma unroll
    for (int i = 1; i < kWaves; ++i) r = argmin_combine(r, scratch[i]);
    if constexpr (kTrail) __syncthreads();
    return r;
}

}  // namespace mpq
