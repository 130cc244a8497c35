// The code of one element at a point's scale (Eq. (10)): the fp64 quotient
// r / a rounded to nearest, ties to even, and clipped to [-M, M].
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>

namespace mpq {

// First in fp32: with 2^-100 <= a <= 2^100, y32 = fl32(r) fl32(1 / a) is
// within |y| 3 2^-24 of r / a, under 2^-12 for |y| < 2^10 (larger quotients
// clip to the same M either way), so unless y32 lies within 2^-12 of a
// half-integer it rounds as r / a does.  Else in fp64: y is within |y| 2^-51
// of the fp64 quotient fl(r / a), and only within 2^-40 of a half-integer is
// the quotient formed.
struct PointCode {
    double ap, ia, Md;
    float ia32, Mf;
    bool fast;

    __device__ __forceinline__ PointCode(float a, int M)
        : ap((double)a), ia(1.0 / (double)a), Md((double)M), ia32((float)(1.0 / (double)a)),
          Mf((float)M), fast((double)a >= 0x1p-100 && (double)a <= 0x1p100)
    {
    }

    __device__ __forceinline__ double operator()(double ru) const
    {
        if (fast) {
            const float y32 = (float)ru * ia32;
            const float c32 = rintf(y32);
            if (fabsf(fabsf(y32 - c32) - 0.5f) > 0x1p-12f) return (double)fminf(fmaxf(c32, -Mf), Mf);
        }
        const double y = ru * ia;
        double c = rint(y);
        if (fabs(fabs(y - c) - 0.5) < 0x1p-40) c = rint(ru / ap);
        return fmin(fmax(c, -Md), Md);
    }
};

}  // namespace mpq
