// Binary64 atan2 of the direction lookup, shared by the render kernels and
// the host-side accuracy test.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>

namespace sqn {

// atan2 in binary64 to within 2e-14 (tests/test_atan2_lookup.py checks it
// against numpy's arctan2 on random pairs of every octant and magnitude and
// on the signed zeros): octant reduction to t = min/max, then t > tan(pi/8)
// to (t - 1)/(t + 1) in one division, and an odd polynomial t + t^3 P(t^2)
// with P a least-squares fit of (atan(t) - t)/t^3 at Chebyshev nodes of
// [0, tan^2(pi/8)].  Signs and zeros follow atan2.  The direction lookup
// needs the angles to about 1e-8.
__host__ __device__ inline double atan2_lookup(double y, double x)
{
    constexpr double kPi = 3.14159265358979323846;
    constexpr double kTanPi8 = 0.41421356237309503;
    const double ax = fabs(x), ay = fabs(y);
    const double mx = fmax(ax, ay), mn = fmin(ax, ay);
    const bool big = mn > kTanPi8 * mx;
    const double num = big ? mn - mx : mn;
    const double den = big ? mn + mx : mx;
    const double t = den > 0.0 ? num / den : 0.0;
    const double s = t * t;
    double p = 0.03139479947774411;
    p = fma(p, s, -0.05926635751528511);
    p = fma(p, s, 0.0757883898701557);
    p = fma(p, s, -0.09080691227325184);
    p = fma(p, s, 0.11110579634656349);
    p = fma(p, s, -0.14285699429416587);
    p = fma(p, s, 0.1999999981132898);
    p = fma(p, s, -0.333333333326259);
    double r = fma(t * s, p, t);
    if (big)
        r += 0.25 * kPi;
    if (ay > ax)
        r = 0.5 * kPi - r;
    if (signbit(x))
        r = kPi - r;
    return copysign(r, y);
}

}  // namespace sqn
