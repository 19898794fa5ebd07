// fp64 terms of the GPD likelihood sums (Grimshaw's reduction of the maximum-likelihood fit):
// for t = x*y > -1, a = t / (1 + t) and b = log1p(t).
#pragma once

#include <hip/hip_runtime.h>
#include <cmath>

namespace enova {

// ln 2 = kLn2Hi + kLn2Lo, kLn2Hi with 32 significant bits so k * kLn2Hi is exact for |k| < 2^21.
constexpr double kLn2Hi = 0x1.62e42fee00000p-1;
constexpr double kLn2Lo = 0x1.a39ef35793c76p-33;

// log1p by the classical argument reduction for logarithms (e.g. J.-M. Muller, Elementary
// Functions: Algorithms and Implementation, the chapter on logarithms): 1 + t = 2^k m with m in
// [sqrt(1/2), sqrt(2)), log m = 2 atanh(s) with s = (m - 1)/(m + 1), |s| <= 0.1716, whose series
// 2s (1 + s^2/3 + ... + s^18/19) is truncated below 2^-54 relative. What rounding 1 + t drops is
// added back to first order, c = (t - ((1 + t) - 1)) / (1 + t); 1/(1 + t) is shared with a.
__host__ __device__ inline void gpd_terms(double t, double &a, double &b)
{
    const double u = 1.0 + t;
    const double r = 1.0 / u;
    a = t * r;
    const double c = (t - (u - 1.0)) * r;
    int k;
    double m = std::frexp(u, &k);   // u = m 2^k, m in [1/2, 1)
    if (m < 0.70710678118654752440) {
        m *= 2.0;
        --k;
    }
    const double s = (m - 1.0) / (m + 1.0);
    const double z = s * s;
    double p = 1.0 / 19.0;
    p = p * z + 1.0 / 17.0;
    p = p * z + 1.0 / 15.0;
    p = p * z + 1.0 / 13.0;
    p = p * z + 1.0 / 11.0;
    p = p * z + 1.0 / 9.0;
    p = p * z + 1.0 / 7.0;
    p = p * z + 1.0 / 5.0;
    p = p * z + 1.0 / 3.0;
    const double lm = 2.0 * s + (2.0 * s * z) * p;
    const double kd = static_cast<double>(k);
    b = kd * kLn2Hi + (kd * kLn2Lo + (lm + c));
}

// Device form of gpd_terms: both quotients from the hardware reciprocal refined by two Newton
// steps (r <- r + r (1 - u r)), the second quotient corrected once more, and the exponent split of
// 1 + t read from its bits (frexp only for a subnormal or non-finite 1 + t); r = 1/(1 + t) is
// returned for the derivatives. The results stay within a few ulps of gpd_terms.
__device__ inline void gpd_terms_fast(double t, double &a, double &b, double &r)
{
    const double u = 1.0 + t;
    r = __builtin_amdgcn_rcp(u);
    r = fma(r, fma(-u, r, 1.0), r);
    r = fma(r, fma(-u, r, 1.0), r);
    a = t * r;
    const double c = (t - (u - 1.0)) * r;
    const long long bits = __double_as_longlong(u);
    const int ebits = static_cast<int>((bits >> 52) & 0x7ff);
    int k;
    double m;
    if (ebits == 0 || ebits == 0x7ff) {
        m = frexp(u, &k);
    } else {
        k = ebits - 1022;
        m = __longlong_as_double((bits & static_cast<long long>(0x800fffffffffffffULL)) | 0x3fe0000000000000LL);
    }
    if (m < 0.70710678118654752440) {
        m *= 2.0;
        --k;
    }
    const double d = m + 1.0, nm = m - 1.0;
    double rd = __builtin_amdgcn_rcp(d);
    rd = fma(rd, fma(-d, rd, 1.0), rd);
    rd = fma(rd, fma(-d, rd, 1.0), rd);
    double s = nm * rd;
    s = fma(rd, fma(-d, s, nm), s);
    const double z = s * s;
    double p = 1.0 / 19.0;
    p = p * z + 1.0 / 17.0;
    p = p * z + 1.0 / 15.0;
    p = p * z + 1.0 / 13.0;
    p = p * z + 1.0 / 11.0;
    p = p * z + 1.0 / 9.0;
    p = p * z + 1.0 / 7.0;
    p = p * z + 1.0 / 5.0;
    p = p * z + 1.0 / 3.0;
    const double lm = 2.0 * s + (2.0 * s * z) * p;
    const double kd = static_cast<double>(k);
    b = kd * kLn2Hi + (kd * kLn2Lo + (lm + c));
}

__device__ inline void gpd_terms_fast(double t, double &a, double &b)
{
    double r;
    gpd_terms_fast(t, a, b, r);
}

}  // namespace enova
