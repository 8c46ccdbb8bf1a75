// Natural logarithm of a positive normal double, about one ulp from the correctly rounded value
// (host and device, so that a host test can check it against the C library).  The method is the
// argument reduction and s = f / (2 + f) form of the public-domain fdlibm e_log.c (Sun
// Microsystems, 1993), with its split of ln 2 into a 32-bit head and a tail; the polynomial here
// is the plain atanh Taylor series, not fdlibm's minimax coefficients.
//
// x = 2^k m with m in [sqrt(1/2), sqrt(2)) and f = m - 1.  With s = f / (2 + f),
//   log(1 + f) = log((1 + s) / (1 - s)) = 2 atanh(s) = 2 s + s R(z),   z = s^2,
// R(z) = sum_{n >= 1} 2 z^n / (2n + 1) (the Taylor series of atanh; |s| <= 0.172 so ten terms
// leave a remainder below 2^-56 of the result), and 2 s = f - s f = f - h + s h with h = f^2 / 2,
// so log(1 + f) = f - (h - s (h + R)): the large terms f and h are exact or nearly so and the
// rounding of the small correction s (h + R) hardly matters.  k ln 2 is added as
// k * ln2_hi + k * ln2_lo with ln2_hi carrying 32 significant bits (exact for |k| < 2^21).
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>

namespace bcpnn {

__host__ __device__ inline double log_positive(double x) {
    constexpr double kLn2Hi = 0x1.62e42fee00000p-1;    // ln 2 to 32 bits
    constexpr double kLn2Lo = 0x1.a39ef35793c76p-33;   // ln 2 - kLn2Hi
    int e;
    double m = frexp(x, &e);                            // [1/2, 1)
    if (m < 0.70710678118654752440) {
        m *= 2.0;
        e -= 1;
    }
    const double f = m - 1.0;
    const double s = f / (2.0 + f);
    const double z = s * s;
    double r = 2.0 / 23;
    r = fma(r, z, 2.0 / 21);
    r = fma(r, z, 2.0 / 19);
    r = fma(r, z, 2.0 / 17);
    r = fma(r, z, 2.0 / 15);
    r = fma(r, z, 2.0 / 13);
    r = fma(r, z, 2.0 / 11);
    r = fma(r, z, 2.0 / 9);
    r = fma(r, z, 2.0 / 7);
    r = fma(r, z, 2.0 / 5);
    r = fma(r, z, 2.0 / 3);
    r *= z;
    const double h = 0.5 * f * f;
    const double k = (double)e;
    return k * kLn2Hi - ((h - fma(s, h + r, k * kLn2Lo)) - f);
}

}  // namespace bcpnn
