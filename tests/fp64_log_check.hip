// Host check of log_positive (paper_2106_05373_amd/csrc/fp64_log.h), the fp64 log of the MI
// kernel, against the C library's log: at most one ulp apart over 6 million arguments (wide
// range, and ratios within 1e-3 and 1e-8 of one, where mutual-information terms sit).
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <cmath>

#include "fp64_log.h"

static int64_t bits(double d) {
    int64_t i;
    memcpy(&i, &d, 8);
    return i;
}

int main() {
    uint64_t st = 88172645463325252ull;
    int64_t worst = 0, differ = 0, n = 0;
    double wx = 0.0;
    for (int it = 0; it < 6000000; ++it) {
        st ^= st << 13;
        st ^= st >> 7;
        st ^= st << 17;
        const double u = (double)(st >> 11) * 0x1p-53;
        const double x = it % 3 == 0 ? std::exp(-40.0 + 80.0 * u)
                       : it % 3 == 1 ? 1.0 + (u - 0.5) * 1e-3
                                     : 1.0 + (u - 0.5) * 1e-8;
        const int64_t d = bits(bcpnn::log_positive(x)) - bits(std::log(x));
        const int64_t a = d < 0 ? -d : d;
        differ += a != 0;
        ++n;
        if (a > worst) {
            worst = a;
            wx = x;
        }
    }
    printf("max ulp difference %lld (x = %.17g), %lld of %lld differ\n", (long long)worst, wx,
           (long long)differ, (long long)n);
    return worst <= 1 ? 0 : 1;
}
