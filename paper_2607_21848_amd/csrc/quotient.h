// Correctly rounded double quotients that share one reciprocal.
//
// q(a, b) = RN(a / b) from y = RN(1 / b) with one correction step:
//     q0 = RN(a y),  r = a - b q0 (exact: one fused multiply-add),
//     q  = RN(q0 + r y)
// Markstein's theorem (P. Markstein, IBM J. Res. Dev. 34(1), 1990; also
// Muller et al., Handbook of Floating-Point Arithmetic, the FMA-based division
// section) gives q = RN(a / b) when y is the correctly rounded reciprocal,
// q0 is within one unit in the last place of a / b, and no intermediate
// underflows or overflows. Callers use it only where they have established
// that range condition (every operand and intermediate well inside the
// normal range, a != -0); everywhere else they divide. One division then
// serves several quotients over the same denominator.
#pragma once

#if defined(__HIP__) || defined(__HIPCC__)
#define REVISIT_HD __host__ __device__
#else
#define REVISIT_HD
#endif

#include <math.h>

namespace revisit {

REVISIT_HD inline double quotient_from_reciprocal(double a, double b, double y) {
    const double q0 = a * y;
    const double r = fma(-q0, b, a);
    return fma(r, y, q0);
}

}  // namespace revisit
