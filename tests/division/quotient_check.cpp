// CPU check of revisit::quotient_from_reciprocal against IEEE division.
// Built with -ffp-contract=off; fma() is the correctly rounded library
// function. Prints the number of mismatches per family and exits 1 if any.
//
// Families (each a mix of signs):
//   config    operands in the ranges the reprojection kernel produces on the
//             configurations' scenes: b (the camera-frame depth) in
//             [1e-3, 1e3], a (the projected coordinate times depth) in
//             [-1e6, 1e6], and the lift's (u - c) / f with |u - c| <= 2^12,
//             f in [1, 4096];
//   wide      |a|, b log-uniform over [2^-500, 2^500];
//   hard      b with significands next to 1 and to 2 (all ones), a equal to
//             b times a small integer, plus or minus a few units, quotients
//             next to binade boundaries;
//   random    random significands with exponents in [-400, 400].
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../paper_2607_21848_amd/csrc/quotient.h"

static uint64_t state = 0x9E3779B97F4A7C15ull;
static uint64_t next_u64() {
    state ^= state << 13;
    state ^= state >> 7;
    state ^= state << 17;
    return state;
}
static double uniform01() { return (double)(next_u64() >> 11) * 0x1.0p-53; }
static double bits_to_double(uint64_t u) {
    double d;
    memcpy(&d, &u, 8);
    return d;
}
static uint64_t double_bits(double d) {
    uint64_t u;
    memcpy(&u, &d, 8);
    return u;
}
static double log_uniform(double lo_exp, double hi_exp) { return exp2(lo_exp + (hi_exp - lo_exp) * uniform01()); }
static double random_sign(double x) { return (next_u64() & 1) ? -x : x; }

static long checked = 0;
static int check(double a, double b, long* bad) {
    const double want = a / b;
    const double got = revisit::quotient_from_reciprocal(a, b, 1.0 / b);
    ++checked;
    if (double_bits(want) != double_bits(got)) {
        if (*bad < 5) fprintf(stderr, "mismatch: a=%a b=%a a/b=%a got %a\n", a, b, want, got);
        ++*bad;
        return 1;
    }
    return 0;
}

int main(int argc, char** argv) {
    const long n = argc > 1 ? atol(argv[1]) : 2000000;
    long bad_config = 0, bad_wide = 0, bad_hard = 0, bad_random = 0;
    for (long i = 0; i < n; ++i) {
        const double b = log_uniform(log2(1e-3), log2(1e3));
        const double a = random_sign(uniform01() * 1e6);
        check(a, b, &bad_config);
        // the lift: (u - c) / f with u a token centre, c, f fp32 intrinsics
        const double u = floor(uniform01() * 4096.0) + 0.5;
        const double c = (double)(float)(uniform01() * 4096.0);
        const double f = (double)(float)(1.0 + uniform01() * 4095.0);
        if (u != c) check(u - c, random_sign(f), &bad_config);
    }
    for (long i = 0; i < n; ++i) check(random_sign(log_uniform(-500, 500)), log_uniform(-500, 500), &bad_wide);
    for (long i = 0; i < n; ++i) {
        // significands next to 1 and to 2
        const uint64_t mant = (next_u64() & 1) ? (next_u64() & 0xFFFu) : (0xFFFFFFFFFFFFFull - (next_u64() & 0xFFFu));
        const int e = (int)(next_u64() % 200) - 100;
        const double b = ldexp(bits_to_double(0x3FF0000000000000ull | mant), e);
        const double k = (double)(1 + next_u64() % 1000);
        double a = b * k;
        const int steps = (int)(next_u64() % 9) - 4;
        for (int s = 0; s < abs(steps); ++s) a = nextafter(a, steps > 0 ? INFINITY : -INFINITY);
        check(random_sign(a), b, &bad_hard);
        // quotients next to powers of two: a = 2^j b (1 +- tiny)
        const double a2 = nextafter(ldexp(b, (int)(next_u64() % 40) - 20), (next_u64() & 1) ? INFINITY : 0.0);
        check(a2, b, &bad_hard);
    }
    for (long i = 0; i < n; ++i) {
        const double a = ldexp(1.0 + uniform01(), (int)(next_u64() % 801) - 400);
        const double b = ldexp(1.0 + uniform01(), (int)(next_u64() % 801) - 400);
        check(random_sign(a), b, &bad_random);
    }
    printf("quotient_from_reciprocal: %ld quotients; mismatches config %ld, wide %ld, hard %ld, random %ld\n",
           checked, bad_config, bad_wide, bad_hard, bad_random);
    return (bad_config | bad_wide | bad_hard | bad_random) ? 1 : 0;
}
