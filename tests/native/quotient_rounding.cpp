// Host check of the fast quotient rounding used by every normalisation kernel: bf16_rne_quotient(v, n,
// quotient_rcp_f32(n)) of a float32 v must equal bf16_rne_from_f64(v / n) bit for bit.  Random quotients,
// quotients placed on bfloat16 rounding midpoints and 0 to 40 float32 units in the last place to either side
// of them, powers of two, norms whose reciprocal is no normal float32, and the subnormal range.  Also checks
// the error bound the fast path rests on: the float32 product stays within 2 float32 units of the double
// quotient.  Prints the number of cases and the largest error seen; exits non-zero on the first failure.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>

#include "common.hpp"

using lacache::bf16_rne_from_f64;
using lacache::bf16_rne_quotient;
using lacache::quotient_rcp_f32;

static double max_err_ulps = 0.0;

static int check(float v, double n, long long& count) {
    ++count;
    const float rnf = quotient_rcp_f32(n);
    const double q = (double)v / n;
    const uint16_t want = bf16_rne_from_f64(q), got = bf16_rne_quotient(v, n, rnf);
    if (want != got) {
        std::printf("MISMATCH v=%.9g n=%.17g want=%04x got=%04x\n", (double)v, n, want, got);
        return 1;
    }
    // the bound behind the fallback window (4 units): |v * rnf - q| in units of the float32 product's binade
    const float f = v * rnf;
    if (rnf != 0.0f && std::fabs(f) >= 0x1p-125) {
        int e;
        std::frexp(std::fabs(f), &e);
        const double err = std::fabs((double)f - q) / std::ldexp(1.0, e - 24);
        if (err > max_err_ulps) max_err_ulps = err;
        if (err > 2.000001) {
            std::printf("BOUND v=%.9g n=%.17g error %.3f units\n", (double)v, n, err);
            return 1;
        }
    }
    return 0;
}

int main(int argc, char** argv) {
    const long long iters = argc > 1 ? std::atoll(argv[1]) : 2000000;
    std::mt19937_64 g(12345);
    std::uniform_real_distribution<double> u(-1.0, 1.0), pos(0.5, 2.0);
    std::uniform_int_distribution<int> ex(-120, 4), step(-40, 40);
    long long count = 0;
    for (long long it = 0; it < iters; ++it) {
        // random float32 value over a norm-like double
        const double n = pos(g) * std::ldexp(1.0, ex(g) / 4 + 3);
        if (check((float)(u(g) * n), n, count)) return 1;

        // quotients on a bfloat16 rounding midpoint (an 8-bit significand plus one half) and 0 .. 40 float32
        // units from it (the fallback window is 4), each from a float32 v and the double norm v / target
        const double mid = std::ldexp((double)(128 + (g() % 128)) + 0.5, ex(g) / 2 - 7);
        const float v = (float)(std::ldexp(u(g), step(g) / 4));
        if (v != 0.0f) {
            int e;
            std::frexp(mid, &e);
            const double unit = std::ldexp(1.0, e - 24);
            static const int offs[] = {0, 1, 2, 3, 4, 5, 6, 7, 8, 12, 16, 20, 24, 32, 40};
            for (int k : offs)
                for (int dir = -1; dir <= 1; dir += 2) {
                    const double t = mid + dir * k * unit;
                    const double nn = std::fabs((double)v / t);
                    if (check(v, nn, count) || check(-v, nn, count)) return 1;
                    // and the norm nudged by a few double units either way
                    double lo = nn, hi = nn;
                    for (int s = 1; s <= 3; ++s) {
                        lo = std::nextafter(lo, 0.0);
                        hi = std::nextafter(hi, 1e300);
                        if (check(v, lo, count) || check(v, hi, count)) return 1;
                    }
                }
        }
        // quotients exactly on a midpoint: v = mid * m * 2^s and n = m * 2^s for a small odd m
        const double m = (double)(2 * (g() % 64) + 1);
        const int s = step(g) / 2;
        const double vm = mid * m * std::ldexp(1.0, s);
        if ((double)(float)vm == vm && check((float)vm, m * std::ldexp(1.0, s), count)) return 1;

        // exact and near powers of two
        const double p2 = std::ldexp(1.0, ex(g));
        const float vp = (float)std::ldexp(pos(g), step(g) / 4);
        if (check(vp, vp / p2, count) || check(vp, std::nextafter(vp / p2, 0.0), count)) return 1;

        // normalisation-shaped: v an input value, n a norm of a vector holding it
        const float w = (float)std::ldexp(u(g), step(g));
        if (check(w, std::sqrt((double)w * w + pos(g)), count)) return 1;

        // norms whose reciprocal is no normal float32 (huge or tiny vectors): every element divides
        const float big = (float)(u(g) * 3e38), tiny = (float)(u(g) * 1e-44);
        if (check(big, std::fabs((double)big) * 1.5 + 1e38, count)) return 1;
        if (check(tiny, std::fabs((double)tiny) * 1.5 + 1e-44, count)) return 1;
        if (check(0.0f, pos(g), count)) return 1;
    }
    std::printf("ok %lld max error %.3f units\n", count, max_err_ulps);
    return 0;
}
