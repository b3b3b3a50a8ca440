// Host check of the fast quotient rounding used by every normalisation kernel: bf16_rne_quotient(v, n, 1/n)
// must equal bf16_rne_from_f64(v / n) bit for bit.  Random quotients, quotients placed on and around bfloat16
// rounding midpoints, powers of two, and the subnormal range.  Prints the number of cases and exits non-zero
// on the first mismatch.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>

#include "common.hpp"

using lacache::bf16_rne_from_f64;
using lacache::bf16_rne_quotient;

static int check(double v, double n, long long& count) {
    ++count;
    const uint16_t want = bf16_rne_from_f64(v / n), got = bf16_rne_quotient(v, n, 1.0 / n);
    if (want != got) {
        std::printf("MISMATCH v=%.17g n=%.17g want=%04x got=%04x\n", v, n, want, got);
        return 1;
    }
    return 0;
}

int main(int argc, char** argv) {
    const long long iters = argc > 1 ? std::atoll(argv[1]) : 2000000;
    std::mt19937_64 g(12345);
    std::uniform_real_distribution<double> u(-1.0, 1.0), pos(0.5, 2.0);
    std::uniform_int_distribution<int> ex(-140, 4), step(-40, 40);
    long long count = 0;
    for (long long it = 0; it < iters; ++it) {
        const double n = pos(g) * std::ldexp(1.0, ex(g) / 8 + 3);
        // random quotient
        if (check(u(g) * n, n, count)) return 1;
        // a quotient on a bfloat16 rounding midpoint (an 8-bit significand plus one half), and nudged by
        // 1 .. 40 units in the last place of a double to either side (the fallback window is 16 units)
        const double m = (double)(128 + (g() % 128)) + 0.5;
        const double mid = std::ldexp(m, ex(g) - 7);
        static const int nudges[] = {0, 1, 2, 3, 8, 15, 16, 17, 20, 40};
        for (int k : nudges) {
            for (int dir = -1; dir <= 1; dir += 2) {
                double q = mid;
                for (int s = 0; s < k; ++s) q = std::nextafter(q, dir > 0 ? 4.0 : 0.0);
                if (check(q * n, n, count) || check(-q * n, n, count)) return 1;
            }
        }
        // exact and near powers of two
        const double p2 = std::ldexp(1.0, ex(g));
        if (check(p2 * n, n, count) || check(std::nextafter(p2, 0.0) * n, n, count)) return 1;
        // integer-ratio inputs as normalisation produces them: v an input value, n a norm
        const double v = std::ldexp(u(g), step(g));
        if (check(v, std::sqrt(v * v + pos(g)), count)) return 1;
    }
    std::printf("ok %lld\n", count);
    return 0;
}
