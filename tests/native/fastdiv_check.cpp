// Host-side check of the launch-constant division used to decode workgroup indices:
// FastDiv::make(d).div(n) must equal n / d for every n < 2^31.  Exhaustive over n for
// small divisors, and over the n that sit next to multiples of d (where an off-by-one
// in the multiplier shows first) for divisors up to 2^24 plus random ones.
#include "fla_swin_internal.h"

#include <cstdio>
#include <cstdint>
#include <random>

static int check(unsigned d, unsigned n) {
    const unsigned got = fla::FastDiv::make(d).div(n);
    if (got != n / d) {
        std::printf("FAIL d=%u n=%u got=%u want=%u\n", d, n, got, n / d);
        return 1;
    }
    return 0;
}

int main() {
    int bad = 0;
    for (unsigned d = 1; d <= 64 && !bad; ++d)
        for (unsigned n = 0; n < (1u << 20) && !bad; ++n) bad |= check(d, n);
    std::mt19937_64 rng(12345);
    const unsigned top = 0x7fffffffu;
    for (int i = 0; i < 200000 && !bad; ++i) {
        unsigned d = i < 100000 ? (unsigned)(rng() % (1u << 24)) + 1 : (unsigned)(rng() % top) + 1;
        const unsigned long long qmax = top / d;
        for (int j = 0; j < 4 && !bad; ++j) {
            const unsigned long long qq = rng() % (qmax + 1);
            const unsigned long long base = qq * d;
            for (long long delta = -1; delta <= 1; ++delta) {
                const long long n = (long long)base + delta;
                if (n >= 0 && n <= (long long)top) bad |= check(d, (unsigned)n);
            }
            bad |= check(d, top);
        }
    }
    std::printf(bad ? "fastdiv FAILED\n" : "fastdiv OK\n");
    return bad;
}
