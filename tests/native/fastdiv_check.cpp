// Host-side check of the launch-constant divisions the kernels use:
// FastDiv::make(d).div(n) must equal n / d for every n < 2^31.  Exhaustive over n for
// small divisors, and over the n that sit next to multiples of d (where an off-by-one
// in the multiplier shows first) for divisors up to 2^24 plus random ones.
// WindowAddr (window-local index t -> byte offset and token index) must split t into
// row t / cols and column t % cols for every window width and every t of its window.
#include "fla_swin_device.h"

#include <cstdio>
#include <cstdint>
#include <algorithm>
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
    // window widths 1 .. 4096, and t over the window-local indices the host admits
    // (t < n with n * cols <= 2^32, n <= 4096 * cols), sampled densely near multiples of cols
    for (int c = 1; c <= 4096 && !bad; ++c) {
        fla::WindowAddr a;
        a.init(c, 1000003u, 7u);
        const unsigned long long nmax = std::min<unsigned long long>(4096ull * c, (1ull << 32) / c);
        const unsigned long long tmax = nmax;
        for (unsigned r = 0; r < 4096 && !bad; r += (c < 64 ? 1 : 37)) {
            for (int dc = -1; dc <= 1 && !bad; ++dc) {
                const long long t = (long long)r * c + (dc < 0 ? c - 1 : dc == 0 ? 0 : c / 2);
                if (t < 0 || (unsigned long long)t >= tmax) continue;
                const unsigned want_r = (unsigned)t / c, want_c = (unsigned)t % c;
                if (a((int)t) != want_r * 1000003u + want_c * 7u || a.token((int)t, 5000u) != want_r * 5000u + want_c) {
                    std::printf("FAIL WindowAddr cols=%d t=%lld\n", c, t);
                    bad = 1;
                }
            }
        }
    }
    std::printf(bad ? "fastdiv FAILED\n" : "fastdiv OK\n");
    return bad;
}
