// Host check of na::FastDiv (paper_2403_04690_amd/csrc/na_fastdiv.h), built and
// run by tests/test_fastdiv.py with the host compiler.
//   * every divisor 1 <= d < 2^20: the device's double-division multiplier
//     equals the host's integer one, and for powers of two both are 1 (the
//     device takes that value without dividing);
//   * for those divisors and sampled larger ones up to 2^31 - 1: n / d is exact
//     for dividends at the edges (0, 1, d - 1, d, d + 1, multiples of d and
//     their neighbours, 2^31 - 1) and for pseudo-random n < 2^31.
// Prints "ok <divisors> <divisions>" or the first failure, and exits nonzero on
// failure.
#include <cstdint>
#include <cstdio>

#include "na_fastdiv.h"

static uint64_t rng_state = 0x9e3779b97f4a7c15ull;
static uint32_t next31() {  // splitmix64, top 31 bits
    uint64_t z = (rng_state += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    z ^= z >> 31;
    return (uint32_t)(z >> 33);
}

static long long divisions = 0;

static bool check_div(int d, int n, uint32_t mul, uint32_t shr) {
    ++divisions;
    const int got = na::FastDiv::divide(n, mul, shr);
    if (got != n / d) {
        std::printf("FAIL d=%d n=%d got %d want %d (mul %u shr %u)\n", d, n, got, n / d, mul, shr);
        return false;
    }
    return true;
}

static bool check_divisor(int d, int randoms) {
    na::FastDiv f;
    f.init(d);  // host build: the integer path
    const uint32_t s = na::FastDiv::shift_for(d);
    if (f.shr != s || f.mul != na::FastDiv::mul_int(d, s)) {
        std::printf("FAIL init d=%d\n", d);
        return false;
    }
    const int edges[] = {0, 1, d - 1, d, d + 1, 2 * d - 1, 2 * d, 0x7fffffff, 0x7ffffffe};
    for (int n : edges)
        if (n >= 0 && !check_div(d, n, f.mul, f.shr)) return false;
    const int64_t top = (int64_t)(0x7fffffff / d) * d;  // largest multiple of d below 2^31
    for (int64_t n = top - 1; n <= top + 1; ++n)
        if (n >= 0 && n <= 0x7fffffff && !check_div(d, (int)n, f.mul, f.shr)) return false;
    for (int i = 0; i < randoms; ++i) {
        const int n = (int)next31();
        if (!check_div(d, n, f.mul, f.shr)) return false;
        const int m = (int)(next31() % (uint32_t)(d < 4096 ? 65536 : d * 4 + 1));
        if (!check_div(d, m & 0x7fffffff, f.mul, f.shr)) return false;
    }
    return true;
}

int main() {
    long long divisors = 0;
    for (int d = 1; d < (1 << 20); ++d, ++divisors) {
        const uint32_t s = na::FastDiv::shift_for(d);
        const uint32_t mi = na::FastDiv::mul_int(d, s), md = na::FastDiv::mul_double(d, s);
        if (mi != md) {
            std::printf("FAIL multiplier d=%d int %u double %u\n", d, mi, md);
            return 1;
        }
        if ((d & (d - 1)) == 0 && (mi != 1u || (1 << s) != d)) {  // the device's power-of-two path
            std::printf("FAIL power of two d=%d mul %u shift %u\n", d, mi, s);
            return 1;
        }
        if (!check_divisor(d, 16)) return 1;
    }
    for (int i = 0; i < 200000; ++i, ++divisors) {  // larger divisors: the integer path only
        const int d = (int)(next31() | 1u) >> (i % 11);
        if (d >= 1 && !check_divisor(d, 16)) return 1;
    }
    const int powers[] = {1 << 20, (1 << 20) + 1, 1 << 30, (1 << 30) + 1, 0x7fffffff};
    for (int d : powers) {
        ++divisors;
        if (!check_divisor(d, 1000)) return 1;
    }
    std::printf("ok %lld %lld\n", divisors, divisions);
    return 0;
}
