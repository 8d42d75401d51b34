// Host check of the library's index division (csrc/nlb_divide.h), the same
// source the kernels compile.  Built and run by tests/test_divide.py.
//
// The kernels split flat indices f < rows * units into (row f / units,
// column f mod units) with rows <= 1024 slot rows per sample tile and
// units <= 65536 copy units per row (rows of up to 2^18 bytes in 4-byte
// units, time encodings of up to 65535 values), and the time-encoding
// stream divides any 32-bit flat index by the units per row and the slot
// row by s (1 included); the insert takes remainders mod s.  Prints
// "ok <checks>" or the first failure.
#include <cstdio>
#include <cstdint>
#include <cstdlib>

#include "nlb_divide.h"

static uint64_t checks = 0;

static void fail(const char *what, uint32_t f, uint32_t d, uint64_t got, uint64_t want) {
    std::printf("FAIL %s f=%u d=%u got=%llu want=%llu\n", what, f, d, (unsigned long long)got,
                (unsigned long long)want);
    std::exit(1);
}

struct Magic {
    uint64_t div, mod;
    explicit Magic(uint32_t d) : div(nlb_div_magic(d)), mod(nlb_mod_magic(d)) {}
};

static void check(uint32_t f, uint32_t d, const Magic &M) {
    const uint32_t q = nlb_div(f, M.div), r = nlb_mod(f, M.mod, d);
    if (q != f / d) fail("div", f, d, q, f / d);
    if (r != f % d) fail("mod", f, d, r, f % d);
    checks++;
}

// The helper the library used first: floor(f * ceil(2^40 / d) / 2^40), exact
// only while f * d < 2^40.  Counted to show that the boundary set below
// finds its errors.
static uint32_t old_div(uint32_t f, uint32_t d) {
    const uint64_t m = ((1ull << 40) + d - 1) / d;
    return (uint32_t)(((uint64_t)f * m) >> 40);
}

int main() {
    uint64_t old_wrong = 0;
    // Every divisor of a row split and every row boundary of a tile: the
    // last unit of row k - 1 and the first of row k.
    for (uint32_t d = 1; d <= 65536; d++) {
        const Magic M(d);
        check(0, d, M);
        for (uint32_t k = 1; k <= 1024; k++) {
            const uint32_t f = k * d;
            check(f - 1, d, M);
            check(f, d, M);
            if (old_div(f - 1, d) != k - 1 || old_div(f, d) != k) old_wrong++;
        }
    }
    // Every numerator below 2^26 (the largest tile range) for a set of
    // divisors: powers of two and their neighbours, and row widths in use.
    const uint32_t some[] = {1, 2, 3, 4, 5, 7, 10, 25, 63, 64, 65, 100, 127, 128, 129, 1023, 1024, 1025,
                             4095, 32767, 32768, 32769, 65535, 65536};
    for (uint32_t d : some) {
        const Magic M(d);
        for (uint32_t f = 0; f < (1u << 26); f++) check(f, d, M);
    }
    // Whole 32-bit range: boundaries of every quotient (sampled for small
    // divisors), and the extremes for all divisors up to 2^20.
    const uint32_t big[] = {1u, 2u, 3u, 10u, 64u, 1000u, 65535u, 65537u, 1u << 20, (1u << 31) - 1,
                            1u << 31, (1u << 31) + 1, 0xC0000001u, 0xFFFFFFFEu, 0xFFFFFFFFu};
    for (uint32_t d : big) {
        const Magic M(d);
        const uint64_t qmax = 0xFFFFFFFFull / d;
        const uint64_t step = qmax > (1u << 22) ? qmax >> 22 : 1;
        for (uint64_t q = 1; q <= qmax; q += step) {
            check((uint32_t)(q * d - 1), d, M);
            check((uint32_t)(q * d), d, M);
        }
        check(0xFFFFFFFFu, d, M);
    }
    for (uint32_t d = 1; d <= (1u << 20); d++) {
        const Magic M(d);
        check(0xFFFFFFFFu, d, M);
        check(0xFFFFFFFFu - 0xFFFFFFFFu % d, d, M);
        check(0xFFFFFFFFu - 0xFFFFFFFFu % d - 1, d, M);
    }
    // The 12-bit form: every numerator below 2^12 for every divisor up to
    // 2^12 (the slot rows of a tile, divided by s).
    for (uint32_t d = 1; d <= 4096; d++) {
        const uint64_t m12 = nlb_div12_magic(d);
        for (uint32_t f = 0; f < 4096; f++) {
            const uint32_t q = nlb_div12(f, m12);
            if (q != f / d) fail("div12", f, d, q, f / d);
            checks++;
        }
    }
    // Seeded random pairs (SplitMix64 output function as the source).
    uint64_t z = 12345;
    for (int i = 0; i < 20000000; i++) {
        uint64_t x = (z += 0x9E3779B97F4A7C15ull);
        x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
        x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
        x ^= x >> 31;
        uint32_t d = (uint32_t)(x >> 32);
        const int shift = (int)(x & 31);
        d >>= shift;
        if (d == 0) d = 1;
        check((uint32_t)x, d, Magic(d));
    }
    std::printf("ok %llu checks; the replaced helper was wrong at %llu row boundaries\n",
                (unsigned long long)checks, (unsigned long long)old_wrong);
    return 0;
}
