// Exhaustive-ish check of the multiply-shift division constants built by
// make_fastdiv (Granlund and Montgomery, PLDI 1994, Fig. 4.1): for every
// divisor tried, n / d == (t + ((n - t) >> s1)) >> s2 with t = mulhi(n, m),
// the form the kernels evaluate.  Prints the number of cases and failures;
// exits non-zero on any failure.
#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

#include "isoq_internal.h"

using isoq::FastDiv;

static uint32_t divide(uint32_t n, const FastDiv &f)
{
    const uint32_t t = (uint32_t)(((uint64_t)n * f.m) >> 32);
    return (t + ((n - t) >> f.s1)) >> f.s2;
}

int main()
{
    std::mt19937_64 rng(1);
    std::vector<uint32_t> ds;
    for (uint32_t d = 1; d <= 5000; d++)
        ds.push_back(d);
    for (int k = 1; k < 32; k++) {
        ds.push_back(1u << k);
        ds.push_back((1u << k) - 1);
        if (k < 31)
            ds.push_back((1u << k) + 1);
    }
    ds.push_back(0xFFFFFFFFu);
    for (int i = 0; i < 2000; i++)
        ds.push_back(1 + (uint32_t)(rng() % 0xFFFFFFFFull));
    long bad = 0, total = 0;
    for (uint32_t d : ds) {
        const FastDiv f = isoq::make_fastdiv(d);
        std::vector<uint32_t> ns = {0, 1, d - 1, d, d + 1, 2 * d - 1, 2 * d, 0x7FFFFFFF, 0xFFFFFFFF, 0xFFFFFFFE};
        for (int i = 0; i < 2000; i++)
            ns.push_back((uint32_t)rng());
        for (int i = 0; i < 200; i++)
            ns.push_back((uint32_t)(rng() % 100000));
        // values just below and at multiples of d, where a wrong rounding shows
        for (int i = 0; i < 50; i++) {
            const uint64_t q = rng() % (0xFFFFFFFFull / d + 1);
            const uint64_t v = q * d;
            if (v <= 0xFFFFFFFFull)
                ns.push_back((uint32_t)v);
            if (v >= 1 && v - 1 <= 0xFFFFFFFFull)
                ns.push_back((uint32_t)(v - 1));
        }
        for (uint32_t n : ns) {
            total++;
            if (divide(n, f) != n / d) {
                if (bad < 5)
                    std::printf("mismatch d=%u n=%u\n", d, n);
                bad++;
            }
        }
    }
    std::printf("checked %ld failures %ld\n", total, bad);
    return bad != 0;
}
