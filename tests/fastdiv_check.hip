// Host-side check of the library's division by launch constants (FastDiv in
// csrc/internal.h) against plain integer division: every divisor below 5000
// with every numerator below 20000 plus 2000 random numerators below 2^31,
// a stride of larger divisors, and the edge numerators near 2^31.
// Prints "ok <count>" and exits 0, or the first mismatch and exits 1.
#include "../paper_1907_02154_amd/csrc/internal.h"

#include <cstdio>

using miconv::FastDiv;

static int check(unsigned n, unsigned d, FastDiv f, unsigned long long *count)
{
    ++*count;
    if (miconv::fdiv(n, f) == n / d) return 0;
    std::printf("mismatch: %u / %u gave %u\n", n, d, miconv::fdiv(n, f));
    return 1;
}

int main()
{
    unsigned long long count = 0;
    unsigned s = 12345u;
    for (unsigned d = 1; d < 70000; d += d < 5000 ? 1 : 37) {
        const FastDiv f = miconv::make_fastdiv(d);
        for (unsigned n = 0; n < 20000; ++n)
            if (check(n, d, f, &count)) return 1;
        for (int i = 0; i < 2000; ++i) {
            s = s * 1664525u + 1013904223u;
            if (check(s & 0x7fffffffu, d, f, &count)) return 1;
        }
        const unsigned top = 0x7fffffffu / d * d;
        const unsigned edge[4] = {0x7fffffffu, 0x7ffffffeu, top, top - 1};
        for (unsigned e : edge)
            if (check(e, d, f, &count)) return 1;
    }
    const unsigned big[5] = {0x40000000u, 0x40000001u, 0x3fffffffu, 1000000007u, 0x7fffffffu};
    for (unsigned d : big) {
        const FastDiv f = miconv::make_fastdiv(d);
        for (int i = 0; i < 100000; ++i) {
            s = s * 1664525u + 1013904223u;
            if (check(s & 0x7fffffffu, d, f, &count)) return 1;
        }
    }
    std::printf("ok %llu\n", count);
    return 0;
}
