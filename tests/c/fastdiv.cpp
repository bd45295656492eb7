// Host-only test of the 32-bit invariant division used by the tree-step decode (FastDiv32):
// exact quotients for every divisor up to 2^16 at the extreme dividends, and for seeded random
// divisors and dividends below 2^31, against the hardware division. Exit status 0 on success.
#include <cstdint>
#include <cstdio>

#include "plan.h"

static uint64_t state = 0x9E3779B97F4A7C15ull;
static uint32_t next32() {  // xorshift64*
    state ^= state >> 12;
    state ^= state << 25;
    state ^= state >> 27;
    return (uint32_t)((state * 0x2545F4914F6CDD1Dull) >> 32);
}

int main() {
    long failures = 0;
    auto check = [&](uint32_t x, uint32_t d) {
        const trivance::FastDiv32 f = trivance::make_fastdiv32(d);
        if (trivance::fastdiv32_host(x, f) != x / d) {
            if (failures < 5) std::fprintf(stderr, "x=%u d=%u: %u != %u\n", x, d,
                                            trivance::fastdiv32_host(x, f), x / d);
            ++failures;
        }
    };
    const uint32_t top = 0x7FFFFFFFu;  // largest dividend
    for (uint32_t d = 1; d <= 65536; ++d) {
        for (uint32_t x : {0u, 1u, d - 1, d, d + 1, 2 * d - 1, top, top - 1, top - d, top / d * d,
                           top / d * d - 1})
            if (x <= top) check(x, d);
        for (int i = 0; i < 8; ++i) check(next32() & top, d);
    }
    for (uint32_t d : {(1u << 31) - 1, 1u << 30, (1u << 30) + 1, 2199u * 2200u, 1000003u}) {
        for (uint32_t x : {0u, 1u, d - 1, d, top}) if (x <= top) check(x, d);
    }
    for (int i = 0; i < 4000000; ++i) {
        const uint32_t d = (next32() >> (next32() % 31)) | 1u;
        check(next32() & top, d);
        check(next32() & top, d + 1 <= top ? d + 1 : d);
    }
    if (failures == 0) std::printf("fastdiv ok\n");
    return failures == 0 ? 0 : 1;
}
