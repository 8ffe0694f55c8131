// Host check of the routing kernel's small-divisor remainder, its Barrett
// constant and its bit select (the same inline functions the kernels use):
// prints one line per case for the test to compare with exact arithmetic.
#include <cstdio>
#include <cstdint>

#include "rr_device.hpp"

static uint64_t next(uint64_t &s)
{
    s ^= s << 13;
    s ^= s >> 7;
    s ^= s << 17;
    return s;
}

int main()
{
    uint64_t s = 0x9E3779B97F4A7C15ull;
    const uint32_t edge_m[] = {1u, 2u, 3u, 255u, 256u, 4095u, 4096u, 8191u, 8192u, 65535u};
    const uint64_t edge_x[] = {0ull, 1ull, 0xFFFFull, 0x10000ull, 0xFFFFFFFFull, 0x100000000ull,
                               0x8000000000000000ull, 0xFFFFFFFFFFFFFFFFull};
    for (uint32_t m : edge_m) {
        std::printf("div %u %llu\n", m, (unsigned long long)rr::max_u64_div_small(m));
        for (uint64_t x : edge_x)
            std::printf("mod %llu %u %u\n", (unsigned long long)x, m, rr::mod_u64_small(x, m));
    }
    for (int i = 0; i < 20000; ++i) {
        const uint64_t x = next(s);
        const uint32_t m = (uint32_t)(next(s) % 65535u) + 1u;
        std::printf("mod %llu %u %u\n", (unsigned long long)x, m, rr::mod_u64_small(x, m));
        if (i % 10 == 0) std::printf("div %u %llu\n", m, (unsigned long long)rr::max_u64_div_small(m));
        uint32_t z = (uint32_t)next(s);
        if (z == 0u) z = 1u;
        const int pc = __builtin_popcount(z);
        const int y = (int)(next(s) % (uint64_t)pc);
        std::printf("sel %u %d %d\n", z, y, rr::select_bit(z, y));
    }
    std::printf("arith driver ok\n");
    return 0;
}
