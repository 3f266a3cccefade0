// Host-side check of the multiply-high remainder the kernels use for ring
// and pool indices (sifar_kernels.h): against the % operator on every
// divisor 1..4096 with edge and random dividends, and on large divisors.
// Built and run by tests/test_divmod.py on the CPU (no GPU call).
#include <cstdio>
#include <cstdint>
#include <random>

#include "sifar_kernels.h"

int main() {
    using sifar::make_div;
    using sifar::mod_u32;
    std::mt19937_64 rng(260708973);
    uint64_t checked = 0;
    auto check = [&](uint32_t d, uint32_t x) -> bool {
        const uint32_t got = mod_u32(x, make_div(d));
        ++checked;
        if (got != x % d) {
            std::printf("FAIL d=%u x=%u got=%u want=%u\n", d, x, got, x % d);
            return false;
        }
        return true;
    };
    const uint32_t edges[] = {0u, 1u, 2u, 3u, 63u, 64u, 65u, 0x7FFFFFFFu, 0x80000000u,
                              0x80000001u, 0xFFFFFFFEu, 0xFFFFFFFFu};
    for (uint32_t d = 1; d <= 4096; ++d) {
        for (uint32_t x : edges)
            if (!check(d, x)) return 1;
        for (uint32_t k = 1; k < 4; ++k)
            if (!check(d, d * k - 1) || !check(d, d * k) || !check(d, d * k + 1)) return 1;
        for (int i = 0; i < 2000; ++i)
            if (!check(d, static_cast<uint32_t>(rng()))) return 1;
    }
    for (int i = 0; i < 200000; ++i) {
        const uint32_t d = static_cast<uint32_t>(rng()) | 1u;
        const uint32_t e = static_cast<uint32_t>(rng()) >> (rng() % 32);
        if (!check(d, static_cast<uint32_t>(rng())) || !check(e ? e : 1u, static_cast<uint32_t>(rng())))
            return 1;
    }
    for (uint32_t x : edges)
        for (uint32_t d : edges)
            if (d && !check(d, x)) return 1;
    std::printf("ok %llu\n", static_cast<unsigned long long>(checked));
    return 0;
}
