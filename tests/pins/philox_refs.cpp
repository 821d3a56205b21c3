// Independent Philox4x32-10 implementations used only to pin the oracle:
// PyTorch's header-only engine (ATen/core/PhiloxRNGEngine.h) and rocRAND's
// header-only engine (rocrand/rocrand_philox4x32_10.h), both open source.
// Reads lines "c0 c1 c2 c3 k0 k1" (hex) from stdin and prints, per line, the
// block from each implementation: "<torch 4 words> <rocrand 4 words or ->".
// rocRAND addresses the counter as (offset / 4, subsequence), so it is only
// asked when the 64-bit block index (c1:c0) is below 2^62.
#include <ATen/core/PhiloxRNGEngine.h>
#include <rocrand/rocrand_philox4x32_10.h>

#include <cinttypes>
#include <cstdio>

int main()
{
    unsigned c0, c1, c2, c3, k0, k1;
    while (std::scanf("%x %x %x %x %x %x", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
        const uint64_t key = (uint64_t)k0 | ((uint64_t)k1 << 32);
        const uint64_t lo = (uint64_t)c0 | ((uint64_t)c1 << 32);
        const uint64_t hi = (uint64_t)c2 | ((uint64_t)c3 << 32);
        at::Philox4_32 t(key, hi, lo);
        unsigned a = t(), b = t(), c = t(), d = t();
        std::printf("%08x %08x %08x %08x", a, b, c, d);
        if (lo < (1ULL << 62)) {
            rocrand_device::philox4x32_10_engine r(key, hi, lo * 4ULL);
            uint4 v = r.next4();
            std::printf(" %08x %08x %08x %08x\n", v.x, v.y, v.z, v.w);
        } else {
            std::printf(" -\n");
        }
    }
    return 0;
}
