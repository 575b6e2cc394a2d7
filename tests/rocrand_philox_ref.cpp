// Independent reference stream for the oracle's Philox4x32-10 counter mapping:
// rocRAND's host-callable engine, seeded with (seed, subsequence = offset,
// skip = 4 * g), returns the block for counter (g lo, g hi, offset lo, offset hi)
// and key (seed lo, seed hi).  Reads "seed offset g" triples (decimal) from
// stdin and prints the four output words in hexadecimal.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>

int main()
{
    unsigned long long seed, offset, g;
    while (std::scanf("%llu %llu %llu", &seed, &offset, &g) == 3) {
        rocrand_device::philox4x32_10_engine eng(seed, offset, 4ull * g);
        uint4 r = eng.next4();
        std::printf("%08x %08x %08x %08x\n", r.x, r.y, r.z, r.w);
    }
    return 0;
}
