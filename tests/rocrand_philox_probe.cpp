// Reference Philox4x32-10 outputs from rocRAND's host-callable engine, used to
// pin the oracle's own Philox.  Reads "seed c0 c1 c2 c3" lines from stdin and
// prints the four output words of Philox(key = seed, counter = (c0..c3)).
// rocRAND positions: the subsequence selects counter words 2-3 and the offset
// (counted in 32-bit outputs, four per counter) selects words 0-1; word 1 is
// reached with four skips of c1 * 2^32 outputs so that no skip overflows.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>

int main()
{
    unsigned long long seed;
    unsigned int c0, c1, c2, c3;
    while (std::scanf("%llu %u %u %u %u", &seed, &c0, &c1, &c2, &c3) == 5) {
        rocrand_state_philox4x32_10 st;
        unsigned long long sub = (unsigned long long)c2 | ((unsigned long long)c3 << 32);
        rocrand_init(seed, sub, 4ull * c0, &st);
        for (int k = 0; k < 4; ++k) skipahead((unsigned long long)c1 << 32, &st);
        uint4 r = rocrand4(&st);
        std::printf("%u %u %u %u\n", r.x, r.y, r.z, r.w);
    }
    return 0;
}
