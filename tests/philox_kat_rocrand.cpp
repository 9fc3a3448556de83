// Known-answer helper for the Philox4x32-10 pin: prints rocRAND's host-side
// Philox4x32-10 block for each "seed c0 c1 c2 c3" line read from stdin.
// rocRAND's engine maps (seed, subsequence, offset) to key = seed words,
// counter.z/w = subsequence words and counter.x/y = offset / 4, so the block
// for counter (c0, c1, c2, c3) is the first next4() after seeding with
// subsequence = c2 | c3 << 32 and offset = 4 * (c0 | c1 << 32).
#include <hip/hip_runtime.h>
#include <rocrand/rocrand_kernel.h>
#include <cstdio>

int main()
{
    unsigned long long seed, c0, c1, c2, c3;
    while (std::scanf("%llu %llu %llu %llu %llu", &seed, &c0, &c1, &c2, &c3) == 5) {
        rocrand_state_philox4x32_10 st;
        rocrand_init(seed, c2 | (c3 << 32), 4ull * (c0 | (c1 << 32)), &st);
        uint4 v = rocrand4(&st);
        std::printf("%u %u %u %u\n", v.x, v.y, v.z, v.w);
    }
    return 0;
}
