// Test aid: prints rocRAND's Philox4x32-10 output blocks, an implementation
// independent of the oracle's, through rocRAND's public engine on the host.
// stdin: lines "seed step param_index block"; stdout: four hex words per line.
// The engine's (seed, subsequence, offset) maps to key (seed_lo, seed_hi) and
// counter (offset/4 as a 64-bit pair, subsequence as a 64-bit pair), so the
// block with counter (block, param_index, step_lo, step_hi) is offset
// 4 * (param_index * 2^32 + block) of subsequence step.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>

int main()
{
    unsigned long long seed, step, pidx, blk;
    while (std::scanf("%llu %llu %llu %llu", &seed, &step, &pidx, &blk) == 4) {
        rocrand_device::philox4x32_10_engine e(seed, step, 4ULL * ((pidx << 32) | blk));
        unsigned a = e.next(), b = e.next(), c = e.next(), d = e.next();
        std::printf("%08x %08x %08x %08x\n", a, b, c, d);
    }
    return 0;
}
