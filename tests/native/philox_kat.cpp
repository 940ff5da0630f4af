// Known-answer source for the oracle's Philox4x32-10: ROCm's open-source
// rocRAND engine, compiled for the host CPU.  Reads lines of
// "seed subsequence offset" (decimal) on stdin and prints the four 32-bit
// words of next4() for each, in hex.  With offset a multiple of 4 the engine
// returns the block whose counter is (offset/4 low, offset/4 high,
// subsequence low, subsequence high) under key (seed low, seed high).
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>

int main() {
    unsigned long long seed, subseq, offset;
    while (std::scanf("%llu %llu %llu", &seed, &subseq, &offset) == 3) {
        rocrand_device::philox4x32_10_engine eng(seed, subseq, offset);
        uint4 w = eng.next4();
        std::printf("%08x %08x %08x %08x\n", w.x, w.y, w.z, w.w);
    }
    return 0;
}
