// Independent Philox4x32-10 implementation for cross-checking the oracle:
// rocRAND's host-callable engine.  Reads lines "seed subsequence x0 x1" (the
// block advance (x1 << 32) | x0) and prints the four words of that block.
// Built and run by the CPU test suite; not part of the library.
#include <rocrand/rocrand_philox4x32_10.h>

#include <cstdio>

int main() {
    unsigned long long seed, subsequence;
    unsigned int x0, x1;
    while (std::scanf("%llx %llx %x %x", &seed, &subsequence, &x0, &x1) == 4) {
        rocrand_device::philox4x32_10_engine engine(seed, subsequence, 0ull);
        unsigned long long blocks = ((unsigned long long)x1 << 32) | x0;
        while (blocks) {
            unsigned long long step = blocks > (1ull << 61) ? (1ull << 61) : blocks;
            engine.discard(step * 4ull);
            blocks -= step;
        }
        unsigned int w0 = engine.next(), w1 = engine.next(), w2 = engine.next(),
                     w3 = engine.next();
        std::printf("%08x %08x %08x %08x\n", w0, w1, w2, w3);
    }
    return 0;
}
