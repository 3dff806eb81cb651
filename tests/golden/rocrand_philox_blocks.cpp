// Prints Philox-4x32-10 blocks computed by rocRAND's host/device engine, for
// the (key, counter) pairs read from stdin, one "seed c0 c1 c2 c3" per line.
// rocrand_init(seed, subsequence, offset) keys the engine with the 64-bit
// seed and sets counter words (x, y) from offset/4 and (z, w) from the
// subsequence; the next four outputs are then the block at that counter.
#include <cstdio>
#include <rocrand/rocrand_kernel.h>

int main() {
    unsigned long long seed, c0, c1, c2, c3;
    while (std::scanf("%llu %llu %llu %llu %llu", &seed, &c0, &c1, &c2, &c3) == 5) {
        rocrand_state_philox4x32_10 st;
        unsigned long long offset = ((c1 << 32) | c0) * 4ull;
        unsigned long long subseq = (c3 << 32) | c2;
        rocrand_init(seed, subseq, offset, &st);
        unsigned a = rocrand(&st), b = rocrand(&st), c = rocrand(&st), d = rocrand(&st);
        std::printf("%u %u %u %u\n", a, b, c, d);
    }
    return 0;
}
