// Independent reference for the Philox4x32-10 pin: prints words produced by
// rocRAND's Philox4x32-10 engine (its (seed, subsequence, offset) state).
// Reads "seed subsequence offset count" lines from stdin and prints `count`
// words per line, in hex.  Host-only use of rocRAND's header.
#include <rocrand/rocrand_kernel.h>
#include <cstdio>

int main() {
    unsigned long long seed, subseq, offset, count;
    while (std::scanf("%llu %llu %llu %llu", &seed, &subseq, &offset, &count) == 4) {
        rocrand_state_philox4x32_10 st;
        rocrand_init(seed, subseq, offset, &st);
        for (unsigned long long i = 0; i < count; ++i) std::printf("%08x\n", rocrand(&st));
    }
    return 0;
}
