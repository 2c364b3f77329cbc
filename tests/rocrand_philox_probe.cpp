// Prints rocRAND's Philox4x32-10 block for counter (b, t, 0, 0) and key = seed,
// one line per (b, t) pair given on the command line. Used by the oracle pins as
// an independent implementation of the generator; host code only.
#include <rocrand/rocrand_philox4x32_10.h>

#include <cstdio>
#include <cstdlib>

int main(int argc, char** argv) {
    if (argc < 2) return 1;
    const unsigned long long seed = strtoull(argv[1], nullptr, 0);
    for (int i = 2; i + 1 < argc; i += 2) {
        const unsigned long long b = strtoull(argv[i], nullptr, 0);
        const unsigned long long t = strtoull(argv[i + 1], nullptr, 0);
        rocrand_state_philox4x32_10 st;
        // rocRAND's counter is (offset/4 low, offset/4 high, subsequence low, high)
        rocrand_init(seed, 0, 4ull * (b + (t << 32)), &st);
        const uint4 r = rocrand4(&st);
        printf("%u %u %u %u\n", r.x, r.y, r.z, r.w);
    }
    return 0;
}
