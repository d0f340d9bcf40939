// Host-side reference stream from rocRAND's philox4x32_10 engine (the library
// routine that pins the oracle's Philox4x32-10).  Usage:
//   rocrand_philox_ref <seed> <subsequence> <offset> <count>
// prints <count> raw 32-bit outputs in hex, one per line.
#include <rocrand/rocrand_kernel.h>
#include <cstdio>
#include <cstdlib>

int main(int argc, char** argv) {
    if (argc != 5) return 2;
    unsigned long long seed = strtoull(argv[1], nullptr, 0);
    unsigned long long subseq = strtoull(argv[2], nullptr, 0);
    unsigned long long offset = strtoull(argv[3], nullptr, 0);
    long count = strtol(argv[4], nullptr, 0);
    rocrand_state_philox4x32_10 st;
    rocrand_init(seed, subseq, offset, &st);
    for (long i = 0; i < count; ++i) printf("%08x\n", rocrand(&st));
    return 0;
}
