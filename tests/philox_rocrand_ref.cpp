// Test helper (not product code): prints Philox4x32-10 words from rocRAND's
// published engine, used to pin the oracle's Philox implementation.
// Usage: philox_rocrand_ref <seed> <subsequence> <offset> <count>
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
#include <cstdlib>

int main(int argc, char** argv) {
    if (argc != 5) return 2;
    unsigned long long seed = strtoull(argv[1], nullptr, 0);
    unsigned long long sub = strtoull(argv[2], nullptr, 0);
    unsigned long long off = strtoull(argv[3], nullptr, 0);
    long n = strtol(argv[4], nullptr, 0);
    rocrand_device::philox4x32_10_engine eng(seed, sub, off);
    for (long i = 0; i < n; ++i) printf("%u\n", eng());
    return 0;
}
