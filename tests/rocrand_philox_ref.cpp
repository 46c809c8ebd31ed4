// Host-only helper: prints rocRAND's Philox4x32-10 output for counters and
// keys read from stdin, one "c0 c1 c2 c3 k0 k1" line (decimal) per query.
// It is an independent implementation used to pin the oracle's generator.
//
// The engine maps (seed, subsequence, offset) to key = (lo32(seed),
// hi32(seed)) and counter = (offset / 4 as a 64-bit value in words 0-1,
// subsequence as a 64-bit value in words 2-3); with offset a multiple of 4
// its first output is exactly Philox4x32-10(counter, key).
#include <rocrand/rocrand_philox4x32_10.h>

#include <cstdio>

int main() {
    unsigned long long c0, c1, c2, c3, k0, k1;
    while (std::scanf("%llu %llu %llu %llu %llu %llu", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
        unsigned long long seed = (k1 << 32) | k0;
        unsigned long long subseq = (c3 << 32) | c2;
        unsigned long long blk = (c1 << 32) | c0;
        rocrand_state_philox4x32_10 st;
        // offset = 4 * blk: the caller keeps blk below 2^62.
        rocrand_init(seed, subseq, blk * 4ull, &st);
        uint4 r = rocrand4(&st);
        std::printf("%u %u %u %u\n", r.x, r.y, r.z, r.w);
    }
    return 0;
}
