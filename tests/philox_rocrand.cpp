// Philox4x32-10 outputs from ROCm's rocRAND host implementation (header
// only; no GPU involved), for pinning the oracle's Philox to an
// implementation written by others.  Reads lines "key ctr_lo ctr_hi"
// (decimal 64-bit words: key = k0 | k1 << 32, ctr_lo = c0 | c1 << 32,
// ctr_hi = c2 | c3 << 32) and prints the four output words of each.
//
// rocRAND's engine takes the key as its seed and keeps a 128-bit counter:
// a subsequence adds to the high 64 bits, a discard of 4 q numbers adds q
// to the low 64 bits (carrying upward).  Starting from counter 0, the low
// half is set by discards of at most 2^61 blocks each, so no addition
// carries.
#include <rocrand/rocrand_philox4x32_10.h>

#include <cstdio>

int main()
{
    unsigned long long key, lo, hi;
    while (std::scanf("%llu %llu %llu", &key, &lo, &hi) == 3) {
        rocrand_device::philox4x32_10_engine e(key, hi, 0);
        while (lo) {
            const unsigned long long q = lo < (1ull << 61) ? lo : (1ull << 61);
            e.discard(4 * q);
            lo -= q;
        }
        const unsigned int w0 = e(), w1 = e(), w2 = e(), w3 = e();
        std::printf("%u %u %u %u\n", w0, w1, w2, w3);
    }
    return 0;
}
