// Host check of the block index used by the kernels (BlockDiv in
// zpp_launch.h): for every block size the library accepts (64 b, b = 1..64),
// the index a kernel computes for element i -- a shift for a power-of-two
// block, else the high half of the 64 x 64-bit product of i >> 6 and the
// magic number, which is what __umul64hi returns on the device -- equals
// i / block, over small i, random i up to 2^64 - 1 and the elements on
// either side of every block boundary near 2^64.  Prints "block index ok".
#include <stdint.h>
#include <stdio.h>

#include <random>

#include "zpp_launch.h"

static uint64_t index_of(const zpp::BlockDiv &d, uint64_t i) {
    if (d.magic)
        return (uint64_t)(((unsigned __int128)(i >> 6) * d.magic) >> 64);
    return i >> d.shift;
}

int main() {
    std::mt19937_64 rng(12345);
    long bad = 0, checked = 0;
    for (uint32_t block = 64; block <= 4096; block += 64) {
        const zpp::BlockDiv d = zpp::make_block_div(block);
        if (d.block != block)
            ++bad;
        auto check = [&](uint64_t i) {
            ++checked;
            if (index_of(d, i) != i / block) {
                if (bad < 10)
                    printf("block %u i %llu: %llu, want %llu\n", block, (unsigned long long)i,
                           (unsigned long long)index_of(d, i), (unsigned long long)(i / block));
                ++bad;
            }
        };
        for (uint64_t i = 0; i < 300000; ++i)
            check(i);
        for (int r = 0; r < 200000; ++r)
            check(rng() >> (rng() % 64));
        // both sides of block boundaries up to the top of the range
        for (uint64_t k = UINT64_MAX / block; k > UINT64_MAX / block - 2000; --k)
            for (int dlt = -2; dlt <= 1; ++dlt)
                check(k * block + (uint64_t)(int64_t)dlt);
        for (int r = 0; r < 20000; ++r) {
            const uint64_t k = rng() / block;
            check(k * block);
            check(k * block - 1);
        }
        check(UINT64_MAX);
    }
    if (bad) {
        printf("%ld of %ld indices wrong\n", bad, checked);
        return 1;
    }
    printf("block index ok (%ld indices)\n", checked);
    return 0;
}
