// Host check of the quantizers' work shape for blocks that are not powers of
// two (zpp_chunk.h): for every such block size and both vector widths (8
// bf16 of the int8 quantizer, 4 fp32 of the int4 one), the shape exists,
// its K blocks fit the 64 V vector slots of a wave and the LDS word of each
// block (K <= 64), and the lane/slot walk of one chunk -- vector j = 64 v +
// l of the chunk for v < V -- covers every element of every block of the
// chunk exactly once, including a last chunk of fewer blocks and a last
// block cut short by the end of the array.  Prints the worst fill of the
// slots and "chunk shapes ok".
#include <stdint.h>
#include <stdio.h>

#include <vector>

#include "zpp_chunk.h"

int main() {
    long bad = 0;
    double worst = 1.0;
    // int8: 8 bf16 per vector, 8 slots; int4: 4 fp32 per group, 8 slots for
    // blocks of up to 2048 values and 16 above (the kernels' two instances)
    const struct { uint32_t w; } kinds[2] = {{8}, {4}};
    for (const auto &kd : kinds) {
        for (uint32_t b = 1; b <= 64; ++b) {
            if ((b & (b - 1)) == 0)
                continue;  // powers of two take the other kernels
            const uint32_t B = 64 * b, vpb = B / kd.w;
            const uint32_t max_v = (kd.w == 8 || vpb <= 64 * 8) ? 8 : 16;
            const zpp::ChunkShape sh = zpp::chunk_shape(vpb, max_v);
            if (sh.K == 0 || sh.K > 64 || sh.V == 0 || sh.V > max_v ||
                (uint64_t)sh.K * vpb > 64ull * sh.V) {
                printf("bad shape: w %u B %u -> K %u V %u\n", kd.w, B, sh.K, sh.V);
                ++bad;
                continue;
            }
            const double fill = (double)sh.K * vpb / (64.0 * sh.V);
            if (fill < worst)
                worst = fill;
            // one array of 2.5 chunks whose last block is short
            const uint64_t n = (uint64_t)B * (sh.K * 2 + sh.K / 2 + 1) - 3 * kd.w - 1;
            std::vector<int> seen(n, 0);
            const uint64_t nblocks = (n + B - 1) / B;
            for (uint64_t k0 = 0; k0 < nblocks; k0 += sh.K) {
                const uint64_t kc = nblocks - k0 < sh.K ? nblocks - k0 : sh.K;
                const uint64_t base = k0 * B, end = base + kc * B < n ? base + kc * B : n;
                for (uint32_t v = 0; v < sh.V; ++v)
                    for (uint32_t l = 0; l < 64; ++l) {
                        const uint64_t i = base + ((uint64_t)v * 64 + l) * kd.w;
                        if (i >= end)
                            continue;
                        const uint64_t kl = i / B - k0;
                        if (kl >= kc || (i + kd.w <= end && (i + kd.w - 1) / B != i / B)) {
                            printf("vector outside its block: w %u B %u i %llu\n", kd.w, B,
                                   (unsigned long long)i);
                            ++bad;
                        }
                        for (uint32_t e = 0; e < kd.w && i + e < end; ++e)
                            ++seen[i + e];
                    }
            }
            for (uint64_t i = 0; i < n; ++i)
                if (seen[i] != 1) {
                    printf("element %llu seen %d times: w %u B %u\n", (unsigned long long)i,
                           seen[i], kd.w, B);
                    ++bad;
                    break;
                }
        }
    }
    printf("worst fill %.4f\n", worst);
    if (bad) {
        printf("%ld failures\n", bad);
        return 1;
    }
    printf("chunk shapes ok\n");
    return 0;
}
