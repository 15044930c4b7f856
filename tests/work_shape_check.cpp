// Host check of the work shapes for blocks that are not powers of two
// (zpp_chunk.h).
//
// Lane-group shapes (the int8 quantizer, 8 bf16 per vector, with and without
// the copy; the int4 quantizer, 4 fp32 per group), with the kernels' own
// parameters: the shape exists, G is 16, 32 or 64, S is at most 16 and at
// least the kernel's minimum where the fill allows it, the G S slots hold
// the block, and the walk -- block k in lanes [G (k % (64 /
// G)), +G) of a wave, lane r holding the block's vectors v G + r for v below
// the kernel's slot count (the power of two at or above S) -- covers every
// element exactly once, the last block cut short included.
//
// Workgroup renumbering per XCD (xcd_grouped): a permutation of [0, grid)
// for every grid and run length tried, and in every complete run of 8 R
// workgroups the ones that XCD x receives (positions x, x + 8, ...) take R
// consecutive numbers.
//
// Prints the worst fills and "work shapes ok".
#include <stdint.h>
#include <stdio.h>

#include <vector>

#include "zpp_chunk.h"

static uint32_t slot_bucket(uint32_t s, uint32_t smallest) {
    uint32_t b = smallest;
    while (b < s)
        b *= 2;
    return b;
}

static long check_groups(uint32_t w, uint32_t min_fill, uint32_t min_s, uint32_t smallest_bucket,
                         const char *what, double &worst) {
    long bad = 0;
    for (uint32_t b = 1; b <= 64; ++b) {
        if ((b & (b - 1)) == 0)
            continue;
        const uint32_t B = 64 * b, vpb = B / w;
        const zpp::GroupShape sh = zpp::group_shape(vpb, 16, min_fill, min_s);
        const bool pow2 = sh.G != 0 && (sh.G & (sh.G - 1)) == 0;
        if (!pow2 || sh.G < 16 || sh.G > 64 || sh.S == 0 || sh.S > 16 ||
            (uint64_t)sh.G * sh.S < vpb || (uint64_t)sh.G * (sh.S - 1) >= vpb) {
            printf("bad group shape: %s B %u -> G %u S %u\n", what, B, sh.G, sh.S);
            ++bad;
            continue;
        }
        const double fill = (double)vpb / ((double)sh.G * sh.S);
        if (fill < worst)
            worst = fill;
        // the rule: a shape with at least min_s slots and the fill asked for
        // is taken whenever one exists, the widest such group first
        for (uint32_t g = 64; g > sh.G; g /= 2) {
            const uint32_t s = (vpb + g - 1) / g;
            if (s >= min_s && s <= 16 && 100ull * vpb >= (uint64_t)min_fill * g * s) {
                printf("wider group passed over: %s B %u G %u (took %u)\n", what, B, g, sh.G);
                ++bad;
            }
        }
        const uint32_t slots = slot_bucket(sh.S, smallest_bucket);
        const uint32_t bpw = 64 / sh.G;
        // 2.5 waves of blocks, the last block short
        const uint64_t n = (uint64_t)B * (bpw * 2 + bpw / 2 + 1) - 3 * w - 1;
        std::vector<int> seen(n, 0);
        const uint64_t nblocks = (n + B - 1) / B;
        for (uint64_t k = 0; k < nblocks; ++k)
            for (uint32_t r = 0; r < sh.G; ++r)
                for (uint32_t v = 0; v < slots; ++v) {
                    const uint64_t j = (uint64_t)v * sh.G + r;
                    const uint64_t i = k * B + j * w;
                    if (j >= vpb || i >= n)
                        continue;
                    if (v >= sh.S) {
                        printf("slot past S holds data: %s B %u\n", what, B);
                        ++bad;
                    }
                    for (uint32_t e = 0; e < w && i + e < n; ++e)
                        ++seen[i + e];
                }
        for (uint64_t i = 0; i < n; ++i)
            if (seen[i] != 1) {
                printf("element %llu seen %d times: %s B %u\n", (unsigned long long)i, seen[i],
                       what, B);
                ++bad;
                break;
            }
    }
    return bad;
}

static long check_xcd_grouped() {
    long bad = 0;
    const size_t runs[] = {0, 1, 2, 4, 16, 128, 1000};
    const size_t grids[] = {1, 7, 8, 9, 63, 64, 65, 1023, 1024, 1025, 8 * 128 * 3 + 5, 99305};
    for (size_t R : runs)
        for (size_t grid : grids) {
            std::vector<int> seen(grid, 0);
            for (size_t w = 0; w < grid; ++w) {
                const size_t t = zpp::xcd_grouped(w, grid, R);
                if (t >= grid) {
                    printf("xcd_grouped out of range: R %zu grid %zu w %zu -> %zu\n", R, grid, w, t);
                    ++bad;
                    continue;
                }
                ++seen[t];
            }
            for (size_t t = 0; t < grid; ++t)
                if (seen[t] != 1) {
                    printf("xcd_grouped not a permutation: R %zu grid %zu\n", R, grid);
                    ++bad;
                    break;
                }
            if (R <= 1)
                continue;
            for (size_t run = 0; (run + 1) * 8 * R <= grid; ++run)
                for (size_t x = 0; x < 8; ++x)
                    for (size_t j = 0; j < R; ++j) {
                        const size_t w = run * 8 * R + x + 8 * j;
                        if (zpp::xcd_grouped(w, grid, R) != run * 8 * R + x * R + j) {
                            printf("xcd_grouped: XCD %zu not consecutive: R %zu grid %zu\n", x,
                                   R, grid);
                            ++bad;
                        }
                    }
        }
    return bad;
}

int main() {
    double worst_i8 = 1.0, worst_i8c = 1.0, worst_i4 = 1.0;
    long bad = 0;
    // the kernels' parameters: int8 fill 75% (55% with the copy), two slots
    // at least, slot instances 2 / 4 / 8 / 16; int4 fill 75%, three slots,
    // instances 4 / 8 / 16
    bad += check_groups(8, 75, 2, 2, "int8", worst_i8);
    bad += check_groups(8, 55, 2, 2, "int8+copy", worst_i8c);
    bad += check_groups(4, 75, 3, 4, "int4", worst_i4);
    bad += check_xcd_grouped();
    printf("worst fill: int8 %.4f, int8+copy %.4f, int4 %.4f\n", worst_i8, worst_i8c, worst_i4);
    if (bad) {
        printf("%ld failures\n", bad);
        return 1;
    }
    printf("work shapes ok\n");
    return 0;
}
