// Work distribution shared by the kernels and the host checks: the lane
// layout of the quantizers for blocks that are not powers of two (any
// multiple of 64 up to 4096), and the renumbering of workgroups per XCD.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace zpp {

// Lane-group shape for blocks that are not powers of two: each block owns an
// aligned group of G lanes of a wave (G = 16, 32 or 64, so 64 / G blocks per
// wave), each lane holding S of the block's vectors (vector j of the block
// in lane j % G of the group, slot j / G); slots past the block's last
// vector stay empty.  The block's absmax is then a reduction over its G
// lanes with cross-lane xor shuffles, as in the power-of-two kernels.
// Chosen on the host: the largest G whose S (at least min_s, at most
// max_s) slots the block fills to at least min_fill_pct percent; failing
// that, the largest fill.  A block of more than 64 max_s vectors has no
// shape (G = 0).
struct GroupShape {
    uint32_t G;  // lanes per block
    uint32_t S;  // vector slots per lane
};

inline GroupShape group_shape(uint32_t vectors_per_block, uint32_t max_s, uint32_t min_fill_pct,
                              uint32_t min_s) {
    GroupShape best = {0, 0};
    uint64_t best_slots = 0;
    for (uint32_t g = 64; g >= 16; g /= 2) {
        const uint32_t s = (vectors_per_block + g - 1) / g;
        if (s > max_s)
            continue;
        if (s >= min_s && 100ull * vectors_per_block >= (uint64_t)min_fill_pct * g * s)
            return {g, s};
        // the same vectors in fewer slots is the larger fill
        if (best.G == 0 || (uint64_t)g * s < best_slots) {
            best = {g, s};
            best_slots = (uint64_t)g * s;
        }
    }
    return best;
}

// The dispatcher hands workgroups to the GPU's 8 XCDs in turn (workgroup w
// to XCD w % 8), each XCD with its own L2.  xcd_grouped(w, grid, R)
// renumbers workgroup w so that in every run of 8 R workgroups each XCD
// takes R consecutive positions (an incomplete last run keeps its order):
// neighbouring workgroups that read the same cache lines -- a line of
// per-block scales serving several tiles -- then fetch them through one L2.
// A permutation of [0, grid) for any R; R <= 1 is the identity.  (constexpr,
// so kernels and host checks call the same function.)
constexpr size_t xcd_grouped(size_t w, size_t grid, size_t R) {
    if (R <= 1)
        return w;
    const size_t run = w / (8 * R), r = w % (8 * R);
    return (run + 1) * 8 * R <= grid ? run * 8 * R + (r % 8) * R + r / 8 : w;
}

}  // namespace zpp
