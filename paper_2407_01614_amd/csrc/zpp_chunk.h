// Work shape of the quantizers for blocks that are not powers of two (any
// multiple of 64 up to 4096): a wave takes K whole blocks at a time, laid
// out as the power-of-two kernels lay out their tiles (vector j of the
// chunk, a 16-byte vector of w elements, in lane j % 64, slot j / 64), so
// every load is a 1 KiB contiguous wave load; V slots per lane.  K and V
// are chosen per block size on the host: the largest share of the 64 V
// vector slots that K blocks fill, then the most blocks.
#pragma once

#include <stdint.h>

namespace zpp {

struct ChunkShape {
    uint32_t K;  // blocks per chunk
    uint32_t V;  // vector slots per lane
};

// vectors_per_block = B / w; at most max_v slots per lane and 64 blocks per
// chunk.  A block of more than 64 max_v vectors has no shape (K = 0).
inline ChunkShape chunk_shape(uint32_t vectors_per_block, uint32_t max_v) {
    ChunkShape best = {0, 0};
    uint64_t best_fill = 0, best_slots = 1;  // compare fill / slots as fractions
    for (uint32_t v = 1; v <= max_v; ++v) {
        uint32_t k = 64 * v / vectors_per_block;
        if (k > 64)
            k = 64;
        if (k == 0)
            continue;
        const uint64_t fill = (uint64_t)k * vectors_per_block, slots = 64ull * v;
        // fill / slots > best_fill / best_slots, or equal with more vectors
        const uint64_t lhs = fill * best_slots, rhs = best_fill * slots;
        if (lhs > rhs || (lhs == rhs && fill > best_fill)) {
            best = {k, v};
            best_fill = fill;
            best_slots = slots;
        }
    }
    return best;
}

}  // namespace zpp
