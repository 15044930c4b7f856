// Dequant-gather: the local half of the backward AllGather(L, P') over the
// node-local secondary shards (Algorithm 1, backward branch), with the qwZ
// dequantization fused in.  1 B + 4/B B read, 2 B written per element.
//
// The shard pointers travel by value in the kernel arguments; blockIdx.y picks
// the shard, so the pointer is a uniform (scalar) load.  Vector kernel: a lane
// turns 16 codes (one 16-byte load) and one scale (shared by the 16 lanes of
// a 256-block, served from cache) into 16 bf16 (two 16-byte stores).
#include "zpp_device.h"
#include "zpp_launch.h"

#ifndef ZPP_GATHER_UNROLL
#define ZPP_GATHER_UNROLL 2
#endif
#ifndef ZPP_GATHER_MAX_GRID_X
#define ZPP_GATHER_MAX_GRID_X (1u << 20)
#endif

namespace zpp {
namespace {

struct GatherArgs {
    GatherShards shards;
    uint16_t *out;
    size_t shard_elems;
    size_t layer_elems;
    uint32_t block_shift;  // log2(block)
};

__device__ __forceinline__ float code_f32(uint32_t w, int byte) {
    return (float)(int)(int8_t)(uint8_t)(w >> (8 * byte));
}

// 4 codes of one word -> 2 words of packed bf16; finite scale, so no NaN
// can arise (finite * finite never is NaN) and the NaN test is skipped.
__device__ __forceinline__ u32x2 dequant_word_finite(uint32_t w, float s) {
    u32x2 r;
    const uint32_t b0 = __float_as_uint(code_f32(w, 0) * s);
    const uint32_t b1 = __float_as_uint(code_f32(w, 1) * s);
    const uint32_t b2 = __float_as_uint(code_f32(w, 2) * s);
    const uint32_t b3 = __float_as_uint(code_f32(w, 3) * s);
    r.x = ((b0 + 0x7FFFu + ((b0 >> 16) & 1u)) >> 16) |
          ((b1 + 0x7FFFu + ((b1 >> 16) & 1u)) & 0xFFFF0000u);
    r.y = ((b2 + 0x7FFFu + ((b2 >> 16) & 1u)) >> 16) |
          ((b3 + 0x7FFFu + ((b3 >> 16) & 1u)) & 0xFFFF0000u);
    return r;
}

__device__ __forceinline__ u32x2 dequant_word_any(uint32_t w, float s) {
    u32x2 r;
    r.x = pack_bf16x2(code_f32(w, 0) * s, code_f32(w, 1) * s);
    r.y = pack_bf16x2(code_f32(w, 2) * s, code_f32(w, 3) * s);
    return r;
}

template <int U>
__global__ __launch_bounds__(kThreads) void gather_vec_kernel(GatherArgs a) {
    constexpr size_t kTile = (size_t)kThreads * 16 * U;
    const uint32_t j = blockIdx.y;
    const size_t lo = (size_t)j * a.shard_elems;
    if (lo >= a.layer_elems)
        return;
    const size_t rest = a.layer_elems - lo;
    const size_t valid = rest < a.shard_elems ? rest : a.shard_elems;
    const int8_t *__restrict__ codes = a.shards.codes[j];
    const float *__restrict__ scales = a.shards.scales[j];
    uint16_t *__restrict__ out = a.out + lo;
    const size_t ntiles = (valid + kTile - 1) / kTile;
    for (size_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const size_t base = t * kTile + (size_t)threadIdx.x * 16;
        if ((t + 1) * kTile <= valid) {
            u32x4 c[U];
            float s[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const size_t i = base + (size_t)u * kThreads * 16;
                c[u] = ld_nt(reinterpret_cast<const u32x4 *>(codes + i));
                s[u] = scales[i >> a.block_shift];
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const size_t i = base + (size_t)u * kThreads * 16;
                u32x2 r0, r1, r2, r3;
                if (__builtin_isfinite(s[u])) {
                    r0 = dequant_word_finite(c[u].x, s[u]);
                    r1 = dequant_word_finite(c[u].y, s[u]);
                    r2 = dequant_word_finite(c[u].z, s[u]);
                    r3 = dequant_word_finite(c[u].w, s[u]);
                } else {
                    r0 = dequant_word_any(c[u].x, s[u]);
                    r1 = dequant_word_any(c[u].y, s[u]);
                    r2 = dequant_word_any(c[u].z, s[u]);
                    r3 = dequant_word_any(c[u].w, s[u]);
                }
                st_nt(reinterpret_cast<u32x4 *>(out + i), u32x4{r0.x, r0.y, r1.x, r1.y});
                st_nt(reinterpret_cast<u32x4 *>(out + i + 8), u32x4{r2.x, r2.y, r3.x, r3.y});
            }
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const size_t i0 = base + (size_t)u * kThreads * 16;
                for (size_t i = i0; i < i0 + 16 && i < valid; ++i) {
                    const float x = (float)codes[i] * scales[i >> a.block_shift];
                    out[i] = (uint16_t)bf16_rne_bits(x);
                }
            }
        }
    }
}

// Any shard length and alignment: one output element per thread.
__global__ __launch_bounds__(kThreads) void gather_scalar_kernel(GatherArgs a) {
    const uint32_t j = blockIdx.y;
    const size_t lo = (size_t)j * a.shard_elems;
    if (lo >= a.layer_elems)
        return;
    const size_t rest = a.layer_elems - lo;
    const size_t valid = rest < a.shard_elems ? rest : a.shard_elems;
    const int8_t *codes = a.shards.codes[j];
    const float *scales = a.shards.scales[j];
    const size_t stride = (size_t)gridDim.x * kThreads;
    for (size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x; i < valid; i += stride) {
        const float x = (float)codes[i] * scales[i >> a.block_shift];
        a.out[lo + i] = (uint16_t)bf16_rne_bits(x);
    }
}

}  // namespace

hipError_t launch_gather(const GatherShards &shards, uint32_t num_shards, size_t shard_elems,
                         uint32_t block, size_t layer_elems, uint16_t *out, bool vector_path,
                         hipStream_t stream) {
    GatherArgs a;
    a.shards = shards;
    a.out = out;
    a.shard_elems = shard_elems;
    a.layer_elems = layer_elems;
    a.block_shift = (uint32_t)__builtin_ctz(block);
    const size_t per_shard = shard_elems < layer_elems ? shard_elems : layer_elems;
    if (vector_path) {
        constexpr size_t kTile = (size_t)kThreads * 16 * ZPP_GATHER_UNROLL;
        const size_t tiles = (per_shard + kTile - 1) / kTile;
        const unsigned gx =
            (unsigned)(tiles < ZPP_GATHER_MAX_GRID_X ? tiles : ZPP_GATHER_MAX_GRID_X);
        hipLaunchKernelGGL((gather_vec_kernel<ZPP_GATHER_UNROLL>), dim3(gx, num_shards),
                           dim3(kThreads), 0, stream, a);
    } else {
        const size_t blocks = (per_shard + kThreads - 1) / kThreads;
        const unsigned gx = (unsigned)(blocks < (1u << 20) ? blocks : (1u << 20));
        hipLaunchKernelGGL(gather_scalar_kernel, dim3(gx, num_shards), dim3(kThreads), 0,
                           stream, a);
    }
    return hipGetLastError();
}

}  // namespace zpp
