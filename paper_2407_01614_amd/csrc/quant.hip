// qwZ quantization of a bf16 weight shard: symmetric absmax int8 per block of
// B elements with one fp32 scale per block (weights are quantized before the
// AllGather, Background section).  2 B read, 1 B + 4/B B written per element.
//
// Vector kernel: one lane holds 8 consecutive bf16 (one 16-byte load), so a
// block of B elements spans L = min(B/8, 64) lanes of one wave and a lane
// holds V = max(1, B/512) vectors.  The absmax is an integer max over the bf16
// magnitude bits (|x| bits are monotone in |x|, and bits >= 0x7F80 mean Inf or
// NaN), reduced across the L lanes with cross-lane xor shuffles; no LDS
// traffic and no float compares are needed.  Every lane then derives the
// block's scale and inverse itself (two correctly rounded divisions per 8
// elements) and writes its 8 codes as one 8-byte store.  Blocks that are
// not powers of two (any multiple of 64 up to 4096) take the same approach
// with the block's width a run-time value: a block owns an aligned group of
// 16 to 64 lanes, each holding up to 16 of its vectors.
//
// The same kernels can also store the bf16 they read to a second array:
// the secondary refresh and its quantization in one pass (2 B read, 2 B +
// 1 B + 4/B B written per element, against 4 + 3 + 4/B B for the two
// calls).
#include "zpp_chunk.h"
#include "zpp_device.h"
#include "zpp_launch.h"
#include "zpp_quant.h"

#ifndef ZPP_QUANT_UNROLL
#define ZPP_QUANT_UNROLL 2
#endif
#ifndef ZPP_QUANT_THREADS
#define ZPP_QUANT_THREADS 256
#endif
// Shape of the kernel for blocks that are not powers of two (zpp_chunk.h):
// at least two vector slots per lane, and the widest lane group whose slots
// the block fills to this percentage.  Swept at the Llama-2-13B partition
// over blocks of 192 to 2112 (median of 20 launches each): the plain
// quantizer streams best with a fill of 75% (93-102 us against 97-120 for
// 55-85% or three slots), the pass with the copy with 55% (167-175 us
// against 168-185); one slot per lane was slower for both (137 against
// 97 us at 448).
#ifndef ZPP_QUANT_GROUP_MIN_FILL
#define ZPP_QUANT_GROUP_MIN_FILL 75
#endif
#ifndef ZPP_QUANT_COPY_GROUP_MIN_FILL
#define ZPP_QUANT_COPY_GROUP_MIN_FILL 55
#endif
#ifndef ZPP_QUANT_MAX_GRID
#define ZPP_QUANT_MAX_GRID (1u << 20)
#endif
// Block-rows in flight per wave of the refresh-and-quantize pass: one, where
// the quantizer alone streams best with two (Llama-2-13B partition: 157.6
// against 164.8 us; the plain quantizer 112 against 94 us with one).
#ifndef ZPP_QUANT_COPY_UNROLL
#define ZPP_QUANT_COPY_UNROLL 1
#endif

namespace zpp {
namespace {

constexpr int kQuantThreads = ZPP_QUANT_THREADS;

// With COPY the loaded bf16 are also stored to `copy`, bit for bit (the
// secondary refresh taken into the quantization's pass).
template <int B, int U, bool COPY>
__global__ __launch_bounds__(kQuantThreads) void quant_vec_kernel(
    const uint16_t *__restrict__ src, size_t n, int8_t *__restrict__ codes,
    float *__restrict__ scales, uint16_t *__restrict__ copy) {
    constexpr int L = (B / 8 < kWave) ? B / 8 : kWave;  // lanes per quant block
    constexpr int V = (B / 8 > kWave) ? B / (8 * kWave) : 1;
    constexpr int kGroupsPerWave = kWave / L;
    constexpr int kGroupsPerRow = kGroupsPerWave * (kQuantThreads / kWave);
    constexpr int kGroupsPerBlock = kGroupsPerRow * U;
    const size_t nblocks = (n + B - 1) / B;
    const int lane = threadIdx.x & (kWave - 1);
    const int gl = lane / L;
    const int li = lane % L;
    const int wave = threadIdx.x / kWave;

    for (size_t g0 = (size_t)blockIdx.x * kGroupsPerBlock; g0 < nblocks;
         g0 += (size_t)gridDim.x * kGroupsPerBlock) {
        // all U rows of loads first, then the reductions and stores
        u32x4 x[U][V];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const size_t k = g0 + (size_t)u * kGroupsPerRow + (size_t)wave * kGroupsPerWave + gl;
            const bool valid = k < nblocks;
#pragma unroll
            for (int v = 0; v < V; ++v) {
                const size_t i = k * B + ((size_t)v * L + li) * 8;
                if (valid && i + 8 <= n) {
                    x[u][v] = ld_nt(reinterpret_cast<const u32x4 *>(src + i));
                } else {
                    uint32_t h[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        h[e] = (valid && i + e < n) ? (uint32_t)src[i + e] : 0u;
                    x[u][v] = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16),
                                    h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
                }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const size_t k = g0 + (size_t)u * kGroupsPerRow + (size_t)wave * kGroupsPerWave + gl;
            const bool valid = k < nblocks;
            u16x2 m2 = {0, 0};
#pragma unroll
            for (int v = 0; v < V; ++v)
                m2 = __builtin_elementwise_max(m2, __builtin_elementwise_max(
                         __builtin_elementwise_max(absbits2(x[u][v].x), absbits2(x[u][v].y)),
                         __builtin_elementwise_max(absbits2(x[u][v].z), absbits2(x[u][v].w))));
            uint32_t mx = max((uint32_t)m2.x, (uint32_t)m2.y);
#pragma unroll
            for (int off = L / 2; off >= 1; off >>= 1)
                mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));

            const BlockQuant q = block_params(mx);
#pragma unroll
            for (int v = 0; v < V; ++v) {
                const size_t i = k * B + ((size_t)v * L + li) * 8;
                u32x2 c;
                c.x = quant_word(x[u][v].x, x[u][v].y, q);
                c.y = quant_word(x[u][v].z, x[u][v].w, q);
                if (valid && i + 8 <= n) {
                    st_nt(reinterpret_cast<u32x2 *>(codes + i), c);
                    if (COPY)
                        st_nt(reinterpret_cast<u32x4 *>(copy + i), x[u][v]);
                } else if (valid) {
                    for (int e = 0; e < 8 && i + e < n; ++e) {
                        codes[i + e] =
                            (int8_t)((e < 4 ? c.x >> (8 * e) : c.y >> (8 * (e - 4))) & 0xFFu);
                        if (COPY)
                            copy[i + e] = src[i + e];
                    }
                }
            }
            if (valid && li == 0)
                scales[k] = q.scale;
        }
    }
}

// Vector path for a block B = 64 b that is not a power of two, lane-group
// layout (zpp_chunk.h): each block owns an aligned group of G lanes, lane r
// of the group holding the block's vectors v G + r for v < S (vectors past
// the block's end stay empty), so a wave load covers 64 / G runs of G
// consecutive vectors.  The block absmax is a reduction over the group's G
// lanes with cross-lane xor shuffles and every lane derives the block's
// parameters itself, as in the power-of-two kernel: no LDS, no atomics and
// no barrier.  Workgroups whose blocks all lie inside the array load each
// vector with one predicated load; only the last one checks every element.
template <int G, int S, bool COPY>
__global__ __launch_bounds__(kQuantThreads) void quant_grp_kernel(
    const uint16_t *__restrict__ src, size_t n, uint32_t B, int8_t *__restrict__ codes,
    float *__restrict__ scales, uint16_t *__restrict__ copy) {
    constexpr int kGroupsPerWave = kWave / G;
    constexpr int kGroupsPerBlock = kGroupsPerWave * (kQuantThreads / kWave);
    const uint32_t vpb = B / 8;
    const size_t nblocks = (n + B - 1) / B;
    const int lane = threadIdx.x & (kWave - 1);
    const int li = lane % G;
    const size_t kw = (size_t)(threadIdx.x / kWave) * kGroupsPerWave + lane / G;
    for (size_t g0 = (size_t)blockIdx.x * kGroupsPerBlock; g0 < nblocks;
         g0 += (size_t)gridDim.x * kGroupsPerBlock) {
        const size_t k = g0 + kw;
        const bool valid = k < nblocks;
        const bool whole = (g0 + kGroupsPerBlock) * B <= n;  // uniform
        u32x4 x[S];
        if (whole) {
#pragma unroll
            for (int v = 0; v < S; ++v) {
                x[v] = u32x4{0u, 0u, 0u, 0u};
                const uint32_t j = (uint32_t)(v * G + li);
                if (j < vpb)
                    x[v] = ld_nt(reinterpret_cast<const u32x4 *>(src + k * B + (size_t)j * 8));
            }
        } else {
#pragma unroll
            for (int v = 0; v < S; ++v) {
                x[v] = u32x4{0u, 0u, 0u, 0u};
                const uint32_t j = (uint32_t)(v * G + li);
                const size_t i = k * B + (size_t)j * 8;
                if (valid && j < vpb) {
                    if (i + 8 <= n) {
                        x[v] = ld_nt(reinterpret_cast<const u32x4 *>(src + i));
                    } else if (i < n) {
                        uint32_t h[8];
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            h[e] = (i + e < n) ? (uint32_t)src[i + e] : 0u;
                        x[v] = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16),
                                     h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
                    }
                }
            }
        }
        u16x2 m2 = {0, 0};
#pragma unroll
        for (int v = 0; v < S; ++v)
            m2 = __builtin_elementwise_max(m2, __builtin_elementwise_max(
                     __builtin_elementwise_max(absbits2(x[v].x), absbits2(x[v].y)),
                     __builtin_elementwise_max(absbits2(x[v].z), absbits2(x[v].w))));
        uint32_t mx = max((uint32_t)m2.x, (uint32_t)m2.y);
#pragma unroll
        for (int off = G / 2; off >= 1; off >>= 1)
            mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
        const BlockQuant q = block_params(mx);
#pragma unroll
        for (int v = 0; v < S; ++v) {
            const uint32_t j = (uint32_t)(v * G + li);
            const size_t i = k * B + (size_t)j * 8;
            if (!valid || j >= vpb || i >= n)
                continue;
            u32x2 c;
            c.x = quant_word(x[v].x, x[v].y, q);
            c.y = quant_word(x[v].z, x[v].w, q);
            if (i + 8 <= n) {
                st_nt(reinterpret_cast<u32x2 *>(codes + i), c);
                if (COPY)
                    st_nt(reinterpret_cast<u32x4 *>(copy + i), x[v]);
            } else {
                for (int e = 0; e < 8 && i + e < n; ++e) {
                    codes[i + e] =
                        (int8_t)((e < 4 ? c.x >> (8 * e) : c.y >> (8 * (e - 4))) & 0xFFu);
                    if (COPY)
                        copy[i + e] = src[i + e];
                }
            }
        }
        if (valid && li == 0)
            scales[k] = q.scale;
    }
}

// Any alignment, any block: one wave per quant block, lanes stride through it
// element by element.
__global__ __launch_bounds__(kThreads) void quant_scalar_kernel(
    const uint16_t *__restrict__ src, size_t n, uint32_t block, int8_t *__restrict__ codes,
    float *__restrict__ scales, uint16_t *__restrict__ copy) {
    const size_t nblocks = (n + block - 1) / block;
    const int lane = threadIdx.x & (kWave - 1);
    const size_t wave0 = (size_t)blockIdx.x * (kThreads / kWave) + threadIdx.x / kWave;
    const size_t nwaves = (size_t)gridDim.x * (kThreads / kWave);
    for (size_t k = wave0; k < nblocks; k += nwaves) {
        const size_t lo = k * block;
        const size_t hi = (lo + block < n) ? lo + block : n;
        uint32_t mx = 0;
        for (size_t i = lo + lane; i < hi; i += kWave)
            mx = max(mx, (uint32_t)src[i] & 0x7FFFu);
        for (int off = kWave / 2; off >= 1; off >>= 1)
            mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
        const BlockQuant q = block_params(mx);
        for (size_t i = lo + lane; i < hi; i += kWave) {
            const uint16_t h = src[i];
            codes[i] = (int8_t)quant_one(bf16_lo((uint32_t)h), q);
            if (copy)
                copy[i] = h;
        }
        if (lane == 0)
            scales[k] = q.scale;
    }
}

template <int B, bool COPY>
void launch_vec(const uint16_t *src, size_t n, int8_t *codes, float *scales, uint16_t *copy,
                hipStream_t stream) {
    constexpr int L = (B / 8 < kWave) ? B / 8 : kWave;
    constexpr int U = COPY ? ZPP_QUANT_COPY_UNROLL : ZPP_QUANT_UNROLL;
    constexpr size_t kGroupsPerBlock = (kWave / L) * (kQuantThreads / kWave) * U;
    const size_t nblocks = (n + B - 1) / B;
    const size_t need = (nblocks + kGroupsPerBlock - 1) / kGroupsPerBlock;
    const unsigned grid = (unsigned)(need < ZPP_QUANT_MAX_GRID ? need : ZPP_QUANT_MAX_GRID);
    hipLaunchKernelGGL((quant_vec_kernel<B, U, COPY>), dim3(grid), dim3(kQuantThreads), 0,
                       stream, src, n, codes, scales, copy);
}

template <int G, int S, bool COPY>
void launch_grp(const uint16_t *src, size_t n, uint32_t block, int8_t *codes, float *scales,
                uint16_t *copy, hipStream_t stream) {
    constexpr size_t kGroupsPerBlock = (kWave / G) * (kQuantThreads / kWave);
    const size_t nblocks = (n + block - 1) / block;
    const size_t need = (nblocks + kGroupsPerBlock - 1) / kGroupsPerBlock;
    const unsigned grid = (unsigned)(need < ZPP_QUANT_MAX_GRID ? need : ZPP_QUANT_MAX_GRID);
    hipLaunchKernelGGL((quant_grp_kernel<G, S, COPY>), dim3(grid), dim3(kQuantThreads), 0,
                       stream, src, n, block, codes, scales, copy);
}

template <int S, bool COPY>
void launch_grp_g(uint32_t G, const uint16_t *src, size_t n, uint32_t block, int8_t *codes,
                  float *scales, uint16_t *copy, hipStream_t stream) {
    switch (G) {
    case 16: launch_grp<16, S, COPY>(src, n, block, codes, scales, copy, stream); break;
    case 32: launch_grp<32, S, COPY>(src, n, block, codes, scales, copy, stream); break;
    default: launch_grp<64, S, COPY>(src, n, block, codes, scales, copy, stream); break;
    }
}

template <bool COPY>
void launch_vector(const uint16_t *src, size_t n, uint32_t block, int8_t *codes, float *scales,
                   uint16_t *copy, hipStream_t stream) {
    switch (block) {
    case 64: launch_vec<64, COPY>(src, n, codes, scales, copy, stream); break;
    case 128: launch_vec<128, COPY>(src, n, codes, scales, copy, stream); break;
    case 256: launch_vec<256, COPY>(src, n, codes, scales, copy, stream); break;
    case 512: launch_vec<512, COPY>(src, n, codes, scales, copy, stream); break;
    case 1024: launch_vec<1024, COPY>(src, n, codes, scales, copy, stream); break;
    case 2048: launch_vec<2048, COPY>(src, n, codes, scales, copy, stream); break;
    case 4096: launch_vec<4096, COPY>(src, n, codes, scales, copy, stream); break;
    default: {
        const GroupShape sh =
            COPY ? group_shape(block / 8, 16, ZPP_QUANT_COPY_GROUP_MIN_FILL, 2)
                 : group_shape(block / 8, 16, ZPP_QUANT_GROUP_MIN_FILL, 2);
        if (sh.S <= 2)
            launch_grp_g<2, COPY>(sh.G, src, n, block, codes, scales, copy, stream);
        else if (sh.S <= 4)
            launch_grp_g<4, COPY>(sh.G, src, n, block, codes, scales, copy, stream);
        else if (sh.S <= 8)
            launch_grp_g<8, COPY>(sh.G, src, n, block, codes, scales, copy, stream);
        else
            launch_grp_g<16, COPY>(sh.G, src, n, block, codes, scales, copy, stream);
    }
    }
}

}  // namespace

hipError_t launch_quantize_copy(const uint16_t *src, size_t n, uint32_t block, int8_t *codes,
                                float *scales, uint16_t *copy, bool vector_path,
                                hipStream_t stream) {
    if (vector_path) {
        if (copy)
            launch_vector<true>(src, n, block, codes, scales, copy, stream);
        else
            launch_vector<false>(src, n, block, codes, scales, nullptr, stream);
    } else {
        const size_t nblocks = (n + block - 1) / block;
        const size_t need = (nblocks + (kThreads / kWave) - 1) / (kThreads / kWave);
        const unsigned grid = (unsigned)(need < (1u << 20) ? need : (1u << 20));
        hipLaunchKernelGGL(quant_scalar_kernel, dim3(grid), dim3(kThreads), 0, stream, src, n,
                           block, codes, scales, copy);
    }
    return hipGetLastError();
}

hipError_t launch_quantize(const uint16_t *src, size_t n, uint32_t block, int8_t *codes,
                           float *scales, bool vector_path, hipStream_t stream) {
    return launch_quantize_copy(src, n, block, codes, scales, nullptr, vector_path, stream);
}

}  // namespace zpp
