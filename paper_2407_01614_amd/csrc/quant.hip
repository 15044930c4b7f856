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
// not powers of two (any multiple of 64 up to 4096) take a one-wave kernel
// that works on several whole blocks at a time, the block absmax folded in
// LDS.
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

// Vector path for a block B = 64 b that is not a power of two: a one-wave
// workgroup takes K whole blocks at a time (zpp_chunk.h), lane l holding the
// 8-element vectors v 64 + l of the chunk for v < V (each wave load 1 KiB
// contiguous, as in the power-of-two kernel).  All loads of a chunk are
// issued first.  Each lane folds each of its vectors' absmax into its
// block's word in LDS (an LDS max), or, when one block fills the chunk
// (K = 1), the wave reduces it with cross-lane shuffles; one lane per block
// then derives its parameters once, stores its scale and leaves the
// parameters in LDS, from which every lane quantizes its vectors.
constexpr int kMaxQuantSlots = 8;  // 4096 / 8 = 512 vectors of a block fit 64 x 8

template <bool COPY>
__global__ __launch_bounds__(kWave) void quant_multi_kernel(
    const uint16_t *__restrict__ src, size_t n, BlockDiv blk, uint32_t K, uint32_t V,
    int8_t *__restrict__ codes, float *__restrict__ scales, uint16_t *__restrict__ copy) {
    __shared__ uint32_t bmax[64];
    __shared__ BlockQuant bq[64];
    const uint32_t lane = threadIdx.x;
    const size_t B = blk.block;
    const size_t nblocks = (n + B - 1) / B;
    for (size_t k0 = (size_t)blockIdx.x * K; k0 < nblocks; k0 += (size_t)gridDim.x * K) {
        const uint32_t kc = (uint32_t)(nblocks - k0 < K ? nblocks - k0 : K);
        const size_t base = k0 * B;
        const size_t end = (base + kc * B < n) ? base + kc * B : n;
        if (lane < kc)
            bmax[lane] = 0u;
        __syncthreads();
        // every load of the chunk first, then the LDS maxima (a max in the
        // same pass would wait for each load in turn)
        u32x4 x[kMaxQuantSlots];
        uint32_t kl[kMaxQuantSlots];
        if (end == base + (size_t)K * B) {
            // a whole chunk: every vector complete, one predicated load each
            const uint32_t nvec = K * (uint32_t)(B / 8);
#pragma unroll
            for (int v = 0; v < kMaxQuantSlots; ++v) {
                x[v] = u32x4{0u, 0u, 0u, 0u};
                const uint32_t j = (uint32_t)v * kWave + lane;
                if ((uint32_t)v < V && j < nvec)
                    x[v] = ld_nt(reinterpret_cast<const u32x4 *>(src + base + (size_t)j * 8));
            }
        } else {
#pragma unroll
            for (int v = 0; v < kMaxQuantSlots; ++v) {
                x[v] = u32x4{0u, 0u, 0u, 0u};
                if ((uint32_t)v < V) {
                    const size_t i = base + ((size_t)v * kWave + lane) * 8;
                    if (i + 8 <= end) {
                        x[v] = ld_nt(reinterpret_cast<const u32x4 *>(src + i));
                    } else if (i < end) {
                        uint32_t h[8];
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            h[e] = (i + e < end) ? (uint32_t)src[i + e] : 0u;
                        x[v] = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16),
                                     h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
                    }
                }
            }
        }
#pragma unroll
        for (int v = 0; v < kMaxQuantSlots; ++v)
            kl[v] = 0u;
        if (K == 1) {
            // one block per chunk: its absmax is a reduction over the wave
            u16x2 m2 = {0, 0};
#pragma unroll
            for (int v = 0; v < kMaxQuantSlots; ++v)
                m2 = __builtin_elementwise_max(m2, __builtin_elementwise_max(
                         __builtin_elementwise_max(absbits2(x[v].x), absbits2(x[v].y)),
                         __builtin_elementwise_max(absbits2(x[v].z), absbits2(x[v].w))));
            uint32_t mx = max((uint32_t)m2.x, (uint32_t)m2.y);
#pragma unroll
            for (int off = kWave / 2; off >= 1; off >>= 1)
                mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
            if (lane == 0) {
                const BlockQuant q = block_params(mx);
                bq[0] = q;
                scales[k0] = q.scale;
            }
        } else {
#pragma unroll
            for (int v = 0; v < kMaxQuantSlots; ++v) {
                const size_t i = base + ((size_t)v * kWave + lane) * 8;
                if ((uint32_t)v < V && i < end) {
                    kl[v] = (uint32_t)(block_of(blk, i) - k0);
                    const u16x2 m2 = __builtin_elementwise_max(
                        __builtin_elementwise_max(absbits2(x[v].x), absbits2(x[v].y)),
                        __builtin_elementwise_max(absbits2(x[v].z), absbits2(x[v].w)));
                    atomicMax(&bmax[kl[v]], max((uint32_t)m2.x, (uint32_t)m2.y));
                }
            }
            __syncthreads();
            if (lane < kc) {
                const BlockQuant q = block_params(bmax[lane]);
                bq[lane] = q;
                scales[k0 + lane] = q.scale;
            }
        }
        __syncthreads();
#pragma unroll
        for (int v = 0; v < kMaxQuantSlots; ++v) {
            if ((uint32_t)v >= V)
                continue;
            const size_t i = base + ((size_t)v * kWave + lane) * 8;
            if (i >= end)
                continue;
            const BlockQuant q = bq[kl[v]];
            u32x2 c;
            c.x = quant_word(x[v].x, x[v].y, q);
            c.y = quant_word(x[v].z, x[v].w, q);
            if (i + 8 <= end) {
                st_nt(reinterpret_cast<u32x2 *>(codes + i), c);
                if (COPY)
                    st_nt(reinterpret_cast<u32x4 *>(copy + i), x[v]);
            } else {
                for (int e = 0; e < 8 && i + e < end; ++e) {
                    codes[i + e] =
                        (int8_t)((e < 4 ? c.x >> (8 * e) : c.y >> (8 * (e - 4))) & 0xFFu);
                    if (COPY)
                        copy[i + e] = src[i + e];
                }
            }
        }
        __syncthreads();  // bmax and bq are rewritten for the next chunk
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
        const ChunkShape sh = chunk_shape(block / 8, kMaxQuantSlots);
        const size_t nblocks = (n + block - 1) / block;
        const size_t need = (nblocks + sh.K - 1) / sh.K;
        const unsigned grid = (unsigned)(need < ZPP_QUANT_MAX_GRID ? need : ZPP_QUANT_MAX_GRID);
        hipLaunchKernelGGL((quant_multi_kernel<COPY>), dim3(grid), dim3(kWave), 0, stream, src,
                           n, make_block_div(block), sh.K, sh.V, codes, scales, copy);
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
