// qgZ, the gradient side of the partition step: blockwise int4 quantization
// of fp32 gradients before the exchange that replaces the ReduceScatter
// (Background section; Algorithm 1, backward loop), and, on the receiving
// rank, the dequantize-and-reduce of the P quantized copies of its partition
// into the fp32 gradient the optimizer step consumes.
//
// Quantize: 4 B read, 0.5 B + 4/B B written per element.  The absmax is an
// integer max of the |x| bit patterns (bits >= 0x7F800000 mean Inf or NaN),
// reduced over the lanes of a block with xor shuffles.  Codes come from the
// same round-to-nearest-even trick as the int8 quantizer (the low bits of
// x*inv + 1.5*2^23), packed four to a 16-bit store.
//
// Dequant-reduce: P * (0.5 B + 4/B B) read, 4 B written per element.  The
// sources' pointers travel by value in the kernel arguments; a lane
// accumulates its elements over the sources in order, one fma each.
//
// The dequant-reduce also reads the P copies from one interleaved receive
// buffer (layout in zpp_i4grad.h): the gradient source of the receive
// kernels forms each float4, so the bits are those of the separate arrays.
//
// Blocks may be any multiple of 64 up to 4096; for those that are not powers
// of two the quantizer gives each block an aligned group of 16 to 64 lanes
// of a wave, each lane holding several of its groups of 4 values.
//
// The power-of-two kernels keep every wave's loads and stores contiguous: on
// this GPU, non-temporal stores that leave gaps inside a wave's footprint
// (16 bytes per lane at a 32- or 64-byte stride) run two to three times
// slower.  The lane-group quantizer's code stores are runs of 2 G bytes per
// block (32 to 128), which the sweep of its shapes measured: groups of 8
// lanes (16-byte runs) were the slow ones and are not used.
#include "zpp_chunk.h"
#include "zpp_device.h"
#include "zpp_i4grad.h"
#include "zpp_launch.h"
#include "zpp_quant.h"

#ifndef ZPP_QGZ_THREADS
#define ZPP_QGZ_THREADS 256
#endif
#ifndef ZPP_QGZ_QUANT_UNROLL
#define ZPP_QGZ_QUANT_UNROLL 4
#endif
#ifndef ZPP_QGZ_REDUCE_GROUPS
#define ZPP_QGZ_REDUCE_GROUPS 2
#endif
#ifndef ZPP_QGZ_REDUCE_IL_GROUPS
#define ZPP_QGZ_REDUCE_IL_GROUPS 2
#endif
// Shape of the quantizer for blocks that are not powers of two
// (zpp_chunk.h): at least three slots per lane, and the widest lane group
// whose slots the block fills to this percentage.  Swept at the Llama-2-13B
// partition over blocks of 192 to 4032 (median of 20 launches each): 149-157
// us with this rule, against up to 173 us with two slots and 220 with
// groups of 8 lanes (16-byte runs of codes per store instruction), and
// 191-228 us for the earlier layout that folded each block's absmax in LDS.
#ifndef ZPP_QGZ_GROUP_MIN_FILL
#define ZPP_QGZ_GROUP_MIN_FILL 75
#endif
#ifndef ZPP_QGZ_MAX_GRID
#define ZPP_QGZ_MAX_GRID (1u << 30)
#endif

namespace zpp {
namespace {

constexpr int kQgzThreads = ZPP_QGZ_THREADS;

struct I4Quant {
    float scale, pre, inv;
    bool zero, tiny;
};

__device__ __forceinline__ I4Quant i4_params(uint32_t absbits) {
    I4Quant q;
    const float a = __uint_as_float(absbits);
    q.tiny = a < 0x1p-100f;
    q.pre = q.tiny ? 0x1p64f : 1.0f;
    q.inv = 7.0f / (a * q.pre);
    if (absbits >= 0x7F800000u) {
        q.scale = __uint_as_float(kScaleNaNBits);
        q.zero = true;
    } else if (absbits == 0u) {
        q.scale = 0.0f;
        q.zero = true;
    } else {
        q.scale = a / 7.0f;
        q.zero = false;
    }
    return q;
}

// 4 values -> 4 int4 codes packed little-endian in 16 bits.  No clamp is
// needed: |x * inv| rounds to at most 7 (1 + 2^-24)^2 < 7.5.
__device__ __forceinline__ uint32_t i4_half(const f32x4 &x, const I4Quant &q) {
#pragma clang fp contract(off)
    uint32_t b[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float xe = q.tiny ? x[e] * q.pre : x[e];
        b[e] = code_bits(xe * q.inv);
    }
    // low bytes side by side, then low nibbles: bytes 0 and 2 of t hold
    // (c0 | c1 << 4) and (c2 | c3 << 4)
    const uint32_t w = pack_low_bytes(b[0], b[1], b[2], b[3]) & 0x0F0F0F0Fu;
    const uint32_t t = w | (w >> 4);
    const uint32_t packed = __builtin_amdgcn_perm(0u, t, 0x0c0c0200u);
    return q.zero ? 0u : packed;
}

__device__ __forceinline__ uint32_t abs_bits_max4(const f32x4 &v) {
    return max(max(__float_as_uint(v.x) & 0x7FFFFFFFu, __float_as_uint(v.y) & 0x7FFFFFFFu),
               max(__float_as_uint(v.z) & 0x7FFFFFFFu, __float_as_uint(v.w) & 0x7FFFFFFFu));
}

// A lane holds groups of 4 consecutive values; group t of lane l in a wave's
// tile starts at 256 t + 4 l, so every load instruction of a wave reads 1 KiB
// and every code store writes 128 contiguous bytes.  A block of B values
// spans L = min(B/4, 64) lanes and G = max(1, B/256) groups per lane; a
// wave covers C = max(B, 256) values per tile and keeps U tiles in flight.
// Where the codes and scale of one source go in a receive buffer of P
// sources interleaved block by block (block k of B elements: source q's B/2
// code bytes at (k P + q) B/2, its scale at k P + q); P = 1, q = 0 is the
// plain layout (byte i / 2, scale k).
__device__ __forceinline__ size_t i4_out_byte(size_t i, uint32_t shift, uint32_t q, uint32_t P) {
    return (((i >> shift) * P + q) << (shift - 1)) + ((i & (((size_t)1 << shift) - 1)) >> 1);
}

// The same for element i of block k of any block size B.
__device__ __forceinline__ size_t i4_out_byte_any(size_t i, size_t k, uint32_t B, uint32_t q,
                                                  uint32_t P) {
    return (k * P + q) * (B / 2) + ((i - k * B) >> 1);
}

template <int B, int U>
__global__ __launch_bounds__(kQgzThreads) void quant_i4_kernel(
    const float *__restrict__ src, size_t n, uint8_t *__restrict__ codes,
    float *__restrict__ scales, uint32_t q_src, uint32_t num_src) {
    constexpr uint32_t kShift = __builtin_ctz(B);
    constexpr int C = B > 256 ? B : 256;
    constexpr int G = C / 256;
    constexpr int L = B < 256 ? B / 4 : kWave;
    constexpr int kWaves = kQgzThreads / kWave;
    const size_t ntiles = (n + C - 1) / C;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    for (size_t t0 = ((size_t)blockIdx.x * kWaves + wave) * U; t0 < ntiles;
         t0 += (size_t)gridDim.x * kWaves * U) {
        f32x4 x[U][G];
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const size_t i = (t0 + u) * C + (size_t)g * 256 + (size_t)lane * 4;
                if (t0 + u < ntiles && i + 4 <= n) {
                    x[u][g] = ld_nt(reinterpret_cast<const f32x4 *>(src + i));
                } else {
                    float h[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        h[e] = (t0 + u < ntiles && i + e < n) ? src[i + e] : 0.0f;
                    x[u][g] = f32x4{h[0], h[1], h[2], h[3]};
                }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const size_t tile = t0 + u;
            uint32_t mx = 0;
#pragma unroll
            for (int g = 0; g < G; ++g)
                mx = max(mx, abs_bits_max4(x[u][g]));
#pragma unroll
            for (int off = L / 2; off >= 1; off >>= 1)
                mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
            const I4Quant q = i4_params(mx);
            if (tile < ntiles) {
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    const size_t i = tile * C + (size_t)g * 256 + (size_t)lane * 4;
                    const uint32_t h = i4_half(x[u][g], q);
                    const size_t byte0 = i4_out_byte(i, kShift, q_src, num_src);
                    // the second byte holds elements i + 2 and i + 3
                    if (i + 2 < n) {
                        st_nt(reinterpret_cast<uint16_t *>(codes + byte0), (uint16_t)h);
                    } else if (i < n) {
                        codes[byte0] = (uint8_t)h;
                    }
                }
                const size_t k = (tile * C + (size_t)lane * 4) / B;
                if (lane % L == 0 && k * B < n)
                    scales[k * num_src + q_src] = q.scale;
            }
        }
    }
}

// Vector path for a block B = 64 b that is not a power of two, lane-group
// layout (zpp_chunk.h): each block owns an aligned group of G lanes, lane r
// of the group holding the block's groups of 4 values v G + r for v < S
// (groups past the block's end stay empty).  The block absmax is a
// reduction over the group's G lanes with cross-lane xor shuffles and every
// lane derives the block's parameters itself, as in the power-of-two
// kernel: no LDS, no atomics and no barrier.  Workgroups whose blocks all
// lie inside the array load each group with one predicated load; only the
// last one checks every element.
template <int G, int S>
__global__ __launch_bounds__(kQgzThreads) void quant_i4_grp_kernel(
    const float *__restrict__ src, size_t n, uint32_t B, uint8_t *__restrict__ codes,
    float *__restrict__ scales, uint32_t q_src, uint32_t num_src) {
    constexpr int kBlocksPerWave = kWave / G;
    constexpr int kBlocksPerGroup = kBlocksPerWave * (kQgzThreads / kWave);
    const uint32_t gpb = B / 4;
    const size_t nblocks = (n + B - 1) / B;
    const int lane = threadIdx.x & (kWave - 1);
    const int li = lane % G;
    const size_t kw = (size_t)(threadIdx.x / kWave) * kBlocksPerWave + lane / G;
    for (size_t g0 = (size_t)blockIdx.x * kBlocksPerGroup; g0 < nblocks;
         g0 += (size_t)gridDim.x * kBlocksPerGroup) {
        const size_t k = g0 + kw;
        const bool valid = k < nblocks;
        const bool whole = (g0 + kBlocksPerGroup) * B <= n;  // uniform
        f32x4 x[S];
        if (whole) {
#pragma unroll
            for (int v = 0; v < S; ++v) {
                x[v] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                const uint32_t j = (uint32_t)(v * G + li);
                if (j < gpb)
                    x[v] = ld_nt(reinterpret_cast<const f32x4 *>(src + k * B + (size_t)j * 4));
            }
        } else {
#pragma unroll
            for (int v = 0; v < S; ++v) {
                x[v] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                const uint32_t j = (uint32_t)(v * G + li);
                const size_t i = k * B + (size_t)j * 4;
                if (valid && j < gpb) {
                    if (i + 4 <= n) {
                        x[v] = ld_nt(reinterpret_cast<const f32x4 *>(src + i));
                    } else if (i < n) {
                        float h[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            h[e] = (i + e < n) ? src[i + e] : 0.0f;
                        x[v] = f32x4{h[0], h[1], h[2], h[3]};
                    }
                }
            }
        }
        uint32_t mx = 0;
#pragma unroll
        for (int v = 0; v < S; ++v)
            mx = max(mx, abs_bits_max4(x[v]));
#pragma unroll
        for (int off = G / 2; off >= 1; off >>= 1)
            mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
        const I4Quant q = i4_params(mx);
#pragma unroll
        for (int v = 0; v < S; ++v) {
            const uint32_t j = (uint32_t)(v * G + li);
            const size_t i = k * B + (size_t)j * 4;
            if (!valid || j >= gpb || i >= n)
                continue;
            const uint32_t h = i4_half(x[v], q);
            const size_t byte0 = i4_out_byte_any(i, k, B, q_src, num_src);
            // the second byte holds elements i + 2 and i + 3
            if (i + 2 < n)
                st_nt(reinterpret_cast<uint16_t *>(codes + byte0), (uint16_t)h);
            else
                codes[byte0] = (uint8_t)h;
        }
        if (valid && li == 0)
            scales[k * num_src + q_src] = q.scale;
    }
}

// Any alignment: one wave per block, lanes stride through it; each code
// byte is written by the lane that owns its even element.
__global__ __launch_bounds__(kQgzThreads) void quant_i4_scalar_kernel(
    const float *__restrict__ src, size_t n, uint32_t block, uint8_t *__restrict__ codes,
    float *__restrict__ scales, uint32_t q_src, uint32_t num_src) {
    const size_t nblocks = (n + block - 1) / block;
    const int lane = threadIdx.x & (kWave - 1);
    const size_t wave0 = (size_t)blockIdx.x * (kQgzThreads / kWave) + threadIdx.x / kWave;
    const size_t nwaves = (size_t)gridDim.x * (kQgzThreads / kWave);
    for (size_t k = wave0; k < nblocks; k += nwaves) {
        const size_t lo = k * block;
        const size_t hi = (lo + block < n) ? lo + block : n;
        uint32_t mx = 0;
        for (size_t i = lo + lane; i < hi; i += kWave)
            mx = max(mx, __float_as_uint(src[i]) & 0x7FFFFFFFu);
        for (int off = kWave / 2; off >= 1; off >>= 1)
            mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
        const I4Quant q = i4_params(mx);
        // block is even, so a code byte never straddles two blocks
        for (size_t i = lo + 2 * lane; i < hi; i += 2 * kWave) {
            const float x0 = src[i];
            const float x1 = (i + 1 < hi) ? src[i + 1] : 0.0f;
            const uint32_t h = i4_half(f32x4{x0, x1, 0.0f, 0.0f}, q);
            codes[i4_out_byte_any(i, k, block, q_src, num_src)] = (uint8_t)(h & 0xFFu);
        }
        if (lane == 0)
            scales[k * num_src + q_src] = q.scale;
    }
}

struct ReduceArgs {
    const uint8_t *codes[kMaxShards];
    const float *scales[kMaxShards];
    uint32_t num_src;
    size_t n;
    BlockDiv block;
    float scale_out;
    float *out;
};

// A lane holds G groups of 4 consecutive elements; group t of lane l in a
// wave's tile starts at 256 t + 4 l, so each source is read as 128-byte
// contiguous wave loads (2 bytes per lane) and every store of the wave
// writes 1 KiB contiguously.  Sources are taken eight at a time, all their
// loads in flight before the fma passes, which keep the order q = 0, 1, ...
// Workgroups are renumbered in runs per XCD (kSeparateXcdRun), so that the
// tiles sharing a line of a source's scales read it through one L2.
template <int G>
__global__ __launch_bounds__(kQgzThreads) void reduce_i4_kernel(ReduceArgs a) {
    constexpr int kBatch = 8;
    constexpr int kWaves = kQgzThreads / kWave;
    constexpr size_t C = 256 * G;
    const size_t ntiles = (a.n + C - 1) / C;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const size_t wg = xcd_grouped(blockIdx.x, gridDim.x, kSeparateXcdRun);
    for (size_t tile = wg * kWaves + wave; tile < ntiles;
         tile += (size_t)gridDim.x * kWaves) {
        const size_t base = tile * C + (size_t)lane * 4;
        const bool full = tile * C + C <= a.n;
        float acc[G][4];
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                acc[g][e] = 0.0f;
        for (uint32_t q0 = 0; q0 < a.num_src; q0 += kBatch) {
            uint32_t w[kBatch][G];
            float s[kBatch][G];
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                const uint32_t q = q0 + j;
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    const size_t i = base + (size_t)g * 256;
                    w[j][g] = 0;
                    s[j][g] = 0.0f;
                    if (q < a.num_src) {
                        if (full) {
                            w[j][g] = ld_nt(reinterpret_cast<const uint16_t *>(a.codes[q] + i / 2));
                        } else {
                            if (i < a.n)
                                w[j][g] = a.codes[q][i / 2];
                            if (i + 2 < a.n)
                                w[j][g] |= (uint32_t)a.codes[q][i / 2 + 1] << 8;
                        }
                        if (i < a.n)
                            s[j][g] = a.scales[q][block_of(a.block, i)];
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                if (q0 + j < a.num_src) {
#pragma unroll
                    for (int g = 0; g < G; ++g)
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            acc[g][e] = __builtin_fmaf(i4_code(w[j][g], e), s[j][g], acc[g][e]);
                }
            }
        }
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const size_t i = base + (size_t)g * 256;
            if (full) {
                st_nt(reinterpret_cast<f32x4 *>(a.out + i),
                      f32x4{acc[g][0] * a.scale_out, acc[g][1] * a.scale_out,
                            acc[g][2] * a.scale_out, acc[g][3] * a.scale_out});
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (i + e < a.n)
                        a.out[i + e] = acc[g][e] * a.scale_out;
            }
        }
    }
}

// Any alignment: one element per thread.
__global__ __launch_bounds__(kQgzThreads) void reduce_i4_scalar_kernel(ReduceArgs a) {
    for (size_t i = (size_t)blockIdx.x * kQgzThreads + threadIdx.x; i < a.n;
         i += (size_t)gridDim.x * kQgzThreads) {
        float acc = 0.0f;
        for (uint32_t q = 0; q < a.num_src; ++q) {
            const uint32_t byte = a.codes[q][i / 2];
            const uint32_t nib = (i % 2 == 0) ? (byte & 0xFu) : (byte >> 4);
            acc = __builtin_fmaf(i4_code(nib, 0), a.scales[q][block_of(a.block, i)], acc);
        }
        a.out[i] = acc * a.scale_out;
    }
}

// The reduction from a gradient source of zpp_i4grad.h: a lane holds G
// groups of 4 consecutive elements at 256 t + 4 l of its wave's tile, as
// above; each group is the source's gradient of those four elements, stored
// as one float4 (1 KiB contiguous per wave store).  Partial tiles go element
// by element.
template <class GS, int G>
__global__ __launch_bounds__(kQgzThreads) void reduce_gs_kernel(GS gs, size_t n,
                                                               float *__restrict__ out) {
    constexpr int kWaves = kQgzThreads / kWave;
    constexpr size_t C = 256 * G;
    const size_t ntiles = (n + C - 1) / C;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    for (size_t tile = (size_t)blockIdx.x * kWaves + wave; tile < ntiles;
         tile += (size_t)gridDim.x * kWaves) {
        const size_t base = tile * C + (size_t)lane * 4;
        if (tile * C + C <= n) {
            f32x4 r[G];
#pragma unroll
            for (int g = 0; g < G; ++g)
                r[g] = grad_load4(gs, base + (size_t)g * 256);
#pragma unroll
            for (int g = 0; g < G; ++g)
                st_nt(reinterpret_cast<f32x4 *>(out + base + (size_t)g * 256), r[g]);
        } else {
#pragma unroll
            for (int g = 0; g < G; ++g)
                for (int e = 0; e < 4; ++e) {
                    const size_t i = base + (size_t)g * 256 + e;
                    if (i < n)
                        out[i] = grad_at(gs, i);
                }
        }
    }
}

// Any alignment: one element per thread.
template <class GS>
__global__ __launch_bounds__(kQgzThreads) void reduce_gs_scalar_kernel(GS gs, size_t n,
                                                                      float *__restrict__ out) {
    for (size_t i = (size_t)blockIdx.x * kQgzThreads + threadIdx.x; i < n;
         i += (size_t)gridDim.x * kQgzThreads)
        out[i] = grad_at(gs, i);
}

template <int B>
void launch_quant_i4_b(const float *src, size_t n, uint8_t *codes, float *scales,
                       uint32_t q_src, uint32_t num_src, hipStream_t stream) {
    constexpr size_t C = B > 256 ? B : 256;
    constexpr size_t kTilesPerBlock = (kQgzThreads / kWave) * ZPP_QGZ_QUANT_UNROLL;
    const size_t ntiles = (n + C - 1) / C;
    const size_t need = (ntiles + kTilesPerBlock - 1) / kTilesPerBlock;
    const unsigned grid = (unsigned)(need < ZPP_QGZ_MAX_GRID ? need : ZPP_QGZ_MAX_GRID);
    hipLaunchKernelGGL((quant_i4_kernel<B, ZPP_QGZ_QUANT_UNROLL>), dim3(grid), dim3(kQgzThreads),
                       0, stream, src, n, codes, scales, q_src, num_src);
}

template <int G, int S>
void launch_quant_i4_grp(const float *src, size_t n, uint32_t block, uint8_t *codes,
                         float *scales, uint32_t q_src, uint32_t num_src, hipStream_t stream) {
    constexpr size_t kBlocksPerGroup = (kWave / G) * (kQgzThreads / kWave);
    const size_t nblocks = (n + block - 1) / block;
    const size_t need = (nblocks + kBlocksPerGroup - 1) / kBlocksPerGroup;
    const unsigned grid = (unsigned)(need < ZPP_QGZ_MAX_GRID ? need : ZPP_QGZ_MAX_GRID);
    hipLaunchKernelGGL((quant_i4_grp_kernel<G, S>), dim3(grid), dim3(kQgzThreads), 0, stream,
                       src, n, block, codes, scales, q_src, num_src);
}

template <int S>
void launch_quant_i4_grp_g(uint32_t G, const float *src, size_t n, uint32_t block,
                           uint8_t *codes, float *scales, uint32_t q_src, uint32_t num_src,
                           hipStream_t stream) {
    switch (G) {
    case 16: launch_quant_i4_grp<16, S>(src, n, block, codes, scales, q_src, num_src, stream); break;
    case 32: launch_quant_i4_grp<32, S>(src, n, block, codes, scales, q_src, num_src, stream); break;
    default: launch_quant_i4_grp<64, S>(src, n, block, codes, scales, q_src, num_src, stream); break;
    }
}

}  // namespace

hipError_t launch_quantize_i4_il(const float *src, size_t n, uint32_t block, uint32_t source,
                                 uint32_t num_src, uint8_t *codes, float *scales,
                                 bool vector_path, hipStream_t stream) {
    if (vector_path) {
        switch (block) {
        case 64: launch_quant_i4_b<64>(src, n, codes, scales, source, num_src, stream); break;
        case 128: launch_quant_i4_b<128>(src, n, codes, scales, source, num_src, stream); break;
        case 256: launch_quant_i4_b<256>(src, n, codes, scales, source, num_src, stream); break;
        case 512: launch_quant_i4_b<512>(src, n, codes, scales, source, num_src, stream); break;
        case 1024: launch_quant_i4_b<1024>(src, n, codes, scales, source, num_src, stream); break;
        case 2048: launch_quant_i4_b<2048>(src, n, codes, scales, source, num_src, stream); break;
        case 4096: launch_quant_i4_b<4096>(src, n, codes, scales, source, num_src, stream); break;
        default: {
            const GroupShape sh = group_shape(block / 4, 16, ZPP_QGZ_GROUP_MIN_FILL, 3);
            if (sh.S <= 4)
                launch_quant_i4_grp_g<4>(sh.G, src, n, block, codes, scales, source, num_src,
                                         stream);
            else if (sh.S <= 8)
                launch_quant_i4_grp_g<8>(sh.G, src, n, block, codes, scales, source, num_src,
                                         stream);
            else
                launch_quant_i4_grp_g<16>(sh.G, src, n, block, codes, scales, source, num_src,
                                          stream);
        }
        }
    } else {
        const size_t nblocks = (n + block - 1) / block;
        const size_t need = (nblocks + (kQgzThreads / kWave) - 1) / (kQgzThreads / kWave);
        const unsigned grid = (unsigned)(need < (1u << 20) ? need : (1u << 20));
        hipLaunchKernelGGL(quant_i4_scalar_kernel, dim3(grid), dim3(kQgzThreads), 0, stream, src,
                           n, block, codes, scales, source, num_src);
    }
    return hipGetLastError();
}

hipError_t launch_quantize_i4(const float *src, size_t n, uint32_t block, uint8_t *codes,
                              float *scales, bool vector_path, hipStream_t stream) {
    return launch_quantize_i4_il(src, n, block, 0, 1, codes, scales, vector_path, stream);
}

hipError_t launch_dequant_reduce_i4(const uint8_t *const *src_codes,
                                    const float *const *src_scales, uint32_t num_src, size_t n,
                                    uint32_t block, float scale_out, float *out,
                                    bool vector_path, hipStream_t stream) {
    ReduceArgs a = {};
    for (uint32_t q = 0; q < num_src; ++q) {
        a.codes[q] = src_codes[q];
        a.scales[q] = src_scales[q];
    }
    a.num_src = num_src;
    a.n = n;
    a.block = make_block_div(block);
    a.scale_out = scale_out;
    a.out = out;
    if (vector_path) {
        constexpr size_t C = 256 * ZPP_QGZ_REDUCE_GROUPS;
        const size_t ntiles = (n + C - 1) / C;
        const size_t waves = kQgzThreads / kWave;
        const size_t need = (ntiles + waves - 1) / waves;
        const unsigned grid = (unsigned)(need < ZPP_QGZ_MAX_GRID ? need : ZPP_QGZ_MAX_GRID);
        hipLaunchKernelGGL((reduce_i4_kernel<ZPP_QGZ_REDUCE_GROUPS>), dim3(grid),
                           dim3(kQgzThreads), 0, stream, a);
    } else {
        const size_t need = (n + kQgzThreads - 1) / kQgzThreads;
        const unsigned grid = (unsigned)(need < (1u << 20) ? need : (1u << 20));
        hipLaunchKernelGGL(reduce_i4_scalar_kernel, dim3(grid), dim3(kQgzThreads), 0, stream, a);
    }
    return hipGetLastError();
}

hipError_t launch_dequant_reduce_i4_il(const uint8_t *codes, const float *scales, uint32_t num_src,
                                       size_t n, uint32_t block, float scale_out, float *out,
                                       bool vector_path, hipStream_t stream) {
    const I4GradIl gs = make_i4grad_il(codes, scales, num_src, block, scale_out);
    if (vector_path) {
        constexpr size_t C = 256 * ZPP_QGZ_REDUCE_IL_GROUPS;
        const size_t ntiles = (n + C - 1) / C;
        const size_t waves = kQgzThreads / kWave;
        const size_t need = (ntiles + waves - 1) / waves;
        const unsigned grid = (unsigned)(need < ZPP_QGZ_MAX_GRID ? need : ZPP_QGZ_MAX_GRID);
        hipLaunchKernelGGL((reduce_gs_kernel<I4GradIl, ZPP_QGZ_REDUCE_IL_GROUPS>), dim3(grid),
                           dim3(kQgzThreads), 0, stream, gs, n, out);
    } else {
        const size_t need = (n + kQgzThreads - 1) / kQgzThreads;
        const unsigned grid = (unsigned)(need < (1u << 20) ? need : (1u << 20));
        hipLaunchKernelGGL(reduce_gs_scalar_kernel<I4GradIl>, dim3(grid), dim3(kQgzThreads), 0,
                           stream, gs, n, out);
    }
    return hipGetLastError();
}

}  // namespace zpp
