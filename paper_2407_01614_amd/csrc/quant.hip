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
// elements) and writes its 8 codes as one 8-byte store.
#include "zpp_device.h"
#include "zpp_launch.h"

#ifndef ZPP_QUANT_MAX_GRID
#define ZPP_QUANT_MAX_GRID (1u << 20)
#endif

namespace zpp {
namespace {

constexpr uint32_t kScaleNaNBits = 0x7FC00000u;

struct BlockQuant {
    float scale;  // value stored for the block
    float pre;    // power-of-two pre-scale of tiny blocks (exact)
    float inv;    // 127 / (absmax * pre)
    bool zero;    // codes are all 0 (zero or non-finite block)
};

// Decisions of one block from the max of its |x| bit patterns.
__device__ __forceinline__ BlockQuant block_params(uint32_t absbits) {
    BlockQuant q;
    const float a = __uint_as_float(absbits << 16);
    q.pre = (a < 0x1p-100f) ? 0x1p64f : 1.0f;
    q.inv = 127.0f / (a * q.pre);
    if (absbits >= 0x7F80u) {
        q.scale = __uint_as_float(kScaleNaNBits);
        q.zero = true;
    } else if (absbits == 0u) {
        q.scale = 0.0f;
        q.zero = true;
    } else {
        q.scale = a / 127.0f;
        q.zero = false;
    }
    return q;
}

__device__ __forceinline__ int quant_one(float x, const BlockQuant &q) {
    float y = __builtin_rintf((x * q.pre) * q.inv);
    y = __builtin_fminf(__builtin_fmaxf(y, -127.0f), 127.0f);
    return q.zero ? 0 : (int)y;
}

__device__ __forceinline__ uint32_t quant_word(uint32_t w0, uint32_t w1, const BlockQuant &q) {
    // 4 bf16 (two 32-bit words) -> 4 int8 codes packed little-endian
    const uint32_t c0 = (uint32_t)quant_one(bf16_lo(w0), q) & 0xFFu;
    const uint32_t c1 = (uint32_t)quant_one(bf16_hi(w0), q) & 0xFFu;
    const uint32_t c2 = (uint32_t)quant_one(bf16_lo(w1), q) & 0xFFu;
    const uint32_t c3 = (uint32_t)quant_one(bf16_hi(w1), q) & 0xFFu;
    return c0 | (c1 << 8) | (c2 << 16) | (c3 << 24);
}

__device__ __forceinline__ uint32_t absbits_max(uint32_t w) {
    return max(w & 0x7FFFu, (w >> 16) & 0x7FFFu);
}

template <int B>
__global__ __launch_bounds__(kThreads) void quant_vec_kernel(const uint16_t *__restrict__ src,
                                                             size_t n, int8_t *__restrict__ codes,
                                                             float *__restrict__ scales) {
    constexpr int L = (B / 8 < kWave) ? B / 8 : kWave;  // lanes per quant block
    constexpr int V = (B / 8 > kWave) ? B / (8 * kWave) : 1;
    constexpr int kGroupsPerWave = kWave / L;
    constexpr int kGroupsPerBlock = kGroupsPerWave * (kThreads / kWave);
    const size_t nblocks = (n + B - 1) / B;
    const int lane = threadIdx.x & (kWave - 1);
    const int gl = lane / L;
    const int li = lane % L;
    const int wave = threadIdx.x / kWave;

    for (size_t g0 = (size_t)blockIdx.x * kGroupsPerBlock; g0 < nblocks;
         g0 += (size_t)gridDim.x * kGroupsPerBlock) {
        const size_t k = g0 + (size_t)wave * kGroupsPerWave + gl;
        const bool valid = k < nblocks;
        u32x4 x[V];
        uint32_t mx = 0;
#pragma unroll
        for (int v = 0; v < V; ++v) {
            const size_t i = k * B + ((size_t)v * L + li) * 8;
            if (valid && i + 8 <= n) {
                x[v] = ld_nt(reinterpret_cast<const u32x4 *>(src + i));
            } else {
                uint32_t h[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    h[e] = (valid && i + e < n) ? (uint32_t)src[i + e] : 0u;
                x[v] = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                             h[6] | (h[7] << 16)};
            }
            mx = max(mx, max(max(absbits_max(x[v].x), absbits_max(x[v].y)),
                             max(absbits_max(x[v].z), absbits_max(x[v].w))));
        }
#pragma unroll
        for (int off = L / 2; off >= 1; off >>= 1)
            mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));

        const BlockQuant q = block_params(mx);
#pragma unroll
        for (int v = 0; v < V; ++v) {
            const size_t i = k * B + ((size_t)v * L + li) * 8;
            u32x2 c;
            c.x = quant_word(x[v].x, x[v].y, q);
            c.y = quant_word(x[v].z, x[v].w, q);
            if (valid && i + 8 <= n) {
                st_nt(reinterpret_cast<u32x2 *>(codes + i), c);
            } else if (valid) {
                for (int e = 0; e < 8 && i + e < n; ++e)
                    codes[i + e] = (int8_t)((e < 4 ? c.x >> (8 * e) : c.y >> (8 * (e - 4))) & 0xFFu);
            }
        }
        if (valid && li == 0)
            scales[k] = q.scale;
    }
}

// Any alignment, any power-of-two block: one wave per quant block, lanes
// stride through it element by element.
__global__ __launch_bounds__(kThreads) void quant_scalar_kernel(const uint16_t *__restrict__ src,
                                                                size_t n, uint32_t block,
                                                                int8_t *__restrict__ codes,
                                                                float *__restrict__ scales) {
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
        for (size_t i = lo + lane; i < hi; i += kWave)
            codes[i] = (int8_t)quant_one(bf16_lo((uint32_t)src[i]), q);
        if (lane == 0)
            scales[k] = q.scale;
    }
}

template <int B>
void launch_vec(const uint16_t *src, size_t n, int8_t *codes, float *scales,
                hipStream_t stream) {
    constexpr int L = (B / 8 < kWave) ? B / 8 : kWave;
    constexpr size_t kGroupsPerBlock = (kWave / L) * (kThreads / kWave);
    const size_t nblocks = (n + B - 1) / B;
    const size_t need = (nblocks + kGroupsPerBlock - 1) / kGroupsPerBlock;
    const unsigned grid = (unsigned)(need < ZPP_QUANT_MAX_GRID ? need : ZPP_QUANT_MAX_GRID);
    hipLaunchKernelGGL((quant_vec_kernel<B>), dim3(grid), dim3(kThreads), 0, stream, src, n,
                       codes, scales);
}

}  // namespace

hipError_t launch_quantize(const uint16_t *src, size_t n, uint32_t block, int8_t *codes,
                           float *scales, bool vector_path, hipStream_t stream) {
    if (vector_path) {
        switch (block) {
        case 64: launch_vec<64>(src, n, codes, scales, stream); break;
        case 128: launch_vec<128>(src, n, codes, scales, stream); break;
        case 256: launch_vec<256>(src, n, codes, scales, stream); break;
        case 512: launch_vec<512>(src, n, codes, scales, stream); break;
        case 1024: launch_vec<1024>(src, n, codes, scales, stream); break;
        case 2048: launch_vec<2048>(src, n, codes, scales, stream); break;
        case 4096: launch_vec<4096>(src, n, codes, scales, stream); break;
        default: return hipErrorInvalidValue;
        }
    } else {
        const size_t nblocks = (n + block - 1) / block;
        const size_t need = (nblocks + (kThreads / kWave) - 1) / (kThreads / kWave);
        const unsigned grid = (unsigned)(need < (1u << 20) ? need : (1u << 20));
        hipLaunchKernelGGL(quant_scalar_kernel, dim3(grid), dim3(kThreads), 0, stream, src, n,
                           block, codes, scales);
    }
    return hipGetLastError();
}

}  // namespace zpp
