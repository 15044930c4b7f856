// qgZ, the gradient side of the partition step: blockwise int4 quantization
// of fp32 gradients before the exchange that replaces the ReduceScatter
// (Background section; Algorithm 1, backward loop), and, on the receiving
// rank, the dequantize-and-reduce of the P quantized copies of its partition
// into the fp32 gradient the optimizer step consumes.
//
// Quantize: 4 B read, 0.5 B + 4/B B written per element.  A lane holds 8
// consecutive values (two 16-byte loads); the absmax is an integer max of the
// |x| bit patterns (bits >= 0x7F800000 mean Inf or NaN), reduced over the
// B/8 lanes of a block with xor shuffles.  Codes come from the same
// round-to-nearest-even trick as the int8 quantizer (the low bits of
// x*inv + 1.5*2^23), and 8 codes are packed into one 32-bit store.
//
// Dequant-reduce: P * (0.5 B + 4/B B) read, 4 B written per element.  The
// sources' pointers travel by value in the kernel arguments; a lane
// accumulates 8 elements over the sources in order, one fma each, loading
// four sources ahead.
#include "zpp_device.h"
#include "zpp_launch.h"
#include "zpp_quant.h"

#ifndef ZPP_QGZ_THREADS
#define ZPP_QGZ_THREADS 256
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

// 8 values -> 8 int4 codes packed little-endian in one word.  No clamp is
// needed: |x * inv| rounds to at most 7 (1 + 2^-24)^2 < 7.5.
__device__ __forceinline__ uint32_t i4_word(const f32x4 &lo, const f32x4 &hi, const I4Quant &q) {
#pragma clang fp contract(off)
    float x[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    uint32_t b[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float xe = q.tiny ? x[e] * q.pre : x[e];
        b[e] = code_bits(xe * q.inv);
    }
    // low bytes of each group of four, then their low nibbles side by side
    const uint32_t w0 = pack_low_bytes(b[0], b[1], b[2], b[3]) & 0x0F0F0F0Fu;
    const uint32_t w1 = pack_low_bytes(b[4], b[5], b[6], b[7]) & 0x0F0F0F0Fu;
    const uint32_t t0 = w0 | (w0 >> 4);  // bytes 0 and 2 hold (c0|c1<<4), (c2|c3<<4)
    const uint32_t t1 = w1 | (w1 >> 4);
    const uint32_t packed = __builtin_amdgcn_perm(t1, t0, 0x06040200u);
    return q.zero ? 0u : packed;
}

__device__ __forceinline__ uint32_t abs_bits_max4(const f32x4 &v) {
    return max(max(__float_as_uint(v.x) & 0x7FFFFFFFu, __float_as_uint(v.y) & 0x7FFFFFFFu),
               max(__float_as_uint(v.z) & 0x7FFFFFFFu, __float_as_uint(v.w) & 0x7FFFFFFFu));
}

template <int B>
__global__ __launch_bounds__(kQgzThreads) void quant_i4_kernel(const float *__restrict__ src,
                                                               size_t n, uint8_t *__restrict__ codes,
                                                               float *__restrict__ scales) {
    constexpr int L = (B / 8 < kWave) ? B / 8 : kWave;  // lanes per block
    constexpr int V = (B / 8 > kWave) ? B / (8 * kWave) : 1;
    constexpr int kGroupsPerWave = kWave / L;
    constexpr int kGroupsPerBlock = kGroupsPerWave * (kQgzThreads / kWave);
    const size_t nblocks = (n + B - 1) / B;
    const size_t nbytes = (n + 1) / 2;
    const int lane = threadIdx.x & (kWave - 1);
    const int gl = lane / L, li = lane % L;
    const int wave = threadIdx.x / kWave;
    for (size_t g0 = (size_t)blockIdx.x * kGroupsPerBlock; g0 < nblocks;
         g0 += (size_t)gridDim.x * kGroupsPerBlock) {
        const size_t k = g0 + (size_t)wave * kGroupsPerWave + gl;
        const bool valid = k < nblocks;
        f32x4 x[V][2];
        uint32_t mx = 0;
#pragma unroll
        for (int v = 0; v < V; ++v) {
            const size_t i = k * B + ((size_t)v * L + li) * 8;
            if (valid && i + 8 <= n) {
                x[v][0] = ld_nt(reinterpret_cast<const f32x4 *>(src + i));
                x[v][1] = ld_nt(reinterpret_cast<const f32x4 *>(src + i + 4));
            } else {
                float h[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    h[e] = (valid && i + e < n) ? src[i + e] : 0.0f;
                x[v][0] = f32x4{h[0], h[1], h[2], h[3]};
                x[v][1] = f32x4{h[4], h[5], h[6], h[7]};
            }
            mx = max(mx, max(abs_bits_max4(x[v][0]), abs_bits_max4(x[v][1])));
        }
#pragma unroll
        for (int off = L / 2; off >= 1; off >>= 1)
            mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
        const I4Quant q = i4_params(mx);
#pragma unroll
        for (int v = 0; v < V; ++v) {
            const size_t i = k * B + ((size_t)v * L + li) * 8;
            const uint32_t w = i4_word(x[v][0], x[v][1], q);
            const size_t byte0 = i / 2;
            if (valid && byte0 + 4 <= nbytes) {
                st_nt(reinterpret_cast<uint32_t *>(codes + byte0), w);
            } else if (valid) {
                for (int e = 0; e < 4 && byte0 + e < nbytes; ++e)
                    codes[byte0 + e] = (uint8_t)(w >> (8 * e));
            }
        }
        if (valid && li == 0)
            scales[k] = q.scale;
    }
}

// Any alignment: one wave per block, lanes stride through it; each code
// byte is written by the lane that owns its even element.
__global__ __launch_bounds__(kQgzThreads) void quant_i4_scalar_kernel(const float *__restrict__ src,
                                                                      size_t n, uint32_t block,
                                                                      uint8_t *__restrict__ codes,
                                                                      float *__restrict__ scales) {
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
            const uint32_t w = i4_word(f32x4{x0, x1, 0.0f, 0.0f}, f32x4{0.0f, 0.0f, 0.0f, 0.0f}, q);
            codes[i / 2] = (uint8_t)(w & 0xFFu);
        }
        if (lane == 0)
            scales[k] = q.scale;
    }
}

struct ReduceArgs {
    const uint8_t *codes[kMaxShards];
    const float *scales[kMaxShards];
    uint32_t num_src;
    size_t n;
    uint32_t block_shift;
    float scale_out;
    float *out;
};

__device__ __forceinline__ float i4_code(uint32_t w, int e) {
    return (float)((int32_t)(w << (28 - 4 * e)) >> 28);
}

__global__ __launch_bounds__(kQgzThreads) void reduce_i4_kernel(ReduceArgs a) {
    const size_t chunks = (a.n + 7) / 8;
    for (size_t c = (size_t)blockIdx.x * kQgzThreads + threadIdx.x; c < chunks;
         c += (size_t)gridDim.x * kQgzThreads) {
        const size_t i = c * 8;
        const bool full = i + 8 <= a.n;
        float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        const size_t kb = i >> a.block_shift;
        for (uint32_t q0 = 0; q0 < a.num_src; q0 += 4) {
            uint32_t w[4];
            float s[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t q = q0 + j;
                if (q < a.num_src) {
                    if (full) {
                        w[j] = ld_nt(reinterpret_cast<const uint32_t *>(a.codes[q] + i / 2));
                    } else {
                        w[j] = 0;
                        for (size_t e = i; e < a.n; e += 2)
                            w[j] |= (uint32_t)a.codes[q][e / 2] << (4 * (e - i));
                    }
                    s[j] = a.scales[q][kb];
                } else {
                    w[j] = 0;
                    s[j] = 0.0f;
                }
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (q0 + j < a.num_src) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        acc[e] = __builtin_fmaf(i4_code(w[j], e), s[j], acc[e]);
                }
            }
        }
        if (full) {
            st_nt(reinterpret_cast<f32x4 *>(a.out + i),
                  f32x4{acc[0] * a.scale_out, acc[1] * a.scale_out, acc[2] * a.scale_out,
                        acc[3] * a.scale_out});
            st_nt(reinterpret_cast<f32x4 *>(a.out + i + 4),
                  f32x4{acc[4] * a.scale_out, acc[5] * a.scale_out, acc[6] * a.scale_out,
                        acc[7] * a.scale_out});
        } else {
            for (size_t e = i; e < a.n; ++e)
                a.out[e] = acc[e - i] * a.scale_out;
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
            acc = __builtin_fmaf(i4_code(nib, 0), a.scales[q][i >> a.block_shift], acc);
        }
        a.out[i] = acc * a.scale_out;
    }
}

template <int B>
void launch_quant_i4_b(const float *src, size_t n, uint8_t *codes, float *scales,
                       hipStream_t stream) {
    constexpr int L = (B / 8 < kWave) ? B / 8 : kWave;
    constexpr size_t kGroupsPerBlock = (kWave / L) * (kQgzThreads / kWave);
    const size_t nblocks = (n + B - 1) / B;
    const size_t need = (nblocks + kGroupsPerBlock - 1) / kGroupsPerBlock;
    const unsigned grid = (unsigned)(need < ZPP_QGZ_MAX_GRID ? need : ZPP_QGZ_MAX_GRID);
    hipLaunchKernelGGL((quant_i4_kernel<B>), dim3(grid), dim3(kQgzThreads), 0, stream, src, n,
                       codes, scales);
}

}  // namespace

hipError_t launch_quantize_i4(const float *src, size_t n, uint32_t block, uint8_t *codes,
                              float *scales, bool vector_path, hipStream_t stream) {
    if (vector_path) {
        switch (block) {
        case 64: launch_quant_i4_b<64>(src, n, codes, scales, stream); break;
        case 128: launch_quant_i4_b<128>(src, n, codes, scales, stream); break;
        case 256: launch_quant_i4_b<256>(src, n, codes, scales, stream); break;
        case 512: launch_quant_i4_b<512>(src, n, codes, scales, stream); break;
        case 1024: launch_quant_i4_b<1024>(src, n, codes, scales, stream); break;
        case 2048: launch_quant_i4_b<2048>(src, n, codes, scales, stream); break;
        case 4096: launch_quant_i4_b<4096>(src, n, codes, scales, stream); break;
        default: return hipErrorInvalidValue;
        }
    } else {
        const size_t nblocks = (n + block - 1) / block;
        const size_t need = (nblocks + (kQgzThreads / kWave) - 1) / (kQgzThreads / kWave);
        const unsigned grid = (unsigned)(need < (1u << 20) ? need : (1u << 20));
        hipLaunchKernelGGL(quant_i4_scalar_kernel, dim3(grid), dim3(kQgzThreads), 0, stream, src,
                           n, block, codes, scales);
    }
    return hipGetLastError();
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
    a.block_shift = (uint32_t)__builtin_ctz(block);
    a.scale_out = scale_out;
    a.out = out;
    if (vector_path) {
        const size_t chunks = (n + 7) / 8;
        const size_t need = (chunks + kQgzThreads - 1) / kQgzThreads;
        const unsigned grid = (unsigned)(need < ZPP_QGZ_MAX_GRID ? need : ZPP_QGZ_MAX_GRID);
        hipLaunchKernelGGL(reduce_i4_kernel, dim3(grid), dim3(kQgzThreads), 0, stream, a);
    } else {
        const size_t need = (n + kQgzThreads - 1) / kQgzThreads;
        const unsigned grid = (unsigned)(need < (1u << 20) ? need : (1u << 20));
        hipLaunchKernelGGL(reduce_i4_scalar_kernel, dim3(grid), dim3(kQgzThreads), 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace zpp
