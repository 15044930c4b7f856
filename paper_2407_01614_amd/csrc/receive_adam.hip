// qgZ receive fused into the partition step: the rank's optimizer step takes
// its gradient straight from the P int4 copies of its partition that the
// exchange replacing the ReduceScatter delivered (Background section: qgZ;
// Algorithm 1, backward loop, and the optimizer.step() closing it), instead
// of reading an fp32 gradient that a separate dequantize-and-reduce wrote.
//
// Per element: 12 B read (p, m, v) plus P (0.5 B + 4/B B) of codes and
// scales, 14 B written (p, m, v, bf16 primary): 30.125 B at P = 8 and block
// 256, against 8.125 + 30 B for the two kernels in sequence, which write the
// fp32 gradient and read it back.  The gradient is formed exactly as the
// dequantize-and-reduce forms it (acc = fma(code, scale, acc) over the
// sources in order from acc = 0, then one multiply by the output scale) and
// the update is the partition step's own, so the results are those of the
// two calls, bit for bit.
//
// Lane layout of the partition step: one wave per 256-element tile, lane l
// holds elements [256 t + 4 l, +4): one 16-byte access per state array, one
// 2-byte load of codes per source (a wave reads 128 contiguous bytes of each
// source) and one scale per source.  Sources are loaded eight at a time, all
// eight in flight before their fma passes.  Residency is capped at
// ZPP_RECV_RESIDENCY workgroups per CU: at the Llama-2-13B partition with 8
// sources 994-1001 us with 12 (13: 995-999, 11: 1001-1008, 14: 1003-1011),
// 1027 us uncapped.  Scales loaded as wave-uniform scalar loads (possible for
// blocks of 256 or more) took 1112-1251 us: the scalar cache's latency is not
// hidden the way the vector loads' is.
#include "zpp_adam.h"
#include "zpp_device.h"
#include "zpp_launch.h"
#include "zpp_quant.h"

#ifndef ZPP_RECV_RESIDENCY
#define ZPP_RECV_RESIDENCY 12
#endif
#ifndef ZPP_RECV_MAX_GRID
#define ZPP_RECV_MAX_GRID (1u << 30)
#endif

namespace zpp {
namespace {

struct RecvArgs {
    const uint8_t *codes[kMaxShards];
    const float *scales[kMaxShards];
    float *p, *m, *v;
    uint16_t *out;
    size_t n;
    uint32_t num_src;
    uint32_t block_shift;  // log2(block)
    float scale_out;
    AdamConsts c;
};

constexpr int kBatch = 8;

// The output scale, applied as its own rounded multiply: the two-kernel
// sequence stores this product to memory before the update reads it, so it
// must not be contracted into an add of the update.
__device__ __forceinline__ float scaled(float acc, float scale_out) {
#pragma clang fp contract(off)
    return acc * scale_out;
}

// The gradient of element i from the sources, one element at a time (tails
// and the any-alignment kernel).
__device__ __forceinline__ float gradient_at(const RecvArgs &a, size_t i) {
    float acc = 0.0f;
    for (uint32_t q = 0; q < a.num_src; ++q) {
        const uint32_t byte = a.codes[q][i / 2];
        const uint32_t nib = (i % 2 == 0) ? (byte & 0xFu) : (byte >> 4);
        acc = __builtin_fmaf(i4_code(nib, 0), a.scales[q][i >> a.block_shift], acc);
    }
    return scaled(acc, a.scale_out);
}

template <bool ADAMW>
__device__ __forceinline__ void scalar_step(const RecvArgs &a, size_t i) {
    const float g = gradient_at(a, i);
    float p = a.p[i], m = a.m[i], v = a.v[i];
    adam_update<ADAMW>(p, m, v, g, a.c);
    a.p[i] = p;
    a.m[i] = m;
    a.v[i] = v;
    a.out[i] = (uint16_t)bf16_rne_bits(p);
}

template <bool ADAMW>
__global__ __launch_bounds__(kWave) void recv_adam_kernel(RecvArgs a) {
    const size_t ntiles = (a.n + 255) / 256;
    const int lane = threadIdx.x;
    for (size_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const size_t i = t * 256 + (size_t)lane * 4;
        if (t * 256 + 256 > a.n) {
            // the last, partial tile: element by element
            for (int e = 0; e < 4; ++e)
                if (i + e < a.n)
                    scalar_step<ADAMW>(a, i + e);
            continue;
        }
        f32x4 P = ld_nt(reinterpret_cast<const f32x4 *>(a.p + i));
        f32x4 M = ld_nt(reinterpret_cast<const f32x4 *>(a.m + i));
        f32x4 V = ld_nt(reinterpret_cast<const f32x4 *>(a.v + i));
        float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        for (uint32_t q0 = 0; q0 < a.num_src; q0 += kBatch) {
            uint32_t w[kBatch];
            float s[kBatch];
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                const uint32_t q = q0 + j;
                w[j] = 0u;
                s[j] = 0.0f;
                if (q < a.num_src) {
                    w[j] = ld_nt(reinterpret_cast<const uint16_t *>(a.codes[q] + i / 2));
                    s[j] = a.scales[q][i >> a.block_shift];
                }
            }
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                if (q0 + j < a.num_src) {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        acc[e] = __builtin_fmaf(i4_code(w[j], e), s[j], acc[e]);
                }
            }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float p = P[e], m = M[e], v = V[e];
            adam_update<ADAMW>(p, m, v, scaled(acc[e], a.scale_out), a.c);
            P[e] = p;
            M[e] = m;
            V[e] = v;
        }
        st_nt(reinterpret_cast<f32x4 *>(a.p + i), P);
        st_nt(reinterpret_cast<f32x4 *>(a.m + i), M);
        st_nt(reinterpret_cast<f32x4 *>(a.v + i), V);
        u32x2 o;
        o.x = pack_bf16x2(P.x, P.y);
        o.y = pack_bf16x2(P.z, P.w);
        st_nt(reinterpret_cast<u32x2 *>(a.out + i), o);
    }
}

// Any alignment: one element per thread, grid-stride.
template <bool ADAMW>
__global__ __launch_bounds__(kThreads) void recv_adam_scalar_kernel(RecvArgs a) {
    const size_t stride = (size_t)gridDim.x * kThreads;
    for (size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x; i < a.n; i += stride)
        scalar_step<ADAMW>(a, i);
}

}  // namespace

hipError_t launch_receive_adam(float *p, float *m, float *v, const uint8_t *const *src_codes,
                               const float *const *src_scales, uint32_t num_src, uint32_t block,
                               float scale_out, uint16_t *out, size_t n, const AdamConsts &c,
                               bool vector_path, hipStream_t stream) {
    RecvArgs a = {};
    for (uint32_t q = 0; q < num_src; ++q) {
        a.codes[q] = src_codes[q];
        a.scales[q] = src_scales[q];
    }
    a.p = p;
    a.m = m;
    a.v = v;
    a.out = out;
    a.n = n;
    a.num_src = num_src;
    a.block_shift = (uint32_t)__builtin_ctz(block);
    a.scale_out = scale_out;
    a.c = c;
    if (vector_path) {
        const size_t tiles = (n + 255) / 256;
        const unsigned grid = (unsigned)(tiles < ZPP_RECV_MAX_GRID ? tiles : ZPP_RECV_MAX_GRID);
        constexpr size_t lds = residency_lds(ZPP_RECV_RESIDENCY);
        if (c.adamw)
            hipLaunchKernelGGL((recv_adam_kernel<true>), dim3(grid), dim3(kWave), lds, stream, a);
        else
            hipLaunchKernelGGL((recv_adam_kernel<false>), dim3(grid), dim3(kWave), lds, stream, a);
    } else {
        const size_t blocks = (n + kThreads - 1) / kThreads;
        const unsigned grid = (unsigned)(blocks < (1u << 20) ? blocks : (1u << 20));
        if (c.adamw)
            hipLaunchKernelGGL((recv_adam_scalar_kernel<true>), dim3(grid), dim3(kThreads), 0,
                               stream, a);
        else
            hipLaunchKernelGGL((recv_adam_scalar_kernel<false>), dim3(grid), dim3(kThreads), 0,
                               stream, a);
    }
    return hipGetLastError();
}

}  // namespace zpp
