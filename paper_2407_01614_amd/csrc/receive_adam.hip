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
// source) and one scale per source (zpp_i4grad.h: sources taken eight at a
// time, all eight in flight before their fma passes).  Residency is capped at
// ZPP_RECV_RESIDENCY workgroups per CU: at the Llama-2-13B partition with 8
// sources 994-1001 us with 12 (13: 995-999, 11: 1001-1008, 14: 1003-1011),
// 1027 us uncapped.  Scales loaded as wave-uniform scalar loads (possible for
// blocks of 256 or more) took 1112-1251 us: the scalar cache's latency is not
// hidden the way the vector loads' is.
//
// The same kernel reads the P copies from one interleaved receive buffer
// (I4GradIl, zpp_i4grad.h: a wave's codes of all sources within one
// contiguous run): 938 us with ZPP_RECV_IL_RESIDENCY = 12 (14: 949, 16: 955,
// uncapped 978) against 981 us from separate arrays in the same run.
#include "zpp_adam.h"
#include "zpp_chunk.h"
#include "zpp_device.h"
#include "zpp_i4grad.h"
#include "zpp_launch.h"

#ifndef ZPP_RECV_RESIDENCY
#define ZPP_RECV_RESIDENCY 12
#endif
#ifndef ZPP_RECV_IL_RESIDENCY
#define ZPP_RECV_IL_RESIDENCY 12
#endif
#ifndef ZPP_RECV_MAX_GRID
#define ZPP_RECV_MAX_GRID (1u << 30)
#endif

namespace zpp {
namespace {

// The gradient comes from `src`: the P int4 copies as separate arrays
// (I4Grad) or interleaved in one receive buffer (I4GradIl, zpp_i4grad.h).
template <class GS>
struct RecvArgs {
    GS src;
    float *p, *m, *v;
    uint16_t *out;
    size_t n;
    AdamConsts c;
};

template <bool ADAMW, class GS>
__device__ __forceinline__ void scalar_step(const RecvArgs<GS> &a, size_t i) {
    const float g = grad_at(a.src, i);
    float p = a.p[i], m = a.m[i], v = a.v[i];
    adam_update<ADAMW>(p, m, v, g, a.c);
    a.p[i] = p;
    a.m[i] = m;
    a.v[i] = v;
    a.out[i] = (uint16_t)bf16_rne_bits(p);
}

// Runs of consecutive workgroups per XCD: grouped for the separate arrays
// (zpp_i4grad.h), plain otherwise.
template <class GS> constexpr size_t recv_xcd_run() { return 0; }
template <> constexpr size_t recv_xcd_run<I4Grad>() { return kSeparateXcdRun; }

template <bool ADAMW, class GS>
__global__ __launch_bounds__(kWave) void recv_adam_kernel(RecvArgs<GS> a) {
    const size_t ntiles = (a.n + 255) / 256;
    const int lane = threadIdx.x;
    for (size_t t = xcd_grouped(blockIdx.x, gridDim.x, recv_xcd_run<GS>()); t < ntiles;
         t += gridDim.x) {
        const size_t i = t * 256 + (size_t)lane * 4;
        if (t * 256 + 256 > a.n) {
            // the last, partial tile: element by element
            for (int e = 0; e < 4; ++e)
                if (i + e < a.n)
                    scalar_step<ADAMW, GS>(a, i + e);
            continue;
        }
        f32x4 P = ld_nt(reinterpret_cast<const f32x4 *>(a.p + i));
        f32x4 M = ld_nt(reinterpret_cast<const f32x4 *>(a.m + i));
        f32x4 V = ld_nt(reinterpret_cast<const f32x4 *>(a.v + i));
        const f32x4 G = grad_load4(a.src, i);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float p = P[e], m = M[e], v = V[e];
            adam_update<ADAMW>(p, m, v, G[e], a.c);
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
template <bool ADAMW, class GS>
__global__ __launch_bounds__(kThreads) void recv_adam_scalar_kernel(RecvArgs<GS> a) {
    const size_t stride = (size_t)gridDim.x * kThreads;
    for (size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x; i < a.n; i += stride)
        scalar_step<ADAMW, GS>(a, i);
}

template <class GS>
hipError_t launch_recv(const RecvArgs<GS> &a, int residency, bool vector_path,
                       hipStream_t stream) {
    if (vector_path) {
        const size_t tiles = (a.n + 255) / 256;
        const unsigned grid = (unsigned)(tiles < ZPP_RECV_MAX_GRID ? tiles : ZPP_RECV_MAX_GRID);
        const size_t lds = residency_lds(residency);
        if (a.c.adamw)
            hipLaunchKernelGGL((recv_adam_kernel<true, GS>), dim3(grid), dim3(kWave), lds, stream,
                               a);
        else
            hipLaunchKernelGGL((recv_adam_kernel<false, GS>), dim3(grid), dim3(kWave), lds,
                               stream, a);
    } else {
        const size_t blocks = (a.n + kThreads - 1) / kThreads;
        const unsigned grid = (unsigned)(blocks < (1u << 20) ? blocks : (1u << 20));
        if (a.c.adamw)
            hipLaunchKernelGGL((recv_adam_scalar_kernel<true, GS>), dim3(grid), dim3(kThreads), 0,
                               stream, a);
        else
            hipLaunchKernelGGL((recv_adam_scalar_kernel<false, GS>), dim3(grid), dim3(kThreads),
                               0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace

I4Grad make_i4grad(const uint8_t *const *src_codes, const float *const *src_scales,
                   uint32_t num_src, uint32_t block, float scale_out) {
    I4Grad s = {};
    for (uint32_t q = 0; q < num_src; ++q) {
        s.codes[q] = src_codes[q];
        s.scales[q] = src_scales[q];
    }
    s.num_src = num_src;
    s.block = make_block_div(block);
    s.scale_out = scale_out;
    return s;
}

hipError_t launch_receive_adam(float *p, float *m, float *v, const uint8_t *const *src_codes,
                               const float *const *src_scales, uint32_t num_src, uint32_t block,
                               float scale_out, uint16_t *out, size_t n, const AdamConsts &c,
                               bool vector_path, hipStream_t stream) {
    RecvArgs<I4Grad> a = {};
    a.src = make_i4grad(src_codes, src_scales, num_src, block, scale_out);
    a.p = p;
    a.m = m;
    a.v = v;
    a.out = out;
    a.n = n;
    a.c = c;
    return launch_recv(a, ZPP_RECV_RESIDENCY, vector_path, stream);
}

I4GradIl make_i4grad_il(const uint8_t *codes, const float *scales, uint32_t num_src,
                        uint32_t block, float scale_out) {
    I4GradIl s = {};
    s.codes = codes;
    s.scales = scales;
    s.num_src = num_src;
    s.block = make_block_div(block);
    s.scale_out = scale_out;
    return s;
}

hipError_t launch_receive_adam_il(float *p, float *m, float *v, const uint8_t *codes,
                                  const float *scales, uint32_t num_src, uint32_t block,
                                  float scale_out, uint16_t *out, size_t n, const AdamConsts &c,
                                  bool vector_path, hipStream_t stream) {
    RecvArgs<I4GradIl> a = {};
    a.src = make_i4grad_il(codes, scales, num_src, block, scale_out);
    a.p = p;
    a.m = m;
    a.v = v;
    a.out = out;
    a.n = n;
    a.c = c;
    return launch_recv(a, ZPP_RECV_IL_RESIDENCY, vector_path, stream);
}

}  // namespace zpp
