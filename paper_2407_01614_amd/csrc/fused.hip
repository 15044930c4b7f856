// Fused partition step: the Adam update of the rank's partition, its bf16
// primary, the hpZ secondary copy and the qwZ int8 quantization of that copy,
// in one pass over HBM (optimizer.step() of Algorithm 1 followed, for the
// same weights, by the secondary copy of the forward loop and the qwZ
// quantization that precedes the gather).
//
// Per element: 16 B read (p, m, v, g); 12 B + 2 B + 2 B + 1 B written (p, m,
// v, primary, secondary, code) plus 4 B per block of scale: 33.016 B at block
// 256, against 30 + 4 + 3.016 = 37.016 B for the three separate kernels,
// which re-read the primary and the secondary from HBM.  The results are
// those of the three separate steps, bit for bit, because the quantization
// reads the same bf16 values the primary holds.
//
// One wave per chunk of C = max(B, 256) consecutive elements: lane l holds
// the 4 elements [chunk + 256 w + 4 l, +4) for w < C / 256.  The bf16 of the
// updated weights stays in registers (two per 4 elements) until the block's
// absmax is known; a 256-block is exactly one wave, so its absmax is a
// six-step cross-lane reduction.  Blocks of 64 to 512 take this kernel.  Any
// other block (1024 and up, or not a power of two) takes two passes: the same
// kernel with the 256-element chunks and no quantization (p, m, v, primary,
// secondary: 32 B per element), then the int8 quantizer over the primary it
// wrote (3 B + 4/B B), in stream order.  The 2 extra bytes per element cost
// less than holding a larger block's values in a wave: at the Llama-2-13B
// partition the two passes took 1094-1104 us at blocks of 192 to 4096, the
// one-pass layouts 1127-1186 us (one wave per chunk of whole blocks, several
// blocks per wave with the maxima in LDS, or workgroups of up to 16 waves
// with one float4 group per thread and a barrier per block), all but 512
// (1073 against 1095 us one pass); the single pass of the qgZ receive took
// 1112-1117 against 1245-1460 us.
// Residency is capped at ZPP_FUSED_RESIDENCY
// workgroups per CU, as for the optimizer step: 1031-1046 us with 12 resident
// at the Llama-2-13B partition (9-20 within 1%), 1127-1145 us uncapped.  With
// the qgZ receive in place of the fp32 gradient (8 int4 sources) the cap is
// ZPP_FUSED_RECV_RESIDENCY: 1111 us with 13, 1118 with 14, 1150 with 12, 1216
// with 11, 1142 uncapped.  From one interleaved receive buffer
// (ZPP_FUSED_RECV_IL_RESIDENCY): 1054 us with 14, 1062 with 16, 1075 with 12,
// 1097 uncapped, against 1096 us from separate arrays in the same run.
#include "zpp_adam.h"
#include "zpp_chunk.h"
#include "zpp_device.h"
#include "zpp_i4grad.h"
#include "zpp_launch.h"
#include "zpp_quant.h"

#ifndef ZPP_FUSED_RESIDENCY
#define ZPP_FUSED_RESIDENCY 12
#endif
#ifndef ZPP_FUSED_RECV_RESIDENCY
#define ZPP_FUSED_RECV_RESIDENCY 13
#endif
#ifndef ZPP_FUSED_RECV_IL_RESIDENCY
#define ZPP_FUSED_RECV_IL_RESIDENCY 14
#endif
#ifndef ZPP_FUSED_MAX_GRID
#define ZPP_FUSED_MAX_GRID (1u << 30)
#endif

namespace zpp {
namespace {

struct FusedArgs {
    float *p, *m, *v;
    uint16_t *primary;
    uint16_t *secondary;  // may be null: no bf16 secondary copy is kept
    int8_t *codes;
    float *scales;
    size_t n;
    AdamConsts c;
};

// Runs of consecutive workgroups per XCD: grouped for the qgZ receive from
// separate arrays (zpp_i4grad.h), plain otherwise.
template <class GS> constexpr size_t fused_xcd_run() { return 0; }
template <> constexpr size_t fused_xcd_run<I4Grad>() { return kSeparateXcdRun; }

// The gradient comes from `gs`: the fp32 array of the partition step
// (F32Grad), or the int4 copies of the qgZ receive (I4Grad, zpp_i4grad.h).
template <bool ADAMW, int B, class GS, bool QUANT = true>
__global__ __launch_bounds__(kWave) void fused_kernel(FusedArgs a, GS gs) {
    constexpr int C = B > 256 ? B : 256;  // elements per chunk (one wave)
    constexpr int W = C / 256;            // float4 groups per lane
    constexpr int L = B < 256 ? B / 4 : kWave;  // lanes per quant block
    const int lane = threadIdx.x;
    const size_t nchunks = (a.n + C - 1) / C;
    for (size_t ch = xcd_grouped(blockIdx.x, gridDim.x, fused_xcd_run<GS>()); ch < nchunks;
         ch += gridDim.x) {
        const size_t base = ch * C;
        const bool full = base + C <= a.n;
        u32x2 pk[W];
        u16x2 m2 = {0, 0};
#pragma unroll
        for (int w = 0; w < W; ++w) {
            const size_t i = base + (size_t)w * 256 + (size_t)lane * 4;
            if (full) {
                f32x4 P = ld_nt(reinterpret_cast<const f32x4 *>(a.p + i));
                f32x4 M = ld_nt(reinterpret_cast<const f32x4 *>(a.m + i));
                f32x4 V = ld_nt(reinterpret_cast<const f32x4 *>(a.v + i));
                const f32x4 G = grad_load4(gs, i);
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
                pk[w] = u32x2{pack_bf16x2(P.x, P.y), pack_bf16x2(P.z, P.w)};
                st_nt(reinterpret_cast<u32x2 *>(a.primary + i), pk[w]);
                if (a.secondary)
                    st_nt(reinterpret_cast<u32x2 *>(a.secondary + i), pk[w]);
            } else {
                // the last, partial chunk: element by element; absent elements
                // hold bf16 zero, which no absmax can see
                uint32_t h[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    h[e] = 0u;
                    if (i + e < a.n) {
                        float p = a.p[i + e], m = a.m[i + e], v = a.v[i + e];
                        adam_update<ADAMW>(p, m, v, grad_at(gs, i + e), a.c);
                        a.p[i + e] = p;
                        a.m[i + e] = m;
                        a.v[i + e] = v;
                        h[e] = bf16_rne_bits(p);
                        a.primary[i + e] = (uint16_t)h[e];
                        if (a.secondary)
                            a.secondary[i + e] = (uint16_t)h[e];
                    }
                }
                pk[w] = u32x2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
            }
            m2 = __builtin_elementwise_max(
                m2, __builtin_elementwise_max(absbits2(pk[w].x), absbits2(pk[w].y)));
        }
        if constexpr (QUANT) {
            uint32_t mx = max((uint32_t)m2.x, (uint32_t)m2.y);
#pragma unroll
            for (int off = L / 2; off >= 1; off >>= 1)
                mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
            const BlockQuant q = block_params(mx);
#pragma unroll
            for (int w = 0; w < W; ++w) {
                const size_t i = base + (size_t)w * 256 + (size_t)lane * 4;
                const uint32_t c4 = quant_word(pk[w].x, pk[w].y, q);
                if (full) {
                    st_nt(reinterpret_cast<uint32_t *>(a.codes + i), c4);
                } else {
                    for (int e = 0; e < 4 && i + e < a.n; ++e)
                        a.codes[i + e] = (int8_t)((c4 >> (8 * e)) & 0xFFu);
                }
            }
            // the first lane of each quant block writes its scale
            const size_t k = (base + (size_t)lane * 4) / B;
            if (lane % L == 0 && k * B < a.n)
                a.scales[k] = q.scale;
        }
    }
}

// Workgroups per CU for each gradient source.
template <class GS> constexpr int fused_residency();
template <> constexpr int fused_residency<F32Grad>() { return ZPP_FUSED_RESIDENCY; }
template <> constexpr int fused_residency<I4Grad>() { return ZPP_FUSED_RECV_RESIDENCY; }
template <> constexpr int fused_residency<I4GradIl>() { return ZPP_FUSED_RECV_IL_RESIDENCY; }

template <int B, class GS, bool QUANT = true>
void launch_fused_b(const FusedArgs &a, const GS &gs, hipStream_t stream) {
    constexpr size_t C = B > 256 ? B : 256;
    const size_t chunks = (a.n + C - 1) / C;
    const unsigned grid = (unsigned)(chunks < ZPP_FUSED_MAX_GRID ? chunks : ZPP_FUSED_MAX_GRID);
    constexpr size_t lds = residency_lds(fused_residency<GS>());
    if (a.c.adamw)
        hipLaunchKernelGGL((fused_kernel<true, B, GS, QUANT>), dim3(grid), dim3(kWave), lds,
                           stream, a, gs);
    else
        hipLaunchKernelGGL((fused_kernel<false, B, GS, QUANT>), dim3(grid), dim3(kWave), lds,
                           stream, a, gs);
}

template <class GS>
hipError_t launch_fused_gs(const FusedArgs &a, const GS &gs, uint32_t block,
                           hipStream_t stream) {
    switch (block) {
    case 64: launch_fused_b<64>(a, gs, stream); break;
    case 128: launch_fused_b<128>(a, gs, stream); break;
    case 256: launch_fused_b<256>(a, gs, stream); break;
    case 512: launch_fused_b<512>(a, gs, stream); break;
    default: {
        // the step and its copies in one pass, then the quantization of
        // the primary it wrote (stream order)
        launch_fused_b<256, GS, false>(a, gs, stream);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
        const bool qvec = reinterpret_cast<uintptr_t>(a.primary) % 16 == 0 &&
                          reinterpret_cast<uintptr_t>(a.codes) % 8 == 0;
        return launch_quantize(a.primary, a.n, block, a.codes, a.scales, qvec, stream);
    }
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_fused(float *p, float *m, float *v, const float *g, uint16_t *primary,
                        uint16_t *secondary, int8_t *codes, float *scales, size_t n,
                        uint32_t block, const AdamConsts &c, bool vector_path,
                        hipStream_t stream) {
    if (!vector_path) {
        // any alignment: the three separate scalar kernels, one after another
        // on the stream, compute the same values
        hipError_t e = launch_adam(p, m, v, g, primary, n, c, false, stream);
        if (e == hipSuccess && secondary)
            e = launch_refresh(secondary, primary, n, false, stream);
        if (e == hipSuccess)
            e = launch_quantize(primary, n, block, codes, scales, false, stream);
        return e;
    }
    const FusedArgs a{p, m, v, primary, secondary, codes, scales, n, c};
    return launch_fused_gs(a, F32Grad{g}, block, stream);
}

hipError_t launch_fused_receive(float *p, float *m, float *v, const uint8_t *const *src_codes,
                                const float *const *src_scales, uint32_t num_src,
                                uint32_t grad_block, float scale_out, uint16_t *primary,
                                uint16_t *secondary, int8_t *codes, float *scales, size_t n,
                                uint32_t block, const AdamConsts &c, bool vector_path,
                                hipStream_t stream) {
    if (!vector_path) {
        // any alignment: the receive step, the refresh and the quantization
        // as scalar kernels, one after another on the stream
        hipError_t e = launch_receive_adam(p, m, v, src_codes, src_scales, num_src, grad_block,
                                           scale_out, primary, n, c, false, stream);
        if (e == hipSuccess && secondary)
            e = launch_refresh(secondary, primary, n, false, stream);
        if (e == hipSuccess)
            e = launch_quantize(primary, n, block, codes, scales, false, stream);
        return e;
    }
    const FusedArgs a{p, m, v, primary, secondary, codes, scales, n, c};
    return launch_fused_gs(a, make_i4grad(src_codes, src_scales, num_src, grad_block, scale_out),
                           block, stream);
}

hipError_t launch_fused_receive_il(float *p, float *m, float *v, const uint8_t *src_codes,
                                   const float *src_scales, uint32_t num_src, uint32_t grad_block,
                                   float scale_out, uint16_t *primary, uint16_t *secondary,
                                   int8_t *codes, float *scales, size_t n, uint32_t block,
                                   const AdamConsts &c, bool vector_path, hipStream_t stream) {
    if (!vector_path) {
        // any alignment: the receive step, the refresh and the quantization
        // as scalar kernels, one after another on the stream
        hipError_t e = launch_receive_adam_il(p, m, v, src_codes, src_scales, num_src, grad_block,
                                              scale_out, primary, n, c, false, stream);
        if (e == hipSuccess && secondary)
            e = launch_refresh(secondary, primary, n, false, stream);
        if (e == hipSuccess)
            e = launch_quantize(primary, n, block, codes, scales, false, stream);
        return e;
    }
    const FusedArgs a{p, m, v, primary, secondary, codes, scales, n, c};
    return launch_fused_gs(a, make_i4grad_il(src_codes, src_scales, num_src, grad_block, scale_out),
                           block, stream);
}

}  // namespace zpp
