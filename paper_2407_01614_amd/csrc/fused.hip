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
// six-step cross-lane reduction.  A block that is not a power of two (any
// multiple of 64 up to 4096) takes fused_multi_kernel: several whole blocks
// per wave at a time, the block absmax folded in LDS.  Blocks of more than
// 1024 values take fused_wg_kernel: a workgroup of several waves, one float4
// group per thread, the block absmax folded in LDS.
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
// The chunked kernel of blocks that are not powers of two keeps up to four
// groups per lane in flight, so fewer of its workgroups share a CU: at the
// Llama-2-13B partition, blocks of 192 / 320 / 960 / 2112 / 4032, 8 per CU
// took 1162 / 1189 / 1178 / 1189 / 1286 us, 6 per CU 1200 / 1195 / 1185 /
// 1180 / 1259, 12 per CU 1193 / 1228 / 1228 / 1220 / 1291, 4 per CU
// 1313-1606; one wave per block (the kernel it replaced) 1424 / 1215 / 1231
// / 1232 / 1284.
#ifndef ZPP_FUSED_MULTI_RESIDENCY
#define ZPP_FUSED_MULTI_RESIDENCY 8
#endif
// Blocks of more than 1024 values take fused_wg_kernel, workgroups of up to
// 16 waves with one float4 group per thread, capped at about this many waves
// per CU.  At the Llama-2-13B partition (median of 20 launches): 1088 /
// 2048 / 2112 / 4032 / 4096 took 1186 / 1180 / 1150 / 1205 / 1188 us with
// 16, against 1282 / 1240 / 1228 / 1343 / 1261 for the one-wave kernels
// (fused_kernel, fused_multi_kernel); with 12 per CU the workgroups of 9
// waves (1088, 2112) fit only once per CU and took 1342-1349 us.  At 1024
// and below it was no faster than the one-wave kernels (192 / 448 / 512 /
// 576 / 1024: 1190 / 1252 / 1106 / 1253 / 1210 against 1180 / 1214 / 1086
// / 1224 / 1178 us): a wave waits at the workgroup's barrier for the
// slowest of its block.
#ifndef ZPP_FUSED_WG_WAVES
#define ZPP_FUSED_WG_WAVES 16
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
template <bool ADAMW, int B, class GS>
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

// A block B = 64 b that is not a power of two: a wave takes K whole blocks at
// a time (zpp_chunk.h), lane l holding the float4 groups v 64 + l of the
// chunk for v < V, so every wave access of p, m, v and the gradient is
// 1 KiB contiguous as in fused_kernel.  The loads of up to four groups per
// lane are issued together; each group is updated and stored as in
// fused_kernel and its bf16 kept in registers; the groups' absmax is folded per block in LDS (or
// across the wave when one block fills the chunk), lane k < K derives block
// k's parameters and scale once, and every lane then stores its codes.  The
// results are those of the three separate kernels.
constexpr int kFusedBatch = 4;  // float4 groups per lane whose loads are in flight at once

template <bool ADAMW, class GS, int MAXV>
__global__ __launch_bounds__(kWave) void fused_multi_kernel(FusedArgs a, GS gs, BlockDiv blk,
                                                            uint32_t K, uint32_t V) {
    __shared__ uint32_t bmax[64];
    __shared__ BlockQuant bq[64];
    const uint32_t lane = threadIdx.x;
    const size_t B = blk.block;
    const size_t nblocks = (a.n + B - 1) / B;
    for (size_t k0 = (size_t)blockIdx.x * K; k0 < nblocks; k0 += (size_t)gridDim.x * K) {
        const uint32_t kc = (uint32_t)(nblocks - k0 < K ? nblocks - k0 : K);
        const size_t base = k0 * B;
        const size_t end = (base + kc * B < a.n) ? base + kc * B : a.n;
        if (lane < kc)
            bmax[lane] = 0u;
        __syncthreads();
        u32x2 pk[MAXV];
        if (end == base + (size_t)K * B) {
            // a whole chunk: every group complete; the loads of up to
            // kFusedBatch groups per lane in flight at once
            const uint32_t ngrp = K * (uint32_t)(B / 4);
#pragma unroll
            for (int v = 0; v < MAXV; ++v)
                pk[v] = u32x2{0u, 0u};
#pragma unroll
            for (int b0 = 0; b0 < MAXV; b0 += kFusedBatch) {
                if ((uint32_t)b0 >= V)
                    break;
                f32x4 P[kFusedBatch], M[kFusedBatch], Q[kFusedBatch], G[kFusedBatch];
#pragma unroll
                for (int u = 0; u < kFusedBatch; ++u) {
                    const uint32_t v = (uint32_t)(b0 + u), j = v * kWave + lane;
                    if (v < V && j < ngrp) {
                        const size_t i = base + (size_t)j * 4;
                        P[u] = ld_nt(reinterpret_cast<const f32x4 *>(a.p + i));
                        M[u] = ld_nt(reinterpret_cast<const f32x4 *>(a.m + i));
                        Q[u] = ld_nt(reinterpret_cast<const f32x4 *>(a.v + i));
                        G[u] = grad_load4(gs, i);
                    }
                }
#pragma unroll
                for (int u = 0; u < kFusedBatch; ++u) {
                    const uint32_t v = (uint32_t)(b0 + u), j = v * kWave + lane;
                    if (v < V && j < ngrp) {
                        const size_t i = base + (size_t)j * 4;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            float p = P[u][e], m = M[u][e], q = Q[u][e];
                            adam_update<ADAMW>(p, m, q, G[u][e], a.c);
                            P[u][e] = p;
                            M[u][e] = m;
                            Q[u][e] = q;
                        }
                        st_nt(reinterpret_cast<f32x4 *>(a.p + i), P[u]);
                        st_nt(reinterpret_cast<f32x4 *>(a.m + i), M[u]);
                        st_nt(reinterpret_cast<f32x4 *>(a.v + i), Q[u]);
                        pk[b0 + u] = u32x2{pack_bf16x2(P[u].x, P[u].y),
                                           pack_bf16x2(P[u].z, P[u].w)};
                        st_nt(reinterpret_cast<u32x2 *>(a.primary + i), pk[b0 + u]);
                        if (a.secondary)
                            st_nt(reinterpret_cast<u32x2 *>(a.secondary + i), pk[b0 + u]);
                    }
                }
            }
        } else {
            // the partition's last chunk: complete groups as above, the last
            // elements one by one
#pragma unroll
            for (int v = 0; v < MAXV; ++v) {
                pk[v] = u32x2{0u, 0u};
                const size_t i = base + ((size_t)v * kWave + lane) * 4;
                if ((uint32_t)v >= V || i >= end)
                    continue;
                if (i + 4 <= end) {
                    f32x4 P = ld_nt(reinterpret_cast<const f32x4 *>(a.p + i));
                    f32x4 M = ld_nt(reinterpret_cast<const f32x4 *>(a.m + i));
                    f32x4 Q = ld_nt(reinterpret_cast<const f32x4 *>(a.v + i));
                    const f32x4 G = grad_load4(gs, i);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        float p = P[e], m = M[e], q = Q[e];
                        adam_update<ADAMW>(p, m, q, G[e], a.c);
                        P[e] = p;
                        M[e] = m;
                        Q[e] = q;
                    }
                    st_nt(reinterpret_cast<f32x4 *>(a.p + i), P);
                    st_nt(reinterpret_cast<f32x4 *>(a.m + i), M);
                    st_nt(reinterpret_cast<f32x4 *>(a.v + i), Q);
                    pk[v] = u32x2{pack_bf16x2(P.x, P.y), pack_bf16x2(P.z, P.w)};
                    st_nt(reinterpret_cast<u32x2 *>(a.primary + i), pk[v]);
                    if (a.secondary)
                        st_nt(reinterpret_cast<u32x2 *>(a.secondary + i), pk[v]);
                } else {
                    uint32_t h[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        h[e] = 0u;
                        if (i + e < end) {
                            float p = a.p[i + e], m = a.m[i + e], q = a.v[i + e];
                            adam_update<ADAMW>(p, m, q, grad_at(gs, i + e), a.c);
                            a.p[i + e] = p;
                            a.m[i + e] = m;
                            a.v[i + e] = q;
                            h[e] = bf16_rne_bits(p);
                            a.primary[i + e] = (uint16_t)h[e];
                            if (a.secondary)
                                a.secondary[i + e] = (uint16_t)h[e];
                        }
                    }
                    pk[v] = u32x2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
                }
            }
        }
        uint32_t kl[MAXV];
#pragma unroll
        for (int v = 0; v < MAXV; ++v)
            kl[v] = 0u;
        if (K == 1) {
            // one block per chunk: its absmax is a reduction over the wave
            u16x2 m2 = {0, 0};
#pragma unroll
            for (int v = 0; v < MAXV; ++v)
                m2 = __builtin_elementwise_max(
                    m2, __builtin_elementwise_max(absbits2(pk[v].x), absbits2(pk[v].y)));
            uint32_t mx = max((uint32_t)m2.x, (uint32_t)m2.y);
#pragma unroll
            for (int off = kWave / 2; off >= 1; off >>= 1)
                mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
            if (lane == 0) {
                const BlockQuant q = block_params(mx);
                bq[0] = q;
                a.scales[k0] = q.scale;
            }
        } else {
#pragma unroll
            for (int v = 0; v < MAXV; ++v) {
                const size_t i = base + ((size_t)v * kWave + lane) * 4;
                if ((uint32_t)v < V && i < end) {
                    kl[v] = (uint32_t)(block_of(blk, i) - k0);
                    const u16x2 m2 =
                        __builtin_elementwise_max(absbits2(pk[v].x), absbits2(pk[v].y));
                    atomicMax(&bmax[kl[v]], max((uint32_t)m2.x, (uint32_t)m2.y));
                }
            }
            __syncthreads();
            if (lane < kc) {
                const BlockQuant q = block_params(bmax[lane]);
                bq[lane] = q;
                a.scales[k0 + lane] = q.scale;
            }
        }
        __syncthreads();
#pragma unroll
        for (int v = 0; v < MAXV; ++v) {
            const size_t i = base + ((size_t)v * kWave + lane) * 4;
            if ((uint32_t)v >= V || i >= end)
                continue;
            const uint32_t c4 = quant_word(pk[v].x, pk[v].y, bq[kl[v]]);
            if (i + 4 <= end) {
                st_nt(reinterpret_cast<uint32_t *>(a.codes + i), c4);
            } else {
                for (int e = 0; e < 4 && i + e < end; ++e)
                    a.codes[i + e] = (int8_t)((c4 >> (8 * e)) & 0xFFu);
            }
        }
        __syncthreads();  // bmax and bq are rewritten for the next chunk
    }
}

// Blocks of more than 1024 values: a workgroup of NW waves (NW = blockDim.x / 64, up to 16) takes kb whole blocks, one
// float4 group per thread, thread t holding the group at 4 t of the
// workgroup's span, so every thread does what a thread of fused_kernel does
// at 256: one group loaded, updated and stored at a time.  The block absmax
// goes through LDS: a wave that lies inside one block reduces it with
// cross-lane shuffles and folds it in with one LDS max, a wave that crosses
// a block boundary folds each lane's in; one barrier later every thread
// reads its block's absmax, derives the parameters and stores its codes.
template <bool ADAMW, class GS>
__global__ __launch_bounds__(1024) void fused_wg_kernel(FusedArgs a, GS gs, uint32_t B,
                                                        uint32_t kb) {
    extern __shared__ uint32_t bmax[];  // kb words at the start of the reservation
    const uint32_t tid = threadIdx.x;
    const uint32_t gpb = B / 4;  // float4 groups per block
    const uint32_t kl = tid / gpb;
    const bool active = kl < kb;
    const size_t nblocks = (a.n + B - 1) / B;
    // the wave lies inside one block of the workgroup (uniform)
    const uint32_t w0 = tid & ~(uint32_t)(kWave - 1);
    const bool wave_in_block = w0 / gpb == (w0 + kWave - 1) / gpb && (w0 + kWave - 1) / gpb < kb;
    for (size_t k0 = (size_t)blockIdx.x * kb; k0 < nblocks; k0 += (size_t)gridDim.x * kb) {
        if (tid < kb)
            bmax[tid] = 0u;
        const size_t i = k0 * B + (size_t)tid * 4;
        const bool live = active && i < a.n;
        u32x2 pk = {0u, 0u};
        if (live && i + 4 <= a.n) {
            f32x4 P = ld_nt(reinterpret_cast<const f32x4 *>(a.p + i));
            f32x4 M = ld_nt(reinterpret_cast<const f32x4 *>(a.m + i));
            f32x4 Q = ld_nt(reinterpret_cast<const f32x4 *>(a.v + i));
            const f32x4 G = grad_load4(gs, i);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                float p = P[e], m = M[e], q = Q[e];
                adam_update<ADAMW>(p, m, q, G[e], a.c);
                P[e] = p;
                M[e] = m;
                Q[e] = q;
            }
            st_nt(reinterpret_cast<f32x4 *>(a.p + i), P);
            st_nt(reinterpret_cast<f32x4 *>(a.m + i), M);
            st_nt(reinterpret_cast<f32x4 *>(a.v + i), Q);
            pk = u32x2{pack_bf16x2(P.x, P.y), pack_bf16x2(P.z, P.w)};
            st_nt(reinterpret_cast<u32x2 *>(a.primary + i), pk);
            if (a.secondary)
                st_nt(reinterpret_cast<u32x2 *>(a.secondary + i), pk);
        } else if (live) {
            // the partition's last elements, one by one; absent ones hold
            // bf16 zero, which no absmax can see
            uint32_t h[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                h[e] = 0u;
                if (i + e < a.n) {
                    float p = a.p[i + e], m = a.m[i + e], q = a.v[i + e];
                    adam_update<ADAMW>(p, m, q, grad_at(gs, i + e), a.c);
                    a.p[i + e] = p;
                    a.m[i + e] = m;
                    a.v[i + e] = q;
                    h[e] = bf16_rne_bits(p);
                    a.primary[i + e] = (uint16_t)h[e];
                    if (a.secondary)
                        a.secondary[i + e] = (uint16_t)h[e];
                }
            }
            pk = u32x2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
        }
        const u16x2 m2 = __builtin_elementwise_max(absbits2(pk.x), absbits2(pk.y));
        uint32_t mx = max((uint32_t)m2.x, (uint32_t)m2.y);
        __syncthreads();  // the zeroed words are visible
        if (wave_in_block) {
#pragma unroll
            for (int off = kWave / 2; off >= 1; off >>= 1)
                mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
            if ((tid & (kWave - 1)) == 0)
                atomicMax(&bmax[kl], mx);
        } else if (active) {
            atomicMax(&bmax[kl], mx);
        }
        __syncthreads();
        if (live) {
            const BlockQuant q = block_params(bmax[kl]);
            const uint32_t c4 = quant_word(pk.x, pk.y, q);
            if (i + 4 <= a.n) {
                st_nt(reinterpret_cast<uint32_t *>(a.codes + i), c4);
            } else {
                for (int e = 0; e < 4 && i + e < a.n; ++e)
                    a.codes[i + e] = (int8_t)((c4 >> (8 * e)) & 0xFFu);
            }
            if (tid == kl * gpb)
                a.scales[k0 + kl] = q.scale;
        }
        __syncthreads();  // the words are zeroed again for the next blocks
    }
}

// Workgroups per CU for each gradient source.
template <class GS> constexpr int fused_residency();
template <> constexpr int fused_residency<F32Grad>() { return ZPP_FUSED_RESIDENCY; }
template <> constexpr int fused_residency<I4Grad>() { return ZPP_FUSED_RECV_RESIDENCY; }
template <> constexpr int fused_residency<I4GradIl>() { return ZPP_FUSED_RECV_IL_RESIDENCY; }

template <int B, class GS>
void launch_fused_b(const FusedArgs &a, const GS &gs, hipStream_t stream) {
    constexpr size_t C = B > 256 ? B : 256;
    const size_t chunks = (a.n + C - 1) / C;
    const unsigned grid = (unsigned)(chunks < ZPP_FUSED_MAX_GRID ? chunks : ZPP_FUSED_MAX_GRID);
    constexpr size_t lds = residency_lds(fused_residency<GS>());
    if (a.c.adamw)
        hipLaunchKernelGGL((fused_kernel<true, B, GS>), dim3(grid), dim3(kWave), lds, stream, a,
                           gs);
    else
        hipLaunchKernelGGL((fused_kernel<false, B, GS>), dim3(grid), dim3(kWave), lds, stream, a,
                           gs);
}

// Workgroup shape of fused_wg_kernel for a block of gpb float4 groups: the
// fewest waves (1 to 16) whose threads the workgroup's whole blocks fill to
// at least 90%, failing that the largest fill.
struct WgShape {
    uint32_t waves, blocks;
};
inline WgShape fused_wg_shape(uint32_t gpb) {
    WgShape best = {0, 0};
    uint64_t best_used = 0, best_threads = 1;
    for (uint32_t nw = 1; nw <= 16; ++nw) {
        const uint32_t kb = nw * kWave / gpb;
        if (kb == 0)
            continue;
        const uint64_t used = (uint64_t)kb * gpb, threads = (uint64_t)nw * kWave;
        if (10 * used >= 9 * threads)
            return {nw, kb};
        if (used * best_threads > best_used * threads) {
            best = {nw, kb};
            best_used = used;
            best_threads = threads;
        }
    }
    return best;
}

template <class GS>
void launch_fused_wg(const FusedArgs &a, const GS &gs, uint32_t block, hipStream_t stream) {
    const WgShape sh = fused_wg_shape(block / 4);
    const size_t nblocks = (a.n + block - 1) / block;
    const size_t need = (nblocks + sh.blocks - 1) / sh.blocks;
    const unsigned grid = (unsigned)(need < ZPP_FUSED_MAX_GRID ? need : ZPP_FUSED_MAX_GRID);
    // about ZPP_FUSED_WG_WAVES waves per CU, as for the one-wave kernel
    int per_cu = (ZPP_FUSED_WG_WAVES + (int)sh.waves / 2) / (int)sh.waves;
    if (per_cu < 1)
        per_cu = 1;
    size_t lds = residency_lds(per_cu);
    if (lds < sh.blocks * sizeof(uint32_t))
        lds = sh.blocks * sizeof(uint32_t);
    const dim3 threads(sh.waves * kWave);
    if (a.c.adamw)
        hipLaunchKernelGGL((fused_wg_kernel<true, GS>), dim3(grid), threads, lds, stream, a, gs,
                           block, sh.blocks);
    else
        hipLaunchKernelGGL((fused_wg_kernel<false, GS>), dim3(grid), threads, lds, stream, a, gs,
                           block, sh.blocks);
}

template <class GS>
hipError_t launch_fused_gs(const FusedArgs &a, const GS &gs, uint32_t block,
                           hipStream_t stream) {
    switch (block) {
    case 64: launch_fused_b<64>(a, gs, stream); break;
    case 128: launch_fused_b<128>(a, gs, stream); break;
    case 256: launch_fused_b<256>(a, gs, stream); break;
    case 512: launch_fused_b<512>(a, gs, stream); break;
    case 1024: launch_fused_b<1024>(a, gs, stream); break;
    default: {
        if (block > 1024) {
            launch_fused_wg(a, gs, block, stream);
            break;
        }
        // blocks of up to 1024 values: at most 4 float4 groups per lane;
        // larger ones 16 (4096 / 4 = 1024 groups fit 64 x 16)
        const bool small = block / 4 <= 64 * 4;
        const ChunkShape sh = chunk_shape(block / 4, small ? 4 : 16);
        const size_t nblocks = (a.n + block - 1) / block;
        const size_t need = (nblocks + sh.K - 1) / sh.K;
        const unsigned grid = (unsigned)(need < ZPP_FUSED_MAX_GRID ? need : ZPP_FUSED_MAX_GRID);
        constexpr size_t lds = residency_lds(ZPP_FUSED_MULTI_RESIDENCY);
        const BlockDiv d = make_block_div(block);
        if (small) {
            if (a.c.adamw)
                hipLaunchKernelGGL((fused_multi_kernel<true, GS, 4>), dim3(grid), dim3(kWave),
                                   lds, stream, a, gs, d, sh.K, sh.V);
            else
                hipLaunchKernelGGL((fused_multi_kernel<false, GS, 4>), dim3(grid), dim3(kWave),
                                   lds, stream, a, gs, d, sh.K, sh.V);
        } else {
            if (a.c.adamw)
                hipLaunchKernelGGL((fused_multi_kernel<true, GS, 16>), dim3(grid), dim3(kWave),
                                   lds, stream, a, gs, d, sh.K, sh.V);
            else
                hipLaunchKernelGGL((fused_multi_kernel<false, GS, 16>), dim3(grid), dim3(kWave),
                                   lds, stream, a, gs, d, sh.K, sh.V);
        }
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
