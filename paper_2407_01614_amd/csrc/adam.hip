// Partition step: Adam(W) over one rank's flat fp32 shard, emitting the bf16
// primary shard (optimizer.step() of Algorithm 1 on the rank's partition).
//
// Pure streaming work: 16 B read + 14 B written per element and about 45
// VALU operations (correctly rounded sqrt and division included), so HBM
// bandwidth is the bound.  Each thread owns U float4 groups per tile; a wave's
// load instruction covers 1 KiB of one array, all 4*U loads of a tile are
// issued before any arithmetic, and every access is non-temporal (nothing is
// reused).  The grid is one-shot (one tile per workgroup): on this GPU a
// persistent grid of a few thousand workgroups streams about 20% slower.
// Residency is capped at ZPP_ADAM_RESIDENCY one-wave workgroups per CU: at
// the Llama-2-13B partition the step takes 923-931 us with 11 resident
// (931-944 with 9, 10 or 12), 1003-1016 us uncapped.
#include "zpp_adam.h"
#include "zpp_device.h"
#include "zpp_launch.h"

#ifndef ZPP_ADAM_UNROLL
#define ZPP_ADAM_UNROLL 1
#endif
#ifndef ZPP_ADAM_THREADS
#define ZPP_ADAM_THREADS 64
#endif
#ifndef ZPP_ADAM_RESIDENCY
#define ZPP_ADAM_RESIDENCY 11
#endif
#ifndef ZPP_ADAM_MAX_GRID
#define ZPP_ADAM_MAX_GRID (1u << 20)
#endif

namespace zpp {
namespace {

struct AdamArgs {
    float *p, *m, *v;
    const float *g;
    uint16_t *out;
    size_t n;
    AdamConsts c;
};

constexpr int kAdamThreads = ZPP_ADAM_THREADS;

template <bool ADAMW, int U>
__global__ __launch_bounds__(kAdamThreads) void adam_vec_kernel(AdamArgs a) {
    constexpr size_t kTile = (size_t)kAdamThreads * 4 * U;
    const size_t ntiles = (a.n + kTile - 1) / kTile;
    for (size_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const size_t base = t * kTile + (size_t)threadIdx.x * 4;
        if ((t + 1) * kTile <= a.n) {
            f32x4 P[U], M[U], V[U], G[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const size_t i = base + (size_t)u * kAdamThreads * 4;
                P[u] = ld_nt(reinterpret_cast<const f32x4 *>(a.p + i));
                M[u] = ld_nt(reinterpret_cast<const f32x4 *>(a.m + i));
                V[u] = ld_nt(reinterpret_cast<const f32x4 *>(a.v + i));
                G[u] = ld_nt(reinterpret_cast<const f32x4 *>(a.g + i));
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const size_t i = base + (size_t)u * kAdamThreads * 4;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    float p = P[u][e], m = M[u][e], v = V[u][e];
                    adam_update<ADAMW>(p, m, v, G[u][e], a.c);
                    P[u][e] = p;
                    M[u][e] = m;
                    V[u][e] = v;
                }
                st_nt(reinterpret_cast<f32x4 *>(a.p + i), P[u]);
                st_nt(reinterpret_cast<f32x4 *>(a.m + i), M[u]);
                st_nt(reinterpret_cast<f32x4 *>(a.v + i), V[u]);
                u32x2 o;
                o.x = pack_bf16x2(P[u].x, P[u].y);
                o.y = pack_bf16x2(P[u].z, P[u].w);
                st_nt(reinterpret_cast<u32x2 *>(a.out + i), o);
            }
        } else {
            // the last, partial tile: element by element
#pragma unroll
            for (int u = 0; u < U; ++u) {
                for (int e = 0; e < 4; ++e) {
                    const size_t i = base + (size_t)u * kAdamThreads * 4 + e;
                    if (i < a.n) {
                        float p = a.p[i], m = a.m[i], v = a.v[i];
                        adam_update<ADAMW>(p, m, v, a.g[i], a.c);
                        a.p[i] = p;
                        a.m[i] = m;
                        a.v[i] = v;
                        a.out[i] = (uint16_t)bf16_rne_bits(p);
                    }
                }
            }
        }
    }
}

// Any alignment: one element per thread, grid-stride.
template <bool ADAMW>
__global__ __launch_bounds__(kThreads) void adam_scalar_kernel(AdamArgs a) {
    const size_t stride = (size_t)gridDim.x * kThreads;
    for (size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x; i < a.n; i += stride) {
        float p = a.p[i], m = a.m[i], v = a.v[i];
        adam_update<ADAMW>(p, m, v, a.g[i], a.c);
        a.p[i] = p;
        a.m[i] = m;
        a.v[i] = v;
        a.out[i] = (uint16_t)bf16_rne_bits(p);
    }
}

}  // namespace

hipError_t launch_adam(float *p, float *m, float *v, const float *g, uint16_t *out, size_t n,
                       const AdamConsts &c, bool vector_path, hipStream_t stream) {
    AdamArgs a{p, m, v, g, out, n, c};
    if (vector_path) {
        constexpr size_t kTile = (size_t)kAdamThreads * 4 * ZPP_ADAM_UNROLL;
        size_t tiles = (n + kTile - 1) / kTile;
        const unsigned grid = (unsigned)(tiles < ZPP_ADAM_MAX_GRID ? tiles : ZPP_ADAM_MAX_GRID);
        constexpr size_t lds = residency_lds(ZPP_ADAM_RESIDENCY);
        if (c.adamw)
            hipLaunchKernelGGL((adam_vec_kernel<true, ZPP_ADAM_UNROLL>), dim3(grid),
                               dim3(kAdamThreads), lds, stream, a);
        else
            hipLaunchKernelGGL((adam_vec_kernel<false, ZPP_ADAM_UNROLL>), dim3(grid),
                               dim3(kAdamThreads), lds, stream, a);
    } else {
        size_t blocks = (n + kThreads - 1) / kThreads;
        const unsigned grid = (unsigned)(blocks < (1u << 20) ? blocks : (1u << 20));
        if (c.adamw)
            hipLaunchKernelGGL((adam_scalar_kernel<true>), dim3(grid), dim3(kThreads), 0,
                               stream, a);
        else
            hipLaunchKernelGGL((adam_scalar_kernel<false>), dim3(grid), dim3(kThreads), 0,
                               stream, a);
    }
    return hipGetLastError();
}

}  // namespace zpp
