// Secondary refresh: bit copy of the local rank's bf16 weights into the hpZ
// secondary partition (Algorithm 1, forward loop; Eq. 1).  2 B read + 2 B
// written per element.  Each thread moves U 16-byte vectors per tile, all
// loads issued before the stores, non-temporal both ways.  Shape, swept at
// the Llama-2-13B partition (813 MB moved): one-wave workgroups with one
// vector per lane, residency left to the hardware, 120.7-123.1 us; four-wave
// workgroups with four vectors per lane 124.3-131.1 us, capped or not.
#include "zpp_device.h"
#include "zpp_launch.h"

#ifndef ZPP_REFRESH_UNROLL
#define ZPP_REFRESH_UNROLL 1
#endif
#ifndef ZPP_REFRESH_THREADS
#define ZPP_REFRESH_THREADS 64
#endif
#ifndef ZPP_REFRESH_RESIDENCY
#define ZPP_REFRESH_RESIDENCY 0
#endif
#ifndef ZPP_REFRESH_MAX_GRID
#define ZPP_REFRESH_MAX_GRID (1u << 20)
#endif

namespace zpp {
namespace {

constexpr int kRefreshThreads = ZPP_REFRESH_THREADS;

template <int U>
__global__ __launch_bounds__(kRefreshThreads) void refresh_vec_kernel(
    uint16_t *__restrict__ dst, const uint16_t *__restrict__ src, size_t count) {
    constexpr size_t kTile = (size_t)kRefreshThreads * 8 * U;  // 8 bf16 per 16-byte vector
    const size_t ntiles = (count + kTile - 1) / kTile;
    for (size_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const size_t base = t * kTile + (size_t)threadIdx.x * 8;
        if ((t + 1) * kTile <= count) {
            u32x4 x[U];
#pragma unroll
            for (int u = 0; u < U; ++u)
                x[u] = ld_nt(reinterpret_cast<const u32x4 *>(src + base +
                                                             (size_t)u * kRefreshThreads * 8));
#pragma unroll
            for (int u = 0; u < U; ++u)
                st_nt(reinterpret_cast<u32x4 *>(dst + base + (size_t)u * kRefreshThreads * 8),
                      x[u]);
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const size_t i0 = base + (size_t)u * kRefreshThreads * 8;
                if (i0 + 8 <= count) {
                    st_nt(reinterpret_cast<u32x4 *>(dst + i0),
                          ld_nt(reinterpret_cast<const u32x4 *>(src + i0)));
                } else {
                    for (size_t i = i0; i < count && i < i0 + 8; ++i)
                        dst[i] = src[i];
                }
            }
        }
    }
}

__global__ __launch_bounds__(kThreads) void refresh_scalar_kernel(uint16_t *__restrict__ dst,
                                                                  const uint16_t *__restrict__ src,
                                                                  size_t count) {
    const size_t stride = (size_t)gridDim.x * kThreads;
    for (size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x; i < count; i += stride)
        dst[i] = src[i];
}

}  // namespace

hipError_t launch_refresh(uint16_t *dst, const uint16_t *src, size_t count, bool vector_path,
                          hipStream_t stream) {
    if (vector_path) {
        constexpr size_t kTile = (size_t)kRefreshThreads * 8 * ZPP_REFRESH_UNROLL;
        const size_t tiles = (count + kTile - 1) / kTile;
        const unsigned grid =
            (unsigned)(tiles < ZPP_REFRESH_MAX_GRID ? tiles : ZPP_REFRESH_MAX_GRID);
        hipLaunchKernelGGL((refresh_vec_kernel<ZPP_REFRESH_UNROLL>), dim3(grid),
                           dim3(kRefreshThreads), residency_lds(ZPP_REFRESH_RESIDENCY), stream,
                           dst, src, count);
    } else {
        const size_t blocks = (count + kThreads - 1) / kThreads;
        const unsigned grid = (unsigned)(blocks < (1u << 20) ? blocks : (1u << 20));
        hipLaunchKernelGGL(refresh_scalar_kernel, dim3(grid), dim3(kThreads), 0, stream, dst,
                           src, count);
    }
    return hipGetLastError();
}

}  // namespace zpp
