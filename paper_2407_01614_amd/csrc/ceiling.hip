// Plain HBM streams (include/zpp_ceiling.h): the read-only, write-only and
// copy ceilings of this GPU, which the partition-path kernels are measured
// against, and the access patterns of three of those kernels with their
// arithmetic taken out.  Built into its own library; not part of the
// partition path.
#include "zpp_ceiling.h"
#include "zpp_device.h"

namespace {

using zpp::f32x4;
using zpp::ld_nt;
using zpp::residency_lds;
using zpp::st_nt;
using zpp::u32x2;
using zpp::u32x4;

constexpr int kReadThreads = 64, kReadVecs = 4, kReadResidency = 16;
constexpr int kWriteThreads = 256, kWriteResidency = 4;
constexpr int kCopyThreads = 64;
constexpr size_t kTileBytes = 4096;  // read and write tiles; a copy tile is 1 KiB
static_assert(kReadThreads * kReadVecs * 16 == kTileBytes, "read tile");
static_assert(kWriteThreads * 16 == kTileBytes, "write tile");

constexpr uint32_t kNeverFolded = 0x9E3779B9u;

__global__ __launch_bounds__(kReadThreads) void read_kernel(const u32x4 *__restrict__ src,
                                                            uint32_t *__restrict__ sink) {
    const size_t base = (size_t)blockIdx.x * (kTileBytes / 16) + threadIdx.x;
    u32x4 x[kReadVecs];
#pragma unroll
    for (int u = 0; u < kReadVecs; ++u)
        x[u] = ld_nt(src + base + (size_t)u * kReadThreads);
    uint32_t acc = 0;
#pragma unroll
    for (int u = 0; u < kReadVecs; ++u)
        acc ^= x[u].x ^ x[u].y ^ x[u].z ^ x[u].w;
    for (int off = 32; off >= 1; off >>= 1)
        acc ^= (uint32_t)__shfl_xor((int)acc, off);
    if (threadIdx.x == 0 && acc == kNeverFolded)
        sink[0] = acc;
}

__global__ __launch_bounds__(kWriteThreads) void write_kernel(u32x4 *__restrict__ dst,
                                                              uint32_t pattern) {
    const size_t i = (size_t)blockIdx.x * (kTileBytes / 16) + threadIdx.x;
    st_nt(dst + i, u32x4{pattern, pattern, pattern, pattern});
}

__global__ __launch_bounds__(kCopyThreads) void copy_kernel(u32x4 *__restrict__ dst,
                                                            const u32x4 *__restrict__ src) {
    const size_t i = (size_t)blockIdx.x * kCopyThreads + threadIdx.x;
    st_nt(dst + i, ld_nt(src + i));
}

// Access patterns.  Each moves exactly the bytes of its kernel in the
// kernel's lane layout, workgroup shape, grid and residency, and replaces the
// arithmetic by one xor per loaded word, so its time is what the memory
// system gives that pattern.

// The Adam step (adam.hip): one-wave workgroups, one 256-element tile each;
// a lane loads one float4 of p, m, v and g, stores float4 p, m, v in place
// and 4 bf16 (8 bytes); at most 11 workgroups per CU (the step's own cap).
constexpr int kAdamPatternResidency = 11;

__global__ __launch_bounds__(64) void adam_pattern_kernel(float *__restrict__ p,
                                                          float *__restrict__ m,
                                                          float *__restrict__ v,
                                                          const float *__restrict__ g,
                                                          uint16_t *__restrict__ out) {
    const size_t i = (size_t)blockIdx.x * 256 + (size_t)threadIdx.x * 4;
    const u32x4 P = ld_nt(reinterpret_cast<const u32x4 *>(p + i));
    const u32x4 M = ld_nt(reinterpret_cast<const u32x4 *>(m + i));
    const u32x4 V = ld_nt(reinterpret_cast<const u32x4 *>(v + i));
    const u32x4 G = ld_nt(reinterpret_cast<const u32x4 *>(g + i));
    const u32x4 P1 = P ^ G;
    st_nt(reinterpret_cast<u32x4 *>(p + i), P1);
    st_nt(reinterpret_cast<u32x4 *>(m + i), M ^ G);
    st_nt(reinterpret_cast<u32x4 *>(v + i), V ^ G);
    st_nt(reinterpret_cast<u32x2 *>(out + i),
          u32x2{(P1.x >> 16) | (P1.y & 0xFFFF0000u), (P1.z >> 16) | (P1.w & 0xFFFF0000u)});
}

// The dequant-gather's row kernel (gather.hip), blocks of 256: one-wave
// workgroups, one 512-element row each; a lane loads 8 codes (8 bytes) and
// stores 8 bf16 (16 bytes); the row's two scales are scalar loads.
__global__ __launch_bounds__(64) void gather_pattern_kernel(const int8_t *__restrict__ codes,
                                                            const float *__restrict__ scales,
                                                            uint16_t *__restrict__ out) {
    const size_t r = blockIdx.x;
    const size_t i = r * 512 + (size_t)threadIdx.x * 8;
    const u32x2 c = ld_nt(reinterpret_cast<const u32x2 *>(codes + i));
    const float s0 = scales[2 * r], s1 = scales[2 * r + 1];  // uniform: scalar loads
    const uint32_t s = __float_as_uint(threadIdx.x < 32 ? s0 : s1);
    st_nt(reinterpret_cast<u32x4 *>(out + i), u32x4{c.x, c.y, c.x ^ s, c.y ^ s});
}

// The int8 quantizer (quant.hip), blocks of 256: four-wave workgroups, two
// rows per wave; a lane loads 8 bf16 (16 bytes) of one row, then stores its
// 8 codes (8 bytes), and the first lane of each 32-lane block its scale.
__global__ __launch_bounds__(256) void quant_pattern_kernel(const uint16_t *__restrict__ src,
                                                            int8_t *__restrict__ codes,
                                                            float *__restrict__ scales) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x / 64;
    // 16 blocks of 256 per workgroup: row u of wave w holds blocks 8 u + 2 w, + 1
    const size_t g0 = (size_t)blockIdx.x * 16;
    u32x4 x[2];
    size_t k[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        k[u] = g0 + (size_t)u * 8 + (size_t)wave * 2 + (size_t)(lane / 32);
        x[u] = ld_nt(reinterpret_cast<const u32x4 *>(src + k[u] * 256 + (size_t)(lane % 32) * 8));
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        st_nt(reinterpret_cast<u32x2 *>(codes + k[u] * 256 + (size_t)(lane % 32) * 8),
              u32x2{x[u].x ^ x[u].z, x[u].y ^ x[u].w});
        if (lane % 32 == 0)
            scales[k[u]] = __uint_as_float(x[u].x & 0x3FFFFFFFu);
    }
}

// Every grid (at most one workgroup per KiB) must fit in 31 bits.
bool bad(const void *p, size_t bytes) {
    return !p || bytes == 0 || bytes % kTileBytes || (uintptr_t)p % 16 ||
           bytes / 1024 > 0x7FFFFFFFu;
}

}  // namespace

extern "C" {

ZPPC_API int zppc_read_stream(const void *src, size_t bytes, uint32_t *sink, hipStream_t stream) {
    if (bad(src, bytes) || !sink)
        return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(read_kernel, dim3((unsigned)(bytes / kTileBytes)), dim3(kReadThreads),
                       residency_lds(kReadResidency), stream,
                       static_cast<const u32x4 *>(src), sink);
    return (int)hipGetLastError();
}

ZPPC_API int zppc_write_stream(void *dst, size_t bytes, uint32_t pattern, hipStream_t stream) {
    if (bad(dst, bytes))
        return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(write_kernel, dim3((unsigned)(bytes / kTileBytes)), dim3(kWriteThreads),
                       residency_lds(kWriteResidency), stream, static_cast<u32x4 *>(dst),
                       pattern);
    return (int)hipGetLastError();
}

ZPPC_API int zppc_copy_stream(void *dst, const void *src, size_t bytes, hipStream_t stream) {
    if (bad(dst, bytes) || bad(src, bytes))
        return (int)hipErrorInvalidValue;
    const char *d = static_cast<const char *>(dst), *s = static_cast<const char *>(src);
    if (d < s + bytes && s < d + bytes)
        return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(copy_kernel, dim3((unsigned)(bytes / (kCopyThreads * 16))),
                       dim3(kCopyThreads), 0, stream, static_cast<u32x4 *>(dst),
                       static_cast<const u32x4 *>(src));
    return (int)hipGetLastError();
}

ZPPC_API int zppc_adam_pattern(float *p, float *m, float *v, const float *g, uint16_t *out,
                               size_t n, hipStream_t stream) {
    if (!p || !m || !v || !g || !out || n == 0 || n % 256 || n / 256 > 0x7FFFFFFFu ||
        (uintptr_t)p % 16 || (uintptr_t)m % 16 || (uintptr_t)v % 16 || (uintptr_t)g % 16 ||
        (uintptr_t)out % 8)
        return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(adam_pattern_kernel, dim3((unsigned)(n / 256)), dim3(64),
                       residency_lds(kAdamPatternResidency), stream, p, m, v, g, out);
    return (int)hipGetLastError();
}

ZPPC_API int zppc_gather_pattern(const int8_t *codes, const float *scales, uint16_t *out,
                                 size_t n, hipStream_t stream) {
    if (!codes || !scales || !out || n == 0 || n % 512 || n / 512 > 0x7FFFFFFFu ||
        (uintptr_t)codes % 8 || (uintptr_t)scales % 4 || (uintptr_t)out % 16)
        return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(gather_pattern_kernel, dim3((unsigned)(n / 512)), dim3(64), 0, stream,
                       codes, scales, out);
    return (int)hipGetLastError();
}

ZPPC_API int zppc_quant_pattern(const uint16_t *src, int8_t *codes, float *scales, size_t n,
                                hipStream_t stream) {
    if (!src || !codes || !scales || n == 0 || n % 4096 || n / 4096 > 0x7FFFFFFFu ||
        (uintptr_t)src % 16 || (uintptr_t)codes % 8 || (uintptr_t)scales % 4)
        return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(quant_pattern_kernel, dim3((unsigned)(n / 4096)), dim3(256), 0, stream,
                       src, codes, scales);
    return (int)hipGetLastError();
}

}  // extern "C"
