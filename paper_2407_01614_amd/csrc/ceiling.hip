// Plain HBM streams (include/zpp_ceiling.h): the read-only, write-only and
// copy ceilings of this GPU, which the partition-path kernels are measured
// against.  Built into its own library; not part of the partition path.
#include "zpp_ceiling.h"
#include "zpp_device.h"

namespace {

using zpp::ld_nt;
using zpp::residency_lds;
using zpp::st_nt;
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

}  // extern "C"
