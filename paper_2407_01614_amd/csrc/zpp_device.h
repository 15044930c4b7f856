// Device-side helpers shared by the partition-path kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "zpp_launch.h"

namespace zpp {

#ifndef ZPP_THREADS
#define ZPP_THREADS 256
#endif
constexpr int kThreads = ZPP_THREADS;  // workgroup size: 4 wave64 by default
constexpr int kWave = 64;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));

// float -> bf16 bits, round to nearest even.  Adding 0x7FFF plus the lowest
// kept bit carries into the kept half exactly when the dropped half is above
// one half ulp, or exactly one half with an odd kept half.  NaN maps to the
// canonical 0x7FC0; +-Inf and overflow come out as +-Inf by the same carry.
__device__ __forceinline__ uint32_t bf16_rne_bits(float f) {
    const uint32_t u = __float_as_uint(f);
    const uint32_t r = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
    return ((u & 0x7FFFFFFFu) > 0x7F800000u) ? 0x7FC0u : r;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return bf16_rne_bits(lo) | (bf16_rne_bits(hi) << 16);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Block index of element i (BlockDiv, zpp_launch.h): the branch is uniform
// across a launch.
__device__ __forceinline__ size_t block_of(const BlockDiv &d, size_t i) {
    return d.magic ? (size_t)__umul64hi((unsigned long long)(i >> 6), d.magic) : i >> d.shift;
}

// Residency cap.  The streaming kernels that keep many HBM streams open at
// once (the optimizer step: four arrays read, four written) run faster with
// fewer workgroups resident per CU than the hardware would otherwise place:
// too many waves in flight oversubscribe the memory channels.  The optimizer
// step, the fused steps, the step with the qgZ receive and the gather use it.  A launch caps
// residency by reserving dynamic LDS that its kernel never touches: a CU then
// holds at most kLdsPerCU / residency_lds(k) = k such workgroups, and the
// dispatcher still hands out the one-shot grid as workgroups retire.
// residency_lds(0) = 0 leaves residency to the hardware.
constexpr size_t kLdsPerCU = 160 * 1024;  // LDS of one gfx950 CU
constexpr size_t residency_lds(int workgroups_per_cu) {
    return workgroups_per_cu <= 0 ? 0 : (kLdsPerCU / workgroups_per_cu) / 1024 * 1024;
}
static_assert(kLdsPerCU / residency_lds(11) == 11 && kLdsPerCU / residency_lds(12) == 12 &&
                  kLdsPerCU / residency_lds(13) == 13 && kLdsPerCU / residency_lds(14) == 14,
              "a reservation caps residency at exactly the requested count");

// Streaming accesses: every byte is touched once, so loads and stores are
// marked non-temporal.
#ifndef ZPP_NT_LOAD
#define ZPP_NT_LOAD 1
#endif
#ifndef ZPP_NT_STORE
#define ZPP_NT_STORE 1
#endif
template <typename T>
__device__ __forceinline__ T ld_nt(const T *p) {
    if constexpr (ZPP_NT_LOAD)
        return __builtin_nontemporal_load(p);
    else
        return *p;
}
template <typename T>
__device__ __forceinline__ void st_nt(T *p, T v) {
    if constexpr (ZPP_NT_STORE)
        __builtin_nontemporal_store(v, p);
    else
        *p = v;
}

}  // namespace zpp
