// The gradient that the qgZ receive delivers to the partition step: the sum,
// over the num_src int4 copies of the rank's partition (one from each sending
// rank, in rank order), of code * scale, accumulated with one fma per source
// from 0, then one multiply by the output scale (1/P for the data-parallel
// mean).  The dequantize-and-reduce kernel forms exactly this value and
// writes it; the kernels that take the receive into the optimizer step form
// it here, so that their results are bit for bit those of the separate calls.
#pragma once

#include "zpp_device.h"
#include "zpp_launch.h"
#include "zpp_quant.h"

namespace zpp {

// Workgroup numbering of the kernels that read the P copies from separate
// arrays (xcd_grouped in zpp_chunk.h): a 128-byte line of one source's
// scales serves 32 blocks, so 32 or more neighbouring tiles read it, and
// runs of this many consecutive workgroups per XCD let one L2 fetch it.  At
// the Llama-2-13B partition with 8 sources (median of 20 launches): the
// dequant-reduce 285 against 305 us, the receive step 990 against 1110, the
// single receive pass 1155 against 1235 (runs of 16 / 32 / 64 in between).
// The interleaved buffer keeps a block's scales of all sources in one
// 32-byte run, and the fused step has no shared lines: both were as fast or
// slower with grouping (the fused step 1079-1152 against 1046 us), so their
// kernels keep the plain numbering.
constexpr size_t kSeparateXcdRun = 128;

struct I4Grad {
    const uint8_t *codes[kMaxShards];  // packed int4, element 2i in the low nibble
    const float *scales[kMaxShards];   // one per block
    uint32_t num_src;
    BlockDiv block;
    float scale_out;
};

// The output scale, applied as its own rounded multiply: the separate calls
// store this product to memory before the update reads it, so it must not be
// contracted into an add of the update.
__device__ __forceinline__ float i4grad_scaled(float acc, float scale_out) {
#pragma clang fp contract(off)
    return acc * scale_out;
}

// The gradient of one element (tails and the any-alignment kernels).
__device__ __forceinline__ float i4grad_at(const I4Grad &s, size_t i) {
    float acc = 0.0f;
    for (uint32_t q = 0; q < s.num_src; ++q) {
        const uint32_t byte = s.codes[q][i / 2];
        const uint32_t nib = (i % 2 == 0) ? (byte & 0xFu) : (byte >> 4);
        acc = __builtin_fmaf(i4_code(nib, 0), s.scales[q][block_of(s.block, i)], acc);
    }
    return i4grad_scaled(acc, s.scale_out);
}

// The gradient of the four consecutive elements i .. i+3 (i a multiple of 4,
// all four in range): one 2-byte code load and one scale per source, the
// sources taken eight at a time with all eight loads in flight before their
// fma passes, which keep the source order.  Whole batches of eight carry no
// per-source test, so their loads issue back to back (the receive step at
// the Llama-2-13B partition: 945 against 974 us, the dequant-reduce 259
// against 270 us); a last partial batch tests each source.
constexpr int kI4Batch = 8;

template <bool FULL>
__device__ __forceinline__ void i4grad_batch(float (&acc)[4], const I4Grad &s, size_t i, size_t k,
                                             uint32_t q0) {
    uint32_t w[kI4Batch];
    float sc[kI4Batch];
#pragma unroll
    for (int j = 0; j < kI4Batch; ++j) {
        const uint32_t q = q0 + j;
        w[j] = 0u;
        sc[j] = 0.0f;
        if (FULL || q < s.num_src) {
            w[j] = ld_nt(reinterpret_cast<const uint16_t *>(s.codes[q] + i / 2));
            sc[j] = s.scales[q][k];
        }
    }
#pragma unroll
    for (int j = 0; j < kI4Batch; ++j) {
        if (FULL || q0 + j < s.num_src) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                acc[e] = __builtin_fmaf(i4_code(w[j], e), sc[j], acc[e]);
        }
    }
}

__device__ __forceinline__ f32x4 i4grad_load4(const I4Grad &s, size_t i) {
    float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    const size_t k = block_of(s.block, i);
    uint32_t q0 = 0;
    for (; q0 + kI4Batch <= s.num_src; q0 += kI4Batch)
        i4grad_batch<true>(acc, s, i, k, q0);
    if (q0 < s.num_src)
        i4grad_batch<false>(acc, s, i, k, q0);
    return f32x4{i4grad_scaled(acc[0], s.scale_out), i4grad_scaled(acc[1], s.scale_out),
                 i4grad_scaled(acc[2], s.scale_out), i4grad_scaled(acc[3], s.scale_out)};
}

// The same P int4 copies interleaved in one receive buffer: for each block k
// of B elements the sources' codes lie side by side (source
// q's B/2 bytes at (k P + q) B/2) and so do their scales (source q's at
// k P + q).  P = 1 is the plain layout of one copy.  A wave's 256-element
// tile then reads all its codes within one run of P x 128 bytes (blocks of
// 256 or fewer) instead of from P separate arrays.  The gradient is formed in
// the same order with the same operations as from separate arrays, so the
// results are the same bits.
struct I4GradIl {
    const uint8_t *codes;
    const float *scales;
    uint32_t num_src;
    BlockDiv block;
    float scale_out;
};

// Byte offset of element i's code of source q, element i in block k (element
// i is in the low nibble when i is even).
__device__ __forceinline__ size_t il_code_byte(const I4GradIl &s, size_t i, size_t k,
                                               uint32_t q) {
    const size_t B = s.block.block;
    return (k * s.num_src + q) * (B / 2) + ((i - k * B) >> 1);
}

__device__ __forceinline__ float i4grad_at(const I4GradIl &s, size_t i) {
    float acc = 0.0f;
    const size_t k = block_of(s.block, i);
    for (uint32_t q = 0; q < s.num_src; ++q) {
        const uint32_t byte = s.codes[il_code_byte(s, i, k, q)];
        const uint32_t nib = (i % 2 == 0) ? (byte & 0xFu) : (byte >> 4);
        acc = __builtin_fmaf(i4_code(nib, 0), s.scales[k * s.num_src + q], acc);
    }
    return i4grad_scaled(acc, s.scale_out);
}

// The gradient of the four consecutive elements i .. i+3 (i a multiple of 4,
// all four in range): the loads of the separate layout (a 2-byte code load
// and a scale per source, sources eight at a time, all loads in flight before
// the fma passes, which keep the source order), addressed in the interleaved
// buffer: a wave's loads of one source are 128 contiguous bytes, and those of
// all sources lie within one run of the buffer.
template <bool FULL>
__device__ __forceinline__ void i4grad_il_batch(float (&acc)[4], const I4GradIl &s,
                                                const uint8_t *base, size_t stride,
                                                const float *sbase, uint32_t q0) {
    uint32_t w[kI4Batch];
    float sc[kI4Batch];
#pragma unroll
    for (int b = 0; b < kI4Batch; ++b) {
        w[b] = 0u;
        sc[b] = 0.0f;
        if (FULL || q0 + b < s.num_src) {
            w[b] = ld_nt(reinterpret_cast<const uint16_t *>(base + (q0 + b) * stride));
            sc[b] = sbase[q0 + b];
        }
    }
#pragma unroll
    for (int b = 0; b < kI4Batch; ++b) {
        if (FULL || q0 + b < s.num_src) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                acc[e] = __builtin_fmaf(i4_code(w[b], e), sc[b], acc[e]);
        }
    }
}

__device__ __forceinline__ f32x4 i4grad_load4(const I4GradIl &s, size_t i) {
    float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    const size_t k = block_of(s.block, i);
    const uint8_t *base = s.codes + il_code_byte(s, i, k, 0);
    const size_t stride = s.block.block / 2;
    const float *sbase = s.scales + k * s.num_src;
    uint32_t q0 = 0;
    for (; q0 + kI4Batch <= s.num_src; q0 += kI4Batch)
        i4grad_il_batch<true>(acc, s, base, stride, sbase, q0);
    if (q0 < s.num_src)
        i4grad_il_batch<false>(acc, s, base, stride, sbase, q0);
    return f32x4{i4grad_scaled(acc[0], s.scale_out), i4grad_scaled(acc[1], s.scale_out),
                 i4grad_scaled(acc[2], s.scale_out), i4grad_scaled(acc[3], s.scale_out)};
}

// The fp32 gradient array the separate partition step reads, behind the same
// interface.
struct F32Grad {
    const float *g;
};

__device__ __forceinline__ float grad_at(const F32Grad &s, size_t i) { return s.g[i]; }
__device__ __forceinline__ f32x4 grad_load4(const F32Grad &s, size_t i) {
    return ld_nt(reinterpret_cast<const f32x4 *>(s.g + i));
}
__device__ __forceinline__ float grad_at(const I4Grad &s, size_t i) { return i4grad_at(s, i); }
__device__ __forceinline__ f32x4 grad_load4(const I4Grad &s, size_t i) {
    return i4grad_load4(s, i);
}
__device__ __forceinline__ float grad_at(const I4GradIl &s, size_t i) { return i4grad_at(s, i); }
__device__ __forceinline__ f32x4 grad_load4(const I4GradIl &s, size_t i) {
    return i4grad_load4(s, i);
}



}  // namespace zpp
