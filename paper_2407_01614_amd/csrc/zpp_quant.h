// Device-side pieces of the blockwise quantization shared by the kernels: the
// int8 decisions of the quantize kernel and the fused optimizer-step
// epilogue, and the int4 decode of the qgZ receive.
#pragma once

#include "zpp_device.h"

namespace zpp {

constexpr uint32_t kScaleNaNBits = 0x7FC00000u;

struct BlockQuant {
    float scale;  // value stored for the block
    float pre;    // power-of-two pre-scale of tiny blocks (exact)
    float inv;    // 127 / (absmax * pre)
    bool zero;    // codes are all 0 (zero or non-finite block)
    bool tiny;    // absmax < 2^-100: values are pre-scaled by 2^64 first
};

// Decisions of one block from the max of its |x| bit patterns.
__device__ __forceinline__ BlockQuant block_params(uint32_t absbits) {
    BlockQuant q;
    const float a = __uint_as_float(absbits << 16);
    q.tiny = a < 0x1p-100f;
    q.pre = q.tiny ? 0x1p64f : 1.0f;
    q.inv = 127.0f / (a * q.pre);
    if (absbits >= 0x7F80u) {
        q.scale = __uint_as_float(kScaleNaNBits);
        q.zero = true;
    } else if (absbits == 0u) {
        q.scale = 0.0f;
        q.zero = true;
    } else {
        q.scale = a / 127.0f;
        q.zero = false;
    }
    return q;
}

// Scalar code of one value (used by the any-alignment kernel).  No clamp is
// needed: |x| <= a and inv <= (127/a)(1 + 2^-24), so |x * inv| rounds to at
// most 127 (1 + 2^-24)^2 < 127.5 and rint stays within [-127, 127].
__device__ __forceinline__ int quant_one(float x, const BlockQuant &q) {
    const float y = __builtin_rintf((x * q.pre) * q.inv);
    return q.zero ? 0 : (int)y;
}

// Adding 1.5 * 2^23 to y (|y| < 2^22) leaves rint(y) in the low bits of the
// sum's bit pattern: the sum's ulp is 1 and the addition rounds to nearest
// even, exactly as rint does; the low byte is then the two's-complement code.
// The product and the addition must stay two roundings (no fma).
constexpr float kRoundMagic = 12582912.0f;

__device__ __forceinline__ uint32_t code_bits(float y) {
#pragma clang fp contract(off)
    return __float_as_uint(y + kRoundMagic);
}

__device__ __forceinline__ uint32_t pack_low_bytes(uint32_t b0, uint32_t b1, uint32_t b2,
                                                   uint32_t b3) {
    const uint32_t w01 = __builtin_amdgcn_perm(b1, b0, 0x0c0c0400u);
    const uint32_t w23 = __builtin_amdgcn_perm(b3, b2, 0x0c0c0400u);
    return __builtin_amdgcn_perm(w23, w01, 0x05040100u);
}

// 4 bf16 (two words) -> 4 int8 codes packed little-endian.
__device__ __forceinline__ uint32_t quant_word(uint32_t w0, uint32_t w1, const BlockQuant &q) {
#pragma clang fp contract(off)
    float x0 = bf16_lo(w0), x1 = bf16_hi(w0), x2 = bf16_lo(w1), x3 = bf16_hi(w1);
    if (q.tiny) {
        x0 *= q.pre;
        x1 *= q.pre;
        x2 *= q.pre;
        x3 *= q.pre;
    }
    const uint32_t packed = pack_low_bytes(code_bits(x0 * q.inv), code_bits(x1 * q.inv),
                                           code_bits(x2 * q.inv), code_bits(x3 * q.inv));
    return q.zero ? 0u : packed;
}

// max of the |x| bit patterns of the two bf16 in a word
__device__ __forceinline__ u16x2 absbits2(uint32_t w) {
    return __builtin_bit_cast(u16x2, w & 0x7FFF7FFFu);
}

// int4 code e (4-bit two's complement, nibble e of w, e = 0 the lowest) as a
// float; shared by the qgZ dequantize-and-reduce and the receive fused into
// the partition step, which must form the same gradient.
__device__ __forceinline__ float i4_code(uint32_t w, int e) {
    return (float)((int32_t)(w << (28 - 4 * e)) >> 28);
}

}  // namespace zpp
