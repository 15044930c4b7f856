// Internal launchers behind the C ABI.  Arguments are already validated; each
// launcher only enqueues its kernel on `stream` and returns the launch error.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace zpp {

// Index of the block of `block` elements that holds element i, for any block
// B = 64 b with b = 1 .. 64: a shift when B is a power of two, otherwise
// floor((i >> 6) / b) as the high half of the 64 x 64-bit product of i >> 6
// and magic = ceil(2^64 / b).  That quotient is exact for every i < 2^64:
// with x = i >> 6 = q b + r (x < 2^58, r < b) the product is
// 2^64 (q + r / b) + x e / b with e = magic b - 2^64 < b <= 64, and
// x e < 2^64 keeps r / b + x e / (b 2^64) below 1.
struct BlockDiv {
    uint64_t magic;  // 0 when the block is a power of two
    uint32_t shift;  // log2(block) when it is
    uint32_t block;
};

inline BlockDiv make_block_div(uint32_t block) {
    BlockDiv d;
    d.block = block;
    if ((block & (block - 1)) == 0) {
        d.magic = 0;
        d.shift = (uint32_t)__builtin_ctz(block);
    } else {
        // block / 64 is not a power of two, so 2^64 / b is not an integer
        // and its ceiling is floor((2^64 - 1) / b) + 1
        d.magic = UINT64_MAX / (block / 64) + 1;
        d.shift = 0;
    }
    return d;
}

struct AdamConsts {
    float lr_wd;      // lr * weight_decay (decoupled decay)
    float wd;         // weight_decay (L2 form)
    float beta1, one_minus_beta1;
    float beta2, one_minus_beta2;
    float step_size;  // lr / (1 - beta1^t)
    float inv_bc2;    // 1 / (1 - beta2^t)
    float eps;
    int adamw;
};

hipError_t launch_adam(float *p, float *m, float *v, const float *g, uint16_t *out, size_t n,
                       const AdamConsts &c, bool vector_path, hipStream_t stream);

hipError_t launch_refresh(uint16_t *dst, const uint16_t *src, size_t count, bool vector_path,
                          hipStream_t stream);

hipError_t launch_quantize(const uint16_t *src, size_t n, uint32_t block, int8_t *codes,
                           float *scales, bool vector_path, hipStream_t stream);

// The quantization that also stores the bf16 it reads to `copy`: the
// secondary refresh and its quantization in one pass.
hipError_t launch_quantize_copy(const uint16_t *src, size_t n, uint32_t block, int8_t *codes,
                                float *scales, uint16_t *copy, bool vector_path,
                                hipStream_t stream);

// Adam step + bf16 primary + optional bf16 secondary + int8 codes/scales of
// the primary, in one pass (vector_path) or as the three scalar kernels.
hipError_t launch_fused(float *p, float *m, float *v, const float *g, uint16_t *primary,
                        uint16_t *secondary, int8_t *codes, float *scales, size_t n,
                        uint32_t block, const AdamConsts &c, bool vector_path,
                        hipStream_t stream);

constexpr uint32_t kMaxShards = 64;

struct GatherShards {
    const int8_t *codes[kMaxShards];
    const float *scales[kMaxShards];
};

hipError_t launch_gather(const GatherShards &shards, uint32_t num_shards, size_t shard_elems,
                         uint32_t block, size_t layer_elems, uint16_t *out, bool vector_path,
                         hipStream_t stream);

// qgZ: int4 quantization of fp32 gradients, and the dequantize-and-reduce
// of num_src quantized copies of one partition.
hipError_t launch_quantize_i4(const float *src, size_t n, uint32_t block, uint8_t *codes,
                              float *scales, bool vector_path, hipStream_t stream);

hipError_t launch_dequant_reduce_i4(const uint8_t *const *src_codes,
                                    const float *const *src_scales, uint32_t num_src, size_t n,
                                    uint32_t block, float scale_out, float *out,
                                    bool vector_path, hipStream_t stream);

struct I4Grad;
struct I4GradIl;

// The int4 gradient sources of the qgZ receive, gathered for a kernel argument.
I4Grad make_i4grad(const uint8_t *const *src_codes, const float *const *src_scales,
                   uint32_t num_src, uint32_t block, float scale_out);

// The fused pass with the qgZ receive: the gradient comes from num_src int4
// copies (blocks of grad_block) instead of an fp32 array, then as
// launch_fused (vector_path) or the receive step, refresh and quantization as
// scalar kernels.
hipError_t launch_fused_receive(float *p, float *m, float *v, const uint8_t *const *src_codes,
                                const float *const *src_scales, uint32_t num_src,
                                uint32_t grad_block, float scale_out, uint16_t *primary,
                                uint16_t *secondary, int8_t *codes, float *scales, size_t n,
                                uint32_t block, const AdamConsts &c, bool vector_path,
                                hipStream_t stream);

// The int4 copies interleaved in one receive buffer (layout in
// zpp_i4grad.h), gathered for a kernel argument.
I4GradIl make_i4grad_il(const uint8_t *codes, const float *scales, uint32_t num_src,
                        uint32_t block, float scale_out);

// The receive step and the fused pass from the interleaved receive buffer.
hipError_t launch_receive_adam_il(float *p, float *m, float *v, const uint8_t *codes,
                                  const float *scales, uint32_t num_src, uint32_t block,
                                  float scale_out, uint16_t *out, size_t n, const AdamConsts &c,
                                  bool vector_path, hipStream_t stream);
hipError_t launch_fused_receive_il(float *p, float *m, float *v, const uint8_t *src_codes,
                                   const float *src_scales, uint32_t num_src, uint32_t grad_block,
                                   float scale_out, uint16_t *primary, uint16_t *secondary,
                                   int8_t *codes, float *scales, size_t n, uint32_t block,
                                   const AdamConsts &c, bool vector_path, hipStream_t stream);

// The dequant-reduce from the interleaved receive buffer.
hipError_t launch_dequant_reduce_i4_il(const uint8_t *codes, const float *scales, uint32_t num_src,
                                       size_t n, uint32_t block, float scale_out, float *out,
                                       bool vector_path, hipStream_t stream);

// int4 quantization of one source's n values into its slots of an
// interleaved receive buffer of num_src sources (num_src = 1: the plain
// layout of launch_quantize_i4).
hipError_t launch_quantize_i4_il(const float *src, size_t n, uint32_t block, uint32_t source,
                                 uint32_t num_src, uint8_t *codes, float *scales,
                                 bool vector_path, hipStream_t stream);

// The qgZ receive fused into the partition step: the gradient of every
// element is the dequantize-and-reduce of the num_src int4 sources (times
// scale_out), fed straight into the Adam update of p, m, v and the bf16 out.
hipError_t launch_receive_adam(float *p, float *m, float *v, const uint8_t *const *src_codes,
                               const float *const *src_scales, uint32_t num_src, uint32_t block,
                               float scale_out, uint16_t *out, size_t n, const AdamConsts &c,
                               bool vector_path, hipStream_t stream);

}  // namespace zpp
