// Internal launchers behind the C ABI.  Arguments are already validated; each
// launcher only enqueues its kernel on `stream` and returns the launch error.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace zpp {

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
