// C ABI of the partition path (declared in include/zpp.h): argument checks,
// stream ordering with events, and dispatch to the kernels.
#include <math.h>
#include <stdint.h>

#include "zpp.h"
#include "zpp_launch.h"

namespace {

thread_local int g_last_hip_error = 0;

zpp_status hip_fail(hipError_t e) {
    g_last_hip_error = (int)e;
    return ZPP_EHIP;
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Do [a, a + abytes) and [b, b + bbytes) share a byte?
bool overlaps(const void *a, size_t abytes, const void *b, size_t bbytes) {
    if (abytes == 0 || bbytes == 0)
        return false;
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + bbytes && b0 < a0 + abytes;
}

// Any multiple of 64 from 64 to 4096.
bool valid_block(uint32_t block) { return block >= 64 && block <= 4096 && block % 64 == 0; }

// Largest element count whose byte ranges (up to 16 B per element) cannot
// overflow a size_t.
constexpr size_t kMaxElems = SIZE_MAX / 16;

bool any_overlap(const void *const *ptrs, const size_t *bytes, int k) {
    for (int x = 0; x < k; ++x)
        for (int y = x + 1; y < k; ++y)
            if (overlaps(ptrs[x], bytes[x], ptrs[y], bytes[y]))
                return true;
    return false;
}

zpp_status check_hparams(const zpp_adam_hparams *hp) {
    if (!hp)
        return ZPP_EINVAL;
    if (!isfinite(hp->lr) || !isfinite(hp->beta1) || !isfinite(hp->beta2) ||
        !isfinite(hp->eps) || !isfinite(hp->weight_decay))
        return ZPP_EINVAL;
    if (hp->beta1 < 0.0f || hp->beta1 >= 1.0f || hp->beta2 < 0.0f || hp->beta2 >= 1.0f ||
        hp->eps < 0.0f || hp->step < 1)
        return ZPP_EINVAL;
    return ZPP_OK;
}

// Step-dependent constants, folded on the host in double and rounded once.
zpp::AdamConsts adam_consts(const zpp_adam_hparams &hp) {
    zpp::AdamConsts c;
    const double b1 = hp.beta1, b2 = hp.beta2, lr = hp.lr, wd = hp.weight_decay;
    const double bc1 = 1.0 - pow(b1, (double)hp.step);
    const double bc2 = 1.0 - pow(b2, (double)hp.step);
    c.lr_wd = (float)(lr * wd);
    c.wd = hp.weight_decay;
    c.beta1 = hp.beta1;
    c.one_minus_beta1 = (float)(1.0 - b1);
    c.beta2 = hp.beta2;
    c.one_minus_beta2 = (float)(1.0 - b2);
    c.step_size = (float)(lr / bc1);
    c.inv_bc2 = (float)(1.0 / bc2);
    c.eps = hp.eps;
    c.adamw = hp.adamw ? 1 : 0;
    return c;
}

zpp_status wait_on(hipStream_t stream, hipEvent_t ev) {
    if (!ev)
        return ZPP_OK;
    const hipError_t e = hipStreamWaitEvent(stream, ev, 0);
    return e == hipSuccess ? ZPP_OK : hip_fail(e);
}

// Bytes of codes and count of scales of an interleaved receive buffer of
// num_src int4 copies of n elements in blocks of `block`.
size_t il_code_bytes(size_t n, uint32_t block, uint32_t num_src) {
    return (n + block - 1) / block * num_src * (block / 2);
}
size_t il_scale_count(size_t n, uint32_t block, uint32_t num_src) {
    return (n + block - 1) / block * num_src;
}

zpp_status record(hipStream_t stream, hipEvent_t ev) {
    if (!ev)
        return ZPP_OK;
    const hipError_t e = hipEventRecord(ev, stream);
    return e == hipSuccess ? ZPP_OK : hip_fail(e);
}

}  // namespace

extern "C" {

ZPP_API zpp_status zpp_adam_partition_step(float *master, float *exp_avg, float *exp_avg_sq,
                                           const float *grad, uint16_t *primary_bf16, size_t n,
                                           const zpp_adam_hparams *hp, hipStream_t stream) {
    zpp_status st = check_hparams(hp);
    if (st != ZPP_OK)
        return st;
    if (n == 0)
        return ZPP_OK;
    if (n > kMaxElems)
        return ZPP_EINVAL;
    if (!master || !exp_avg || !exp_avg_sq || !grad || !primary_bf16)
        return ZPP_EINVAL;
    if (!aligned(master, 4) || !aligned(exp_avg, 4) || !aligned(exp_avg_sq, 4) ||
        !aligned(grad, 4) || !aligned(primary_bf16, 2))
        return ZPP_EALIGN;
    const void *ptrs[5] = {master, exp_avg, exp_avg_sq, grad, primary_bf16};
    const size_t bytes[5] = {4 * n, 4 * n, 4 * n, 4 * n, 2 * n};
    if (any_overlap(ptrs, bytes, 5))
        return ZPP_EOVERLAP;
    const bool vec = aligned(master, 16) && aligned(exp_avg, 16) && aligned(exp_avg_sq, 16) &&
                     aligned(grad, 16) && aligned(primary_bf16, 16);
    const hipError_t e = zpp::launch_adam(master, exp_avg, exp_avg_sq, grad, primary_bf16, n,
                                          adam_consts(*hp), vec, stream);
    return e == hipSuccess ? ZPP_OK : hip_fail(e);
}

ZPP_API zpp_status zpp_adam_step_refresh_quantize(float *master, float *exp_avg, float *exp_avg_sq,
                                                  const float *grad, uint16_t *primary_bf16,
                                                  uint16_t *secondary_bf16, int8_t *codes,
                                                  float *scales, size_t n, uint32_t block,
                                                  const zpp_adam_hparams *hp, hipStream_t stream,
                                                  hipEvent_t wait_before, hipEvent_t done_after) {
    zpp_status st = check_hparams(hp);
    if (st != ZPP_OK)
        return st;
    if (!valid_block(block) || n > kMaxElems)
        return ZPP_EINVAL;
    const size_t nblocks = (n + block - 1) / block;
    if (n) {
        if (!master || !exp_avg || !exp_avg_sq || !grad || !primary_bf16 || !codes || !scales)
            return ZPP_EINVAL;
        if (!aligned(master, 4) || !aligned(exp_avg, 4) || !aligned(exp_avg_sq, 4) ||
            !aligned(grad, 4) || !aligned(primary_bf16, 2) || !aligned(secondary_bf16, 2) ||
            !aligned(scales, 4))
            return ZPP_EALIGN;
        const void *ptrs[8] = {master, exp_avg, exp_avg_sq, grad, primary_bf16, codes, scales,
                               secondary_bf16};
        const size_t bytes[8] = {4 * n, 4 * n, 4 * n, 4 * n, 2 * n, n, 4 * nblocks,
                                 secondary_bf16 ? 2 * n : 0};
        if (any_overlap(ptrs, bytes, 8))
            return ZPP_EOVERLAP;
    }
    st = wait_on(stream, wait_before);
    if (st != ZPP_OK)
        return st;
    if (n) {
        const bool vec = aligned(master, 16) && aligned(exp_avg, 16) && aligned(exp_avg_sq, 16) &&
                         aligned(grad, 16) && aligned(primary_bf16, 8) &&
                         aligned(secondary_bf16, 8) && aligned(codes, 4);
        const hipError_t e =
            zpp::launch_fused(master, exp_avg, exp_avg_sq, grad, primary_bf16, secondary_bf16,
                              codes, scales, n, block, adam_consts(*hp), vec, stream);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    return record(stream, done_after);
}

ZPP_API zpp_status zpp_refresh_secondary(uint16_t *secondary_bf16, const uint16_t *src_bf16,
                                         size_t count, hipStream_t stream, hipEvent_t wait_before,
                                         hipEvent_t done_after) {
    if (count > kMaxElems)
        return ZPP_EINVAL;
    if (count) {
        if (!secondary_bf16 || !src_bf16)
            return ZPP_EINVAL;
        if (!aligned(secondary_bf16, 2) || !aligned(src_bf16, 2))
            return ZPP_EALIGN;
        if (overlaps(secondary_bf16, 2 * count, src_bf16, 2 * count))
            return ZPP_EOVERLAP;
    }
    zpp_status st = wait_on(stream, wait_before);
    if (st != ZPP_OK)
        return st;
    if (count) {
        const bool vec = aligned(secondary_bf16, 16) && aligned(src_bf16, 16);
        const hipError_t e = zpp::launch_refresh(secondary_bf16, src_bf16, count, vec, stream);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    return record(stream, done_after);
}

ZPP_API zpp_status zpp_quantize_blockwise_i8(const uint16_t *src_bf16, size_t n, uint32_t block,
                                             int8_t *codes, float *scales, hipStream_t stream,
                                             hipEvent_t wait_before, hipEvent_t done_after) {
    if (!valid_block(block) || n > kMaxElems)
        return ZPP_EINVAL;
    const size_t nblocks = (n + block - 1) / block;
    if (n) {
        if (!src_bf16 || !codes || !scales)
            return ZPP_EINVAL;
        if (!aligned(src_bf16, 2) || !aligned(scales, 4))
            return ZPP_EALIGN;
        if (overlaps(src_bf16, 2 * n, codes, n) || overlaps(src_bf16, 2 * n, scales, 4 * nblocks) ||
            overlaps(codes, n, scales, 4 * nblocks))
            return ZPP_EOVERLAP;
    }
    zpp_status st = wait_on(stream, wait_before);
    if (st != ZPP_OK)
        return st;
    if (n) {
        const bool vec = aligned(src_bf16, 16) && aligned(codes, 8);
        const hipError_t e = zpp::launch_quantize(src_bf16, n, block, codes, scales, vec, stream);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    return record(stream, done_after);
}

ZPP_API zpp_status zpp_refresh_quantize_i8(uint16_t *secondary_bf16, const uint16_t *src_bf16,
                                           size_t n, uint32_t block, int8_t *codes, float *scales,
                                           hipStream_t stream, hipEvent_t wait_before,
                                           hipEvent_t done_after) {
    if (!valid_block(block) || n > kMaxElems)
        return ZPP_EINVAL;
    const size_t nblocks = (n + block - 1) / block;
    if (n) {
        if (!secondary_bf16 || !src_bf16 || !codes || !scales)
            return ZPP_EINVAL;
        if (!aligned(secondary_bf16, 2) || !aligned(src_bf16, 2) || !aligned(scales, 4))
            return ZPP_EALIGN;
        const void *ptrs[4] = {secondary_bf16, src_bf16, codes, scales};
        const size_t bytes[4] = {2 * n, 2 * n, n, 4 * nblocks};
        if (any_overlap(ptrs, bytes, 4))
            return ZPP_EOVERLAP;
    }
    zpp_status st = wait_on(stream, wait_before);
    if (st != ZPP_OK)
        return st;
    if (n) {
        const bool vec = aligned(src_bf16, 16) && aligned(secondary_bf16, 16) && aligned(codes, 8);
        const hipError_t e =
            zpp::launch_quantize_copy(src_bf16, n, block, codes, scales, secondary_bf16, vec,
                                      stream);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    return record(stream, done_after);
}

ZPP_API zpp_status zpp_dequant_gather_layer(const int8_t *const *shard_codes,
                                            const float *const *shard_scales, uint32_t num_shards,
                                            size_t shard_elems, uint32_t block, size_t layer_elems,
                                            uint16_t *out_bf16, hipStream_t stream,
                                            const hipEvent_t *wait_events, uint32_t num_wait,
                                            hipEvent_t done_after) {
    if (num_shards == 0 || num_shards > ZPP_MAX_SHARDS || !valid_block(block))
        return ZPP_EINVAL;
    if (shard_elems == 0 || shard_elems > kMaxElems / num_shards)
        return ZPP_EINVAL;
    if (layer_elems > (size_t)num_shards * shard_elems)
        return ZPP_EINVAL;
    if (num_wait > ZPP_MAX_WAIT_EVENTS || (num_wait && !wait_events))
        return ZPP_EINVAL;
    for (uint32_t w = 0; w < num_wait; ++w)
        if (!wait_events[w])
            return ZPP_EINVAL;
    if (!shard_codes || !shard_scales)
        return ZPP_EINVAL;
    const size_t nblocks = (shard_elems + block - 1) / block;
    zpp::GatherShards shards = {};
    bool vec = (shard_elems % 16 == 0) && aligned(out_bf16, 16);
    for (uint32_t j = 0; j < num_shards; ++j) {
        if (!shard_codes[j] || !shard_scales[j])
            return ZPP_EINVAL;
        if (!aligned(shard_scales[j], 4))
            return ZPP_EALIGN;
        shards.codes[j] = shard_codes[j];
        shards.scales[j] = shard_scales[j];
        vec = vec && aligned(shard_codes[j], 16);
    }
    if (layer_elems) {
        if (!out_bf16)
            return ZPP_EINVAL;
        if (!aligned(out_bf16, 2))
            return ZPP_EALIGN;
        for (uint32_t j = 0; j < num_shards; ++j)
            if (overlaps(out_bf16, 2 * layer_elems, shard_codes[j], shard_elems) ||
                overlaps(out_bf16, 2 * layer_elems, shard_scales[j], 4 * nblocks))
                return ZPP_EOVERLAP;
    }
    for (uint32_t w = 0; w < num_wait; ++w) {
        const zpp_status st = wait_on(stream, wait_events[w]);
        if (st != ZPP_OK)
            return st;
    }
    if (layer_elems) {
        const hipError_t e = zpp::launch_gather(shards, num_shards, shard_elems, block,
                                                layer_elems, out_bf16, vec, stream);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    return record(stream, done_after);
}

ZPP_API zpp_status zpp_quantize_blockwise_i4(const float *src, size_t n, uint32_t block,
                                             uint8_t *codes, float *scales, hipStream_t stream,
                                             hipEvent_t wait_before, hipEvent_t done_after) {
    if (!valid_block(block) || n > kMaxElems)
        return ZPP_EINVAL;
    const size_t nblocks = (n + block - 1) / block;
    const size_t nbytes = (n + 1) / 2;
    if (n) {
        if (!src || !codes || !scales)
            return ZPP_EINVAL;
        if (!aligned(src, 4) || !aligned(scales, 4))
            return ZPP_EALIGN;
        const void *ptrs[3] = {src, codes, scales};
        const size_t bytes[3] = {4 * n, nbytes, 4 * nblocks};
        if (any_overlap(ptrs, bytes, 3))
            return ZPP_EOVERLAP;
    }
    zpp_status st = wait_on(stream, wait_before);
    if (st != ZPP_OK)
        return st;
    if (n) {
        const bool vec = aligned(src, 16) && aligned(codes, 2);
        const hipError_t e = zpp::launch_quantize_i4(src, n, block, codes, scales, vec, stream);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    return record(stream, done_after);
}

ZPP_API zpp_status zpp_dequant_reduce_i4(const uint8_t *const *src_codes,
                                         const float *const *src_scales, uint32_t num_src, size_t n,
                                         uint32_t block, float scale_out, float *out,
                                         hipStream_t stream, const hipEvent_t *wait_events,
                                         uint32_t num_wait, hipEvent_t done_after) {
    if (num_src == 0 || num_src > ZPP_MAX_SHARDS || !valid_block(block) || n > kMaxElems)
        return ZPP_EINVAL;
    if (!isfinite(scale_out))
        return ZPP_EINVAL;
    if (num_wait > ZPP_MAX_WAIT_EVENTS || (num_wait && !wait_events))
        return ZPP_EINVAL;
    for (uint32_t w = 0; w < num_wait; ++w)
        if (!wait_events[w])
            return ZPP_EINVAL;
    if (!src_codes || !src_scales)
        return ZPP_EINVAL;
    const size_t nblocks = (n + block - 1) / block;
    const size_t nbytes = (n + 1) / 2;
    bool vec = aligned(out, 16);
    for (uint32_t q = 0; q < num_src; ++q) {
        if (!src_codes[q] || !src_scales[q])
            return ZPP_EINVAL;
        if (!aligned(src_scales[q], 4))
            return ZPP_EALIGN;
        vec = vec && aligned(src_codes[q], 2);
    }
    if (n) {
        if (!out)
            return ZPP_EINVAL;
        if (!aligned(out, 4))
            return ZPP_EALIGN;
        for (uint32_t q = 0; q < num_src; ++q)
            if (overlaps(out, 4 * n, src_codes[q], nbytes) ||
                overlaps(out, 4 * n, src_scales[q], 4 * nblocks))
                return ZPP_EOVERLAP;
    }
    for (uint32_t w = 0; w < num_wait; ++w) {
        const zpp_status st = wait_on(stream, wait_events[w]);
        if (st != ZPP_OK)
            return st;
    }
    if (n) {
        const hipError_t e = zpp::launch_dequant_reduce_i4(src_codes, src_scales, num_src, n,
                                                           block, scale_out, out, vec, stream);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    return record(stream, done_after);
}

ZPP_API zpp_status zpp_qgz_receive_adam_step(float *master, float *exp_avg, float *exp_avg_sq,
                                             const uint8_t *const *src_codes,
                                             const float *const *src_scales, uint32_t num_src,
                                             uint32_t block, float scale_out,
                                             uint16_t *primary_bf16, size_t n,
                                             const zpp_adam_hparams *hp, hipStream_t stream,
                                             const hipEvent_t *wait_events, uint32_t num_wait,
                                             hipEvent_t done_after) {
    zpp_status st = check_hparams(hp);
    if (st != ZPP_OK)
        return st;
    if (num_src == 0 || num_src > ZPP_MAX_SHARDS || !valid_block(block) || n > kMaxElems)
        return ZPP_EINVAL;
    if (!isfinite(scale_out))
        return ZPP_EINVAL;
    if (num_wait > ZPP_MAX_WAIT_EVENTS || (num_wait && !wait_events))
        return ZPP_EINVAL;
    for (uint32_t w = 0; w < num_wait; ++w)
        if (!wait_events[w])
            return ZPP_EINVAL;
    if (!src_codes || !src_scales)
        return ZPP_EINVAL;
    const size_t nblocks = (n + block - 1) / block;
    const size_t nbytes = (n + 1) / 2;
    bool vec = aligned(master, 16) && aligned(exp_avg, 16) && aligned(exp_avg_sq, 16) &&
               aligned(primary_bf16, 8);
    for (uint32_t q = 0; q < num_src; ++q) {
        if (!src_codes[q] || !src_scales[q])
            return ZPP_EINVAL;
        if (!aligned(src_scales[q], 4))
            return ZPP_EALIGN;
        vec = vec && aligned(src_codes[q], 2);
    }
    if (n) {
        if (!master || !exp_avg || !exp_avg_sq || !primary_bf16)
            return ZPP_EINVAL;
        if (!aligned(master, 4) || !aligned(exp_avg, 4) || !aligned(exp_avg_sq, 4) ||
            !aligned(primary_bf16, 2))
            return ZPP_EALIGN;
        const void *outs[4] = {master, exp_avg, exp_avg_sq, primary_bf16};
        const size_t out_bytes[4] = {4 * n, 4 * n, 4 * n, 2 * n};
        if (any_overlap(outs, out_bytes, 4))
            return ZPP_EOVERLAP;
        for (int o = 0; o < 4; ++o)
            for (uint32_t q = 0; q < num_src; ++q)
                if (overlaps(outs[o], out_bytes[o], src_codes[q], nbytes) ||
                    overlaps(outs[o], out_bytes[o], src_scales[q], 4 * nblocks))
                    return ZPP_EOVERLAP;
    }
    for (uint32_t w = 0; w < num_wait; ++w) {
        st = wait_on(stream, wait_events[w]);
        if (st != ZPP_OK)
            return st;
    }
    if (n) {
        const hipError_t e = zpp::launch_receive_adam(master, exp_avg, exp_avg_sq, src_codes,
                                                      src_scales, num_src, block, scale_out,
                                                      primary_bf16, n, adam_consts(*hp), vec,
                                                      stream);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    return record(stream, done_after);
}

ZPP_API zpp_status zpp_qgz_receive_step_refresh_quantize(
    float *master, float *exp_avg, float *exp_avg_sq, const uint8_t *const *src_codes,
    const float *const *src_scales, uint32_t num_src, uint32_t grad_block, float scale_out,
    uint16_t *primary_bf16, uint16_t *secondary_bf16, int8_t *codes, float *scales, size_t n,
    uint32_t block, const zpp_adam_hparams *hp, hipStream_t stream, const hipEvent_t *wait_events,
    uint32_t num_wait, hipEvent_t done_after) {
    zpp_status st = check_hparams(hp);
    if (st != ZPP_OK)
        return st;
    if (num_src == 0 || num_src > ZPP_MAX_SHARDS || !valid_block(grad_block) ||
        !valid_block(block) || n > kMaxElems)
        return ZPP_EINVAL;
    if (!isfinite(scale_out))
        return ZPP_EINVAL;
    if (num_wait > ZPP_MAX_WAIT_EVENTS || (num_wait && !wait_events))
        return ZPP_EINVAL;
    for (uint32_t w = 0; w < num_wait; ++w)
        if (!wait_events[w])
            return ZPP_EINVAL;
    if (!src_codes || !src_scales)
        return ZPP_EINVAL;
    const size_t gblocks = (n + grad_block - 1) / grad_block;
    const size_t nblocks = (n + block - 1) / block;
    const size_t nbytes = (n + 1) / 2;
    bool vec = aligned(master, 16) && aligned(exp_avg, 16) && aligned(exp_avg_sq, 16) &&
               aligned(primary_bf16, 8) && aligned(secondary_bf16, 8) && aligned(codes, 4);
    for (uint32_t q = 0; q < num_src; ++q) {
        if (!src_codes[q] || !src_scales[q])
            return ZPP_EINVAL;
        if (!aligned(src_scales[q], 4))
            return ZPP_EALIGN;
        vec = vec && aligned(src_codes[q], 2);
    }
    if (n) {
        if (!master || !exp_avg || !exp_avg_sq || !primary_bf16 || !codes || !scales)
            return ZPP_EINVAL;
        if (!aligned(master, 4) || !aligned(exp_avg, 4) || !aligned(exp_avg_sq, 4) ||
            !aligned(primary_bf16, 2) || !aligned(secondary_bf16, 2) || !aligned(scales, 4))
            return ZPP_EALIGN;
        const void *outs[7] = {master, exp_avg, exp_avg_sq, primary_bf16, codes, scales,
                               secondary_bf16};
        const size_t out_bytes[7] = {4 * n, 4 * n, 4 * n, 2 * n, n, 4 * nblocks,
                                     secondary_bf16 ? 2 * n : 0};
        if (any_overlap(outs, out_bytes, 7))
            return ZPP_EOVERLAP;
        for (int o = 0; o < 7; ++o)
            for (uint32_t q = 0; q < num_src; ++q)
                if (overlaps(outs[o], out_bytes[o], src_codes[q], nbytes) ||
                    overlaps(outs[o], out_bytes[o], src_scales[q], 4 * gblocks))
                    return ZPP_EOVERLAP;
    }
    for (uint32_t w = 0; w < num_wait; ++w) {
        st = wait_on(stream, wait_events[w]);
        if (st != ZPP_OK)
            return st;
    }
    if (n) {
        const hipError_t e = zpp::launch_fused_receive(
            master, exp_avg, exp_avg_sq, src_codes, src_scales, num_src, grad_block, scale_out,
            primary_bf16, secondary_bf16, codes, scales, n, block, adam_consts(*hp), vec, stream);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    return record(stream, done_after);
}

ZPP_API zpp_status zpp_quantize_blockwise_i4_interleaved(const float *src, size_t n,
                                                         uint32_t block, uint32_t source,
                                                         uint32_t num_src, uint8_t *codes,
                                                         float *scales, hipStream_t stream,
                                                         hipEvent_t wait_before,
                                                         hipEvent_t done_after) {
    if (!valid_block(block) || num_src == 0 || num_src > ZPP_MAX_SHARDS || source >= num_src)
        return ZPP_EINVAL;
    if (n > kMaxElems / num_src)
        return ZPP_EINVAL;
    if (n) {
        if (!src || !codes || !scales)
            return ZPP_EINVAL;
        if (!aligned(src, 4) || !aligned(scales, 4))
            return ZPP_EALIGN;
        const void *ptrs[3] = {src, codes, scales};
        const size_t bytes[3] = {4 * n, il_code_bytes(n, block, num_src),
                                 4 * il_scale_count(n, block, num_src)};
        if (any_overlap(ptrs, bytes, 3))
            return ZPP_EOVERLAP;
    }
    zpp_status st = wait_on(stream, wait_before);
    if (st != ZPP_OK)
        return st;
    if (n) {
        const bool vec = aligned(src, 16) && aligned(codes, 2);
        const hipError_t e = zpp::launch_quantize_i4_il(src, n, block, source, num_src, codes,
                                                        scales, vec, stream);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    return record(stream, done_after);
}

ZPP_API zpp_status zpp_dequant_reduce_i4_interleaved(const uint8_t *codes, const float *scales,
                                                     uint32_t num_src, size_t n, uint32_t block,
                                                     float scale_out, float *out,
                                                     hipStream_t stream,
                                                     const hipEvent_t *wait_events,
                                                     uint32_t num_wait, hipEvent_t done_after) {
    if (num_src == 0 || num_src > ZPP_MAX_SHARDS || !valid_block(block))
        return ZPP_EINVAL;
    if (n > kMaxElems / num_src || !isfinite(scale_out))
        return ZPP_EINVAL;
    if (num_wait > ZPP_MAX_WAIT_EVENTS || (num_wait && !wait_events))
        return ZPP_EINVAL;
    for (uint32_t w = 0; w < num_wait; ++w)
        if (!wait_events[w])
            return ZPP_EINVAL;
    if (!codes || !scales)
        return ZPP_EINVAL;
    if (!aligned(scales, 4))
        return ZPP_EALIGN;
    if (n) {
        if (!out)
            return ZPP_EINVAL;
        if (!aligned(out, 4))
            return ZPP_EALIGN;
        if (overlaps(out, 4 * n, codes, il_code_bytes(n, block, num_src)) ||
            overlaps(out, 4 * n, scales, 4 * il_scale_count(n, block, num_src)))
            return ZPP_EOVERLAP;
    }
    for (uint32_t w = 0; w < num_wait; ++w) {
        const zpp_status st = wait_on(stream, wait_events[w]);
        if (st != ZPP_OK)
            return st;
    }
    if (n) {
        const bool vec = aligned(out, 16) && aligned(codes, 2);
        const hipError_t e = zpp::launch_dequant_reduce_i4_il(codes, scales, num_src, n, block,
                                                              scale_out, out, vec, stream);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    return record(stream, done_after);
}

ZPP_API zpp_status zpp_qgz_receive_adam_step_interleaved(
    float *master, float *exp_avg, float *exp_avg_sq, const uint8_t *codes, const float *scales,
    uint32_t num_src, uint32_t block, float scale_out, uint16_t *primary_bf16, size_t n,
    const zpp_adam_hparams *hp, hipStream_t stream, const hipEvent_t *wait_events,
    uint32_t num_wait, hipEvent_t done_after) {
    zpp_status st = check_hparams(hp);
    if (st != ZPP_OK)
        return st;
    if (num_src == 0 || num_src > ZPP_MAX_SHARDS || !valid_block(block))
        return ZPP_EINVAL;
    if (n > kMaxElems / num_src || !isfinite(scale_out))
        return ZPP_EINVAL;
    if (num_wait > ZPP_MAX_WAIT_EVENTS || (num_wait && !wait_events))
        return ZPP_EINVAL;
    for (uint32_t w = 0; w < num_wait; ++w)
        if (!wait_events[w])
            return ZPP_EINVAL;
    if (!codes || !scales)
        return ZPP_EINVAL;
    if (!aligned(scales, 4))
        return ZPP_EALIGN;
    if (n) {
        if (!master || !exp_avg || !exp_avg_sq || !primary_bf16)
            return ZPP_EINVAL;
        if (!aligned(master, 4) || !aligned(exp_avg, 4) || !aligned(exp_avg_sq, 4) ||
            !aligned(primary_bf16, 2))
            return ZPP_EALIGN;
        const void *ptrs[6] = {master, exp_avg, exp_avg_sq, primary_bf16, codes, scales};
        const size_t bytes[6] = {4 * n, 4 * n, 4 * n, 2 * n, il_code_bytes(n, block, num_src),
                                 4 * il_scale_count(n, block, num_src)};
        // the two inputs may share bytes with each other, not with an output
        for (int o = 0; o < 4; ++o)
            for (int x = o + 1; x < 6; ++x)
                if (overlaps(ptrs[o], bytes[o], ptrs[x], bytes[x]))
                    return ZPP_EOVERLAP;
    }
    for (uint32_t w = 0; w < num_wait; ++w) {
        st = wait_on(stream, wait_events[w]);
        if (st != ZPP_OK)
            return st;
    }
    if (n) {
        const bool vec = aligned(master, 16) && aligned(exp_avg, 16) && aligned(exp_avg_sq, 16) &&
                         aligned(primary_bf16, 8) && aligned(codes, 2);
        const hipError_t e = zpp::launch_receive_adam_il(master, exp_avg, exp_avg_sq, codes,
                                                         scales, num_src, block, scale_out,
                                                         primary_bf16, n, adam_consts(*hp), vec,
                                                         stream);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    return record(stream, done_after);
}

ZPP_API zpp_status zpp_qgz_receive_step_refresh_quantize_interleaved(
    float *master, float *exp_avg, float *exp_avg_sq, const uint8_t *src_codes,
    const float *src_scales, uint32_t num_src, uint32_t grad_block, float scale_out,
    uint16_t *primary_bf16, uint16_t *secondary_bf16, int8_t *codes, float *scales, size_t n,
    uint32_t block, const zpp_adam_hparams *hp, hipStream_t stream, const hipEvent_t *wait_events,
    uint32_t num_wait, hipEvent_t done_after) {
    zpp_status st = check_hparams(hp);
    if (st != ZPP_OK)
        return st;
    if (num_src == 0 || num_src > ZPP_MAX_SHARDS || !valid_block(grad_block) ||
        !valid_block(block))
        return ZPP_EINVAL;
    if (n > kMaxElems / num_src || !isfinite(scale_out))
        return ZPP_EINVAL;
    if (num_wait > ZPP_MAX_WAIT_EVENTS || (num_wait && !wait_events))
        return ZPP_EINVAL;
    for (uint32_t w = 0; w < num_wait; ++w)
        if (!wait_events[w])
            return ZPP_EINVAL;
    if (!src_codes || !src_scales)
        return ZPP_EINVAL;
    if (!aligned(src_scales, 4))
        return ZPP_EALIGN;
    if (n) {
        if (!master || !exp_avg || !exp_avg_sq || !primary_bf16 || !codes || !scales)
            return ZPP_EINVAL;
        if (!aligned(master, 4) || !aligned(exp_avg, 4) || !aligned(exp_avg_sq, 4) ||
            !aligned(primary_bf16, 2) || !aligned(secondary_bf16, 2) || !aligned(scales, 4))
            return ZPP_EALIGN;
        const size_t nblocks = (n + block - 1) / block;
        const void *ptrs[9] = {master, exp_avg, exp_avg_sq, primary_bf16, codes, scales,
                               secondary_bf16, src_codes, src_scales};
        const size_t bytes[9] = {4 * n, 4 * n, 4 * n, 2 * n, n, 4 * nblocks,
                                 secondary_bf16 ? 2 * n : 0,
                                 il_code_bytes(n, grad_block, num_src),
                                 4 * il_scale_count(n, grad_block, num_src)};
        // the two inputs may share bytes with each other, not with an output
        for (int o = 0; o < 7; ++o)
            for (int x = o + 1; x < 9; ++x)
                if (overlaps(ptrs[o], bytes[o], ptrs[x], bytes[x]))
                    return ZPP_EOVERLAP;
    }
    for (uint32_t w = 0; w < num_wait; ++w) {
        st = wait_on(stream, wait_events[w]);
        if (st != ZPP_OK)
            return st;
    }
    if (n) {
        const bool vec = aligned(master, 16) && aligned(exp_avg, 16) && aligned(exp_avg_sq, 16) &&
                         aligned(primary_bf16, 8) && aligned(secondary_bf16, 8) &&
                         aligned(codes, 4) && aligned(src_codes, 2);
        const hipError_t e = zpp::launch_fused_receive_il(
            master, exp_avg, exp_avg_sq, src_codes, src_scales, num_src, grad_block, scale_out,
            primary_bf16, secondary_bf16, codes, scales, n, block, adam_consts(*hp), vec, stream);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    return record(stream, done_after);
}

ZPP_API const char *zpp_status_string(int status) {
    switch (status) {
    case ZPP_OK: return "ok";
    case ZPP_EINVAL: return "invalid argument";
    case ZPP_EALIGN: return "misaligned pointer";
    case ZPP_EOVERLAP: return "overlapping buffers";
    case ZPP_EHIP: return "HIP runtime error";
    }
    return "unknown status";
}

ZPP_API int zpp_last_hip_error(void) { return g_last_hip_error; }

}  // extern "C"
