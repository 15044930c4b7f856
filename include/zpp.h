/*
 * zpp.h - C ABI of the one-rank partition path of the modified ZeRO++ hpZ
 * scheme (arXiv 2407.01614), built for AMD Instinct MI355X (gfx950).
 *
 * The path, per rank and iteration:
 *   1. zpp_adam_partition_step   optimizer.step() on the rank's partition
 *                                (Algorithm 1, last statement of the loop):
 *                                fp32 master/moments in place, bf16 primary out.
 *   2. zpp_refresh_secondary     fill the hpZ secondary copy (Algorithm 1,
 *                                forward loop: allocate |L|/P' and copy the
 *                                local rank's weights asynchronously; Eq. 1).
 *   3. zpp_quantize_blockwise_i8 qwZ: quantize weights before they are
 *                                gathered (Background section).
 *   4. zpp_dequant_gather_layer  backward AllGather(L, P') over the
 *                                node-local secondary shards, dequantizing
 *                                on the way (Algorithm 1, backward branch of
 *                                PrefetchAllGather).
 * The ordering fix of the paper (the gather of a secondary copy may only
 * start once the copy that fills it has finished; Algorithm 1, the wait in
 * PrefetchAllGather, and the synchronization operator of the Algorithm
 * section) is expressed with HIP events: steps 2 and 3 record `done_after`,
 * step 4 makes its stream wait on `wait_events` on the device, without
 * blocking the host.
 *
 * Conventions common to every call:
 *   - All array pointers are DEVICE pointers (HBM of the current device),
 *     owned by the caller.  The library never allocates, frees or blocks the
 *     host; every call only enqueues work on `stream` and returns.
 *   - bf16 values are passed as their uint16_t bit patterns.
 *   - `stream == NULL` is the null stream.  Events are created by the caller;
 *     a NULL event means "no event".
 *   - Validation is synchronous and happens before anything is enqueued; on
 *     any validation error nothing is enqueued (no kernel, no event).
 *   - A size of 0 is a valid no-op that still honours the wait events and
 *     records `done_after`, so a waiter never hangs.
 *   - If the HIP runtime rejects a launch, the call returns ZPP_EHIP and
 *     zpp_last_hip_error() gives the hipError_t (per host thread).  Work
 *     enqueued before the failing HIP call stays enqueued.  Faults inside a
 *     kernel surface at the caller's next synchronization, as for any HIP
 *     stream operation.
 */
#ifndef ZPP_H
#define ZPP_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Symbols of this header are the only ones the library exports. */
#define ZPP_API __attribute__((visibility("default")))

typedef enum {
    ZPP_OK = 0,
    ZPP_EINVAL = 1,   /* bad argument: NULL pointer with a non-zero size, bad size or block */
    ZPP_EALIGN = 2,   /* a pointer is not aligned to its element type */
    ZPP_EOVERLAP = 3, /* an output range overlaps another argument's range */
    ZPP_EHIP = 4      /* the HIP runtime returned an error; see zpp_last_hip_error() */
} zpp_status;

/* Hyperparameters of one Adam step, read at call time (the struct may be
 * reused or freed as soon as the call returns).  The paper does not name the
 * optimizer: this is Adam (Kingma & Ba) with decoupled weight decay
 * (Loshchilov & Hutter) when adamw != 0, or with the L2 term wd * p added to
 * the gradient when adamw == 0.  Bias correction uses the 1-based step t.
 * Requirements: all floats finite, 0 <= beta1, beta2 < 1, eps >= 0,
 * step >= 1; otherwise ZPP_EINVAL. */
typedef struct {
    float lr;
    float beta1;
    float beta2;
    float eps;
    float weight_decay;
    int32_t adamw;
    int64_t step;
} zpp_adam_hparams;

/* Partition step: optimizer.step() on one rank's ZeRO partition (Algorithm 1;
 * the optimizer states are sharded over the P ranks, Background section).
 * For every i < n, in fp32:
 *     adamw ? p -= lr*wd*p : g += wd*p
 *     m = beta1*m + (1-beta1)*g ;  v = beta2*v + (1-beta2)*g*g
 *     p -= (lr / (1-beta1^t)) * m / (sqrt(v / (1-beta2^t)) + eps)
 *     primary_bf16[i] = bf16(p)   (round to nearest even; NaN -> 0x7FC0)
 * master, exp_avg, exp_avg_sq: float[n], updated in place (three distinct
 *   arrays).  grad: float[n], read only.  primary_bf16: uint16_t[n] out, the
 *   rank's slice of the layer the forward AllGather(L, P) assembles.
 * None of the five ranges may overlap another (ZPP_EOVERLAP).  Pointers must
 * be aligned to their element size (ZPP_EALIGN); 16-byte alignment of all
 * five selects the vector kernel.  hp must be non-NULL. */
ZPP_API zpp_status zpp_adam_partition_step(float *master, float *exp_avg, float *exp_avg_sq,
                                           const float *grad, uint16_t *primary_bf16, size_t n,
                                           const zpp_adam_hparams *hp, hipStream_t stream);

/* Secondary refresh: the copy into the hpZ secondary partition
 * L_{i,second} of |L_i|/P' elements (Eq. 1) of the weights that belong to
 * the local rank, taken out of the full parameter tensor (Algorithm 1,
 * forward loop).  secondary_bf16[i] = src_bf16[i] bit for bit, i < count.
 * Order on `stream`: wait for `wait_before` (e.g. the previous gather that
 * still reads this buffer), copy, then record `done_after`, which the gather
 * of this copy must wait on (the paper's fix).
 * The two ranges must not overlap (ZPP_EOVERLAP); pointers 2-byte aligned
 * (ZPP_EALIGN). */
ZPP_API zpp_status zpp_refresh_secondary(uint16_t *secondary_bf16, const uint16_t *src_bf16,
                                         size_t count, hipStream_t stream, hipEvent_t wait_before,
                                         hipEvent_t done_after);

/* qwZ quantization of a weight shard before it is gathered (Background
 * section: weights are quantized before AllGather).  Symmetric absmax int8
 * over consecutive blocks of `block` elements (the last block may be
 * shorter), one fp32 scale per block, all decisions in fp32:
 *   block holds an Inf or NaN  -> scale = NaN (0x7FC00000), codes 0
 *   a = max |x| == 0           -> scale = 0, codes 0
 *   otherwise                  -> scale = a / 127, inv = 127 / a (both
 *       correctly rounded), code = rint(x * inv) (ties to even) in
 *       [-127, 127]; when a < 2^-100, x and a are first multiplied by 2^64.
 * src_bf16: uint16_t[n].  codes: int8_t[n] out.  scales: float[ceil(n/block)]
 * out.  block: a multiple of 64 in [64, 4096], else ZPP_EINVAL.
 * Order on `stream`: wait `wait_before`, quantize, record `done_after`.
 * No two of the three ranges may overlap (ZPP_EOVERLAP).  Alignment: src 2,
 * scales 4 (ZPP_EALIGN); src 16 and codes 8 bytes select the vector kernel. */
ZPP_API zpp_status zpp_quantize_blockwise_i8(const uint16_t *src_bf16, size_t n, uint32_t block,
                                             int8_t *codes, float *scales, hipStream_t stream,
                                             hipEvent_t wait_before, hipEvent_t done_after);

/* The secondary refresh and its qwZ quantization in one pass: the same
 * results, bit for bit, as zpp_refresh_secondary(secondary_bf16, src_bf16, n)
 * followed by zpp_quantize_blockwise_i8(secondary_bf16, n, block, codes,
 * scales) (Algorithm 1: the D2D copy of the local rank's weights into
 * L_{i,second}; Background: qwZ quantizes them before the gather), reading
 * src_bf16 once: 5.016 instead of 7.016 bytes of HBM traffic per element for
 * block 256.  secondary_bf16: uint16_t[n] out; src_bf16: uint16_t[n];
 * codes: int8_t[n] out; scales: float[ceil(n/block)] out; block: a multiple
 * of 64 in [64, 4096], else ZPP_EINVAL.  Order on `stream`: wait
 * `wait_before` (e.g. the last gather that read the codes), copy and
 * quantize, record `done_after`, which the gather of these codes must wait
 * on (the paper's fix).  No two of the four ranges may overlap
 * (ZPP_EOVERLAP).  Alignment: secondary and src 2 bytes, scales 4
 * (ZPP_EALIGN); src and secondary 16 and codes 8 bytes select the vector
 * kernel. */
ZPP_API zpp_status zpp_refresh_quantize_i8(uint16_t *secondary_bf16, const uint16_t *src_bf16,
                                           size_t n, uint32_t block, int8_t *codes, float *scales,
                                           hipStream_t stream, hipEvent_t wait_before,
                                           hipEvent_t done_after);

/* Fused partition step: zpp_adam_partition_step, then the secondary refresh
 * and the qwZ quantization of the new bf16 weights, in one pass over HBM
 * (optimizer.step() of Algorithm 1, the secondary copy of the forward loop
 * and the quantization that precedes the gather, applied to the same
 * weights).  Results are bit for bit those of the three separate calls
 * (zpp_adam_partition_step into primary_bf16, zpp_refresh_secondary from it,
 * zpp_quantize_blockwise_i8 of it), at 33.016 instead of 37.016 bytes of HBM
 * traffic per element for block 256.  Blocks of 64 to 512 take one pass;
 * any other block takes two kernels in stream order, the step with its
 * copies and then the quantization of primary_bf16 (2 more bytes read per
 * element, which measured faster than one pass for such blocks).
 * master, exp_avg, exp_avg_sq: float[n] in place; grad: float[n];
 * primary_bf16: uint16_t[n] out; secondary_bf16: uint16_t[n] out, or NULL to
 * keep no bf16 secondary copy; codes: int8_t[n] out; scales:
 * float[ceil(n/block)] out.  block: a multiple of 64 in [64, 4096].  hp as for
 * zpp_adam_partition_step.
 * Order on `stream`: wait `wait_before`, run, record `done_after` (the event
 * a gather of the codes waits on).
 * No two ranges may overlap (ZPP_EOVERLAP).  Alignment: floats 4, bf16 2
 * bytes (ZPP_EALIGN); 16-byte fp32 arrays, 8-byte bf16 arrays and 4-byte
 * codes select the single-pass kernel (for the two-kernel blocks, the
 * quantization's vector kernel further needs a 16-byte primary_bf16 and
 * 8-byte codes), otherwise the three scalar kernels run one after
 * another. */
ZPP_API zpp_status zpp_adam_step_refresh_quantize(float *master, float *exp_avg, float *exp_avg_sq,
                                                  const float *grad, uint16_t *primary_bf16,
                                                  uint16_t *secondary_bf16, int8_t *codes,
                                                  float *scales, size_t n, uint32_t block,
                                                  const zpp_adam_hparams *hp, hipStream_t stream,
                                                  hipEvent_t wait_before, hipEvent_t done_after);

/* Maximum number of shards one gather accepts (the secondary group P'). */
#define ZPP_MAX_SHARDS 64u
/* Maximum number of events one gather waits on. */
#define ZPP_MAX_WAIT_EVENTS 64u

/* Backward AllGather(L, P') of one layer over its P' node-local secondary
 * shards (Algorithm 1, backward branch; hpZ keeps this exchange inside a
 * node), with the qwZ dequantization fused in:
 *     out[j*shard_elems + i] = bf16(float(codes_j[i]) * scales_j[i / block])
 * for all j*shard_elems + i < layer_elems: one fp32 multiply, then round to
 * nearest even (NaN -> 0x7FC0).  The padding of the last shard past
 * layer_elems is dropped.
 * shard_codes, shard_scales: HOST arrays of num_shards DEVICE pointers
 *   (int8_t[shard_elems] and float[ceil(shard_elems/block)] each); they are
 *   read during the call only.  num_shards in [1, ZPP_MAX_SHARDS]; every
 *   pointer non-NULL.  out_bf16: uint16_t[layer_elems] out.
 * shard_elems >= 1, layer_elems <= num_shards * shard_elems (layer_elems 0
 *   is a no-op), block a multiple of 64 in [64, 4096] (ZPP_EINVAL otherwise).
 * Order on `stream`: wait for every event of wait_events[0..num_wait) on the
 * device (the paper's fix: no gather before the copies it reads are
 * complete), gather, record `done_after` (lets the next refresh of these
 * buffers wait for this read).  num_wait <= ZPP_MAX_WAIT_EVENTS, every event
 * non-NULL.
 * out must not overlap any shard range (ZPP_EOVERLAP).  Alignment: out 2,
 * scales 4 (ZPP_EALIGN); shard_elems % 16 == 0 with 16-byte aligned codes
 * and out selects the vector kernel. */
ZPP_API zpp_status zpp_dequant_gather_layer(const int8_t *const *shard_codes,
                                            const float *const *shard_scales, uint32_t num_shards,
                                            size_t shard_elems, uint32_t block, size_t layer_elems,
                                            uint16_t *out_bf16, hipStream_t stream,
                                            const hipEvent_t *wait_events, uint32_t num_wait,
                                            hipEvent_t done_after);

/* qgZ, sending side: quantize a rank's fp32 gradient of one destination
 * partition before the exchange that replaces the ReduceScatter (Background
 * section: gradients are quantized before ReduceScatter; Algorithm 1,
 * backward loop: an INT4 all-to-all takes its place).  Symmetric absmax int4
 * over consecutive blocks of `block` values (the last block may be short),
 * one fp32 scale per block, decisions in fp32:
 *   block holds an Inf or NaN  -> scale = NaN (0x7FC00000), codes 0
 *   a = max |x| == 0           -> scale = 0, codes 0
 *   otherwise                  -> scale = a / 7, inv = 7 / a (correctly
 *       rounded), code = rint(x * inv) (ties to even) in [-7, 7]; when
 *       a < 2^-100, x and a are first multiplied by 2^64.
 * Packing: two codes per byte, element 2i in the low nibble, 2i+1 in the high
 * nibble, 4-bit two's complement; an odd n leaves the last high nibble 0.
 * src: float[n].  codes: uint8_t[ceil(n/2)] out.  scales:
 * float[ceil(n/block)] out.  block: a multiple of 64 in [64, 4096].
 * Order on `stream`: wait `wait_before`, quantize, record `done_after`.
 * No two ranges may overlap (ZPP_EOVERLAP).  Alignment: src and scales 4
 * bytes (ZPP_EALIGN); 16-byte src and 2-byte codes select the vector kernel. */
ZPP_API zpp_status zpp_quantize_blockwise_i4(const float *src, size_t n, uint32_t block,
                                             uint8_t *codes, float *scales, hipStream_t stream,
                                             hipEvent_t wait_before, hipEvent_t done_after);

/* qgZ, receiving side: the num_src quantized copies of this rank's n-element
 * gradient partition (one from each sending rank, in rank order) are
 * dequantized and reduced into the fp32 gradient the partition step reads:
 *     acc = 0;  for q in 0..num_src-1: acc = fma(code_q[i], scale_q[i/block], acc)
 *     out[i] = acc * scale_out          (1 for a sum, 1/P for the mean)
 * each fma one rounding, the final product another; the order is fixed.
 * src_codes, src_scales: HOST arrays of num_src DEVICE pointers
 * (uint8_t[ceil(n/2)] and float[ceil(n/block)] each), read during the call
 * only; num_src in [1, ZPP_MAX_SHARDS].  out: float[n].  scale_out finite.
 * Order on `stream`: wait for every event of wait_events[0..num_wait) (the
 * exchange that delivered the sources), reduce, record `done_after`.
 * out must not overlap any source range (ZPP_EOVERLAP).  Alignment: out and
 * scales 4 bytes (ZPP_EALIGN); 16-byte out and 2-byte codes select the vector
 * kernel. */
ZPP_API zpp_status zpp_dequant_reduce_i4(const uint8_t *const *src_codes,
                                         const float *const *src_scales, uint32_t num_src, size_t n,
                                         uint32_t block, float scale_out, float *out,
                                         hipStream_t stream, const hipEvent_t *wait_events,
                                         uint32_t num_wait, hipEvent_t done_after);

/* qgZ receive fused into the partition step: the rank's optimizer step takes
 * its gradient straight from the num_src int4 copies of its partition that
 * the exchange replacing the ReduceScatter delivered (Background section:
 * qgZ; Algorithm 1, backward loop and the closing optimizer.step()).
 * Results are bit for bit those of zpp_dequant_reduce_i4(src_codes,
 * src_scales, num_src, n, block, scale_out, g) into an fp32 buffer g
 * followed by zpp_adam_partition_step(master, exp_avg, exp_avg_sq, g,
 * primary_bf16, n, hp), without the buffer: for every i < n
 *     acc = 0;  for q in 0..num_src-1: acc = fma(code_q[i], scale_q[i/block], acc)
 *     g = acc * scale_out;  then the Adam(W) update of zpp_adam_partition_step
 * at 26 B + num_src * (0.5 B + 4/block B) of HBM traffic per element instead
 * of 30 B + num_src * (0.5 B + 4/block B) + 4 B + 4 B.
 * master, exp_avg, exp_avg_sq: float[n] in place.  src_codes, src_scales:
 * HOST arrays of num_src DEVICE pointers (uint8_t[ceil(n/2)], packed as
 * zpp_quantize_blockwise_i4 writes them, and float[ceil(n/block)] each),
 * read during the call only; num_src in [1, ZPP_MAX_SHARDS].  block: a
 * multiple of 64 in [64, 4096].  scale_out finite (1/num_src for the data-parallel
 * mean).  primary_bf16: uint16_t[n] out.  hp as for zpp_adam_partition_step.
 * Order on `stream`: wait for every event of wait_events[0..num_wait) (the
 * exchange that delivered the sources), step, record `done_after`.
 * No two of the four outputs may overlap, nor any output a source range
 * (ZPP_EOVERLAP).  Alignment: floats and scales 4, bf16 2 bytes
 * (ZPP_EALIGN); 16-byte state arrays, an 8-byte primary and 2-byte codes
 * select the vector kernel. */
ZPP_API zpp_status zpp_qgz_receive_adam_step(float *master, float *exp_avg, float *exp_avg_sq,
                                             const uint8_t *const *src_codes,
                                             const float *const *src_scales, uint32_t num_src,
                                             uint32_t block, float scale_out,
                                             uint16_t *primary_bf16, size_t n,
                                             const zpp_adam_hparams *hp, hipStream_t stream,
                                             const hipEvent_t *wait_events, uint32_t num_wait,
                                             hipEvent_t done_after);

/* The whole pass of one rank's partition with the qgZ receive: the partition
 * step taking its gradient from the int4 copies (as
 * zpp_qgz_receive_adam_step), then the secondary refresh and the qwZ
 * quantization of the new bf16 weights (as zpp_adam_step_refresh_quantize),
 * in one pass over HBM.  Results are bit for bit those of
 * zpp_qgz_receive_adam_step into primary_bf16, zpp_refresh_secondary from
 * it and zpp_quantize_blockwise_i8 of it, at 29 B + num_src * (0.5 B +
 * 4/grad_block B) + 4/block B of HBM traffic per element instead of
 * 33 B + num_src * (0.5 B + 4/grad_block B) + 4/block B.  An int8 block
 * other than 64 to 512 takes two kernels in stream order, as for
 * zpp_adam_step_refresh_quantize.
 * master, exp_avg, exp_avg_sq: float[n] in place.  src_codes, src_scales,
 * num_src, scale_out: as for zpp_qgz_receive_adam_step, with int4 blocks of
 * grad_block (a multiple of 64 in [64, 4096]).  primary_bf16: uint16_t[n] out;
 * secondary_bf16: uint16_t[n] out, or NULL to keep no bf16 secondary copy;
 * codes: int8_t[n] out; scales: float[ceil(n/block)] out, int8 blocks of
 * block (a multiple of 64 in [64, 4096]).  hp as for zpp_adam_partition_step.
 * Order on `stream`: wait for every event of wait_events[0..num_wait),
 * run, record `done_after` (the event a gather of the codes waits on).
 * No two outputs may overlap, nor any output a source range (ZPP_EOVERLAP).
 * Alignment: floats and scales 4, bf16 2 bytes (ZPP_EALIGN); 16-byte state
 * arrays, 8-byte bf16 arrays, 4-byte codes and 2-byte source codes select
 * the single-pass kernel, otherwise the three scalar kernels run one after
 * another. */
ZPP_API zpp_status zpp_qgz_receive_step_refresh_quantize(
    float *master, float *exp_avg, float *exp_avg_sq, const uint8_t *const *src_codes,
    const float *const *src_scales, uint32_t num_src, uint32_t grad_block, float scale_out,
    uint16_t *primary_bf16, uint16_t *secondary_bf16, int8_t *codes, float *scales, size_t n,
    uint32_t block, const zpp_adam_hparams *hp, hipStream_t stream, const hipEvent_t *wait_events,
    uint32_t num_wait, hipEvent_t done_after);

/* The qgZ receive buffer interleaved: the num_src int4 copies of an n-element
 * partition in ONE buffer, block by block, instead of num_src separate
 * arrays.  With B = the int4 block and k = i / B:
 *   source q's code of element i: byte (k * num_src + q) * B/2 + (i mod B)/2,
 *       low nibble for even i, high nibble for odd i (packing as
 *       zpp_quantize_blockwise_i4);
 *   source q's scale of block k:  float (k * num_src + q).
 * Codes: uint8_t[ceil(n/B) * num_src * B/2]; scales:
 * float[ceil(n/B) * num_src].  With num_src = 1 it is the plain layout of
 * zpp_quantize_blockwise_i4.  A receiving kernel then reads each block's
 * codes of all sources within one contiguous run rather than from num_src
 * separate arrays.  The exchange that fills it (each sending rank writing its
 * slots, e.g. by peer stores within a node) is not part of this library;
 * zpp_quantize_blockwise_i4_interleaved writes one source's slots. */

/* zpp_quantize_blockwise_i4 (same blocks, scales, codes and rules) writing
 * source `source` of num_src into an interleaved receive buffer (layout
 * above); the other sources' slots are left as they are.  num_src in
 * [1, ZPP_MAX_SHARDS], source < num_src, n <= SIZE_MAX / 16 / num_src.
 * Order on `stream`: wait `wait_before`, quantize, record `done_after`.
 * No two of src, the codes buffer and the scales buffer may overlap
 * (ZPP_EOVERLAP).  Alignment: src and scales 4 bytes (ZPP_EALIGN); 16-byte
 * src and 2-byte codes select the vector kernel. */
ZPP_API zpp_status zpp_quantize_blockwise_i4_interleaved(const float *src, size_t n,
                                                         uint32_t block, uint32_t source,
                                                         uint32_t num_src, uint8_t *codes,
                                                         float *scales, hipStream_t stream,
                                                         hipEvent_t wait_before,
                                                         hipEvent_t done_after);

/* zpp_dequant_reduce_i4 with its num_src int4 copies in one interleaved
 * receive buffer (layout above): the same arithmetic in the same order, so
 * the same bits.  codes, scales: DEVICE pointers to the interleaved buffer,
 * B = block.  n <= SIZE_MAX / 16 / num_src.  out: float[n], which must not
 * overlap the buffer (ZPP_EOVERLAP).  Order on `stream`: wait for every
 * event of wait_events[0..num_wait), reduce, record `done_after`.
 * Alignment: out and scales 4 bytes (ZPP_EALIGN); 16-byte out and 2-byte
 * codes select the vector kernel. */
ZPP_API zpp_status zpp_dequant_reduce_i4_interleaved(const uint8_t *codes, const float *scales,
                                                     uint32_t num_src, size_t n, uint32_t block,
                                                     float scale_out, float *out,
                                                     hipStream_t stream,
                                                     const hipEvent_t *wait_events,
                                                     uint32_t num_wait, hipEvent_t done_after);

/* zpp_qgz_receive_adam_step with its num_src int4 copies in one interleaved
 * receive buffer (layout above): the same arithmetic in the same order, so
 * the same bits.  codes, scales: DEVICE pointers to the interleaved buffer,
 * B = block.  n <= SIZE_MAX / 16 / num_src.  Everything else as for
 * zpp_qgz_receive_adam_step, alignment included; the two input ranges may
 * overlap each other, not an output. */
ZPP_API zpp_status zpp_qgz_receive_adam_step_interleaved(
    float *master, float *exp_avg, float *exp_avg_sq, const uint8_t *codes, const float *scales,
    uint32_t num_src, uint32_t block, float scale_out, uint16_t *primary_bf16, size_t n,
    const zpp_adam_hparams *hp, hipStream_t stream, const hipEvent_t *wait_events,
    uint32_t num_wait, hipEvent_t done_after);

/* zpp_qgz_receive_step_refresh_quantize with its num_src int4 copies in one
 * interleaved receive buffer (src_codes, src_scales; layout above, B =
 * grad_block): the same bits.  Everything else as there, alignment
 * included. */
ZPP_API zpp_status zpp_qgz_receive_step_refresh_quantize_interleaved(
    float *master, float *exp_avg, float *exp_avg_sq, const uint8_t *src_codes,
    const float *src_scales, uint32_t num_src, uint32_t grad_block, float scale_out,
    uint16_t *primary_bf16, uint16_t *secondary_bf16, int8_t *codes, float *scales, size_t n,
    uint32_t block, const zpp_adam_hparams *hp, hipStream_t stream, const hipEvent_t *wait_events,
    uint32_t num_wait, hipEvent_t done_after);

/* Static, NUL-terminated description of a status code.  Takes any int, so
 * that a caller may pass whatever status value it holds: a value that is not
 * one of zpp_status gives "unknown status". */
ZPP_API const char *zpp_status_string(int status);

/* hipError_t (as int) of the last call on this host thread that returned
 * ZPP_EHIP; 0 if none. */
ZPP_API int zpp_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ZPP_H */
