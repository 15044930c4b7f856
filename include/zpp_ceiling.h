/*
 * Plain HBM streams for measurement: the bandwidth ceilings that the
 * partition-path kernels of zpp.h are compared against.  Not part of the
 * partition path; bench.py loads libzpp_ceiling.so to time them beside the
 * path's kernels.
 *
 * All three move 16-byte vectors with non-temporal loads and stores, every
 * wave's accesses contiguous, in the launch shapes that stream fastest on
 * MI355X (measured):
 *   zppc_read_stream   one-wave workgroups, four 16-byte loads per lane in
 *                      flight, at most 16 workgroups per compute unit;
 *   zppc_write_stream  four-wave workgroups, one 16-byte store per lane, at
 *                      most 4 workgroups per compute unit;
 *   zppc_copy_stream   one-wave workgroups, one 16-byte load and store per
 *                      lane, residency left to the hardware.
 *
 * Beside them, the access patterns of three partition-path kernels with
 * their arithmetic taken out: the same loads and stores in the same lane
 * layout, workgroup shape, one-shot grid and residency cap, each loaded word
 * folded by one xor (what is stored is not meaningful):
 *   zppc_adam_pattern   the Adam step: per element 16 bytes read (p, m, v, g)
 *                       and 14 written (p, m, v in place, a bf16); n a
 *                       multiple of 256;
 *   zppc_gather_pattern the dequant-gather row kernel for blocks of 256:
 *                       n int8 codes and n/256 fp32 scales read, n bf16
 *                       written; n a multiple of 512;
 *   zppc_quant_pattern  the int8 quantizer for blocks of 256: n bf16 read,
 *                       n int8 codes and n/256 fp32 scales written; n a
 *                       multiple of 4096.
 * Their pointers are device pointers aligned to their element vectors (16
 * bytes for fp32 and bf16 arrays read or written 16 bytes per lane, 8 for
 * codes and the bf16 output of the Adam pattern, 4 for scales).
 *
 * Pointers are device pointers owned by the caller, 16-byte aligned; `bytes`
 * is a non-zero multiple of 4096.  The read stream folds what it reads into
 * one word per workgroup and stores it to sink[0] only when that word equals
 * a value no stream of ones produces, so it reads everything and writes
 * (next to) nothing; sink is a device uint32_t[1].  The write stream stores
 * `pattern` in every 32-bit word.  Each call only enqueues its kernel on
 * `stream` and returns the launch's hipError_t as an int (0 = success, or
 * hipErrorInvalidValue for a bad size or alignment, checked before
 * anything is enqueued).
 */
#ifndef ZPP_CEILING_H
#define ZPP_CEILING_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ZPPC_API __attribute__((visibility("default")))

ZPPC_API int zppc_read_stream(const void *src, size_t bytes, uint32_t *sink, hipStream_t stream);
ZPPC_API int zppc_write_stream(void *dst, size_t bytes, uint32_t pattern, hipStream_t stream);
ZPPC_API int zppc_copy_stream(void *dst, const void *src, size_t bytes, hipStream_t stream);
ZPPC_API int zppc_adam_pattern(float *p, float *m, float *v, const float *g, uint16_t *out,
                               size_t n, hipStream_t stream);
ZPPC_API int zppc_gather_pattern(const int8_t *codes, const float *scales, uint16_t *out,
                                 size_t n, hipStream_t stream);
ZPPC_API int zppc_quant_pattern(const uint16_t *src, int8_t *codes, float *scales, size_t n,
                                hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif
