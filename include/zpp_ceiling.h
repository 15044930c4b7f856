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

#ifdef __cplusplus
}
#endif

#endif
