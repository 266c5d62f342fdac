/*
 * dkv_probe.h -- achievable-bandwidth probes (measurement aids; not part of
 * the Distance-KV method).
 *
 * A plain streaming read of device memory with the same load instructions
 * and cache policy as the decode kernel's K/V stream (16-byte non-temporal
 * buffer loads), and a plain copy (16-byte non-temporal loads and stores).  The benchmark times the read on buffers of one decode launch's
 * size to report what a launch of that size reaches on this GPU, next to the
 * HBM specification, and the copy on the bytes the one-time pack moves, the
 * rate a gather of retained rows can at best approach.  Conventions (device pointers, asynchronous on `stream`,
 * host-side argument checks, status codes) are those of dkv.h.
 */
#ifndef DKV_PROBE_H
#define DKV_PROBE_H

#include <stddef.h>
#include <stdint.h>

#include "dkv.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Reads bytes [0, bytes) at `src` in blocks of 256 x G 16-byte granules
 * (G = granules_per_thread: 4, 8, 16 or 32 KiB), one block per workgroup of
 * 256 threads, with the decode kernel's K/V load (16-byte non-temporal buffer
 * loads); each thread issues its G loads and the workgroup retires.  The
 * loaded data is folded into a value that is stored to `sink` (16 bytes) only
 * if it equals an impossible constant, so the loads cannot be removed; the
 * content of `sink` is unspecified.
 *   src, sink  device pointers, 16-byte aligned; src holds `bytes` bytes.
 *   bytes      multiple of 16, >= 0 (0: nothing is enqueued).
 *   granules_per_thread  1, 2, 4 or 8.
 * Errors: DKV_ERR_INVALID_ARG (null pointer, bytes < 0 or not a multiple of
 * 16, G not one of the four), DKV_ERR_UNSUPPORTED (more than 2^31 - 1
 * blocks), DKV_ERR_MISALIGNED, DKV_ERR_HIP (launch refused). */
dkv_status dkv_probe_stream_read(const void* src, int64_t bytes, void* sink, int32_t granules_per_thread,
                                 void* stream);

/* Copies bytes [0, bytes) from `src` to `dst` in blocks of 256 x G 16-byte
 * granules (G = granules_per_thread: 4, 8, 16 or 32 KiB), one block per
 * workgroup of 256 threads: each thread loads its G granules non-temporally,
 * then stores them, and the grid has one workgroup per block.
 *   src, dst   device pointers, 16-byte aligned, `bytes` bytes each, not
 *              overlapping (the caller owns both; dst is overwritten).
 *   bytes      multiple of 16, >= 0 (0: nothing is enqueued).
 *   granules_per_thread  1, 2, 4 or 8.
 * Errors: DKV_ERR_INVALID_ARG (null pointer, overlapping buffers, bytes < 0
 * or not a multiple of 16, G not one of the four), DKV_ERR_MISALIGNED,
 * DKV_ERR_UNSUPPORTED (more than 2^31 - 1 blocks), DKV_ERR_HIP (launch
 * refused). */
dkv_status dkv_probe_copy(const void* src, void* dst, int64_t bytes, int32_t granules_per_thread, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DKV_PROBE_H */
