/*
 * dkv_probe.h -- achievable-bandwidth probe (a measurement aid; not part of
 * the Distance-KV method).
 *
 * A plain streaming read of device memory with the same load instructions
 * and cache policy as the decode kernel's K/V stream (16-byte non-temporal
 * buffer loads).  The benchmark times it on buffers of one decode launch's
 * size to report what a launch of that size reaches on this GPU, next to the
 * HBM specification.  Conventions (device pointers, asynchronous on `stream`,
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

/* Reads bytes [0, bytes) at `src` with `workgroups` workgroups of 256
 * threads; workgroup w streams the w-th of `workgroups` equal contiguous
 * slices (16-byte granules), each thread keeping eight 16-byte loads in
 * flight.  The loaded data is folded into a value that is stored to `sink`
 * (16 bytes) only if it equals an impossible constant, so the loads cannot be
 * removed; the content of `sink` is unspecified.
 *   src, sink  device pointers, 16-byte aligned; src holds `bytes` bytes.
 *   bytes      multiple of 16, >= 0 (0: nothing is enqueued).
 *   workgroups 1 .. 65535; a slice may not exceed 2^31 bytes.
 * Errors: DKV_ERR_INVALID_ARG (null pointer, bytes < 0 or not a multiple of
 * 16, workgroups out of range), DKV_ERR_UNSUPPORTED (slice over 2^31 bytes),
 * DKV_ERR_MISALIGNED, DKV_ERR_HIP (launch refused). */
dkv_status dkv_probe_stream_read(const void* src, int64_t bytes, void* sink, int32_t workgroups,
                                 void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DKV_PROBE_H */
