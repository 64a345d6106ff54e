/*
 * ctx_hbm_probe.h -- streaming kernels that measure the practical HBM ceiling
 * of the device the library runs on.
 *
 * The decode step is bound by reading the KV cache (and, per step, the
 * student's weights) from HBM once.  The rollout engine model of the
 * scheduling simulator prices each decode step's weight streaming at the
 * device's read rate and the attention at its measured cost (the calibrated
 * rollout estimate, eq:calibrated-rollout-speedup, with the step model of App.
 * finite concurrency); these two kernels give the read rate, and the rate of
 * an equal mix of reads and writes (the OPD loss kernel reads the logits and
 * writes their gradient), measured in the caller's process.
 *
 * Conventions: device pointers on the current HIP device, owned by the caller;
 * `stream` is a hipStream_t passed as void* (NULL = default stream); the calls
 * are asynchronous (no host sync, no allocation) and return ctx_status codes.
 */
#ifndef CTX_HBM_PROBE_H_
#define CTX_HBM_PROBE_H_

#include <stddef.h>
#include <stdint.h>

#include "ctx_decode_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Bytes of `sink` that ctx_hbm_read writes per workgroup (one 16-byte word per wave). */
#define CTX_HBM_SINK_BYTES_PER_WORKGROUP 64u
/* ctx_hbm_read / ctx_hbm_copy flag: non-temporal loads (and stores), as the decode kernel streams its cache */
#define CTX_HBM_NONTEMPORAL 1u

/*
 * Read `bytes` from src once (16-byte loads, every byte exactly once) and
 * write the XOR of each wave's data to sink, so that no load can be dropped.
 *   src         16-byte aligned; bytes a multiple of 16, > 0
 *   sink        16-byte aligned, workgroups * CTX_HBM_SINK_BYTES_PER_WORKGROUP bytes
 *   workgroups  grid size, 1 .. 65536 (workgroups of 256 threads, grid-stride loop)
 *   flags       0 or CTX_HBM_NONTEMPORAL
 * Errors: INVALID_ARG (sizes, flags, NULL), ALIGNMENT, HIP.
 */
int ctx_hbm_read(const void* src, size_t bytes, void* sink, int32_t workgroups, uint32_t flags, void* stream);

/*
 * dst[0 .. bytes) = src[0 .. bytes): every byte read once and written once.
 * Same arguments and errors as ctx_hbm_read; src and dst must not overlap.
 */
int ctx_hbm_copy(const void* src, void* dst, size_t bytes, int32_t workgroups, uint32_t flags, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CTX_HBM_PROBE_H_ */
