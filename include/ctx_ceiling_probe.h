/*
 * ctx_ceiling_probe.h -- kernels that measure the practical ceilings of the
 * device the library runs on: HBM streaming and the bf16 matrix-core rate.
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
#ifndef CTX_CEILING_PROBE_H_
#define CTX_CEILING_PROBE_H_

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

/*
 * Matrix-core rate: every wave of `workgroups` workgroups of 256 threads runs
 * `iterations` rounds of 8 independent bf16 MFMAs with fp32 accumulation and
 * writes one 16-byte word per wave to sink, like ctx_hbm_read.  The causal
 * prefill of the reference observation (Sec. 4.1,
 * eq:reference-conditioned-action) is a dense contraction on these units;
 * this gives the rate they sustain on this device for its instruction shapes.
 *   shape       CTX_MFMA_16X16X32 (8 x v_mfma_f32_16x16x32_bf16 per round: 131,072
 *               flops per wave) or CTX_MFMA_32X32X16 (8 x v_mfma_f32_32x32x16_bf16:
 *               262,144 flops per wave)
 *   workgroups  1 .. 65536; iterations 1 .. 1<<20
 *   sink        16-byte aligned, workgroups * CTX_HBM_SINK_BYTES_PER_WORKGROUP bytes
 * Flops per call = workgroups * 4 * iterations * (flops per wave per round).
 * Errors: INVALID_ARG (shape, sizes, NULL), ALIGNMENT, HIP.
 */
#define CTX_MFMA_16X16X32 0
#define CTX_MFMA_32X32X16 1
int ctx_mfma_bf16(int32_t shape, int32_t workgroups, int32_t iterations, void* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CTX_CEILING_PROBE_H_ */
