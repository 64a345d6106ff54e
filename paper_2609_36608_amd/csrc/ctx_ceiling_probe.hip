// ctx_ceiling_probe.hip -- kernels for gfx950 (MI355X) that measure the
// device's practical ceilings (streaming read and copy; the bf16 matrix-core
// rate), behind the C ABI declared in include/ctx_ceiling_probe.h.
//
// Both kernels run a grid-stride loop over tiles of kProbeThreads x
// kProbeUnroll 16-byte words: every thread issues kProbeUnroll independent
// 16-byte loads before using any of them, consecutive threads touch
// consecutive words (each wave reads 1 KiB contiguous per load instruction),
// and the tiles of one workgroup are gridDim apart, so the whole grid sweeps
// the buffer front to back.  The read kernel folds its words by XOR into one
// word per wave, written to the sink, so that no load is dead.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "ctx_attn_common.h"
#include "ctx_ceiling_probe.h"

namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 8;
constexpr int kProbeMaxGrid = 65536;

template <bool kNt>
__device__ __forceinline__ u32x4 probe_load(const u32x4* p) {
  if (kNt) return __builtin_nontemporal_load(p);
  return *p;
}

template <bool kNt>
__device__ __forceinline__ void probe_store(u32x4* p, u32x4 v) {
  if (kNt)
    __builtin_nontemporal_store(v, p);
  else
    *p = v;
}

template <bool kNt>
__global__ __launch_bounds__(kProbeThreads) void hbm_read_kernel(const u32x4* __restrict__ src, size_t words,
                                                                 u32x4* __restrict__ sink) {
  const size_t tile = (size_t)kProbeThreads * kProbeUnroll;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (size_t base = (size_t)blockIdx.x * tile; base < words; base += (size_t)gridDim.x * tile) {
    u32x4 r[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) {
      const size_t i = base + (size_t)u * kProbeThreads + threadIdx.x;
      r[u] = i < words ? probe_load<kNt>(src + i) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) acc ^= r[u];
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    acc.x ^= __shfl_xor(acc.x, off);
    acc.y ^= __shfl_xor(acc.y, off);
    acc.z ^= __shfl_xor(acc.z, off);
    acc.w ^= __shfl_xor(acc.w, off);
  }
  const int lane = threadIdx.x & 63;
  if (lane == 0) sink[(size_t)blockIdx.x * (kProbeThreads / 64) + (threadIdx.x >> 6)] = acc;
}

template <bool kNt>
__global__ __launch_bounds__(kProbeThreads) void hbm_copy_kernel(const u32x4* __restrict__ src,
                                                                 u32x4* __restrict__ dst, size_t words) {
  const size_t tile = (size_t)kProbeThreads * kProbeUnroll;
  for (size_t base = (size_t)blockIdx.x * tile; base < words; base += (size_t)gridDim.x * tile) {
    u32x4 r[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) {
      const size_t i = base + (size_t)u * kProbeThreads + threadIdx.x;
      if (i < words) r[u] = probe_load<kNt>(src + i);
    }
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) {
      const size_t i = base + (size_t)u * kProbeThreads + threadIdx.x;
      if (i < words) probe_store<kNt>(dst + i, r[u]);
    }
  }
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
constexpr int kMfmaChains = 8;

// 8 independent accumulation chains per wave, operands that vary per lane;
// the results are folded into one word per wave so that no MFMA is dead.
template <int kShape>
__global__ __launch_bounds__(kProbeThreads) void mfma_probe_kernel(int iterations, u32x4* __restrict__ sink) {
  bf16x8 a, b;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    a[j] = (__bf16)((float)((threadIdx.x + j) & 7) * 0.125f);
    b[j] = (__bf16)((float)((threadIdx.x * 3 + j) & 7) * 0.0625f);
  }
  float fold = 0.f;
  if (kShape == CTX_MFMA_16X16X32) {
    f32x4 acc[kMfmaChains];
#pragma unroll
    for (int k = 0; k < kMfmaChains; ++k) acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < iterations; ++it) {
#pragma unroll
      for (int k = 0; k < kMfmaChains; ++k) acc[k] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[k], 0, 0, 0);
    }
#pragma unroll
    for (int k = 0; k < kMfmaChains; ++k) fold += acc[k][0] + acc[k][3];
  } else {
    f32x16 acc[kMfmaChains];
#pragma unroll
    for (int k = 0; k < kMfmaChains; ++k) acc[k] = f32x16{};
    for (int it = 0; it < iterations; ++it) {
#pragma unroll
      for (int k = 0; k < kMfmaChains; ++k) acc[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[k], 0, 0, 0);
    }
#pragma unroll
    for (int k = 0; k < kMfmaChains; ++k) fold += acc[k][0] + acc[k][15];
  }
  u32x4 w = {__float_as_uint(fold), 0u, 0u, 0u};
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) w.x ^= __shfl_xor(w.x, off);
  if ((threadIdx.x & 63) == 0) sink[(size_t)blockIdx.x * (kProbeThreads / 64) + (threadIdx.x >> 6)] = w;
}

int check_probe(const void* src, const void* other, size_t bytes, int32_t workgroups, uint32_t flags) {
  ctx_clear_error();
  if (src == nullptr || other == nullptr) return fail(CTX_ERR_INVALID_ARG, "NULL pointer");
  if (bytes == 0 || bytes % 16 != 0) return fail(CTX_ERR_INVALID_ARG, "bytes %zu must be a positive multiple of 16", bytes);
  if (workgroups < 1 || workgroups > kProbeMaxGrid)
    return fail(CTX_ERR_INVALID_ARG, "workgroups %d outside 1..%d", workgroups, kProbeMaxGrid);
  if ((flags & ~CTX_HBM_NONTEMPORAL) != 0) return fail(CTX_ERR_INVALID_ARG, "unknown flags 0x%x", flags);
  if (!aligned16(src) || !aligned16(other)) return fail(CTX_ERR_ALIGNMENT, "pointers must be 16-byte aligned");
  return CTX_OK;
}

}  // namespace

extern "C" int ctx_hbm_read(const void* src, size_t bytes, void* sink, int32_t workgroups, uint32_t flags,
                            void* stream) {
  int rc = check_probe(src, sink, bytes, workgroups, flags);
  if (rc != CTX_OK) return rc;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const u32x4* sp = static_cast<const u32x4*>(src);
  u32x4* kp = static_cast<u32x4*>(sink);
  if (flags & CTX_HBM_NONTEMPORAL)
    hipLaunchKernelGGL(hbm_read_kernel<true>, dim3(workgroups), dim3(kProbeThreads), 0, s, sp, bytes / 16, kp);
  else
    hipLaunchKernelGGL(hbm_read_kernel<false>, dim3(workgroups), dim3(kProbeThreads), 0, s, sp, bytes / 16, kp);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return CTX_OK;
}

extern "C" int ctx_hbm_copy(const void* src, void* dst, size_t bytes, int32_t workgroups, uint32_t flags,
                            void* stream) {
  int rc = check_probe(src, dst, bytes, workgroups, flags);
  if (rc != CTX_OK) return rc;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const u32x4* sp = static_cast<const u32x4*>(src);
  u32x4* dp = static_cast<u32x4*>(dst);
  if (flags & CTX_HBM_NONTEMPORAL)
    hipLaunchKernelGGL(hbm_copy_kernel<true>, dim3(workgroups), dim3(kProbeThreads), 0, s, sp, dp, bytes / 16);
  else
    hipLaunchKernelGGL(hbm_copy_kernel<false>, dim3(workgroups), dim3(kProbeThreads), 0, s, sp, dp, bytes / 16);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return CTX_OK;
}

extern "C" int ctx_mfma_bf16(int32_t shape, int32_t workgroups, int32_t iterations, void* sink, void* stream) {
  ctx_clear_error();
  if (sink == nullptr) return fail(CTX_ERR_INVALID_ARG, "NULL sink");
  if (shape != CTX_MFMA_16X16X32 && shape != CTX_MFMA_32X32X16) return fail(CTX_ERR_INVALID_ARG, "unknown shape %d", shape);
  if (workgroups < 1 || workgroups > kProbeMaxGrid)
    return fail(CTX_ERR_INVALID_ARG, "workgroups %d outside 1..%d", workgroups, kProbeMaxGrid);
  if (iterations < 1 || iterations > (1 << 20)) return fail(CTX_ERR_INVALID_ARG, "iterations %d outside 1..2^20", iterations);
  if (!aligned16(sink)) return fail(CTX_ERR_ALIGNMENT, "sink must be 16-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  u32x4* kp = static_cast<u32x4*>(sink);
  if (shape == CTX_MFMA_16X16X32)
    hipLaunchKernelGGL(mfma_probe_kernel<CTX_MFMA_16X16X32>, dim3(workgroups), dim3(kProbeThreads), 0, s, iterations, kp);
  else
    hipLaunchKernelGGL(mfma_probe_kernel<CTX_MFMA_32X32X16>, dim3(workgroups), dim3(kProbeThreads), 0, s, iterations, kp);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return CTX_OK;
}
