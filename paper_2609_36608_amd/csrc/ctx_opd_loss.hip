// ctx_opd_loss.hip -- fused OPD token loss and logits gradient for gfx950
// (MI355X), behind the C ABI declared in include/ctx_opd_loss.h.
//
// The loss of App. OPD Optimization needs, per supervised token, the
// student's log-probability of the sampled token, i.e. a log-sum-exp over the
// whole vocabulary row (151,936 bf16 logits = 297 KiB for the Qwen3 students),
// and back-propagation writes a gradient row of the same size.  Everything
// else is a handful of scalars per token, so the work is bound by HBM, and
// the least traffic is one read of each logits row and one write of each
// gradient row.
//
// Design:
//   * opd_weight_kernel: one workgroup per response counts its supervised
//     tokens and writes w_j = m_j / (B (M_b + eps)).
//   * opd_row_kernel<C>: a persistent 1024-thread workgroup per CU walks the
//     token rows; it holds a whole row in registers (thread t owns the
//     16-byte chunks t + 1024 k, k < C: coalesced, non-temporal loads).  It reduces the row maximum and
//     the sum of exp over the registers (wave shuffles, then 16 partials
//     through LDS, always in the same order), forms lp, the clipped ratio,
//     the dual-clip loss and the per-row gradient scale g, and writes the
//     gradient row g (onehot - softmax) from the same registers, rounded to
//     bf16.  A row whose g is 0 (a flat clipping regime or A = 0) writes
//     zeros without the second exp pass; a masked row is not read at all.
//     At 128 VGPRs a CU holds one such workgroup, so the next row's loads are
//     issued chunk by chunk as the gradient pass frees the registers: its
//     HBM reads overlap this row's exps and gradient stores.
//   * opd_reduce_kernel: loss = sum_j w_j l_j in double precision, one
//     workgroup, fixed order (deterministic, no atomics).

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>

#include "ctx_opd_loss.h"

// the library's per-thread last-error message (defined with the attention entry points)
__attribute__((visibility("hidden"))) int ctx_report_error(int code, const char* msg);
__attribute__((visibility("hidden"))) void ctx_clear_error();

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kRowThreads = 1024;
constexpr int kRowWaves = kRowThreads / 64;
constexpr int kChunk = 8;  // bf16 per 16-byte chunk
constexpr int kMaxChunksPerThread = 19;  // 76 VGPRs of row data: 128 VGPRs at 16 waves per CU
constexpr int64_t kMaxVocab = (int64_t)kRowThreads * kChunk * kMaxChunksPerThread;  // 155,648
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct OpdParams {
  float clip_log;
  float delta;
  float kappa;
  float eps;
};

__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// round to nearest even, two floats into one word (a low, b high)
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

// Block reductions over kRowWaves partials in a fixed order.
__device__ __forceinline__ float block_max(float x, float* red) {
  x = wave_max(x);
  const int wave = threadIdx.x >> 6;
  __syncthreads();  // red is free (previous reduction read it)
  if ((threadIdx.x & 63) == 0) red[wave] = x;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < kRowWaves; ++w) r = fmaxf(r, red[w]);
  return r;
}

__device__ __forceinline__ float block_sum(float x, float* red) {
  x = wave_sum(x);
  const int wave = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[wave] = x;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < kRowWaves; ++w) r += red[w];
  return r;
}

__global__ __launch_bounds__(256) void opd_weight_kernel(const uint8_t* __restrict__ mask,
                                                         const int32_t* __restrict__ seq_starts,
                                                         int32_t num_seqs, float eps,
                                                         float* __restrict__ weight) {
  __shared__ int red[4];
  const int b = blockIdx.x;
  const int s0 = seq_starts[b], s1 = seq_starts[b + 1];
  int cnt = 0;
  for (int j = s0 + (int)threadIdx.x; j < s1; j += 256) cnt += mask[j] ? 1 : 0;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = cnt;
  __syncthreads();
  const int mb = red[0] + red[1] + red[2] + red[3];
  const float w = (float)(1.0 / ((double)num_seqs * ((double)mb + (double)eps)));
  for (int j = s0 + (int)threadIdx.x; j < s1; j += 256) weight[j] = mask[j] ? w : 0.f;
}

// eq:opd-dual-clip for one token: the loss and d loss / d rho
__device__ __forceinline__ void dual_clip_loss(float rho, float a, const OpdParams& p, float* loss,
                                               float* dloss) {
  const float lo = 1.f - p.delta, hi = 1.f + p.delta;
  const float clipped = fminf(fmaxf(rho, lo), hi);
  const float dclipped = (rho > lo && rho < hi) ? 1.f : 0.f;
  const float unclipped_term = rho * a, clipped_term = clipped * a;
  float l, d;
  if (unclipped_term <= clipped_term) {
    l = -unclipped_term;
    d = -a;
  } else {
    l = -clipped_term;
    d = -a * dclipped;
  }
  if (a < 0.f && -p.kappa * a < l) {
    l = -p.kappa * a;
    d = 0.f;
  }
  *loss = l;
  *dloss = d;
}

// Buffer resource over `bytes` bytes from a wave-uniform base: loads past
// the end return zeros and stores past it are dropped.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  const uint64_t u = ((uint64_t)hi << 32) | lo;
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(u), (short)0,
                                           (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

constexpr int kNonTemporal = 2;  // buffer cache-policy bits: streamed once
// Chunk offsets go in the VGPR offset, which the buffer range check covers;
// the SGPR offset stays 0.
constexpr int kWaitVmcnt0 = 0x0F70;  // s_waitcnt vmcnt(0), expcnt and lgkmcnt left open

// An empty asm that "may change" every chunk of the row: the compiler then
// recomputes the cheap bf16 -> fp32 unpacking in each pass instead of keeping
// eight unpacked floats per chunk alive across passes (two rows' worth of
// registers).  It emits no instruction.
template <int C>
__device__ __forceinline__ void opaque(u32x4 (&x)[C]) {
#pragma unroll
  for (int k = 0; k < C; ++k) asm volatile("" : "+v"(x[k]));
}

template <int C>
__global__ __launch_bounds__(kRowThreads) void opd_row_kernel(
    const uint16_t* __restrict__ logits, int64_t row_stride, int32_t vocab, int32_t num_rows,
    const int32_t* __restrict__ tokens, const float* __restrict__ old_logp,
    const float* __restrict__ teacher_logp, const uint8_t* __restrict__ mask,
    const float* __restrict__ weight, OpdParams prm, float* __restrict__ token_logp,
    float* __restrict__ token_loss, uint16_t* __restrict__ grad, int64_t grad_stride) {
  __shared__ float red[kRowWaves];
  const int tid = threadIdx.x;
  const int nchunks = (vocab + kChunk - 1) / kChunk;
  const int nwhole = vocab / kChunk;  // chunks with 8 columns below vocab
  // C = ceil(nchunks / 1024): rounds k < C - 1 give every thread a whole
  // chunk; only the last round tests chunks and columns against vocab
  constexpr int kwhole = C - 1;
  const uint32_t load_bytes = (uint32_t)nchunks * 16u;   // loads: every chunk (the partial one padded)
  const uint32_t store_bytes = (uint32_t)nwhole * 16u;   // stores: whole chunks; a partial one apart
  const int voff = tid * 16;

  // Persistent: rows blockIdx.x, + gridDim.x, ...  The row is held in x; the
  // next row's loads are issued chunk by chunk as the gradient pass frees x.
  u32x4 x[C];
  int j = blockIdx.x;
  if (j >= num_rows) return;
  bool sup = mask[j] != 0;
  if (sup) {
    const __amdgpu_buffer_rsrc_t rr = row_rsrc(logits + (size_t)j * row_stride, load_bytes);
#pragma unroll
    for (int k = 0; k < C; ++k)
      x[k] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rr, voff + k * kRowThreads * 16, 0,
                                                                              kNonTemporal));
  }
#pragma nounroll
  for (; j < num_rows; j += gridDim.x) {
    // per-row copy of the lane index, opaque to the compiler: lane-dependent
    // masks and offsets are recomputed per row (a few instructions) instead of
    // being hoisted out of the row loop, where they would occupy registers
    int t = tid;
    asm volatile("" : "+v"(t));
    const int vo = t * 16;
    const int jn = j + (int)gridDim.x;
    const bool next_sup = jn < num_rows && mask[jn] != 0;
    float g = 0.f, lse2 = 0.f;
    int tok = -1;
    if (sup) {
      float mx = -INFINITY;
#pragma unroll
      for (int k = 0; k < C; ++k) {
        if (k < kwhole) {
#pragma unroll
          for (int i = 0; i < 4; ++i) mx = fmaxf(mx, fmaxf(lo_bf16(x[k][i]), hi_bf16(x[k][i])));
        } else {
          const int c0 = (t + k * kRowThreads) * kChunk;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if (c0 + 2 * i < vocab) mx = fmaxf(mx, lo_bf16(x[k][i]));
            if (c0 + 2 * i + 1 < vocab) mx = fmaxf(mx, hi_bf16(x[k][i]));
          }
        }
        __builtin_amdgcn_sched_barrier(0);  // chunk by chunk: bounded live ranges
      }
      const float m2 = block_max(mx, red) * kLog2e;
      opaque(x);
      float s = 0.f;
#pragma unroll
      for (int k = 0; k < C; ++k) {
        if (k < kwhole) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            s += __builtin_amdgcn_exp2f(fmaf(lo_bf16(x[k][i]), kLog2e, -m2)) +
                 __builtin_amdgcn_exp2f(fmaf(hi_bf16(x[k][i]), kLog2e, -m2));
        } else {
          const int c0 = (t + k * kRowThreads) * kChunk;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if (c0 + 2 * i < vocab) s += __builtin_amdgcn_exp2f(fmaf(lo_bf16(x[k][i]), kLog2e, -m2));
            if (c0 + 2 * i + 1 < vocab) s += __builtin_amdgcn_exp2f(fmaf(hi_bf16(x[k][i]), kLog2e, -m2));
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      lse2 = m2 + __log2f(block_sum(s, red));  // log2 of sum_v exp(z_v)
      opaque(x);

      // per-token scalars (every thread computes them; they are uniform)
      tok = tokens[j];
      const bool tok_ok = tok >= 0 && tok < vocab;
      const float zt = tok_ok ? __uint_as_float((uint32_t)logits[(size_t)j * row_stride + tok] << 16)
                              : __builtin_nanf("");
      const float lp = zt - lse2 * kLn2;
      const float old = old_logp[j];
      const float a = teacher_logp[j] - old;
      const float r = lp - old;
      const float rc = fminf(fmaxf(r, -prm.clip_log), prm.clip_log);
      const float rho = expf(rc);
      const float drho = (r > -prm.clip_log && r < prm.clip_log) ? rho : 0.f;
      float l, dl;
      dual_clip_loss(rho, a, prm, &l, &dl);
      g = weight[j] * dl * drho;
      if (t == 0) {
        if (token_logp != nullptr) token_logp[j] = lp;
        token_loss[j] = l;
      }
    } else if (t == 0) {  // no loss, no gradient, logits not read
      if (token_logp != nullptr) token_logp[j] = 0.f;
      token_loss[j] = 0.f;
    }

    // gradient row g (onehot(tok) - exp(z - lse)); zeros when g = 0 (masked
    // rows, flat clipping regimes); then the next row's chunk k into x[k]
    const bool has_grad = grad != nullptr;
    const __amdgpu_buffer_rsrc_t gr = row_rsrc(has_grad ? grad + (size_t)j * grad_stride : grad, store_bytes);
    const __amdgpu_buffer_rsrc_t nr = row_rsrc(logits + (size_t)(next_sup ? jn : j) * row_stride, load_bytes);
    const float ng = -g;
    // Every load of this row has landed (the passes above read them); saying
    // so here lets the compiler issue the chunk-by-chunk refills below without
    // waiting on each other (on the masked-row path it could not tell).
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
#pragma unroll
    for (int k = 0; k < C; ++k) {
      const int q = t + k * kRowThreads;
      if (has_grad) {
        u32x4 o = {0u, 0u, 0u, 0u};
        if (g != 0.f) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            o[i] = pack_bf16x2(ng * __builtin_amdgcn_exp2f(fmaf(lo_bf16(x[k][i]), kLog2e, -lse2)),
                               ng * __builtin_amdgcn_exp2f(fmaf(hi_bf16(x[k][i]), kLog2e, -lse2)));
          if (q == tok / kChunk) {  // the sampled token's entry: g (1 - p)
            const int e = tok - q * kChunk;
            const uint32_t w = o[e >> 1];
            const float zv = (e & 1) ? hi_bf16(x[k][e >> 1]) : lo_bf16(x[k][e >> 1]);
            const float gv = fmaf(ng, __builtin_amdgcn_exp2f(fmaf(zv, kLog2e, -lse2)), g);
            const uint32_t hv = pack_bf16x2(gv, gv) & 0xffffu;
            o[e >> 1] = (e & 1) ? (w & 0xffffu) | (hv << 16) : (w & 0xffff0000u) | hv;
          }
        }
        if (k < C - 1 || q < nwhole) {
          __builtin_amdgcn_raw_buffer_store_b128(
              __builtin_bit_cast(__attribute__((ext_vector_type(4))) unsigned, o), gr, vo + k * kRowThreads * 16, 0,
              kNonTemporal);
        } else if (q == nwhole && nwhole < nchunks) {  // the partial chunk: its columns below vocab
          uint16_t* gp = grad + (size_t)j * grad_stride + (size_t)nwhole * kChunk;
          for (int e = 0; e < vocab - nwhole * kChunk; ++e)
            gp[e] = (uint16_t)(e & 1 ? o[e >> 1] >> 16 : o[e >> 1] & 0xffffu);
        }
      }
      if (next_sup)
        x[k] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(nr, vo + k * kRowThreads * 16, 0,
                                                                                kNonTemporal));
      // keep the refill of x[k] after its last use: hoisting the loads would
      // need a second row's worth of registers
      __builtin_amdgcn_sched_barrier(0);
    }
    sup = next_sup;
  }
}

__global__ __launch_bounds__(1024) void opd_reduce_kernel(const float* __restrict__ weight,
                                                          const float* __restrict__ token_loss,
                                                          int32_t n, float* __restrict__ loss) {
  __shared__ double red[16];
  double acc = 0.0;
  for (int j = threadIdx.x; j < n; j += 1024) acc += (double)weight[j] * (double)token_loss[j];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int w = 0; w < 16; ++w) t += red[w];
    *loss = (float)t;
  }
}

int fail(int code, const char* fmt, ...) {
  char msg[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(msg, sizeof msg, fmt, ap);
  va_end(ap);
  return ctx_report_error(code, msg);
}

bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

template <int C>
void launch_rows(int32_t n, int grid, hipStream_t s, const uint16_t* logits, int64_t stride, int32_t vocab,
                 const int32_t* tokens, const float* old_lp, const float* tea_lp, const uint8_t* mask,
                 const float* weight, OpdParams prm, float* token_logp, float* token_loss, uint16_t* grad,
                 int64_t grad_stride) {
  hipLaunchKernelGGL(opd_row_kernel<C>, dim3((unsigned)grid), dim3(kRowThreads), 0, s, logits, stride, vocab, n,
                     tokens, old_lp, tea_lp, mask, weight, prm, token_logp, token_loss, grad, grad_stride);
}

}  // namespace

extern "C" int ctx_opd_loss_run(const void* logits, int64_t row_stride, int32_t vocab, const int32_t* tokens,
                                const float* old_logp, const float* teacher_logp, const uint8_t* mask,
                                const int32_t* seq_starts, int32_t num_seqs, int32_t num_tokens,
                                const ctx_opd_loss_params* params, float* token_logp, float* token_weight,
                                float* token_loss, float* loss, void* grad_logits, int64_t grad_row_stride,
                                void* stream) {
  ctx_clear_error();
  if (params == nullptr) return fail(CTX_ERR_INVALID_ARG, "params is NULL");
  const ctx_opd_loss_params p = *params;
  if (!(std::isfinite(p.log_ratio_clip) && p.log_ratio_clip > 0.f))
    return fail(CTX_ERR_INVALID_ARG, "log_ratio_clip must be finite and > 0");
  if (!(std::isfinite(p.clip_delta) && p.clip_delta >= 0.f && p.clip_delta < 1.f))
    return fail(CTX_ERR_INVALID_ARG, "clip_delta must be in [0, 1)");
  if (!(std::isfinite(p.dual_clip) && p.dual_clip > 1.f))
    return fail(CTX_ERR_INVALID_ARG, "dual_clip must be finite and > 1");
  if (!(std::isfinite(p.eps) && p.eps >= 0.f)) return fail(CTX_ERR_INVALID_ARG, "eps must be finite and >= 0");
  if (num_seqs < 0 || num_tokens < 0) return fail(CTX_ERR_INVALID_ARG, "negative num_seqs or num_tokens");
  if (num_seqs == 0 && num_tokens > 0) return fail(CTX_ERR_INVALID_ARG, "tokens without responses");
  if (vocab <= 0) return fail(CTX_ERR_INVALID_ARG, "vocab %d <= 0", vocab);
  if (vocab > kMaxVocab) return fail(CTX_ERR_UNSUPPORTED, "vocab %d > %lld", vocab, (long long)kMaxVocab);
  if (row_stride < vocab || row_stride % kChunk != 0)
    return fail(CTX_ERR_INVALID_ARG, "row_stride %lld must be >= vocab and a multiple of 8", (long long)row_stride);
  if (loss == nullptr || seq_starts == nullptr) return fail(CTX_ERR_INVALID_ARG, "NULL loss or seq_starts");
  // per-token arrays of an empty batch are never touched and may be NULL
  if (num_tokens > 0 && (token_weight == nullptr || token_loss == nullptr))
    return fail(CTX_ERR_INVALID_ARG, "NULL token_weight or token_loss");
  if (num_tokens > 0 && (logits == nullptr || tokens == nullptr || old_logp == nullptr ||
                         teacher_logp == nullptr || mask == nullptr))
    return fail(CTX_ERR_INVALID_ARG, "NULL per-token input");
  if (grad_logits != nullptr && (grad_row_stride < vocab || grad_row_stride % kChunk != 0))
    return fail(CTX_ERR_INVALID_ARG, "grad_row_stride %lld must be >= vocab and a multiple of 8",
                (long long)grad_row_stride);
  if ((logits != nullptr && !aligned16(logits)) || (grad_logits != nullptr && !aligned16(grad_logits)))
    return fail(CTX_ERR_ALIGNMENT, "logits and grad_logits must be 16-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const OpdParams prm{p.log_ratio_clip, p.clip_delta, p.dual_clip, p.eps};
  if (num_tokens > 0) {
    hipLaunchKernelGGL(opd_weight_kernel, dim3((unsigned)num_seqs), dim3(256), 0, s, mask, seq_starts, num_seqs,
                       p.eps, token_weight);
    const int64_t per_thread = ((int64_t)vocab + kChunk * kRowThreads - 1) / (kChunk * kRowThreads);
    // one resident workgroup per CU (about 128 VGPRs x 16 waves fill it)
    int device = 0, cus = 0;
    hipError_t e = hipGetDevice(&device);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
    if (e != hipSuccess) return fail(CTX_ERR_HIP, "device query: %s", hipGetErrorString(e));
    const int grid = num_tokens < cus ? num_tokens : cus;
    const uint16_t* lg = static_cast<const uint16_t*>(logits);
    uint16_t* gr = static_cast<uint16_t*>(grad_logits);
#define CTX_OPD_ROWS(C)                                                                                 \
  launch_rows<C>(num_tokens, grid, s, lg, row_stride, vocab, tokens, old_logp, teacher_logp, mask, token_weight, \
                 prm, token_logp, token_loss, gr, grad_row_stride)
    switch (per_thread) {  // exactly ceil(chunks / 1024) chunks per thread
      case 1: CTX_OPD_ROWS(1); break;
      case 2: CTX_OPD_ROWS(2); break;
      case 3: CTX_OPD_ROWS(3); break;
      case 4: CTX_OPD_ROWS(4); break;
      case 5: CTX_OPD_ROWS(5); break;
      case 6: CTX_OPD_ROWS(6); break;
      case 7: CTX_OPD_ROWS(7); break;
      case 8: CTX_OPD_ROWS(8); break;
      case 9: CTX_OPD_ROWS(9); break;
      case 10: CTX_OPD_ROWS(10); break;
      case 11: CTX_OPD_ROWS(11); break;
      case 12: CTX_OPD_ROWS(12); break;
      case 13: CTX_OPD_ROWS(13); break;
      case 14: CTX_OPD_ROWS(14); break;
      case 15: CTX_OPD_ROWS(15); break;
      case 16: CTX_OPD_ROWS(16); break;
      case 17: CTX_OPD_ROWS(17); break;
      case 18: CTX_OPD_ROWS(18); break;
      default: CTX_OPD_ROWS(19); break;
    }
#undef CTX_OPD_ROWS
  }
  hipLaunchKernelGGL(opd_reduce_kernel, dim3(1), dim3(1024), 0, s, token_weight, token_loss, num_tokens, loss);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(CTX_ERR_HIP, "kernel launch: %s", hipGetErrorString(e));
  return CTX_OK;
}
