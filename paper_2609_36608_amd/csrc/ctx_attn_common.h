// ctx_attn_common.h -- device helpers, the handle and host-side checks shared
// by the attention translation units of the library (decode-step split and
// merge in ctx_decode_attn.hip, causal prefill in ctx_prefill_attn.hip).
// Internal: not part of the C ABI.
#ifndef CTX_ATTN_COMMON_H_
#define CTX_ATTN_COMMON_H_

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>

#include "ctx_decode_attn.h"

// the library's per-thread last-error message (defined with the decode entry points)
__attribute__((visibility("hidden"))) int ctx_report_error(int code, const char* msg);
__attribute__((visibility("hidden"))) void ctx_clear_error();

struct ctx_decode_attn {
  ctx_decode_attn_desc desc;
  int device;
  int num_cus;
  int32_t ranges_auto[2];  // ranges of the balanced split: contiguous, paged layout
  int64_t max_ranges;   // most ranges any run call can use
  int32_t split_wgw;    // waves (KV heads of one range) per split workgroup
  float* o_ws;
  float2* ml_ws;
};

namespace {

constexpr int kHeadDim = 128;
constexpr float kLazyRescale = 8.0f;  // log2 headroom before the running max moves
constexpr int kXcds = 8;              // XCDs per MI355X; workgroups are dealt to them round-robin

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// ------------------------------------------------------------ math helpers

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  bf16x2 v = {(__bf16)a, (__bf16)b};  // round to nearest even
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ s16x4 pack_bf16x4(float a, float b, float c, float d) {
  u32x2 u = {pack_bf16x2(a, b), pack_bf16x2(c, d)};
  return __builtin_bit_cast(s16x4, u);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// LDS transpose read (gfx950): in each 16-lane group, lane l receives element
// l % 4 of the 8-byte rows addressed by lanes l / 4, 4 + l / 4, 8 + l / 4 and
// 12 + l / 4 -- four tokens of one dimension when those rows are four
// dimensions of four consecutive tokens.
__device__ __forceinline__ s16x4 lds_read_tr16(const uint16_t* p) {
  typedef s16x4 __attribute__((address_space(3))) * lds_s16x4;
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4)(p));
}

// Swizzle of the LDS K/V tiles: a tile row holds one token's 16 chunks of 8
// dimensions, chunk ch of token t at slot ch ^ tile_swizzle(t).  Conflict-free
// for the staging writes (16 lanes per token row), the MFMA operand reads of
// one chunk of 16 consecutive tokens (ds_read_b128) and the transpose reads of
// 8 tokens x 2 chunks per 32 lanes (ds_read_b64_tr_b16).
__device__ __forceinline__ int tile_swizzle(int t) { return ((t & 7) << 1) | ((t >> 3) & 1); }

// 16-byte load of data read once (non-temporal)
__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

// Buffer resources: a wave-uniform base and byte size; loads past the size
// return zeros, which covers the ragged last block of a segment.
constexpr int kRsrcWord3 = 0x00020000;  // raw buffer, 32-bit data format
constexpr int kLoadAux = 2;  // cache policy of streamed K/V loads: non-temporal (read once)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const uint16_t* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  const uint64_t u = ((uint64_t)hi << 32) | lo;
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(u), (short)0,
                                           (int)__builtin_amdgcn_readfirstlane(bytes), kRsrcWord3);
}

// Softmax state of one lane: query head n of the group (lanes with n >= g
// carry unused columns), for the 4 tokens 4c..4c+3 of each block.
struct Softmax {
  float m;  // running max (log2 units), uniform over the 4 lanes of a query
  float l;  // this lane's share of the running sum
};

template <typename OutT>
__device__ __forceinline__ void store4(OutT* dst, f32x4 v);

template <>
__device__ __forceinline__ void store4<float>(float* dst, f32x4 v) {
  *reinterpret_cast<f32x4*>(dst) = v;
}

template <>
__device__ __forceinline__ void store4<uint16_t>(uint16_t* dst, f32x4 v) {
  u32x2 u = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
  *reinterpret_cast<u32x2*>(dst) = u;
}

template <typename OutT>
__device__ __forceinline__ void store2(OutT* dst, float a, float b);

template <>
__device__ __forceinline__ void store2<float>(float* dst, float a, float b) {
  *reinterpret_cast<float2*>(dst) = make_float2(a, b);
}

template <>
__device__ __forceinline__ void store2<uint16_t>(uint16_t* dst, float a, float b) {
  *reinterpret_cast<uint32_t*>(dst) = pack_bf16x2(a, b);
}

// ------------------------------------------------------------ host helpers

int fail(int code, const char* fmt, ...) {
  char msg[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(msg, sizeof msg, fmt, ap);
  va_end(ap);
  return ctx_report_error(code, msg);
}

int hip_fail(hipError_t e, const char* what) {
  return fail(CTX_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// Checks shared by every call on a handle; they clear the last error first.
int check_common(ctx_decode_attn* h, int32_t num_seqs, float scale) {
  ctx_clear_error();
  if (h == nullptr) return fail(CTX_ERR_INVALID_ARG, "handle is NULL");
  if (num_seqs < 0) return fail(CTX_ERR_INVALID_ARG, "num_seqs %d < 0", num_seqs);
  if (num_seqs > h->desc.max_batch)
    return fail(CTX_ERR_CAPACITY, "num_seqs %d > max_batch %d", num_seqs, h->desc.max_batch);
  if (!std::isfinite(scale)) return fail(CTX_ERR_INVALID_ARG, "scale is not finite");
  return CTX_OK;
}

int check_device(ctx_decode_attn* h) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != h->device)
    return fail(CTX_ERR_INVALID_ARG, "current device %d is not the handle's device %d", dev, h->device);
  return CTX_OK;
}

}  // namespace

#endif  // CTX_ATTN_COMMON_H_
