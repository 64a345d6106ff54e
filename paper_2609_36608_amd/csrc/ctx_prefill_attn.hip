// ctx_prefill_attn.hip -- causal prefill attention for gfx950 (MI355X),
// behind ctx_prefill_attn_run in the C ABI declared in include/ctx_decode_attn.h.
//
// Causal prefill of each sequence's newest tokens (the reference next
// observation the fast action conditions on) against its cache, which already
// holds their K/V rows.  The columns of the 16-column MFMA tiles are the
// consecutive (query position, head) pairs of one KV group, column c being
// position c / g and head c % g, so every column carries work for any group
// size g (a position's heads may straddle two workgroups).  A workgroup of kPrefillWaves waves covers kPrefillCols
// columns of one (sequence, KV head) and streams 32-token K/V blocks, up to
// its last query position, through a three-stage LDS tile that all its
// waves share; the blocks are loaded straight into LDS, two blocks ahead of
// the math.  Per 32 tokens and 16 columns a wave computes
//   S^T = K Q^T                 (8 MFMA 16x16x32, K rows straight from LDS)
//   causal mask, lazy online softmax
//   O^T += V^T P^T              (8 MFMA 16x16x32 per bf16 term of P)
// where the V^T operand comes from the row-major LDS tile through the LDS
// transpose read, whose 4 values per lane are tokens 4c..4c+3 of one
// dimension -- the rows the S^T tile gives each lane.  P enters the product
// either as one bf16 term (rounded to nearest even; the row sum is taken over
// the rounded weights, so each output row stays a convex combination of V
// rows) or, with CTX_PREFILL_SPLIT_P, as P_hi + P_lo (16 significant bits, a
// second set of 8 MFMAs).

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "ctx_attn_common.h"

namespace {

// K/V block loads use the default (cached) policy: the query tiles of one
// (sequence, KV head) re-read the same blocks, mostly from L2.
constexpr int kPrefillLoadAux = 0;

constexpr int kWaitVmcnt0 = 0x0F70;  // s_waitcnt vmcnt(0), expcnt and lgkmcnt left open
typedef __attribute__((address_space(3))) void lds_void;
constexpr int kPrefillWaves = 4;  // waves per workgroup
constexpr int kPrefillTiles = 3;  // 16-column tiles per wave
constexpr int kPrefillCols = kPrefillWaves * kPrefillTiles * 16;
constexpr int kPrefillBlock = 32;  // tokens per LDS stage
// 16-byte chunks each thread stages per K (and per V) block
constexpr int kPrefillLoads = kPrefillBlock * 16 / (64 * kPrefillWaves);
// s_waitcnt vmcnt(N): all but this wave's N most recent loads (one block) have landed
constexpr int kWaitVmcnt4p = 0x0F70 | (2 * kPrefillLoads);
static_assert(kPrefillLoads >= 1 && kPrefillLoads * 64 * kPrefillWaves == kPrefillBlock * 16,
              "the workgroup must tile a block's chunks exactly");

struct PrefillPlan {
  int32_t hq;
  int32_t hkv;
  int32_t group;
  int32_t tiles;  // workgroups per (sequence, KV head)
  int32_t units;  // sequences x KV heads
  float scale_log2;
};

// Workgroup barrier with no memory fence: the caller has already waited for
// its own loads into LDS that the other waves will read, and a fence would
// also wait for the loads of later blocks still in flight.  The memory clobber
// keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Split a pair of non-negative floats into bf16 hi = the value with its low 16
// bits cleared and bf16 lo = round-to-nearest-even of the exact remainder, so
// that hi + lo carries 16 significant bits; both packed as (a, b).
__device__ __forceinline__ void split_bf16x2(float a, float b, uint32_t* hi, uint32_t* lo) {
  const uint32_t ua = __float_as_uint(a), ub = __float_as_uint(b);
  *hi = __builtin_amdgcn_perm(ub, ua, 0x07060302u);  // high halves of a and b
  *lo = pack_bf16x2(a - __uint_as_float(ua & 0xffff0000u), b - __uint_as_float(ub & 0xffff0000u));
}

// Largest of 8 logits with the NaN-propagating maximum, which gfx950 has as a
// three-input instruction (fmaxf would first quiet each input).  A NaN logit
// gives a NaN weight either way.
__device__ __forceinline__ float max8(float a, float b, float c, float d, float e, float f, float g, float h) {
  const auto mx = [](float x, float y) { return __builtin_elementwise_maximum(x, y); };
  // grouped so that the three-input form covers it in 4 instructions
  return mx(mx(mx(mx(a, b), c), mx(mx(d, e), f)), mx(g, h));
}

template <typename OutT, bool kSplitP>
__global__ __launch_bounds__(64 * kPrefillWaves) __attribute__((amdgpu_waves_per_eu(2))) void prefill_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc,
    const int32_t* __restrict__ offs, const int32_t* __restrict__ lens,
    const int32_t* __restrict__ q_starts, const int32_t* __restrict__ q_lens, PrefillPlan pp,
    OutT* __restrict__ out) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 15;
  const int c = lane >> 4;
  const int g = pp.group;
  // consecutive workgroups go to different XCDs; keep every tile of a unit on
  // one XCD so that its L2 serves the tiles' re-reads of the unit's K/V
  const int slot = blockIdx.x / kXcds;
  const int tile = slot % pp.tiles;
  const int unit = (slot / pp.tiles) * kXcds + (int)(blockIdx.x % kXcds);
  if (unit >= pp.units) return;
  const int kv = unit % pp.hkv;
  const int b = unit / pp.hkv;
  const int nq = q_lens[b];
  // query positions of the workgroup's columns, tile * kPrefillCols onwards
  const int first_q = tile * kPrefillCols / g;
  if (first_q >= nq) return;  // the whole workgroup: nothing to do
  const int seq_len = lens[b];
  const int hist = seq_len - nq;  // position of query 0
  // one past the last column's position; min(q_end, nq) - 1 rather than
  // min(q_end - 1, nq - 1), a form that compiles to 8 more registers
  const int q_end = (tile * kPrefillCols + kPrefillCols - 1) / g + 1;
  const int last_q = (q_end < nq ? q_end : nq) - 1;
  const int kv_end = hist + last_q + 1;  // tokens any query of the workgroup attends to
  const size_t row_elems = (size_t)pp.hkv * kHeadDim;
  const int row_bytes = (int)(row_elems * 2);
  const uint16_t* kseq = kc + (size_t)offs[b] * row_elems + (size_t)kv * kHeadDim;
  const uint16_t* vseq = vc + (size_t)offs[b] * row_elems + (size_t)kv * kHeadDim;

  __shared__ __attribute__((aligned(16))) uint16_t lds_k0[kPrefillBlock * kHeadDim];
  __shared__ __attribute__((aligned(16))) uint16_t lds_v0[kPrefillBlock * kHeadDim];
  __shared__ __attribute__((aligned(16))) uint16_t lds_k1[kPrefillBlock * kHeadDim];
  __shared__ __attribute__((aligned(16))) uint16_t lds_v1[kPrefillBlock * kHeadDim];
  __shared__ __attribute__((aligned(16))) uint16_t lds_k2[kPrefillBlock * kHeadDim];
  __shared__ __attribute__((aligned(16))) uint16_t lds_v2[kPrefillBlock * kHeadDim];

  // logits in log2 units are s * cs with cs >= 0: a negative scale flips the
  // sign of q instead (exact in bf16), so that max(s) * cs = max(s * cs)
  const float cs = fabsf(pp.scale_log2);
  const uint32_t qflip = pp.scale_log2 < 0.f ? 0x80008000u : 0u;

  // this lane's query column in each tile: query index qi, head kv * g + hh,
  // attending to positions 0 .. last_pos (columns past the last query attend
  // to the whole block range and are not written)
  int qi[kPrefillTiles], hh[kPrefillTiles], last_pos[kPrefillTiles];
  bf16x8 qb[kPrefillTiles][4];
#pragma unroll
  for (int ct = 0; ct < kPrefillTiles; ++ct) {
    const int col = tile * kPrefillCols + (wave * kPrefillTiles + ct) * 16 + n;
    qi[ct] = col / g;
    hh[ct] = col - qi[ct] * g;
    const bool valid = qi[ct] < nq;
    last_pos[ct] = valid ? hist + qi[ct] : kv_end - 1;
    if (valid) {
      const uint16_t* qrow =
          q + ((size_t)(q_starts[b] + qi[ct]) * pp.hq + (size_t)kv * g + hh[ct]) * kHeadDim + 8 * c;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) qb[ct][kk] = as_bf16x8(load16(qrow + 32 * kk) ^ qflip);
    } else {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) qb[ct][kk] = as_bf16x8(u32x4{0u, 0u, 0u, 0u});
    }
  }
  // the wave's query positions: tokens at or below mask_from are seen by every
  // column; tokens from wave_end on by none (a wave past the last query idles)
  const int wave_q0 = (tile * kPrefillCols + wave * kPrefillTiles * 16) / g;
  const int wave_q1 = (tile * kPrefillCols + (wave + 1) * kPrefillTiles * 16 - 1) / g;
  const bool wave_active = wave_q0 < nq;
  const int mask_from = hist + wave_q0;
  const int wave_end = hist + (wave_q1 < last_q ? wave_q1 : last_q) + 1;

  Softmax st[kPrefillTiles];
  f32x4 o[kPrefillTiles][8];
  // lazy-rescale thresholds: the running max plus 2^8, in log2 units (for
  // masked blocks, whose logits are scaled first) and divided by cs (for the
  // raw logits of unmasked blocks); both move only with the running max
  float thr[kPrefillTiles], thr_raw[kPrefillTiles];
#pragma unroll
  for (int ct = 0; ct < kPrefillTiles; ++ct) {
    thr[ct] = -INFINITY;
    thr_raw[ct] = -INFINITY;
    st[ct] = Softmax{-INFINITY, 0.f};
#pragma unroll
    for (int nb = 0; nb < 8; ++nb) o[ct][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // Block loads go straight from memory into the LDS tile (buffer loads with
  // the LDS flag, no registers held).  Such a load writes lane L's 16 bytes at
  // LDS base + 16 L: wave w's round r fills slots 0..15 of tokens
  // 16 r + 4 w + L / 16, so each lane fetches the chunk that the swizzle puts
  // at its slot.  Past kv_end the buffer bound writes zeros.
  int dvo[kPrefillLoads];
#pragma unroll
  for (int r = 0; r < kPrefillLoads; ++r) {
    const int t = (tid >> 4) + r * 4 * kPrefillWaves;
    dvo[r] = t * row_bytes + (((tid & 15) ^ tile_swizzle(t)) << 4);
  }
  auto issue = [&](int tb, uint16_t* dk, uint16_t* dv) {
    // a block past kv_end gets an empty range: no memory access, zeros in LDS
    const int rem = kv_end - tb;
    const uint32_t bytes = (uint32_t)((rem <= 0 ? 0 : rem < kPrefillBlock ? rem : kPrefillBlock) * row_bytes);
    const __amdgpu_buffer_rsrc_t rk = make_rsrc(kseq + (size_t)tb * row_elems, bytes);
    const __amdgpu_buffer_rsrc_t rv = make_rsrc(vseq + (size_t)tb * row_elems, bytes);
#pragma unroll
    for (int r = 0; r < kPrefillLoads; ++r) {
      const int row0 = r * 4 * kPrefillWaves + 4 * wave;  // first token row of this wave's round
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void*)&dk[row0 * kHeadDim], 16, dvo[r], 0, 0, kPrefillLoadAux);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void*)&dv[row0 * kHeadDim], 16, dvo[r], 0, 0, kPrefillLoadAux);
    }
  };
  issue(0, lds_k0, lds_v0);
  issue(kPrefillBlock, lds_k1, lds_v1);

  // per-lane LDS offsets of the operand reads within a 16-token half block
  int k_off[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) k_off[kk] = n * kHeadDim + (((4 * kk + c) ^ tile_swizzle(n)) << 3);
  const int v_tok = 4 * c + (n >> 2);
  const int v_row = v_tok * kHeadDim + 4 * (n & 1);
  const int v_swz = tile_swizzle(v_tok);
  const int v_ch = (n & 3) >> 1;

  // One 32-token block: wait for this wave's loads of it, then the barrier
  // (every wave's loads have landed, and every wave is done with the stage
  // read in the previous step); the loads of the block two ahead go into that
  // stage, in flight for two steps of math.  The three stages are distinct LDS
  // arrays named at compile time, so the compiler's wait before the reads
  // covers only this stage's loads.
  auto step = [&](int t0, const uint16_t* kt, const uint16_t* vt, uint16_t* nk, uint16_t* nv) {
    // Every step issues the loads of the block two ahead (an empty range past
    // kv_end), so this wave's loads of this block are all but its newest
    // block's worth; the barrier then makes everyone's visible.
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt4p);
    lds_barrier();
    issue(t0 + 2 * kPrefillBlock, nk, nv);
    if (wave_active && t0 < wave_end) {
      // S^T of tokens t0 + 16 h + 4c + i (i < 4) for every column tile
      f32x4 sc[kPrefillTiles][2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        u32x4 kr[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          kr[kk] = *reinterpret_cast<const u32x4*>(kt + 16 * h * kHeadDim + k_off[kk]);
#pragma unroll
        for (int ct = 0; ct < kPrefillTiles; ++ct) sc[ct][h] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
#pragma unroll
          for (int ct = 0; ct < kPrefillTiles; ++ct)
            sc[ct][h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kr[kk]), qb[ct][kk], sc[ct][h], 0, 0, 0);
      }
      const bool masked = t0 + kPrefillBlock - 1 > mask_from;
      u32x4 phi[kPrefillTiles], plo[kPrefillTiles];
#pragma unroll
      for (int ct = 0; ct < kPrefillTiles; ++ct) {
        float x[8];
        float lmax;
        bool grow;
        if (masked) {  // blocks on the causal diagonal (or past kv_end)
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              x[4 * h + i] = (t0 + 16 * h + 4 * c + i > last_pos[ct]) ? -INFINITY : sc[ct][h][i] * cs;
          lmax = max8(x[0], x[1], x[2], x[3], x[4], x[5], x[6], x[7]);
          grow = lmax > thr[ct];
        } else {
          const f32x4 a = sc[ct][0], e = sc[ct][1];
          lmax = max8(a[0], a[1], a[2], a[3], e[0], e[1], e[2], e[3]);
          grow = lmax > thr_raw[ct];
        }
        // lazy rescale: only when some logit exceeds the running max by 2^8;
        // the column max (across the 4 lanes of a column) only then
        if (__any(grow)) {
          if (!masked) lmax *= cs;
          float mx = fmaxf(lmax, __shfl_xor(lmax, 16));
          mx = fmaxf(mx, __shfl_xor(mx, 32));
          const float m_new = fmaxf(st[ct].m, mx);
          const float alpha = fast_exp2(st[ct].m - m_new);
          st[ct].l *= alpha;
#pragma unroll
          for (int nb = 0; nb < 8; ++nb) o[ct][nb] *= alpha;
          st[ct].m = m_new;
          thr[ct] = m_new + kLazyRescale;
          thr_raw[ct] = thr[ct] / cs;  // +inf for a zero scale: all logits are 0 then
        }
        float pr[8];
        if (masked) {
#pragma unroll
          for (int i = 0; i < 8; ++i) pr[i] = fast_exp2(x[i] - st[ct].m);
        } else {
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int i = 0; i < 4; ++i) pr[4 * h + i] = fast_exp2(fmaf(sc[ct][h][i], cs, -st[ct].m));
        }
        if (kSplitP) {
          st[ct].l += ((pr[0] + pr[1]) + (pr[2] + pr[3])) + ((pr[4] + pr[5]) + (pr[6] + pr[7]));
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            uint32_t hw, lw;
            split_bf16x2(pr[2 * j], pr[2 * j + 1], &hw, &lw);
            phi[ct][j] = hw;
            plo[ct][j] = lw;
          }
        } else {
          // one bf16 term; the row sum adds the rounded weights the product
          // uses, a pair per dot product with (1, 1)
          const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
          float l = st[ct].l;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const bf16x2 pair = {(__bf16)pr[2 * j], (__bf16)pr[2 * j + 1]};  // round to nearest even
            phi[ct][j] = __builtin_bit_cast(uint32_t, pair);
            l = __builtin_amdgcn_fdot2_f32_bf16(pair, ones, l, false);
          }
          st[ct].l = l;
        }
      }
      // O^T += V^T P^T: the K dimension holds tokens 4c..4c+3 of both halves.
      // The MFMA stream runs at raised wave priority, so that the other wave
      // on this SIMD fills the matrix core's issue gaps with its softmax.
      __builtin_amdgcn_s_setprio(1);
      // The V^T reads of dimension group nb + 1 are issued before the
      // products of group nb (the scheduling barrier keeps the compiler from
      // sinking them to their use), so their latency hides behind those.
      auto read_vt = [&](int nb, s16x4& v0, s16x4& v1) {
        const int off = v_row + (((2 * nb + v_ch) ^ v_swz) << 3);
        v0 = lds_read_tr16(vt + off);
        v1 = lds_read_tr16(vt + 16 * kHeadDim + off);
      };
      s16x4 nv0, nv1;
      read_vt(0, nv0, nv1);
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) {
        const bf16x8 va = __builtin_bit_cast(bf16x8, __builtin_shufflevector(nv0, nv1, 0, 1, 2, 3, 4, 5, 6, 7));
        if (nb + 1 < 8) read_vt(nb + 1, nv0, nv1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int ct = 0; ct < kPrefillTiles; ++ct)
          o[ct][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, as_bf16x8(phi[ct]), o[ct][nb], 0, 0, 0);
        if (kSplitP) {
#pragma unroll
          for (int ct = 0; ct < kPrefillTiles; ++ct)
            o[ct][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, as_bf16x8(plo[ct]), o[ct][nb], 0, 0, 0);
        }
      }
      __builtin_amdgcn_s_setprio(0);
    }
  };
  // block j in stage j % 3; step j issues block j + 2 into stage (j + 2) % 3
  for (int t0 = 0; t0 < kv_end; t0 += 3 * kPrefillBlock) {
    step(t0, lds_k0, lds_v0, lds_k2, lds_v2);
    if (t0 + kPrefillBlock >= kv_end) break;
    step(t0 + kPrefillBlock, lds_k1, lds_v1, lds_k0, lds_v0);
    if (t0 + 2 * kPrefillBlock >= kv_end) break;
    step(t0 + 2 * kPrefillBlock, lds_k2, lds_v2, lds_k1, lds_v1);
  }
  // no load may land in LDS after the workgroup has released it
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);

#pragma unroll
  for (int ct = 0; ct < kPrefillTiles; ++ct) {
    float l_tot = st[ct].l + __shfl_xor(st[ct].l, 16);
    l_tot += __shfl_xor(l_tot, 32);
    if (qi[ct] < nq) {
      const float inv = 1.0f / l_tot;
      OutT* orow = out + ((size_t)(q_starts[b] + qi[ct]) * pp.hq + (size_t)kv * g + hh[ct]) * kHeadDim + 4 * c;
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) store4<OutT>(orow + 16 * nb, o[ct][nb] * inv);
    }
  }
}

}  // namespace

extern "C" int ctx_prefill_attn_run(ctx_decode_attn* h, const void* q, const void* k_cache, const void* v_cache,
                         const int32_t* seq_offsets, const int32_t* seq_lens, const int32_t* q_starts,
                         const int32_t* q_lens, int32_t num_seqs, int32_t max_q_len, float scale,
                         uint32_t flags, void* out, void* stream) {
  int rc = check_common(h, num_seqs, scale);
  if (rc != CTX_OK) return rc;
  const ctx_decode_attn_desc& d = h->desc;
  const int g = d.num_q_heads / d.num_kv_heads;
  if (max_q_len < 0) return fail(CTX_ERR_INVALID_ARG, "max_q_len %d < 0", max_q_len);
  if ((flags & ~CTX_PREFILL_SPLIT_P) != 0) return fail(CTX_ERR_INVALID_ARG, "unknown prefill flags 0x%x", flags);
  if (num_seqs == 0 || max_q_len == 0) return CTX_OK;
  if (q == nullptr || k_cache == nullptr || v_cache == nullptr || seq_offsets == nullptr ||
      seq_lens == nullptr || q_starts == nullptr || q_lens == nullptr || out == nullptr)
    return fail(CTX_ERR_INVALID_ARG, "NULL data pointer");
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out))
    return fail(CTX_ERR_ALIGNMENT, "q, k_cache, v_cache and out must be 16-byte aligned");
  rc = check_device(h);
  if (rc != CTX_OK) return rc;
  PrefillPlan pp;
  pp.hq = d.num_q_heads;
  pp.hkv = d.num_kv_heads;
  pp.group = g;
  pp.tiles = (int32_t)(((int64_t)max_q_len * g + kPrefillCols - 1) / kPrefillCols);
  pp.scale_log2 = (float)((double)scale * 1.4426950408889634);
  pp.units = num_seqs * d.num_kv_heads;
  const int64_t blocks = round_up(pp.units, kXcds) * pp.tiles;  // units padded to whole XCD rounds
  if (blocks > INT32_MAX) return fail(CTX_ERR_INVALID_ARG, "prefill grid too large");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const uint16_t* qp = static_cast<const uint16_t*>(q);
  const uint16_t* kp = static_cast<const uint16_t*>(k_cache);
  const uint16_t* vp = static_cast<const uint16_t*>(v_cache);
  const dim3 grid((unsigned)blocks), block(64 * kPrefillWaves);
  const bool split_p = (flags & CTX_PREFILL_SPLIT_P) != 0;
  if (d.out_dtype == CTX_DTYPE_F32) {
    float* op = static_cast<float*>(out);
    if (split_p)
      hipLaunchKernelGGL((prefill_kernel<float, true>), grid, block, 0, s, qp, kp, vp, seq_offsets, seq_lens,
                         q_starts, q_lens, pp, op);
    else
      hipLaunchKernelGGL((prefill_kernel<float, false>), grid, block, 0, s, qp, kp, vp, seq_offsets, seq_lens,
                         q_starts, q_lens, pp, op);
  } else {
    uint16_t* op = static_cast<uint16_t*>(out);
    if (split_p)
      hipLaunchKernelGGL((prefill_kernel<uint16_t, true>), grid, block, 0, s, qp, kp, vp, seq_offsets, seq_lens,
                         q_starts, q_lens, pp, op);
    else
      hipLaunchKernelGGL((prefill_kernel<uint16_t, false>), grid, block, 0, s, qp, kp, vp, seq_offsets,
                         seq_lens, q_starts, q_lens, pp, op);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return CTX_OK;
}
