// ctx_decode_attn.hip -- decode-step GQA attention over ragged KV caches for
// gfx950 (MI355X), behind the C ABI declared in include/ctx_decode_attn.h.
//
// One decode step: every request's new token (Hq query heads) attends over the
// request's token context c_{t,j} (Sec. 3, eq:token-context), i.e. its rows of
// a shared [R, Hkv, D] bf16 cache; query head h reads KV head h / g.
//
// Design (flash-decoding split-K, register resident):
//   * Work split.  The batch's tokens, flattened sequence after sequence, are
//     cut into equal ranges, one wave per (range, KV head), sized so the
//     whole grid is resident at once; a workgroup holds the waves of up to 8
//     KV heads of one range (whole 2 KiB token rows for Hkv = 8), each with
//     its own LDS tiles.  Every wave derives its ranges from seq_lens on the device,
//     so no host sync is needed and the call is graph-capturable.  A range
//     that holds a whole sequence writes that sequence's output directly;
//     otherwise each piece writes an fp32 partial (m, l, o) to the workspace
//     and a second kernel merges the pieces of each (sequence, head).
//   * Per 16-token block, all g query heads of the KV group are processed at
//     once on the matrix cores:
//       S^T[16 tok x 16]  = K_blk[16 x 128] . Q^T          4 x mfma 16x16x32 bf16
//       O^T[16 dim x 16]  += V^T . [P_hi; P_lo]^T          8 x mfma 16x16x32 bf16
//         (one per 16 dimensions; the K index runs over the 16 tokens twice,
//         against P_hi and P_lo, both bf16, so P keeps ~16 mantissa bits)
//     K and V are read from HBM exactly once, with coalesced 16-byte loads
//     (16 lanes per 256-byte token row), and pass through a wave-private,
//     XOR-swizzled LDS tile: K is read back in the MFMA operand layout, V^T
//     by the LDS transpose read, so every output dimension is computed from
//     its own V column only.
//   * A wave's issue priority falls by quarters of its token range, so that
//     waves dispatched late are not starved by the older ones and the grid
//     drains together.
//   * Online softmax in base 2 (scale * log2 e folded into the fp32 logits)
//     with fp32 running max and sum.  The running max is raised only when a
//     block's maximum exceeds it by more than 2^8, so probabilities stay
//     <= 256 and the rescale of the accumulators is rare; the merge uses the
//     same stale maxima, so the result is unchanged.
//   * Merge: out = sum_s o_s 2^(m_s - M) / sum_s l_s 2^(m_s - M), M = max_s m_s,
//     in fixed segment order (deterministic; no atomics).

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <mutex>
#include <new>

#include "ctx_attn_common.h"

namespace {

constexpr int kBlock = 16;        // tokens per MFMA block
constexpr int kMaxGroup = 16;     // query heads per KV head (MFMA N dimension)
constexpr int kMinRange = 64;     // smallest balanced range, tokens
constexpr int kMergeWaves = 4;
constexpr int kWgWaves = 8;  // most waves (KV heads of one range) per split workgroup
constexpr int kTileBytes = 2 * kBlock * kHeadDim * 2;  // one wave's K and V tiles in LDS
// Waves per SIMD the split kernel is compiled for: 3 for contiguous caches
// (167 VGPRs); the paged kernel's page bookkeeping needs more registers and
// spills at 3, so it is compiled for 2.  An 8-wave workgroup (Hkv = 8) is one
// workgroup per CU either way.
constexpr int kWavesPerEu = 3;
constexpr int kPagedWavesPerEu = 2;

struct Plan {
  int32_t num_seqs;
  int32_t hq;
  int32_t hkv;
  int32_t group;
  int32_t num_ranges;    // ranges in the grid (each = hkv workgroups)
  int32_t forced_width;  // > 0: fixed tokens per range
  int32_t pad;           // sequences occupy round_up(L, pad) tokens of the flattened batch
  float scale_log2;      // scale * log2(e)
};

// Paged layout: token t of sequence b is row block_tables[b][t / P] * P + t % P.
struct Paged {
  const int32_t* block_tables;  // [num_seqs, max_pages]
  int32_t max_pages;
  int32_t page_tokens;          // P, a multiple of kBlock
  const uint16_t* k_new;        // [num_seqs, Hkv, D] appended token, or null
  const uint16_t* v_new;
  uint16_t* k_cache;            // the caches, for writing the appended row
  uint16_t* v_cache;
};

// ------------------------------------------------------------ wave helpers

__device__ __forceinline__ int64_t wave_sum(int64_t x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}

// Tokens a sequence of length len occupies in the flattened batch.  pad is 1
// (contiguous caches) or kBlock (paged), a power of two, so rounding up is a
// mask: a 64-bit division by a run-time value is a long instruction sequence
// on the critical path of every wave's length scan.
__device__ __forceinline__ int64_t padded(int64_t len, int pad) { return (len + pad - 1) & ~(int64_t)(pad - 1); }

// sum of the padded lens[0 .. n)
__device__ __forceinline__ int64_t sum_lens(const int32_t* __restrict__ lens, int n, int lane, int pad) {
  int64_t acc = 0;
  for (int i = lane; i < n; i += 64) acc += padded(lens[i], pad);
  return wave_sum(acc);
}

// First sequence b whose flattened span [P_b, P_b + L_b) contains pos; *start = P_b.
// Returns n if none.
__device__ int find_sequence(const int32_t* __restrict__ lens, int n, int64_t pos, int lane,
                             int64_t* start, int pad) {
  int64_t carry = 0;
  for (int base = 0; base < n; base += 64) {
    const int i = base + lane;
    const int64_t len = i < n ? padded(lens[i], pad) : 0;
    int64_t incl = len;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int64_t y = __shfl_up(incl, off);
      if (lane >= off) incl += y;
    }
    const int64_t excl = incl - len;
    const unsigned long long hit = __ballot(carry + excl <= pos && pos < carry + incl);
    if (hit) {
      const int src = __ffsll(hit) - 1;
      *start = __shfl(carry + excl, src);
      return base + src;
    }
    carry += __shfl(incl, 63);
  }
  *start = carry;
  return n;
}

// Padded lengths of the first 64 sequences, one per lane (0 past n), with their
// inclusive prefix sums: one load round answers totals and offsets for
// batches of up to 64 sequences.
struct LaneScan {
  int64_t len;
  int64_t incl;
};

__device__ __forceinline__ LaneScan scan_lane_lens(const int32_t* __restrict__ lens, int n, int lane,
                                                   int pad) {
  LaneScan r;
  r.len = lane < n ? padded(lens[lane], pad) : 0;
  int64_t incl = r.len;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int64_t y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  r.incl = incl;
  return r;
}

__device__ __forceinline__ int64_t range_width(int64_t total, const Plan& p) {
  if (p.forced_width > 0) return p.forced_width;
  int64_t w = (total + p.num_ranges - 1) / p.num_ranges;
  w = (w + kBlock - 1) / kBlock * kBlock;
  return w < kMinRange ? kMinRange : w;
}

// ------------------------------------------------------------ math helpers

__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kLoadAux));
}

// Process one 16-token block.  `valid` = tokens of the block inside the segment;
// lds_v points at this lane's transpose-read address in the block's V tile
// (token 4c + n / 4, dimensions 4 (n % 4) .. 4 (n % 4) + 3 of dimension group 0),
// v_step(nb) the element offset of dimension group nb from it.
__device__ __forceinline__ void attend_block(const u32x4 (&kr)[4], const uint16_t* lds_v, const int (&v_off)[8],
                                             const bf16x8 (&qb)[4], int valid, int c, float scale_log2,
                                             Softmax& st, f32x4 (&o)[8]) {
  // logits: lane (c, n) gets tokens 4c+i, query n
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < 4; ++kk)
    s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kr[kk]), qb[kk], s, 0, 0, 0);

  float x[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[i] = s[i] * scale_log2;
    if (4 * c + i >= valid) x[i] = -INFINITY;
  }
  float mx = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  if (__any(mx > st.m + kLazyRescale)) {
    const float m_new = fmaxf(st.m, mx);
    const float alpha = fast_exp2(st.m - m_new);  // 0 on the first block (m = -inf)
#pragma unroll
    for (int nb = 0; nb < 8; ++nb) o[nb] *= alpha;
    st.l *= alpha;
    st.m = m_new;
  }
  float p[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) p[i] = fast_exp2(x[i] - st.m);
  st.l += (p[0] + p[1]) + (p[2] + p[3]);

  // P as the B operand of a 16x16x32 MFMA whose K index 8c + j is token 4c + j
  // of P_hi (j < 4) and of P_lo (j >= 4): P = P_hi + P_lo keeps ~16 significant
  // bits, and one product takes both terms.
  float hi[4], lo[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    hi[i] = (float)(__bf16)p[i];
    lo[i] = p[i] - hi[i];
  }
  const s16x4 p_hi = pack_bf16x4(hi[0], hi[1], hi[2], hi[3]);
  const s16x4 p_lo = pack_bf16x4(lo[0], lo[1], lo[2], lo[3]);
  const bf16x8 pb = __builtin_bit_cast(bf16x8, __builtin_shufflevector(p_hi, p_lo, 0, 1, 2, 3, 4, 5, 6, 7));

  // V^T straight from the LDS tile: the transpose read gives lane (c, n)
  // V[token 4c + j][dimension 16 nb + n], j < 4, taken twice (against P_hi and P_lo)
#pragma unroll
  for (int nb = 0; nb < 8; ++nb) {
    const s16x4 vt = lds_read_tr16(lds_v + v_off[nb]);
    const bf16x8 va = __builtin_bit_cast(bf16x8, __builtin_shufflevector(vt, vt, 0, 1, 2, 3, 0, 1, 2, 3));
    o[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb, o[nb], 0, 0, 0);
  }
}


// ------------------------------------------------------------ split kernel

template <typename OutT, bool kPaged>
__global__ __launch_bounds__(64 * kWgWaves) __attribute__((amdgpu_waves_per_eu(kPaged ? kPagedWavesPerEu : kWavesPerEu))) void decode_split_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
    const uint16_t* __restrict__ vc, const int32_t* __restrict__ offs,
    const int32_t* __restrict__ lens, Plan p, Paged pg, float* __restrict__ o_ws,
    float2* __restrict__ ml_ws, OutT* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int n = lane & 15;
  const int c = lane >> 4;
  // A workgroup holds wgw waves, KV heads hg * wgw .. hg * wgw + wgw - 1 of
  // one range w, so that a CU reads several heads' slices of the same token
  // rows at once.  Range-major order: consecutive workgroups take consecutive
  // ranges of one head group.  Workgroups are dealt round-robin over the XCDs
  // (id % kXcds) and num_ranges % kXcds == 0, so every head of a range lands on
  // the same XCD (range w on XCD w % kXcds).  Measured on MI355X this order
  // streams the cache fastest.
  const int wgw = (int)(blockDim.x >> 6);
  const int wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int hg = blockIdx.x / p.num_ranges;
  const int w = blockIdx.x - hg * p.num_ranges;
  const int kv = hg * wgw + wv;
  const int g = p.group;
  // each wave owns a K and a V tile in the workgroup's (dynamic) LDS; its LDS
  // instructions execute in order, so staging a block needs no barrier
  extern __shared__ __attribute__((aligned(16))) uint16_t lds_tiles[];
  uint16_t* lds_k = lds_tiles + (size_t)wv * (kTileBytes / 2);
  uint16_t* lds_v = lds_k + kBlock * kHeadDim;

  // this wave's token range [ws, we) and the first sequence b it overlaps (span starts at pos)
  int64_t total, width, ws, pos;
  int b;
  if (p.num_seqs <= 64) {
    const LaneScan sc = scan_lane_lens(lens, p.num_seqs, lane, p.pad);
    total = __shfl(sc.incl, 63);
    width = range_width(total, p);
    ws = (int64_t)w * width;
    if (ws >= total) return;
    const unsigned long long hit = __ballot(sc.incl - sc.len <= ws && ws < sc.incl);
    b = __ffsll(hit) - 1;
    pos = __shfl(sc.incl - sc.len, b);
  } else {
    total = sum_lens(lens, p.num_seqs, lane, p.pad);
    width = range_width(total, p);
    ws = (int64_t)w * width;
    if (ws >= total) return;
    b = find_sequence(lens, p.num_seqs, ws, lane, &pos, p.pad);
  }
  const int64_t we = ws + width < total ? ws + width : total;

  // LDS offsets of this lane's operand reads: K rows (token n, chunk 4kk + c)
  // and the V transpose reads (token 4c + n / 4, dimensions 16 nb + 4 (n % 4) ..)
  int k_off[4], v_off[8];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) k_off[kk] = n * kHeadDim + (((4 * kk + c) ^ tile_swizzle(n)) << 3);
  {
    const int v_tok = 4 * c + (n >> 2);
#pragma unroll
    for (int nb = 0; nb < 8; ++nb)
      v_off[nb] = v_tok * kHeadDim + (((2 * nb + ((n & 3) >> 1)) ^ tile_swizzle(v_tok)) << 3) + 4 * (n & 1);
  }

  const size_t row_elems = (size_t)p.hkv * kHeadDim;
  while (b < p.num_seqs && pos < we) {
    const int seq_len = lens[b];
    const int64_t s0 = ws > pos ? ws - pos : 0;
    const int64_t s1 = we - pos < seq_len ? we - pos : seq_len;
    if (s1 > s0) {
      const int len = (int)(s1 - s0);
      bf16x8 qb[4];
      if (n < g) {
        const uint16_t* qrow = q + ((size_t)b * p.hq + (size_t)kv * g + n) * kHeadDim + 8 * c;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) qb[kk] = as_bf16x8(load16(qrow + 32 * kk));
      } else {
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) qb[kk] = as_bf16x8(u32x4{0u, 0u, 0u, 0u});
      }
      Softmax st{-INFINITY, 0.f};
      f32x4 o[8];
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) o[nb] = f32x4{0.f, 0.f, 0.f, 0.f};

      const int row_bytes = (int)(row_elems * 2);
      // Contiguous layout: the segment's rows follow each other from row
      // offs[b] + s0.  Paged layout: s0 is a multiple of kBlock (lengths are
      // padded to kBlock in the range plan), so every block lies inside one
      // page; the page numbers of up to 64 pages of the segment are held one
      // per lane and refreshed when the segment runs past them.
      const uint16_t* kseg = kc + (size_t)kv * kHeadDim;
      const uint16_t* vseg = vc + (size_t)kv * kHeadDim;
      int page_lane = 0, page_base = 0;
      if (kPaged) {
        page_base = (int)(s0 / pg.page_tokens);
        const int used = (int)((seq_len + pg.page_tokens - 1) / pg.page_tokens);
        const int j = page_base + lane;
        page_lane = j < used && j < pg.max_pages ? pg.block_tables[(size_t)b * pg.max_pages + j] : 0;
      } else {
        kseg += ((size_t)offs[b] + (size_t)s0) * row_elems;
        vseg += ((size_t)offs[b] + (size_t)s0) * row_elems;
      }
      // the appended token (paged, with k_new): the last token of a sequence
      const bool append = kPaged && pg.k_new != nullptr && s1 == seq_len;

      const int voff = (lane >> 4) * row_bytes + (lane & 15) * 16;
      const int ld_tok = lane >> 4;
      // Coalesced loads: 16 lanes cover one token's 256-byte head slice, four
      // tokens per instruction.  The block goes through a wave-private LDS
      // tile (16-byte chunks XOR-swizzled by token, conflict-free both ways)
      // and is read back in the MFMA operand layout.  The next block's loads
      // are issued as soon as the current block is in LDS, so they are in
      // flight during its math.
      u32x4 pk[4], pv[4];
      // Issue the loads of the block at segment token t into pk, pv and return
      // its first cache row.  Past the segment end the range is empty: the
      // loads return zeros and touch no memory.
      auto issue = [&](int t) __attribute__((always_inline)) -> size_t {
        const int v = len - t < kBlock ? len - t : kBlock;
        size_t row = 0;
        if (v > 0) {
          if (kPaged) {
            const int64_t tok = s0 + t;
            int pj = (int)(tok / pg.page_tokens) - page_base;
            if (pj >= 64) {  // the segment ran past the pages held in registers
              page_base += 64;
              pj -= 64;
              const int used = (int)((seq_len + pg.page_tokens - 1) / pg.page_tokens);
              const int j = page_base + lane;
              page_lane = j < used && j < pg.max_pages ? pg.block_tables[(size_t)b * pg.max_pages + j] : 0;
            }
            const int page = __builtin_amdgcn_readlane(page_lane, pj);
            row = (size_t)page * pg.page_tokens + (size_t)(tok % pg.page_tokens);
          } else {
            row = (size_t)t;
          }
        }
        const uint32_t bytes = v > 0 ? (uint32_t)(v * row_bytes) : 0u;
        const __amdgpu_buffer_rsrc_t rk = make_rsrc(kseg + row * row_elems, bytes);
        const __amdgpu_buffer_rsrc_t rv = make_rsrc(vseg + row * row_elems, bytes);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          pk[u] = buf_load16(rk, voff, 4 * u * row_bytes);
          pv[u] = buf_load16(rv, voff, 4 * u * row_bytes);
        }
        return row;
      };
      size_t blk_row = issue(0);
      for (int t = 0; t < len; t += kBlock) {
        const int valid = len - t < kBlock ? len - t : kBlock;
        {
          // Issue priority falls as the wave works through its range.  Waves
          // dispatched earlier otherwise win the SIMD's arbitration and finish
          // well before the younger ones, leaving the last part of the launch
          // to a few waves; lagging waves now go first, so they finish together.
          const int done = __builtin_amdgcn_readfirstlane((int)(pos + s0 + t - ws));
          const int quarter = __builtin_amdgcn_readfirstlane((int)(width >> 2));
          if (done < quarter) __builtin_amdgcn_s_setprio(3);
          else if (done < 2 * quarter) __builtin_amdgcn_s_setprio(2);
          else if (done < 3 * quarter) __builtin_amdgcn_s_setprio(1);
          else __builtin_amdgcn_s_setprio(0);
        }
        __builtin_amdgcn_wave_barrier();  // keep the previous block's LDS reads before these writes
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int tok = 4 * u + ld_tok;
          const int slot = tok * kHeadDim + (((lane & 15) ^ tile_swizzle(tok)) << 3);
          *reinterpret_cast<u32x4*>(&lds_k[slot]) = pk[u];
          *reinterpret_cast<u32x4*>(&lds_v[slot]) = pv[u];
        }
        if (append && t + kBlock >= len) {
          // the block holding the newest token: attend to the appended row and
          // write it into the cache (16 lanes, 16 bytes each)
          const int tok = valid - 1;
          if (lane < 16) {
            const size_t src = ((size_t)b * p.hkv + kv) * kHeadDim + 8 * lane;
            const u32x4 nk = load16(pg.k_new + src);
            const u32x4 nv = load16(pg.v_new + src);
            const int slot = tok * kHeadDim + ((lane ^ tile_swizzle(tok)) << 3);
            *reinterpret_cast<u32x4*>(&lds_k[slot]) = nk;
            *reinterpret_cast<u32x4*>(&lds_v[slot]) = nv;
            const size_t dst = (blk_row + tok) * row_elems + (size_t)kv * kHeadDim + 8 * lane;
            *reinterpret_cast<u32x4*>(pg.k_cache + dst) = nk;
            *reinterpret_cast<u32x4*>(pg.v_cache + dst) = nv;
          }
        }
        const size_t next_row = issue(t + kBlock);
        __builtin_amdgcn_wave_barrier();
        u32x4 kr[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) kr[kk] = *reinterpret_cast<const u32x4*>(&lds_k[k_off[kk]]);
        attend_block(kr, lds_v, v_off, qb, valid, c, p.scale_log2, st, o);
        blk_row = next_row;
      }

      float l_tot = st.l + __shfl_xor(st.l, 16);
      l_tot += __shfl_xor(l_tot, 32);
      if (s0 == 0 && s1 == seq_len) {
        // the whole sequence is in this range: final output
        if (n < g) {
          const float inv = 1.0f / l_tot;
          OutT* orow = out + ((size_t)b * p.hq + (size_t)kv * g + n) * kHeadDim + 4 * c;
#pragma unroll
          for (int nb = 0; nb < 8; ++nb) store4<OutT>(orow + 16 * nb, o[nb] * inv);
        }
      } else {
        const size_t idx = ((size_t)(w + b) * p.hkv + kv) * g + n;
        if (n < g) {
          float* orow = o_ws + idx * kHeadDim + 4 * c;
#pragma unroll
          for (int nb = 0; nb < 8; ++nb) *reinterpret_cast<f32x4*>(orow + 16 * nb) = o[nb];
          if (c == 0) ml_ws[idx] = make_float2(st.m, l_tot);
        }
      }
    }
    pos += padded(seq_len, p.pad);
    ++b;
  }
}

// ------------------------------------------------------------ merge kernel

__device__ __forceinline__ float lane_value(float x, int src) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), src));
}

// One wave per (sequence, query head); lane l owns dims 2l, 2l+1.  Segment
// weights are computed one segment per lane; partial outputs are read in
// batches of kMergeBatch segments, the next batch in flight while the current
// one is accumulated.
constexpr int kMergeBatch = 16;

__device__ __forceinline__ void load_partials(float2 (&dst)[kMergeBatch], const float* __restrict__ o_ws,
                                              size_t first, size_t stride, int s0, int cnt, int lane) {
#pragma unroll
  for (int u = 0; u < kMergeBatch; ++u)
    dst[u] = s0 + u < cnt
                 ? reinterpret_cast<const float2*>(o_ws + (first + (size_t)(s0 + u) * stride) * kHeadDim)[lane]
                 : make_float2(0.f, 0.f);
}

template <typename OutT>
__global__ __launch_bounds__(64 * kMergeWaves) void decode_merge_kernel(
    const int32_t* __restrict__ lens, Plan p, const float* __restrict__ o_ws,
    const float2* __restrict__ ml_ws, OutT* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int gw = blockIdx.x * kMergeWaves + (threadIdx.x >> 6);
  if (gw >= p.num_seqs * p.hq) return;
  const int b = gw / p.hq;
  const int h = gw - b * p.hq;
  const int kv = h / p.group;
  const int qi = h - kv * p.group;
  int64_t seq_len, total, pos;
  seq_len = lens[b];
  if (p.num_seqs <= 64) {
    const LaneScan sc = scan_lane_lens(lens, p.num_seqs, lane, p.pad);
    total = __shfl(sc.incl, 63);
    pos = __shfl(sc.incl - sc.len, b);
  } else {
    total = sum_lens(lens, p.num_seqs, lane, p.pad);
    pos = sum_lens(lens, b, lane, p.pad);
  }
  float r0 = 0.f, r1 = 0.f;
  if (seq_len > 0) {
    const int64_t width = range_width(total, p);
    const int64_t wf = pos / width;
    int64_t wl = (pos + seq_len - 1) / width;
    if (wf == wl) return;  // written by the split kernel
    // only reachable when seq_lens breaks the max_seq_len contract: stay in the workspace
    if (wl >= p.num_ranges) wl = p.num_ranges - 1;
    const int nseg = (int)(wl - wf + 1);
    // partial (m, l, o) of segment j lives at slot wf + j + b
    const size_t first = ((size_t)(wf + b) * p.hkv + kv) * p.group + qi;
    const size_t stride = (size_t)p.hkv * p.group;
    float2 cur[kMergeBatch];
    load_partials(cur, o_ws, first, stride, 0, nseg < 64 ? nseg : 64, lane);
    const float2 ml0 = lane < nseg ? ml_ws[first + (size_t)lane * stride] : make_float2(-INFINITY, 0.f);
    float m = ml0.x;
    for (int j = lane + 64; j < nseg; j += 64) m = fmaxf(m, ml_ws[first + (size_t)j * stride].x);
    m = wave_max(m);
    float lsum = 0.f;
    for (int base = 0; base < nseg; base += 64) {
      const int cnt = nseg - base < 64 ? nseg - base : 64;
      const float2 ml = base == 0 ? ml0
                                  : (lane < cnt ? ml_ws[first + (size_t)(base + lane) * stride]
                                                : make_float2(-INFINITY, 0.f));
      const float wj = lane < cnt ? fast_exp2(ml.x - m) : 0.f;
      lsum += wj * ml.y;
      if (base > 0) load_partials(cur, o_ws, first + (size_t)base * stride, stride, 0, cnt, lane);
      for (int s0 = 0; s0 < cnt; s0 += kMergeBatch) {
        float2 nxt[kMergeBatch];
        const bool more = s0 + kMergeBatch < cnt;
        if (more) load_partials(nxt, o_ws, first + (size_t)base * stride, stride, s0 + kMergeBatch, cnt, lane);
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) {
          const float wgt = lane_value(wj, (s0 + u) & 63);
          r0 += wgt * cur[u].x;
          r1 += wgt * cur[u].y;
        }
        if (more) {
#pragma unroll
          for (int u = 0; u < kMergeBatch; ++u) cur[u] = nxt[u];
        }
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) lsum += __shfl_xor(lsum, off);
    const float inv = 1.0f / lsum;
    r0 *= inv;
    r1 *= inv;
  }
  store2<OutT>(out + ((size_t)b * p.hq + h) * kHeadDim + 2 * lane, r0, r1);
}

// ------------------------------------------------------------ host side

thread_local char g_last_error[512] = "";

// Waves (KV heads of one range) per split workgroup: 8, 4, 2 or 1, a divisor of Hkv.
int split_waves(int hkv) {
  int wgw = kWgWaves;
  while (hkv % wgw != 0) wgw >>= 1;
  return wgw;
}

// Resident waves per CU of the split kernel for the contiguous ([0]) and
// paged ([1]) layouts with wgw-wave workgroups; they depend on the output
// dtype and wgw only.
int resident_waves(int32_t out_dtype, int wgw, int64_t per_cu[2]) {
  const void* kernels[2] = {
      out_dtype == CTX_DTYPE_F32 ? reinterpret_cast<const void*>(&decode_split_kernel<float, false>)
                                 : reinterpret_cast<const void*>(&decode_split_kernel<uint16_t, false>),
      out_dtype == CTX_DTYPE_F32 ? reinterpret_cast<const void*>(&decode_split_kernel<float, true>)
                                 : reinterpret_cast<const void*>(&decode_split_kernel<uint16_t, true>)};
  for (int layout = 0; layout < 2; ++layout) {
    int n = 0;
    hipError_t e =
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernels[layout], 64 * wgw, (size_t)wgw * kTileBytes);
    if (e != hipSuccess) return hip_fail(e, "hipOccupancyMaxActiveBlocksPerMultiprocessor");
    per_cu[layout] = n < 1 ? 1 : (int64_t)n * wgw;
  }
  return CTX_OK;
}

// Ranges of the balanced split: enough that one wave per (range, KV head) is
// resident at once, in whole multiples of the XCD count.
int64_t ranges_for(int cus, int64_t per_cu, int hkv) {
  const int64_t r = (int64_t)cus * per_cu / hkv / kXcds * kXcds;
  return r < kXcds ? kXcds : r;
}

// Ranges of the balanced split for the contiguous ([0]) and paged ([1]) kernels.
int balanced_ranges(const ctx_decode_attn_desc& d, int cus, int wgw, int64_t ranges[2]) {
  int64_t per_cu[2];
  const int rc = resident_waves(d.out_dtype, wgw, per_cu);
  if (rc != CTX_OK) return rc;
  for (int layout = 0; layout < 2; ++layout) ranges[layout] = ranges_for(cus, per_cu[layout], d.num_kv_heads);
  return CTX_OK;
}

// Checks of a descriptor shared by ctx_decode_attn_create and the
// allocation-free entry point.
int check_desc(const ctx_decode_attn_desc& d) {
  if (d.num_q_heads <= 0 || d.num_kv_heads <= 0)
    return fail(CTX_ERR_INVALID_ARG, "head counts must be positive (Hq=%d, Hkv=%d)",
                d.num_q_heads, d.num_kv_heads);
  if (d.head_dim != kHeadDim)
    return fail(CTX_ERR_UNSUPPORTED, "head_dim %d unsupported (only %d)", d.head_dim, kHeadDim);
  if (d.num_q_heads % d.num_kv_heads != 0)
    return fail(CTX_ERR_UNSUPPORTED, "Hq=%d is not a multiple of Hkv=%d", d.num_q_heads,
                d.num_kv_heads);
  if (d.num_q_heads / d.num_kv_heads > kMaxGroup)
    return fail(CTX_ERR_UNSUPPORTED, "group size %d > %d", d.num_q_heads / d.num_kv_heads,
                kMaxGroup);
  if (d.max_batch <= 0 || d.max_seq_len <= 0)
    return fail(CTX_ERR_INVALID_ARG, "max_batch and max_seq_len must be positive");
  if (d.out_dtype != CTX_DTYPE_BF16 && d.out_dtype != CTX_DTYPE_F32)
    return fail(CTX_ERR_INVALID_ARG, "unknown out_dtype %d", (int)d.out_dtype);
  if (d.split_tokens < 0 || (d.split_tokens > 0 && d.split_tokens < kBlock))
    return fail(CTX_ERR_INVALID_ARG, "split_tokens must be 0 or >= %d", kBlock);
  if (d.page_tokens < 0 || d.page_tokens % kBlock != 0)
    return fail(CTX_ERR_INVALID_ARG, "page_tokens must be 0 or a positive multiple of %d", kBlock);
  if (d.page_tokens > 0 && d.split_tokens % kBlock != 0)
    return fail(CTX_ERR_INVALID_ARG, "with page_tokens, split_tokens must be a multiple of %d", kBlock);
  return CTX_OK;
}

}  // namespace

// The last-error message is shared with the library's other entry points
// (prefill, the OPD loss, the rollout simulator), which report through these
// two functions.
__attribute__((visibility("hidden"))) int ctx_report_error(int code, const char* msg) {
  snprintf(g_last_error, sizeof g_last_error, "%s", msg);
  return code;
}

__attribute__((visibility("hidden"))) void ctx_clear_error() { g_last_error[0] = '\0'; }

extern "C" {

const char* ctx_decode_attn_status_string(int status) {
  switch (status) {
    case CTX_OK: return "ok";
    case CTX_ERR_INVALID_ARG: return "invalid argument";
    case CTX_ERR_UNSUPPORTED: return "unsupported shape";
    case CTX_ERR_CAPACITY: return "num_seqs exceeds max_batch";
    case CTX_ERR_ALIGNMENT: return "pointer not 16-byte aligned";
    case CTX_ERR_HIP: return "HIP runtime error";
    case CTX_ERR_OOM: return "out of device memory";
    default: return "unknown status";
  }
}

const char* ctx_decode_attn_last_error(void) { return g_last_error; }

int ctx_decode_attn_create(const ctx_decode_attn_desc* desc, ctx_decode_attn** out_handle) {
  ctx_clear_error();
  if (out_handle == nullptr) return fail(CTX_ERR_INVALID_ARG, "out_handle is NULL");
  *out_handle = nullptr;
  if (desc == nullptr) return fail(CTX_ERR_INVALID_ARG, "desc is NULL");
  const ctx_decode_attn_desc d = *desc;
  int rc = check_desc(d);
  if (rc != CTX_OK) return rc;

  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  int cus = 0;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
  const int wgw = split_waves(d.num_kv_heads);
  int64_t ranges_auto[2];
  rc = balanced_ranges(d, cus, wgw, ranges_auto);
  if (rc != CTX_OK) return rc;
  int64_t max_ranges = ranges_auto[0] > ranges_auto[1] ? ranges_auto[0] : ranges_auto[1];
  if (d.split_tokens > 0)
    max_ranges = round_up(((int64_t)d.max_batch * round_up(d.max_seq_len, kBlock) + d.split_tokens - 1) /
                              d.split_tokens, kXcds);
  if (max_ranges * d.num_kv_heads > INT32_MAX)
    return fail(CTX_ERR_INVALID_ARG, "split_tokens %d too small for max_batch x max_seq_len",
                d.split_tokens);

  const int64_t slots = max_ranges + d.max_batch;
  const size_t o_bytes = (size_t)slots * d.num_q_heads * kHeadDim * sizeof(float);
  const size_t ml_bytes = (size_t)slots * d.num_q_heads * sizeof(float2);

  ctx_decode_attn* h = new (std::nothrow) ctx_decode_attn{};
  if (h == nullptr) return fail(CTX_ERR_OOM, "host allocation failed");
  h->desc = d;
  h->device = dev;
  h->num_cus = cus;
  h->ranges_auto[0] = (int32_t)ranges_auto[0];
  h->ranges_auto[1] = (int32_t)ranges_auto[1];
  h->max_ranges = max_ranges;
  h->split_wgw = wgw;
  e = hipMalloc(reinterpret_cast<void**>(&h->o_ws), o_bytes);
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&h->ml_ws), ml_bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    if (h->o_ws) (void)hipFree(h->o_ws);
    delete h;
    return fail(CTX_ERR_OOM, "workspace of %zu bytes: %s", o_bytes + ml_bytes, hipGetErrorString(e));
  }
  *out_handle = h;
  return CTX_OK;
}

}  // extern "C"

namespace {

template <bool kPaged>
int launch(ctx_decode_attn* h, const void* q, const void* k, const void* v, const int32_t* offs,
           const int32_t* lens, int32_t num_seqs, float scale, void* out, void* stream, const Paged& pg) {
  const ctx_decode_attn_desc& d = h->desc;
  Plan p;
  p.num_seqs = num_seqs;
  p.hq = d.num_q_heads;
  p.hkv = d.num_kv_heads;
  p.group = d.num_q_heads / d.num_kv_heads;
  p.forced_width = d.split_tokens;
  p.num_ranges = d.split_tokens > 0
                     ? (int32_t)round_up(((int64_t)num_seqs * round_up(d.max_seq_len, kPaged ? kBlock : 1) +
                                          d.split_tokens - 1) / d.split_tokens, kXcds)
                     : h->ranges_auto[kPaged ? 1 : 0];
  p.pad = kPaged ? kBlock : 1;
  p.scale_log2 = (float)((double)scale * 1.4426950408889634);

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int wgw = h->split_wgw;
  const size_t split_lds = (size_t)wgw * kTileBytes;
  const dim3 split_grid((unsigned)(p.num_ranges * p.hkv / wgw));
  const dim3 merge_grid((unsigned)(((int64_t)num_seqs * p.hq + kMergeWaves - 1) / kMergeWaves));
  const uint16_t* qp = static_cast<const uint16_t*>(q);
  const uint16_t* kp = static_cast<const uint16_t*>(k);
  const uint16_t* vp = static_cast<const uint16_t*>(v);
  if (d.out_dtype == CTX_DTYPE_F32) {
    float* op = static_cast<float*>(out);
    hipLaunchKernelGGL((decode_split_kernel<float, kPaged>), split_grid, dim3(64 * wgw), split_lds, s, qp, kp, vp,
                       offs, lens, p, pg, h->o_ws, h->ml_ws, op);
    hipLaunchKernelGGL(decode_merge_kernel<float>, merge_grid, dim3(64 * kMergeWaves), 0, s, lens, p,
                       h->o_ws, h->ml_ws, op);
  } else {
    uint16_t* op = static_cast<uint16_t*>(out);
    hipLaunchKernelGGL((decode_split_kernel<uint16_t, kPaged>), split_grid, dim3(64 * wgw), split_lds, s, qp, kp, vp,
                       offs, lens, p, pg, h->o_ws, h->ml_ws, op);
    hipLaunchKernelGGL(decode_merge_kernel<uint16_t>, merge_grid, dim3(64 * kMergeWaves), 0, s, lens, p,
                       h->o_ws, h->ml_ws, op);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return CTX_OK;
}

}  // namespace

extern "C" {

int ctx_decode_attn_run(ctx_decode_attn* h, const void* q, const void* k_cache,
                        const void* v_cache, const int32_t* seq_offsets, const int32_t* seq_lens,
                        int32_t num_seqs, float scale, void* out, void* stream) {
  int rc = check_common(h, num_seqs, scale);
  if (rc != CTX_OK || num_seqs == 0) return rc;
  if (q == nullptr || k_cache == nullptr || v_cache == nullptr || seq_offsets == nullptr ||
      seq_lens == nullptr || out == nullptr)
    return fail(CTX_ERR_INVALID_ARG, "NULL data pointer");
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out))
    return fail(CTX_ERR_ALIGNMENT, "q, k_cache, v_cache and out must be 16-byte aligned");
  rc = check_device(h);
  if (rc != CTX_OK) return rc;
  Paged pg{};
  return launch<false>(h, q, k_cache, v_cache, seq_offsets, seq_lens, num_seqs, scale, out, stream, pg);
}

int ctx_decode_attn_run_paged(ctx_decode_attn* h, const void* q, void* k_pages, void* v_pages,
                              const int32_t* block_tables, int32_t max_pages_per_seq,
                              const int32_t* seq_lens, int32_t num_seqs, const void* k_new,
                              const void* v_new, float scale, void* out, void* stream) {
  int rc = check_common(h, num_seqs, scale);
  if (rc != CTX_OK) return rc;
  if (h->desc.page_tokens <= 0)
    return fail(CTX_ERR_UNSUPPORTED, "the handle was created without page_tokens");
  if (num_seqs == 0) return CTX_OK;
  if (q == nullptr || k_pages == nullptr || v_pages == nullptr || block_tables == nullptr ||
      seq_lens == nullptr || out == nullptr)
    return fail(CTX_ERR_INVALID_ARG, "NULL data pointer");
  if ((k_new == nullptr) != (v_new == nullptr))
    return fail(CTX_ERR_INVALID_ARG, "k_new and v_new must both be given or both be NULL");
  if (max_pages_per_seq <= 0) return fail(CTX_ERR_INVALID_ARG, "max_pages_per_seq must be positive");
  if (!aligned16(q) || !aligned16(k_pages) || !aligned16(v_pages) || !aligned16(out) ||
      !aligned16(k_new) || !aligned16(v_new))
    return fail(CTX_ERR_ALIGNMENT, "q, k_pages, v_pages, k_new, v_new and out must be 16-byte aligned");
  rc = check_device(h);
  if (rc != CTX_OK) return rc;
  Paged pg;
  pg.block_tables = block_tables;
  pg.max_pages = max_pages_per_seq;
  pg.page_tokens = h->desc.page_tokens;
  pg.k_new = static_cast<const uint16_t*>(k_new);
  pg.v_new = static_cast<const uint16_t*>(v_new);
  pg.k_cache = static_cast<uint16_t*>(k_pages);
  pg.v_cache = static_cast<uint16_t*>(v_pages);
  return launch<true>(h, q, k_pages, v_pages, nullptr, seq_lens, num_seqs, scale, out, stream, pg);
}

int ctx_decode_attn_destroy(ctx_decode_attn* h) {
  if (h == nullptr) return CTX_OK;
  int rc = CTX_OK;
  int prev = -1;
  if (hipGetDevice(&prev) == hipSuccess && prev != h->device) (void)hipSetDevice(h->device);
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) rc = hip_fail(e, "hipDeviceSynchronize");
  if (h->o_ws) (void)hipFree(h->o_ws);
  if (h->ml_ws) (void)hipFree(h->ml_ws);
  if (prev >= 0 && prev != h->device) (void)hipSetDevice(prev);
  delete h;
  return rc;
}

}  // extern "C"

// ------------------------------------------------------------ allocation-free entry point
//
// ctx_decode_attn_run_static runs the same kernels as ctx_decode_attn_run with
// the split workspace in `scratch`, a file-scope device array (one copy per
// device, held until the process ends), instead of a handle's allocation.  In
// host code `scratch` names a host-side stand-in, so its device address is
// looked up once per device (hipGetSymbolAddress, with that device current)
// and only that address is handed to kernels.

namespace {

constexpr size_t kScratchBytes = (size_t)CTX_STATIC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

struct StaticDevice {
  bool ready;
  int cus;
  unsigned char* scratch;     // device address of `scratch` on this device
  int64_t per_cu[2][kWgWaves + 1];  // resident split waves per CU by out dtype and waves per workgroup (0: not yet known)
};

StaticDevice g_static[kMaxDevices];
std::mutex g_static_mutex;

// The device's scratch address and CU count, set up on its first call.
int static_device(int dev, StaticDevice** out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(CTX_ERR_UNSUPPORTED, "device %d >= %d", dev, kMaxDevices);
  StaticDevice& sd = g_static[dev];
  if (!sd.ready) {
    void* ptr = nullptr;
    hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
    sd.scratch = static_cast<unsigned char*>(ptr);
    sd.cus = cus;
    sd.ready = true;
  }
  *out = &sd;
  return CTX_OK;
}

}  // namespace

extern "C" int ctx_decode_attn_run_static(const ctx_decode_attn_desc* desc, const void* q, const void* k_cache,
                                          const void* v_cache, const int32_t* seq_offsets, const int32_t* seq_lens,
                                          int32_t num_seqs, float scale, void* out, void* stream) {
  ctx_clear_error();
  if (desc == nullptr) return fail(CTX_ERR_INVALID_ARG, "desc is NULL");
  const ctx_decode_attn_desc d = *desc;
  int rc = check_desc(d);
  if (rc != CTX_OK) return rc;
  if (d.split_tokens != 0 || d.page_tokens != 0)
    return fail(CTX_ERR_UNSUPPORTED, "the allocation-free entry point takes split_tokens = 0 and page_tokens = 0");
  if (num_seqs < 0) return fail(CTX_ERR_INVALID_ARG, "num_seqs %d < 0", num_seqs);
  if (num_seqs > d.max_batch)
    return fail(CTX_ERR_CAPACITY, "num_seqs %d > max_batch %d", num_seqs, d.max_batch);
  if (!std::isfinite(scale)) return fail(CTX_ERR_INVALID_ARG, "scale is not finite");
  if (num_seqs == 0) return CTX_OK;
  if (q == nullptr || k_cache == nullptr || v_cache == nullptr || seq_offsets == nullptr ||
      seq_lens == nullptr || out == nullptr)
    return fail(CTX_ERR_INVALID_ARG, "NULL data pointer");
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out))
    return fail(CTX_ERR_ALIGNMENT, "q, k_cache, v_cache and out must be 16-byte aligned");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");

  ctx_decode_attn h{};
  {
    std::lock_guard<std::mutex> lock(g_static_mutex);
    StaticDevice* sd = nullptr;
    rc = static_device(dev, &sd);
    if (rc != CTX_OK) return rc;
    const int wgw = split_waves(d.num_kv_heads);
    int64_t& per_cu = sd->per_cu[d.out_dtype == CTX_DTYPE_F32 ? 1 : 0][wgw];
    if (per_cu == 0) {
      int64_t r[2];
      rc = resident_waves(d.out_dtype, wgw, r);
      if (rc != CTX_OK) return rc;
      per_cu = r[0];
    }
    // the same split as a handle made from this descriptor on this device
    const int64_t ranges = ranges_for(sd->cus, per_cu, d.num_kv_heads);
    h.desc = d;
    h.device = dev;
    h.num_cus = sd->cus;
    h.ranges_auto[0] = (int32_t)ranges;
    h.ranges_auto[1] = 0;  // paged layout: not served here
    h.max_ranges = ranges;
    h.split_wgw = wgw;
    h.o_ws = reinterpret_cast<float*>(sd->scratch);
  }
  // the workspace of this call: partial outputs, then their (max, sum) pairs
  const int64_t slots = (int64_t)h.max_ranges + num_seqs;
  const size_t o_bytes = (size_t)round_up((int64_t)slots * d.num_q_heads * kHeadDim * (int64_t)sizeof(float), 256);
  const size_t ml_bytes = (size_t)slots * d.num_q_heads * sizeof(float2);
  if (o_bytes + ml_bytes > kScratchBytes)
    return fail(CTX_ERR_CAPACITY,
                "workspace of %zu bytes (%lld ranges + %d sequences, %d query heads) exceeds the static %zu bytes",
                o_bytes + ml_bytes, (long long)h.max_ranges, num_seqs, d.num_q_heads, kScratchBytes);
  h.ml_ws = reinterpret_cast<float2*>(reinterpret_cast<unsigned char*>(h.o_ws) + o_bytes);
  Paged pg{};
  return launch<false>(&h, q, k_cache, v_cache, seq_offsets, seq_lens, num_seqs, scale, out, stream, pg);
}
