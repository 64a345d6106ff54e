"""Seeded synthetic inputs for decode-step attention over multi-turn contexts.

This module only draws inputs: context lengths, cache layouts and bf16 q/K/V
bits.  It holds none of the attention arithmetic, so both the HIP path and the
CPU oracle can consume the same bits without sharing any computation.

Workload shapes follow the paper's rollout setting: a Qwen3 student decodes
one new token per in-flight request over its interaction context
c_t = q + h_t + o_t (Sec. 3, eq:agent-history), grown by the response prefix
(eq:token-context); the ID fast action additionally conditions on the
reference next observation o^ref_{t+1} (Sec. 4.1,
eq:reference-conditioned-action).  Rollouts run in bf16 with up to 256
concurrent requests (App. rollout-efficiency settings,
tab:scheduling-hyperparameters), 30/15/30-turn episodes (Sec. 5.1) and a
384+128-token thinking budget (App. thinking budget).  The model shapes and
length distributions are the five configurations listed below.

Every random stream is keyed by (seed, config index, layer, tensor id, ...)
through numpy's SeedSequence spawn keys, so any sequence's rows can be drawn
on their own and always come out the same.  The default seed is 42, the
rollout engine seed of the paper's training table (tab:training-hyperparameters).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

DEFAULT_SEED = 42
HEAD_DIM = 128

# tensor ids used in spawn keys
_T_Q, _T_K, _T_V, _T_MASK, _T_LEN, _T_EXTRA, _T_LAYOUT, _T_DEVICE, _T_OPD, _T_OPD_LOGITS = range(10)

BF16_NAN = np.uint16(0x7FC0)


@dataclass(frozen=True)
class Workload:
    """One synthetic decode workload (shapes of a Qwen3 student's attention)."""

    name: str
    index: int
    layers: int
    batch: int
    num_q_heads: int
    num_kv_heads: int
    steps: int
    length_kind: str           # "uniform" or "loguniform"
    length_lo: int
    length_hi: int
    extra_lo: int = 0          # appended reference next observation (config 4)
    extra_hi: int = 0
    peaky_frac: float = 0.0    # fraction of positions whose key row is scaled
    peaky_gain: float = 4.0
    head_dim: int = HEAD_DIM
    description: str = field(default="", compare=False)

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)


WORKLOADS = {
    "tiny": Workload(
        "tiny", 0, layers=1, batch=4, num_q_heads=16, num_kv_heads=8, steps=1,
        length_kind="uniform", length_lo=256, length_hi=1024,
        description="1 layer, batch 4, 16/8 heads, lengths U{256..1024}, 1 decode step"),
    "student_0p6b_1p7b": Workload(
        "student_0p6b_1p7b", 1, layers=28, batch=64, num_q_heads=16, num_kv_heads=8, steps=1,
        length_kind="uniform", length_lo=1024, length_hi=4096,
        description="0.6B/1.7B student shape: 28 layers, batch 64, 16/8 heads, "
                    "early-turn contexts U{1024..4096}, 1 decode step"),
    "student_4b": Workload(
        "student_4b", 2, layers=36, batch=64, num_q_heads=32, num_kv_heads=8, steps=1,
        length_kind="uniform", length_lo=2048, length_hi=8192,
        description="4B student shape: 36 layers, batch 64, 32/8 heads, "
                    "mid-episode contexts U{2048..8192}, 1 decode step"),
    "act_first_burst": Workload(
        "act_first_burst", 3, layers=36, batch=256, num_q_heads=32, num_kv_heads=8, steps=8,
        length_kind="uniform", length_lo=4096, length_hi=12288, extra_lo=128, extra_hi=512,
        peaky_frac=0.05, peaky_gain=4.0,
        description="act-first short-action burst: 36 layers, batch 256, 32/8 heads, "
                    "history U{4096..12288} + reference observation U{128..512}, "
                    "8 decode steps, 5% of key rows x4"),
    "long_ragged": Workload(
        "long_ragged", 4, layers=36, batch=32, num_q_heads=32, num_kv_heads=8, steps=64,
        length_kind="loguniform", length_lo=512, length_hi=32768,
        description="long-horizon ragged batch: 36 layers, batch 32, 32/8 heads, "
                    "lengths log-uniform in [512, 32768], 64 decode steps"),
}


def rng_for(seed: int, *key: int) -> np.random.Generator:
    """Independent PCG64 stream for a spawn key."""
    ss = np.random.SeedSequence(entropy=seed, spawn_key=tuple(int(k) for k in key))
    return np.random.Generator(np.random.PCG64(ss))


# ---------------------------------------------------------------- bf16 bits

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round to nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    out = ((u + bias) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = BF16_NAN
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_bf16(rng: np.random.Generator, shape) -> np.ndarray:
    return f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))


# ----------------------------------------------------------------- lengths

def draw_lengths(w: Workload, seed: int = DEFAULT_SEED) -> np.ndarray:
    """Context length of every sequence at decode step 0 (current token included)."""
    rng = rng_for(seed, w.index, 0, _T_LEN)
    if w.length_kind == "uniform":
        lens = rng.integers(w.length_lo, w.length_hi + 1, size=w.batch)
    elif w.length_kind == "loguniform":
        u = rng.uniform(math.log(w.length_lo), math.log(w.length_hi), size=w.batch)
        lens = np.clip(np.floor(np.exp(u)), w.length_lo, w.length_hi)
    else:
        raise ValueError(w.length_kind)
    if w.extra_hi > 0:
        lens = lens + draw_extra(w, seed)
    return lens.astype(np.int32)


def draw_extra(w: Workload, seed: int = DEFAULT_SEED) -> np.ndarray:
    """Tokens of the appended reference next observation of every sequence
    (the newest tokens, already counted in draw_lengths); zeros if none."""
    if w.extra_hi <= 0:
        return np.zeros(w.batch, np.int32)
    rng_x = rng_for(seed, w.index, 0, _T_EXTRA)
    return rng_x.integers(w.extra_lo, w.extra_hi + 1, size=w.batch).astype(np.int32)


@dataclass
class Layout:
    """Where each sequence's rows live in a [rows, Hkv, D] cache."""

    lens: np.ndarray        # int32 [B], rows attended at decode step 0
    capacity: np.ndarray    # int32 [B], rows reserved (lens + steps - 1)
    offsets: np.ndarray     # int32 [B], first row of each sequence
    num_rows: int
    steps: int

    def lens_at(self, step: int) -> np.ndarray:
        if not 0 <= step < self.steps:
            raise ValueError(f"step {step} outside [0, {self.steps})")
        return (self.lens + step).astype(np.int32)

    @property
    def max_seq_len(self) -> int:
        return int(self.capacity.max()) if len(self.capacity) else 0


def make_layout(lens, steps: int = 1, *, gap_max: int = 0, shuffle: bool = False,
                rng: np.random.Generator | None = None) -> Layout:
    """Place sequences in one cache: capacity lens+steps-1 rows each, optionally
    in a shuffled order and with random gaps (unused rows) between regions."""
    lens = np.asarray(lens, dtype=np.int32)
    cap = (lens + (steps - 1)).astype(np.int64)
    b = len(lens)
    order = np.arange(b)
    if shuffle or gap_max:
        if rng is None:
            raise ValueError("rng required for shuffle/gaps")
    if shuffle:
        order = rng.permutation(b)
    offsets = np.zeros(b, dtype=np.int64)
    row = 0
    for i in order:
        if gap_max:
            row += int(rng.integers(0, gap_max + 1))
        offsets[i] = row
        row += int(cap[i])
    if gap_max:
        row += int(rng.integers(0, gap_max + 1))
    if row >= 2**31:
        raise ValueError("cache too large for int32 row offsets")
    return Layout(lens=lens, capacity=cap.astype(np.int32), offsets=offsets.astype(np.int32),
                  num_rows=int(row), steps=steps)


def workload_layout(w: Workload, seed: int = DEFAULT_SEED, **kw) -> Layout:
    return make_layout(draw_lengths(w, seed), w.steps, **kw)


# ----------------------------------------------------------- q / K / V bits

def query_bits(w: Workload, layer: int, step: int = 0, seed: int = DEFAULT_SEED,
               batch: int | None = None) -> np.ndarray:
    """bf16 bits [B, Hq, D] of the new token's queries."""
    bsz = w.batch if batch is None else batch
    return normal_bf16(rng_for(seed, w.index, layer, _T_Q, step), (bsz, w.num_q_heads, w.head_dim))


def sequence_kv_bits(w: Workload, layer: int, b: int, rows: int, seed: int = DEFAULT_SEED):
    """bf16 bits [rows, Hkv, D] of one sequence's K and V rows.

    For workloads with peaky keys, each position's K row (all heads, all dims) is
    multiplied by `peaky_gain` with probability `peaky_frac`; a power-of-two gain
    is exact in bf16."""
    shape = (rows, w.num_kv_heads, w.head_dim)
    k = normal_bf16(rng_for(seed, w.index, layer, _T_K, b), shape)
    v = normal_bf16(rng_for(seed, w.index, layer, _T_V, b), shape)
    if w.peaky_frac > 0:
        mask = rng_for(seed, w.index, layer, _T_MASK, b).random(rows) < w.peaky_frac
        if mask.any():
            kf = bf16_bits_to_f32(k[mask]) * np.float32(w.peaky_gain)
            k[mask] = f32_to_bf16_bits(kf)
    return k, v


def peaky_mask(w: Workload, layer: int, b: int, rows: int, seed: int = DEFAULT_SEED) -> np.ndarray:
    return rng_for(seed, w.index, layer, _T_MASK, b).random(rows) < w.peaky_frac


def layer_kv_bits(w: Workload, layout: Layout, layer: int, seed: int = DEFAULT_SEED,
                  fill: np.uint16 | None = None):
    """Whole-layer host caches [num_rows, Hkv, D]; rows outside every sequence's
    capacity are set to `fill` (default: random normals)."""
    shape = (layout.num_rows, w.num_kv_heads, w.head_dim)
    if fill is None:
        rng = rng_for(seed, w.index, layer, _T_LAYOUT)
        k = normal_bf16(rng, shape)
        v = normal_bf16(rng, shape)
    else:
        k = np.full(shape, fill, dtype=np.uint16)
        v = np.full(shape, fill, dtype=np.uint16)
    for b in range(len(layout.lens)):
        cap = int(layout.capacity[b])
        off = int(layout.offsets[b])
        kb, vb = sequence_kv_bits(w, layer, b, cap, seed)
        k[off:off + cap] = kb
        v[off:off + cap] = vb
    return k, v


def small_workload(base: Workload, *, name: str | None = None, batch: int | None = None,
                   lengths: tuple[int, int] | None = None, steps: int | None = None,
                   index_offset: int = 100) -> Workload:
    """A reduced copy of a workload (same heads, value distribution and length
    kind) for parity runs the oracle finishes in seconds."""
    lo, hi = lengths if lengths is not None else (base.length_lo, base.length_hi)
    return Workload(
        name=name or f"{base.name}_small", index=base.index + index_offset, layers=1,
        batch=batch or base.batch, num_q_heads=base.num_q_heads, num_kv_heads=base.num_kv_heads,
        steps=steps or base.steps, length_kind=base.length_kind, length_lo=lo, length_hi=hi,
        extra_lo=base.extra_lo if lengths is None else 0,
        extra_hi=base.extra_hi if lengths is None else 0,
        peaky_frac=base.peaky_frac, peaky_gain=base.peaky_gain, head_dim=base.head_dim,
        description=f"reduced {base.name}")


# ------------------------------------------------------ device-side filling

def _device_generator(device, seed: int, *key: int):
    import torch

    g = torch.Generator(device=device)
    h = 0
    for x in (seed, *key):
        h = (h * 1000003 + int(x) + 1) % (2**63 - 1)
    g.manual_seed(h)
    return g


def fill_normal_bf16_device(t, seed: int, *key: int) -> None:
    """Fill a CUDA bf16 tensor with N(0,1) values from torch's seeded device
    generator (full-size layers; tests copy them to the host for the oracle)."""
    g = _device_generator(t.device, seed, *key)
    flat = t.view(-1)
    chunk = 1 << 28
    for s in range(0, flat.numel(), chunk):
        e = min(s + chunk, flat.numel())
        flat[s:e].normal_(generator=g)


def apply_peaky_keys_device(k, w: Workload, layer: int, seed: int = DEFAULT_SEED) -> None:
    """Multiply each cache row's key (all heads and dims) by `peaky_gain` with
    probability `peaky_frac`, drawn on the device; no-op for workloads without
    peaky keys.  k is [rows, Hkv, D] or paged [pages, P, Hkv, D] bf16; a
    power-of-two gain is exact in bf16."""
    import torch

    if w.peaky_frac <= 0:
        return
    rows = k.numel() // (w.num_kv_heads * w.head_dim)
    g = _device_generator(k.device, seed, w.index, layer, _T_MASK)
    peaky = torch.rand(rows, generator=g, device=k.device) < w.peaky_frac
    gain = torch.ones(rows, dtype=torch.bfloat16, device=k.device)
    gain.masked_fill_(peaky, w.peaky_gain)
    k.view(rows, -1).mul_(gain[:, None])


def fill_kv_device(k, v, w: Workload, layer: int, seed: int = DEFAULT_SEED) -> None:
    """A full-size layer's caches drawn on the device: N(0,1) bf16 keys and
    values, and the workload's peaky keys."""
    fill_normal_bf16_device(k, seed, w.index, layer, 1)
    fill_normal_bf16_device(v, seed, w.index, layer, 2)
    apply_peaky_keys_device(k, w, layer, seed)


# ----------------------------------------------------------------- OPD loss batches
# An optimization batch of turn-level full responses (App. OPD Optimization;
# tab:training-hyperparameters: 64 responses per batch, full-response limit 512
# tokens, Qwen3 students with a 151,936-entry vocabulary, bf16).  Half of the
# responses carry an inserted span (the thinking-budget close, App. thinking)
# that stays in the context but is not supervised.


@dataclass(frozen=True)
class OpdWorkload:
    name: str
    index: int
    responses: int
    length_lo: int
    length_hi: int
    vocab: int
    row_stride: int
    logit_std: float = 2.0
    inserted_frac: float = 0.5    # responses with an inserted (masked) span
    inserted_len: int = 8
    outlier_frac: float = 0.03    # tokens whose stored log-probability is far off
    description: str = field(default="", compare=False)


OPD_WORKLOADS = {
    "opd_tiny": OpdWorkload("opd_tiny", 20, responses=6, length_lo=0, length_hi=48, vocab=1003,
                            row_stride=1008, inserted_len=4, outlier_frac=0.2,
                            description="6 responses of U{0..48} tokens, vocabulary 1,003 in rows of 1,008"),
    "opd_qwen3": OpdWorkload("opd_qwen3", 21, responses=64, length_lo=64, length_hi=512, vocab=151936,
                             row_stride=151936,
                             description="OPD batch: 64 turn-level full responses of U{64..512} tokens, "
                                         "Qwen3 vocabulary 151,936, bf16 logits N(0, 2^2)"),
}


@dataclass
class OpdBatch:
    seq_starts: np.ndarray   # int32 [B + 1]
    tokens: np.ndarray       # int32 [N] sampled tokens
    mask: np.ndarray         # uint8 [N] 1 = supervised
    lp_target: np.ndarray    # float64 [N] where the student's log-probability of the token is placed
    old_lp: np.ndarray       # float32 [N] stored sampling log-probabilities
    teacher_lp: np.ndarray   # float32 [N] teacher log-probabilities

    @property
    def num_tokens(self) -> int:
        return int(self.seq_starts[-1])


def opd_batch(w: OpdWorkload, seed: int = DEFAULT_SEED) -> OpdBatch:
    """Lengths, masks, tokens and the stored log-probabilities of a batch.
    The sampled token's log-probability is drawn from -Exp(1); the stored one
    is that plus N(0, 0.1^2), with outlier_frac of the tokens moved by
    +-U(1, 30) (stale samples, exercising every clipping regime); the teacher's
    is the stored one plus N(0, 1)."""
    rng = rng_for(seed, w.index, 0, _T_OPD)
    lens = rng.integers(w.length_lo, w.length_hi + 1, size=w.responses)
    starts = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    n = int(starts[-1])
    mask = np.ones(n, np.uint8)
    for b in range(w.responses):
        if lens[b] > w.inserted_len and rng.random() < w.inserted_frac:
            pos = int(rng.integers(0, lens[b] - w.inserted_len + 1))
            mask[starts[b] + pos: starts[b] + pos + w.inserted_len] = 0
    tokens = rng.integers(0, w.vocab, size=n).astype(np.int32)
    lp_target = -rng.exponential(1.0, size=n)
    old = lp_target + rng.normal(0.0, 0.1, size=n)
    out = rng.random(n) < w.outlier_frac
    old[out] += rng.choice([-1.0, 1.0], size=int(out.sum())) * rng.uniform(1.0, 30.0, size=int(out.sum()))
    teacher = old + rng.normal(0.0, 1.0, size=n)
    return OpdBatch(starts, tokens, mask, lp_target, old.astype(np.float32), teacher.astype(np.float32))


def _opd_token_logit(w: OpdWorkload, batch: OpdBatch) -> np.ndarray:
    # an N(0, s^2) row of V logits has log-sum-exp close to log V + s^2 / 2;
    # the sampled token's logit goes that far above its target log-probability
    return batch.lp_target + math.log(w.vocab) + 0.5 * w.logit_std ** 2


def opd_logits_host(w: OpdWorkload, batch: OpdBatch, seed: int = DEFAULT_SEED) -> np.ndarray:
    """bf16 bits [N, row_stride]: N(0, s^2) logits with the sampled token placed;
    columns >= vocab and masked rows hold NaN (never read)."""
    rng = rng_for(seed, w.index, 1, _T_OPD_LOGITS)
    n = batch.num_tokens
    z = rng.standard_normal((n, w.row_stride), dtype=np.float32) * np.float32(w.logit_std)
    z[np.arange(n), batch.tokens] = _opd_token_logit(w, batch).astype(np.float32)
    z[:, w.vocab:] = np.nan
    z[batch.mask == 0] = np.nan
    return f32_to_bf16_bits(z)


def opd_logits_device(w: OpdWorkload, batch: OpdBatch, device, seed: int = DEFAULT_SEED):
    """The same kind of logits drawn on the device (full-size batches): bf16
    [N, row_stride] torch tensor, every entry finite."""
    import torch

    n = batch.num_tokens
    t = torch.empty((n, w.row_stride), dtype=torch.bfloat16, device=device)
    fill_normal_bf16_device(t, seed, w.index, 1, _T_OPD_LOGITS)
    t.mul_(w.logit_std)
    rows = torch.arange(n, device=device)
    cols = torch.from_numpy(batch.tokens.astype(np.int64)).to(device)
    t[rows, cols] = torch.from_numpy(_opd_token_logit(w, batch).astype(np.float32)).to(device).to(torch.bfloat16)
    return t
