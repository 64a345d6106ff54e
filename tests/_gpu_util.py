"""Helpers shared by the GPU tests: uploads, sampled full-size layers, error stats."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2609_36608_amd import workloads as wl

MAX_ABS = 1e-2     # parity gate, max-abs over every checked element
MEAN_ABS = 1e-3    # parity gate, mean-abs over every checked element
TIGHT_MAX_ABS = 2e-4  # fp32-accumulated attention lands far below the gate; above this is a bug


def dev():
    return torch.device("cuda", torch.cuda.current_device())


def up_bf16(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev()).view(torch.bfloat16)


def up_i32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev())


def bf16_to_f32(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy()


def errors(got: np.ndarray, ref: np.ndarray):
    err = np.abs(got.astype(np.float64) - ref)
    return float(err.max()), float(err.mean())


def assert_parity(got, ref, what="", tight=True):
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    mx, mean = errors(got, ref)
    print(f"{what}: max-abs {mx:.3e} mean-abs {mean:.3e}", flush=True)
    assert mx <= MAX_ABS and mean <= MEAN_ABS, f"{what}: parity gate failed ({mx:.3e}, {mean:.3e})"
    if tight:
        assert mx <= TIGHT_MAX_ABS, f"{what}: max-abs {mx:.3e} far above fp32 rounding"


class SampledLayer:
    """A full-size layer on the GPU: every row drawn on the device, except the
    rows of a few sampled sequences, which come from the seeded host generator
    so the oracle can recompute those sequences."""

    def __init__(self, w: wl.Workload, layer: int = 0, n_sample: int = 6, seed: int = wl.DEFAULT_SEED):
        self.w = w
        self.layout = wl.workload_layout(w, seed)
        lay = self.layout
        rng = np.random.default_rng(1000 + w.index)
        lens = lay.lens
        # the longest, the shortest and the one placed last (highest cache offsets)
        picks = {int(np.argmax(lens)), int(np.argmin(lens)), int(np.argmax(lay.offsets))}
        others = [b for b in range(w.batch) if b not in picks]
        picks |= set(int(x) for x in rng.choice(others, size=min(n_sample - len(picks), len(others)), replace=False))
        self.sample = sorted(picks)
        shape = (lay.num_rows, w.num_kv_heads, w.head_dim)
        self.k = torch.empty(shape, dtype=torch.bfloat16, device=dev())
        self.v = torch.empty(shape, dtype=torch.bfloat16, device=dev())
        wl.fill_normal_bf16_device(self.k, seed, w.index, layer, 1)
        wl.fill_normal_bf16_device(self.v, seed, w.index, layer, 2)
        # compact host cache of the sampled sequences for the oracle
        caps = [int(lay.capacity[b]) for b in self.sample]
        self.host_offsets = np.concatenate([[0], np.cumsum(caps)[:-1]]).astype(np.int32)
        hk = np.empty((sum(caps), w.num_kv_heads, w.head_dim), np.uint16)
        hv = np.empty_like(hk)
        for i, b in enumerate(self.sample):
            kb, vb = wl.sequence_kv_bits(w, layer, b, caps[i], seed)
            o = int(self.host_offsets[i])
            hk[o:o + caps[i]] = kb
            hv[o:o + caps[i]] = vb
            go = int(lay.offsets[b])
            self.k[go:go + caps[i]] = up_bf16(kb)
            self.v[go:go + caps[i]] = up_bf16(vb)
        self.hk, self.hv = hk, hv
        self.offsets = up_i32(lay.offsets)
        self.layer = layer
        self.seed = seed

    def query(self, step: int):
        qh = wl.query_bits(self.w, self.layer, step, self.seed)
        return qh, up_bf16(qh)

    def reference(self, qh: np.ndarray, step: int) -> np.ndarray:
        """Oracle output [len(sample), Hq, D] at a decode step."""
        lens = self.layout.lens_at(step)
        sl = np.array([lens[b] for b in self.sample], np.int32)
        return oracle.decode_attn(qh[self.sample], self.hk, self.hv, self.host_offsets, sl, self.w.scale)


def paged_copy(k: np.ndarray, v: np.ndarray, lay, page_tokens: int, rng, spare_pages: int = 7,
               fill=wl.BF16_NAN):
    """Scatter every sequence's rows of a contiguous cache into randomly chosen
    pages [num_pages, P, Hkv, D]; unused pages and slots hold `fill`.
    Returns (k_pages, v_pages, block_tables) with -1 in unused table entries."""
    caps = [int(c) for c in lay.capacity]
    npages = [-(-c // page_tokens) for c in caps]
    total = sum(npages) + spare_pages
    perm = rng.permutation(total)
    hkv, d = k.shape[1], k.shape[2]
    kp = np.full((total, page_tokens, hkv, d), fill, np.uint16)
    vp = np.full_like(kp, fill)
    bt = np.full((len(caps), max(npages) + 3), -1, np.int32)
    nxt = 0
    for b, cap in enumerate(caps):
        o = int(lay.offsets[b])
        for j in range(npages[b]):
            page = perm[nxt]
            nxt += 1
            bt[b, j] = page
            n = min(page_tokens, cap - j * page_tokens)
            kp[page, :n] = k[o + j * page_tokens: o + j * page_tokens + n]
            vp[page, :n] = v[o + j * page_tokens: o + j * page_tokens + n]
    return kp, vp, bt
