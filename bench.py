#!/usr/bin/env python3
"""Benchmark of decode-step GQA attention over ragged multi-turn KV caches on one MI355X.

A step is one decode step of the student's rollout across all layers: for every
layer, one ctx_decode_attn_run call over the whole batch (every sequence's new
token attends over its cached context).  Inputs are synthetic, seeded, and
resident in HBM before the timed region starts.  Prints one JSON line:
value = algorithmic HBM GB/s of the whole timed region (K and V read once,
q read, fp32 out written, offsets and lengths), plus decode-steps/s, the
fraction of the 8 TB/s HBM peak, the roofline of the attention kernel and the
CPU oracle's rate on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2609_36608_amd import workloads as wl  # noqa: E402

METRIC = "decode-attention HBM GB/s (fraction of 8 TB/s peak) + decode-steps/sec, 1 MI355X"
HBM_PEAK_GBS = 8000.0
REPEATS = 20  # individually timed graph replays reported beside the main timed region
HBM_BUDGET_BYTES = 240 * 2**30  # leave headroom below 288 GB for the rest of the process


def algorithmic_bytes(lens: np.ndarray, w: wl.Workload, out_bytes: int = 4) -> int:
    """K and V rows read once (bf16), q read (bf16), out written, offsets + lengths.
    (The paged layout reads one block-table entry per page instead of an offset
    and, when appending, reads and writes one K and V row per sequence; these
    are left out so both layouts count the same bytes.)"""
    kv = int(lens.astype(np.int64).sum()) * w.num_kv_heads * w.head_dim * 2 * 2
    b = len(lens)
    return kv + b * w.num_q_heads * w.head_dim * (2 + out_bytes) + 8 * b


def profiled_traffic(workload: str, kernel: str = "decode_split_kernel"):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary, or None if that summary is for another workload or kernel or for
    an older version of the kernel source."""
    import glob
    import hashlib

    for path in glob.glob(os.path.join(ROOT, "profiles", "*hbm_traffic*.md")):
        fields = {}
        for line in open(path):
            if ":" in line and not line.startswith(("|", "#", "`")):
                k, _, v = line.partition(":")
                fields[k.strip()] = v.strip()
        src = os.path.join(ROOT, fields.get("kernel_source", "paper_2609_36608_amd/csrc/ctx_decode_attn.hip"))
        if not os.path.exists(src):
            continue
        digest = hashlib.sha256(open(src, "rb").read()).hexdigest()
        if (fields.get("kernel_source_sha256") == digest and fields.get("workload") == workload
                and fields.get("kernel", "decode_split_kernel") == kernel):
            t = int(fields["traffic_bytes_per_launch"])
            a = int(fields["algorithmic_bytes_per_launch"])
            return {"bytes_per_launch": t, "ratio_to_algorithmic": round(t / a, 4),
                    "source": os.path.relpath(path, ROOT)}
    return None


def traffic_fields(workload: str, kernel: str = "decode_split_kernel") -> dict:
    """The roofline's `traffic` (HBM bytes per launch from the counters, or
    None) and, beside it, where that figure comes from."""
    d = profiled_traffic(workload, kernel)
    return {"traffic": d["bytes_per_launch"] if d else None, "traffic_detail": d}


def cpu_baseline(w: wl.Workload, layout: wl.Layout, target_s: float, threads: int,
                 single_thread_s: float = 3.0) -> dict:
    """Time the CPU oracle on layer 0 / step 0 for a fixed sample of sequences,
    repeated until about target_s seconds of CPU work have run on `threads`
    threads, then for about single_thread_s seconds on one thread."""
    import oracle

    rng = np.random.default_rng(7)
    lens = layout.lens
    order = np.argsort(lens)
    n = min(len(lens), 8)
    sample = sorted(set([int(order[-1]), int(order[0])] + [int(x) for x in rng.choice(len(lens), n, replace=False)]))[:n]
    caps = [int(lens[b]) for b in sample]
    offs = np.concatenate([[0], np.cumsum(caps)[:-1]]).astype(np.int32)
    k = np.empty((sum(caps), w.num_kv_heads, w.head_dim), np.uint16)
    v = np.empty_like(k)
    for i, b in enumerate(sample):
        kb, vb = wl.sequence_kv_bits(w, 0, b, caps[i])
        k[offs[i]:offs[i] + caps[i]] = kb
        v[offs[i]:offs[i] + caps[i]] = vb
    q = wl.query_bits(w, 0)[sample]
    sl = np.array(caps, np.int32)
    nbytes = algorithmic_bytes(sl, w)
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.decode_attn(q, k, v, offs, sl, w.scale, threads=threads)
        reps += 1
        el = time.perf_counter() - t0
        if el >= target_s or el / reps * (reps + 1) > 3 * target_s:
            break
    gbs = nbytes * reps / el / 1e9
    # the same sample on one thread, for a shorter while
    reps1, t1 = 0, time.perf_counter()
    while True:
        oracle.decode_attn(q, k, v, offs, sl, w.scale, threads=1)
        reps1 += 1
        el1 = time.perf_counter() - t1
        if el1 >= single_thread_s:
            break
    full_step_bytes = algorithmic_bytes(lens, w) * w.layers
    return {
        "value": round(gbs, 4),
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"layer 0, decode step 0, {len(sample)} of {w.batch} sequences "
                   f"({int(sl.sum())} tokens), all {w.num_q_heads} heads, run {reps}x in {el:.1f} s; "
                   f"float64 C oracle, OpenMP over (sequence, head)"),
        "decode_steps_per_s": round(gbs * 1e9 / full_step_bytes, 6),
        "single_thread": {"value": round(nbytes * reps1 / el1 / 1e9, 4), "unit": "GB/s", "cores": 1,
                          "runs": reps1, "seconds": round(el1, 1)},
        "cpu_model": cpu_model(),
    }


def cpu_model() -> str:
    """The host CPU's model name as /proc/cpuinfo reports it ("" if unreadable)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


def read_ceiling(torch, dev, achieved_gbs: float) -> dict:
    """The device's streaming-read rate (ctx_hbm_read: non-temporal 16-byte
    loads over 4 GiB, median of 8 launches), measured in this process, and the
    fraction of it that `achieved_gbs` reaches."""
    from paper_2609_36608_amd import rollout_calibration as rcal

    r = rcal.measure_hbm(torch, dev, gib=4.0, reps=8)
    return {"read_gbs": r["gbs"], "best_gbs": r["best_gbs"], "frac": round(achieved_gbs / r["gbs"], 4),
            "source": f"ctx_hbm_read, 4 GiB, {r['workgroups']} workgroups, median of {r['reps']} in this process"}


def copy_ceiling(torch, dev, achieved_gbs: float) -> dict:
    """The device's 1:1 read/write streaming rate (ctx_hbm_copy over 4 GiB,
    bytes read plus written, median of 8 launches) in this process."""
    from paper_2609_36608_amd import rollout_calibration as rcal

    r = rcal.measure_hbm(torch, dev, gib=4.0, reps=8, copy=True)
    return {"copy_gbs": r["gbs"], "best_gbs": r["best_gbs"], "frac": round(achieved_gbs / r["gbs"], 4),
            "source": f"ctx_hbm_copy, 4 GiB read + 4 GiB written, {r['workgroups']} workgroups, "
                      f"median of {r['reps']} in this process"}


def mfma_ceiling(torch, dev, achieved_tflops: float) -> dict:
    """The bf16 matrix-core rate the prefill kernel's instruction shape
    (v_mfma_f32_16x16x32_bf16) sustains on this device (ctx_mfma_bf16, 2 waves
    per SIMD as the prefill kernel runs, median of 5 launches) in this process,
    and the fraction of it that `achieved_tflops` reaches."""
    from paper_2609_36608_amd import binding
    from paper_2609_36608_amd import rollout_calibration as rcal

    r = rcal.measure_mfma(torch, dev, binding.CTX_MFMA_16X16X32, waves_per_simd=2)
    return {"mfma_tflops": r["tflops"], "best_tflops": r["best_tflops"], "frac": round(achieved_tflops / r["tflops"], 4),
            "source": "ctx_mfma_bf16 (8 chains of v_mfma_f32_16x16x32_bf16 per wave, 2 waves per SIMD), "
                      "median of 5 in this process"}


CEILING_METRIC = "HBM streaming ceiling GB/s (fraction of 8 TB/s peak), 1 MI355X"


def bench_ceiling(args) -> int:
    """Read-only and 1:1 read/write streaming kernels of the library
    (ctx_hbm_read, ctx_hbm_copy) over 8 GiB, each launched --steps times."""
    import torch

    from paper_2609_36608_amd import binding
    from paper_2609_36608_amd import rollout_calibration as rcal

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    res = {}
    for name, copy, nt in (("read_nt", False, True), ("read_cached", False, False), ("copy_nt", True, True),
                           ("copy_cached", True, False)):
        res[name] = rcal.measure_hbm(torch, dev, gib=8.0, reps=args.steps, copy=copy, nontemporal=nt)
    mfma = {}
    for shape, name in ((binding.CTX_MFMA_16X16X32, "mfma_16x16x32"), (binding.CTX_MFMA_32X32X16, "mfma_32x32x16")):
        for wps in (1, 2):
            mfma[f"{name}_{wps}w"] = rcal.measure_mfma(torch, dev, shape, waves_per_simd=wps, reps=args.steps)
    best = res["read_nt"]
    result = {
        "metric": CEILING_METRIC,
        "value": best["gbs"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": 1,
        "ms_per_step": round(best["bytes"] / best["gbs"] / 1e6, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "config": {"workload": "8 GiB buffer streamed once per launch (copy: 8 GiB read + 8 GiB written)",
                   "parallelism": "none (1 GPU)"},
        "frac_of_hbm_peak": round(best["gbs"] / HBM_PEAK_GBS, 4),
        "kernels": {k: {kk: v[kk] for kk in ("gbs", "best_gbs", "workgroups", "nontemporal", "kernel")}
                    for k, v in res.items()},
        "matrix_cores": {**mfma, "peak_tflops": MFMA_BF16_PEAK_TFLOPS},
        "device": device_info(torch, dev),
    }
    print(json.dumps(result), flush=True)
    return 0


PREFILL_METRIC = "causal prefill attention TFLOP/s (fraction of 2.5 PFLOP/s bf16 MFMA peak), 1 MI355X"
MFMA_BF16_PEAK_TFLOPS = 2500.0


def prefill_flops(lens: np.ndarray, nq: np.ndarray, w: wl.Workload) -> int:
    """Algorithmic flops of one prefill call: query i of sequence b attends to
    L_b - nq_b + i + 1 positions, each costing 2*D for q.k and 2*D for p.v per head."""
    L = lens.astype(np.int64)
    n = nq.astype(np.int64)
    positions = n * (L - n) + n * (n + 1) // 2
    return int(positions.sum()) * 4 * w.head_dim * w.num_q_heads


def prefill_cpu_baseline(w, lens, nq, target_s, threads) -> dict:
    """The CPU oracle on the reference-observation prefill of a few whole sequences."""
    import oracle

    picks = [0, 1, 2, 3]
    sl = lens[picks].astype(np.int32)
    sq = nq[picks].astype(np.int32)
    offs = np.concatenate([[0], np.cumsum(sl)[:-1]]).astype(np.int32)
    qs = np.concatenate([[0], np.cumsum(sq)[:-1]]).astype(np.int32)
    k = np.empty((int(sl.sum()), w.num_kv_heads, w.head_dim), np.uint16)
    v = np.empty_like(k)
    for i, b in enumerate(picks):
        kb, vb = wl.sequence_kv_bits(w, 0, b, int(sl[i]))
        k[offs[i]:offs[i] + sl[i]] = kb
        v[offs[i]:offs[i] + sl[i]] = vb
    rng = np.random.default_rng(7)
    q = wl.normal_bf16(rng, (int(sq.sum()), w.num_q_heads, w.head_dim))
    flops = prefill_flops(sl, sq, w)
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.prefill_attn(q, k, v, offs, sl, qs, sq, w.scale, threads=threads)
        reps += 1
        el = time.perf_counter() - t0
        if el >= target_s or el / reps * (reps + 1) > 3 * target_s:
            break
    return {
        "value": round(flops * reps / el / 1e12, 6),
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"layer 0, sequences {picks} of {w.batch} ({int(sq.sum())} new tokens over "
                   f"{int(sl.sum())} cached), all {w.num_q_heads} heads, run {reps}x in {el:.1f} s; "
                   f"float64 C oracle, OpenMP over (query, head)"),
    }


def bench_prefill(args) -> int:
    """Per layer one ctx_prefill_attn_run: every sequence's appended reference
    observation (its newest U{128..512} tokens) attends causally over its whole
    cached history.  A step = all layers."""
    import torch

    from paper_2609_36608_amd.binding import DecodeAttention

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    w = wl.WORKLOADS[args.workload]
    if w.extra_hi <= 0:
        print(f"bench.py: --prefill needs a workload with an appended observation (act_first_burst)",
              file=sys.stderr)
        return 2
    lens = wl.draw_lengths(w)
    nq = wl.draw_extra(w)
    layout = wl.make_layout(lens, 1)
    B = w.batch
    layer_bytes = layout.num_rows * w.num_kv_heads * w.head_dim * 2 * 2
    n_buf = max(1, min(w.layers, HBM_BUDGET_BYTES // layer_bytes))
    t_setup = time.perf_counter()
    ks, vs = [], []
    for i in range(n_buf):
        k = torch.empty((layout.num_rows, w.num_kv_heads, w.head_dim), dtype=torch.bfloat16, device=dev)
        v = torch.empty_like(k)
        wl.fill_kv_device(k, v, w, i)
        ks.append(k)
        vs.append(v)
    total_q = int(nq.sum())
    q_starts = np.concatenate([[0], np.cumsum(nq)[:-1]]).astype(np.int32)
    q = torch.empty((total_q, w.num_q_heads, w.head_dim), dtype=torch.bfloat16, device=dev)
    wl.fill_normal_bf16_device(q, wl.DEFAULT_SEED, w.index, 0, 0)
    out = torch.empty((total_q, w.num_q_heads, w.head_dim), dtype=torch.float32, device=dev)
    t_offs = torch.from_numpy(layout.offsets).to(dev)
    t_lens = torch.from_numpy(lens).to(dev)
    t_qs = torch.from_numpy(q_starts).to(dev)
    t_nq = torch.from_numpy(nq).to(dev)
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t_setup
    attn = DecodeAttention(w.num_q_heads, w.num_kv_heads, B, int(lens.max()))
    stream = torch.cuda.current_stream()
    max_q = int(nq.max())

    def step(split_p: bool) -> None:
        for layer in range(w.layers):
            attn.prefill(q, ks[layer % n_buf], vs[layer % n_buf], t_offs, t_lens, t_qs, t_nq, max_q,
                         w.scale, out, stream=stream, split_p=split_p)

    def time_mode(split_p: bool) -> float:
        for _ in range(args.warmup):
            step(split_p)
        torch.cuda.synchronize()
        start = torch.cuda.Event(enable_timing=True)
        stop = torch.cuda.Event(enable_timing=True)
        start.record(stream)
        for _ in range(args.steps):
            step(split_p)
        stop.record(stream)
        stop.synchronize()
        torch.cuda.synchronize()
        return start.elapsed_time(stop) / 1e3

    # the default precision (bf16 softmax weights) gives `value`; the two-term
    # weights (CTX_PREFILL_SPLIT_P) are timed beside it
    split_s = time_mode(True) if args.prefill_p in ("both", "split") else None
    elapsed_s = time_mode(False) if args.prefill_p in ("both", "bf16") else split_s
    calls = args.steps * w.layers
    flops = prefill_flops(lens, nq, w)
    if args.calibrate_copy_gib > 0:
        ncopy = int(args.calibrate_copy_gib * 2**30) // 4
        src = torch.ones(ncopy, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    tflops = flops * calls / elapsed_s / 1e12
    kv_bytes = int(lens.astype(np.int64).sum()) * w.num_kv_heads * w.head_dim * 4
    result = {
        "metric": PREFILL_METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed_s * 1e3 / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": (f"reference-observation prefill of {w.name}: {w.layers} layers, batch {B}, "
                         f"{w.num_q_heads}/{w.num_kv_heads} heads, history U{{{w.length_lo}..{w.length_hi}}} "
                         f"+ U{{{w.extra_lo}..{w.extra_hi}}} new tokens attending causally"),
            "name": w.name,
            "new_tokens": total_q,
            "cached_tokens": int(lens.sum()),
            "distinct_layer_buffers": n_buf,
            "seed": wl.DEFAULT_SEED,
            "parallelism": "none (1 GPU)",
        },
        "tokens_per_s": round(total_q * w.layers * args.steps / elapsed_s / w.layers, 1),
        "roofline": {
            "bound": "mfma",
            "achieved": round(flops / (elapsed_s / calls) / 1e12, 2),
            "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(flops / (elapsed_s / calls) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
            "ceiling": mfma_ceiling(torch, dev, flops / (elapsed_s / calls) / 1e12),
            **traffic_fields(w.name, "prefill_kernel"),
            "kernel": ("prefill_kernel (one ctx_prefill_attn_run call per layer, "
                       + ("two-term softmax weights)" if args.prefill_p == "split" else "bf16 softmax weights)")),
            "flops_per_launch": flops,
            "kv_bytes_per_launch": kv_bytes,
            "avg_launch_us": round(elapsed_s / calls * 1e6, 3),
        },
        "setup_s": round(setup_s, 1),
    }
    if split_s is not None and args.prefill_p == "both":
        result["split_p"] = {
            "value": round(flops * calls / split_s / 1e12, 2),
            "ms_per_step": round(split_s * 1e3 / args.steps, 4),
            "avg_launch_us": round(split_s / calls * 1e6, 3),
            "frac": round(flops * calls / split_s / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
        }
    if not args.no_cpu_baseline:
        threads = len(os.sched_getaffinity(0))
        result["cpu_baseline"] = prefill_cpu_baseline(w, lens, nq, args.cpu_seconds, threads)
    print(json.dumps(result), flush=True)
    attn.close()
    return 0


OPD_METRIC = "fused OPD token loss + logits gradient HBM GB/s (fraction of 8 TB/s peak), 1 MI355X"


def opd_bytes(b: wl.OpdBatch, vocab: int, grad: bool = True) -> int:
    """Bytes a call must move at least: every supervised logits row read once,
    every gradient row written once (masked rows: zeros), the per-token inputs
    (token, two log-probabilities, mask) and outputs (lp, weight, loss)."""
    n = b.num_tokens
    sup = int(b.mask.sum())
    return sup * vocab * 2 + (n * vocab * 2 if grad else 0) + n * (4 + 4 + 4 + 1) + n * 12 + 4 * len(b.seq_starts)


def opd_cpu_baseline(w, b: wl.OpdBatch, z_host_fn, target_s: float, threads: int) -> dict:
    """The CPU oracle (loss over a sub-batch of whole responses, then the
    gradient rows of those tokens), repeated for about target_s seconds."""
    import oracle

    r = 4
    end = int(b.seq_starts[r])
    sub = wl.OpdBatch(b.seq_starts[:r + 1].copy(), b.tokens[:end], b.mask[:end], b.lp_target[:end],
                      b.old_lp[:end], b.teacher_lp[:end])
    zh = z_host_fn(end)
    nbytes = opd_bytes(sub, w.vocab)
    reps, t0 = 0, time.perf_counter()
    while True:
        ref = oracle.opd_loss(zh, sub.tokens, sub.old_lp, sub.teacher_lp, sub.mask, sub.seq_starts, threads=threads)
        oracle.opd_grad_rows(zh, sub.tokens, sub.mask, ref["dlp"], np.arange(end), threads=threads)
        reps += 1
        el = time.perf_counter() - t0
        if el >= target_s or el / reps * (reps + 1) > 3 * target_s:
            break
    return {
        "value": round(nbytes * reps / el / 1e9, 4),
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"responses 0..{r - 1} of {w.responses} ({end} tokens x {w.vocab} logits): loss, per-token "
                   f"values and every gradient row, run {reps}x in {el:.1f} s; float64 C oracle, OpenMP over tokens"),
    }


def bench_opd(args) -> int:
    """Per step one ctx_opd_loss_run over a full OPD batch: loss, per-token
    values and the bf16 logits gradient."""
    import torch

    from paper_2609_36608_amd import binding

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    w = wl.OPD_WORKLOADS["opd_qwen3"]
    b = wl.opd_batch(w)
    n = b.num_tokens
    t_setup = time.perf_counter()
    z = wl.opd_logits_device(w, b, dev)
    up = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dt)  # noqa: E731
    tok, old, tea = up(b.tokens, torch.int32), up(b.old_lp, torch.float32), up(b.teacher_lp, torch.float32)
    msk, st = up(b.mask, torch.uint8), up(b.seq_starts, torch.int32)
    out = {"grad_logits": torch.empty((n, w.row_stride), dtype=torch.bfloat16, device=dev),
           "loss": torch.empty(1, dtype=torch.float32, device=dev),
           "token_logp": torch.empty(n, dtype=torch.float32, device=dev),
           "token_weight": torch.empty(n, dtype=torch.float32, device=dev),
           "token_loss": torch.empty(n, dtype=torch.float32, device=dev)}
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t_setup
    stream = torch.cuda.current_stream()

    def step() -> None:
        binding.opd_loss(z, tok, old, tea, msk, st, out=out, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(args.steps):
        step()
    stop.record(stream)
    stop.synchronize()
    torch.cuda.synchronize()
    elapsed_s = start.elapsed_time(stop) / 1e3
    if args.calibrate_copy_gib > 0:
        ncopy = int(args.calibrate_copy_gib * 2**30) // 4
        src = torch.ones(ncopy, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    nbytes = opd_bytes(b, w.vocab)
    call_s = elapsed_s / args.steps
    gbs = nbytes / call_s / 1e9
    result = {
        "metric": OPD_METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(call_s * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.description,
            "name": w.name,
            "tokens": n,
            "supervised_tokens": int(b.mask.sum()),
            "vocab": w.vocab,
            "seed": wl.DEFAULT_SEED,
            "parallelism": "none (1 GPU)",
        },
        "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
        "tokens_per_s": round(n / call_s, 1),
        "roofline": {
            "bound": "hbm",
            "achieved": round(gbs, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(gbs / HBM_PEAK_GBS, 4),
            "ceiling": copy_ceiling(torch, dev, gbs),
            **traffic_fields(w.name, "opd_row_kernel"),
            "kernel": "opd_row_kernel (+ opd_weight_kernel, opd_reduce_kernel: one ctx_opd_loss_run call)",
            "bytes_per_launch": nbytes,
            "avg_launch_us": round(call_s * 1e6, 3),
        },
        "setup_s": round(setup_s, 1),
    }
    if not args.no_cpu_baseline:
        threads = len(os.sched_getaffinity(0))
        zfn = lambda rows: z[:rows].view(torch.int16).cpu().numpy().view(np.uint16)  # noqa: E731
        result["cpu_baseline"] = opd_cpu_baseline(w, b, zfn, args.cpu_seconds, threads)
    print(json.dumps(result), flush=True)
    return 0


SIM_METRIC = ("simulated rollout speedup, ActFirst-OPD over think-then-act (16 tasks, T=30, b_max=256, "
              "16-token fast actions, 512-token full responses), engine model with MI355X-measured attention cost")
SIM_CALIBRATIONS = 3  # independent calibrations; the headline is reported for each


def sim_contexts(n: int, turns: int, seed: int = wl.DEFAULT_SEED) -> np.ndarray:
    """Fixed interaction contexts reused across the virtual turns (as in the
    rollout-efficiency study): one ALFWorld-like prompt of U{1500..3000} tokens per task."""
    rng = wl.rng_for(seed, 30, 0, 0)
    return np.repeat(rng.integers(1500, 3001, size=n)[:, None], turns, axis=1).astype(np.int32)


def bench_sim(args) -> int:
    """Calibrate the engine model on the GPU (decode attention cost, read
    ceiling, prefill rate; all measured in this process), SIM_CALIBRATIONS
    times, then run the rollout scans of the rollout-efficiency study through
    the native engine-model simulator with each calibration."""
    import torch

    from paper_2609_36608_amd import binding
    from paper_2609_36608_amd import rollout_calibration as rcal

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    cals = [rcal.calibrate_engine(torch, dev) for _ in range(SIM_CALIBRATIONS)]
    n = 16

    def speedup(eng, turns, b_max, full_tokens):
        ctx = sim_contexts(n, turns)
        v = binding.rollout_simulate_engine(binding.ROLLOUT_VANILLA, ctx, 16, full_tokens, b_max, **eng)
        a = binding.rollout_simulate_engine(binding.ROLLOUT_ACTFIRST, ctx, 16, full_tokens, b_max, **eng)
        return v["completion"] / a["completion"], v, a

    heads = [speedup(c["engine"], 30, 256, 512)[0] for c in cals]
    cal = cals[int(np.argsort(heads)[len(heads) // 2])]  # the median calibration drives the scans
    eng = cal["engine"]
    t0 = time.perf_counter()
    conc = {ft: {b: round(speedup(eng, 30, b, ft)[0], 3) for b in (16, 32, 64, 128, 256)} for ft in (128, 512)}
    hor = {ft: {t: round(speedup(eng, t, 256, ft)[0], 3) for t in (1, 2, 4, 8, 16, 30)} for ft in (128, 512)}
    head, v, a = speedup(eng, 30, 256, 512)
    native_s = time.perf_counter() - t0
    nsim = 2 * (5 + 6) * 2 + 2
    requests = 2 * n * 30
    att = cal["attention"]
    result = {
        "metric": SIM_METRIC,
        "value": round(head, 4),
        "unit": "x",
        "n_gpus": 1,
        "steps": 1,
        "warmup": 0,
        "ms_per_step": round(native_s / nsim * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {
            "workload": "rollout-efficiency scans: 16 tasks, fixed contexts U{1500..3000} tokens, 16-token fast "
                        "actions, 128- or 512-token full responses; b_max scan at T=30, T scan at b_max=256",
            "engine": {k: float(f"{x:.6g}") for k, x in eng.items()},
            "engine_sources": cal["sources"],
            "parallelism": "none (1 GPU)",
        },
        "calibrations": [{"speedup": round(h, 4), "engine": {k: float(f"{x:.6g}") for k, x in c["engine"].items()},
                          "read_ceiling_gbs": c["read_ceiling"]["gbs"],
                          "prefill_tflops": round(c["prefill"]["tflops"], 1),
                          "attention_gbs": round(c["attention"]["achieved_gbs"], 1)} for h, c in zip(heads, cals)],
        "speedup_spread": {"min": round(min(heads), 4), "median": round(float(np.median(heads)), 4),
                           "max": round(max(heads), 4)},
        "speedup_vs_b_max_T30": conc,
        "speedup_vs_T_b_max256": hor,
        "paper_measured_A100_vllm": {"b_max16_to_256_128tok": [0.80, 1.49], "b_max16_to_256_512tok": [0.92, 2.42]},
        "completion_s": {"vanilla": round(v["completion"], 4), "actfirst": round(a["completion"], 4)},
        "simulations_per_s": round(nsim / native_s, 2),
        "requests_per_s": round(nsim * requests / native_s, 1),
        "roofline": {
            "bound": "hbm",
            "achieved": round(att["achieved_gbs"], 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(att["achieved_gbs"] / HBM_PEAK_GBS, 4),
            "ceiling": {"read_gbs": cal["read_ceiling"]["gbs"], "source": "ctx_hbm_read in this process"},
            "traffic": None,
            "kernel": ("ctx_decode_attn_run calls of the calibration (Qwen3-1.7B shape, 16/8 heads, batches 16..256, "
                       "distinct caches of >= 1 GiB in rotation per point)"),
            "bytes_per_launch": round(att["bytes_per_call"]),
            "avg_launch_us": round(att["avg_call_us"], 3),
        },
    }
    if not args.no_cpu_baseline:
        from oracle import oracle_sched as sch

        ctx = sim_contexts(n, 30).tolist()
        t1 = time.perf_counter()
        reps = 0
        while True:
            sch.simulate_engine(sch.VANILLA, ctx, 16, 512, 256, eng["step_base"], eng["step_per_kv_token"],
                                eng["prefill_per_token"])
            sch.simulate_engine(sch.ACTFIRST, ctx, 16, 512, 256, eng["step_base"], eng["step_per_kv_token"],
                                eng["prefill_per_token"])
            reps += 1
            el = time.perf_counter() - t1
            if el >= args.cpu_seconds or el / reps * (reps + 1) > 3 * args.cpu_seconds:
                break
        result["cpu_baseline"] = {
            "value": round(2 * reps * requests / el, 1),
            "unit": "requests/s",
            "cores": 1,
            "kind": "oracle",
            "sample": f"the headline pair of simulations (Vanilla and ActFirst, T=30, b_max=256, 512 tokens), "
                      f"{reps}x in {el:.1f} s; pure-Python oracle",
        }
    print(json.dumps(result), flush=True)
    return 0


def device_info(torch, dev) -> dict:
    """What the measurement ran on, as the runtime reports it."""
    pr = torch.cuda.get_device_properties(dev)
    return {
        "name": pr.name,
        "arch": getattr(pr, "gcnArchName", ""),
        "compute_units": pr.multi_processor_count,
        "hbm_gib": round(pr.total_memory / 2**30, 1),
    }


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64, help="decode steps timed (each = all layers)")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="long_ragged", choices=sorted(wl.WORKLOADS))
    ap.add_argument("--launch", choices=("both", "stream", "graph"), default="both",
                    help="decode: time stream launches, a HIP-graph replay of the same steps, or both "
                         "(default; `value` is then the graph replay)")
    ap.add_argument("--graph", action="store_const", dest="launch", const="graph",
                    help="decode: time the HIP-graph replay only")
    ap.add_argument("--paged", type=int, default=0, metavar="P",
                    help="use P-token pages (shuffled block tables) and append each step's token")
    ap.add_argument("--prefill", action="store_true",
                    help="time the causal prefill of the appended reference observation instead "
                         "(act_first_burst)")
    ap.add_argument("--prefill-p", choices=("both", "bf16", "split"), default="both",
                    help="with --prefill: softmax-weight precision(s) to time; `value` is the bf16 "
                         "weights (the default of ctx_prefill_attn_run) unless only split is timed")
    ap.add_argument("--opd", action="store_true",
                    help="time the fused OPD token loss + logits gradient instead (64 responses, Qwen3 vocabulary)")
    ap.add_argument("--sim", action="store_true",
                    help="calibrate the decode-step cost on the GPU and run the rollout scheduling scans")
    ap.add_argument("--ceiling", action="store_true",
                    help="time the library's streaming read and copy kernels (the practical HBM ceiling) instead")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--calibrate-copy-gib", type=float, default=0.0,
                    help="also run one device copy of this many GiB (HBM counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU (got --gpus {args.gpus}): the decode attention shards by "
              f"sequence with no exchange between GPUs, so run one process per GPU.",
              file=sys.stderr)
        return 2
    if args.steps < 1 or args.warmup < 0:
        print("bench.py: --steps must be >= 1 and --warmup >= 0", file=sys.stderr)
        return 2

    if args.prefill:
        return bench_prefill(args)
    if args.opd:
        return bench_opd(args)
    if args.sim:
        return bench_sim(args)
    if args.ceiling:
        return bench_ceiling(args)

    import torch

    from paper_2609_36608_amd.binding import DecodeAttention

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    w = wl.WORKLOADS[args.workload]
    layout = wl.workload_layout(w)
    B = w.batch

    # paged layout: each sequence's capacity rounded up to whole pages
    cache_rows = layout.num_rows
    if args.paged:
        if args.paged <= 0 or args.paged % 16:
            print("bench.py: --paged takes a positive multiple of 16", file=sys.stderr)
            return 2
        npages = -(-layout.capacity.astype(np.int64) // args.paged)
        cache_rows = int(npages.sum()) * args.paged
    # distinct per-layer caches; cycle fewer buffers if all layers exceed HBM
    layer_bytes = cache_rows * w.num_kv_heads * w.head_dim * 2 * 2
    n_buf = max(1, min(w.layers, HBM_BUDGET_BYTES // layer_bytes))
    t_setup = time.perf_counter()
    ks, vs = [], []
    for i in range(n_buf):
        k = torch.empty((cache_rows, w.num_kv_heads, w.head_dim), dtype=torch.bfloat16, device=dev)
        v = torch.empty_like(k)
        wl.fill_kv_device(k, v, w, i)  # N(0,1), plus the workload's peaky keys
        ks.append(k)
        vs.append(v)
    qs = []
    for layer in range(w.layers):
        q = torch.empty((B, w.num_q_heads, w.head_dim), dtype=torch.bfloat16, device=dev)
        wl.fill_normal_bf16_device(q, wl.DEFAULT_SEED, w.index, layer, 0)
        qs.append(q)
    outs = [torch.empty((B, w.num_q_heads, w.head_dim), dtype=torch.float32, device=dev) for _ in range(w.layers)]
    offsets = torch.from_numpy(layout.offsets).to(dev)
    lens_steps = torch.from_numpy(np.stack([layout.lens_at(s) for s in range(w.steps)])).to(dev)
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t_setup

    attn = DecodeAttention(w.num_q_heads, w.num_kv_heads, B, layout.max_seq_len, page_tokens=args.paged)
    stream = torch.cuda.current_stream()

    if args.paged:
        # the same rows, viewed as pages: sequence b's capacity is cut into P-token
        # pages whose block-table entries are shuffled over the whole cache
        P = args.paged
        rng = np.random.default_rng(wl.DEFAULT_SEED)
        num_pages = cache_rows // P
        perm = rng.permutation(num_pages).astype(np.int32)
        bt = np.zeros((B, int(npages.max())), np.int32)
        nxt = 0
        for b in range(B):
            bt[b, :npages[b]] = perm[nxt:nxt + npages[b]]
            nxt += npages[b]
        block_tables = torch.from_numpy(bt).to(dev)
        pages_k = [k.view(num_pages, P, w.num_kv_heads, w.head_dim) for k in ks]
        pages_v = [v.view(num_pages, P, w.num_kv_heads, w.head_dim) for v in vs]
        new_k = torch.empty((B, w.num_kv_heads, w.head_dim), dtype=torch.bfloat16, device=dev)
        new_v = torch.empty_like(new_k)
        wl.fill_normal_bf16_device(new_k, wl.DEFAULT_SEED, w.index, 0, 3)
        wl.fill_normal_bf16_device(new_v, wl.DEFAULT_SEED, w.index, 0, 4)

    def step(s: int) -> None:
        lens = lens_steps[s % w.steps]
        for layer in range(w.layers):
            if args.paged:
                attn.run_paged(qs[layer], pages_k[layer % n_buf], pages_v[layer % n_buf], block_tables, lens,
                               w.scale, outs[layer], k_new=new_k, v_new=new_v, stream=stream)
            else:
                attn.run(qs[layer], ks[layer % n_buf], vs[layer % n_buf], offsets, lens, w.scale,
                         outs[layer], stream=stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    def time_steps(use_graph: bool) -> float:
        """Seconds for exactly args.steps decode steps (all layers), HIP events on
        the launch stream; with use_graph the steps are captured once and the
        graph is replayed (after one untimed warm replay)."""
        nonlocal stream
        graph = None
        if use_graph:
            graph = torch.cuda.CUDAGraph()
            side = torch.cuda.Stream()
            side.wait_stream(stream)
            with torch.cuda.stream(side):
                with torch.cuda.graph(graph, stream=side):
                    saved = stream
                    stream = side
                    for s in range(args.steps):
                        step(s)
                    stream = saved
            torch.cuda.synchronize()
            graph.replay()  # warm replay
            torch.cuda.synchronize()
        start = torch.cuda.Event(enable_timing=True)
        stop = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(stream)
        if graph is not None:
            graph.replay()
        else:
            for s in range(args.steps):
                step(s)
        stop.record(stream)
        stop.synchronize()
        torch.cuda.synchronize()
        if graph is not None:
            # the spread: the same graph replayed REPEATS more times, each timed alone
            for _ in range(REPEATS):
                a = torch.cuda.Event(enable_timing=True)
                z = torch.cuda.Event(enable_timing=True)
                a.record(stream)
                graph.replay()
                z.record(stream)
                z.synchronize()
                repeat_s.append(a.elapsed_time(z) / 1e3)
        return start.elapsed_time(stop) / 1e3

    # stream launches, then (by default) the same steps replayed from one graph,
    # the way a serving engine runs its decode steps; `value` is the graph replay
    repeat_s: list[float] = []
    modes = {"both": (True, True), "stream": (True, False), "graph": (False, True)}[args.launch]
    stream_s = time_steps(False) if modes[0] else None
    graph_s = time_steps(True) if modes[1] else None
    elapsed_s = graph_s if graph_s is not None else stream_s

    step_bytes = [algorithmic_bytes(layout.lens_at(s % w.steps), w) * w.layers for s in range(args.steps)]
    total_bytes = float(sum(step_bytes))
    gbs = total_bytes / elapsed_s / 1e9
    calls = args.steps * w.layers
    call_s = elapsed_s / calls
    per_call_bytes = total_bytes / calls
    ms_per_step = elapsed_s * 1e3 / args.steps

    if args.calibrate_copy_gib > 0:
        n = int(args.calibrate_copy_gib * 2**30) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    ceiling = read_ceiling(torch, dev, per_call_bytes / call_s / 1e9)

    result = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.description,
            "name": w.name,
            "layers": w.layers,
            "batch": B,
            "num_q_heads": w.num_q_heads,
            "num_kv_heads": w.num_kv_heads,
            "head_dim": w.head_dim,
            "decode_steps": w.steps,
            "tokens_per_layer_step0": int(layout.lens.sum()),
            "distinct_layer_buffers": n_buf,
            "seed": wl.DEFAULT_SEED,
            "launch": "hip_graph" if graph_s is not None else "stream",
            "kv_layout": f"paged, {args.paged}-token pages, appends each step's token" if args.paged else "contiguous",
            "parallelism": "none (1 GPU)",
        },
        "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
        "decode_steps_per_s": round(args.steps / elapsed_s, 3),
        "tokens_per_s": round(B * args.steps / elapsed_s, 1),
        "roofline": {
            "bound": "hbm",
            "achieved": round(per_call_bytes / call_s / 1e9, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(per_call_bytes / call_s / 1e9 / HBM_PEAK_GBS, 4),
            "ceiling": ceiling,
            **traffic_fields(w.name, f"decode_split_kernel paged {args.paged}" if args.paged else "decode_split_kernel"),
            "kernel": "one ctx_decode_attn_run call (decode_split_kernel + decode_merge_kernel)",
            "bytes_per_launch": round(per_call_bytes),
            "avg_launch_us": round(call_s * 1e6, 3),
        },
        "setup_s": round(setup_s, 1),
        "device": device_info(torch, dev),
    }
    if repeat_s:
        rates = sorted(total_bytes / t / 1e9 for t in repeat_s)
        result["graph_repeats"] = {
            "n": len(rates),
            "median_gbs": round(float(np.median(rates)), 2),
            "min_gbs": round(rates[0], 2),
            "max_gbs": round(rates[-1], 2),
        }
    if graph_s is not None and stream_s is not None:
        result["stream_launches"] = {
            "value": round(total_bytes / stream_s / 1e9, 2),
            "ms_per_step": round(stream_s * 1e3 / args.steps, 4),
            "avg_launch_us": round(stream_s / calls * 1e6, 3),
        }
    if not args.no_cpu_baseline:
        threads = len(os.sched_getaffinity(0))
        result["cpu_baseline"] = cpu_baseline(w, layout, args.cpu_seconds, threads)
    print(json.dumps(result), flush=True)
    attn.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
