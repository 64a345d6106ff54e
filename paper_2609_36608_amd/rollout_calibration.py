"""Engine parameters of the rollout scheduling simulator, measured on this GPU.

The engine model of ctx_rollout_simulate_engine prices one decode step as

    step_base + step_per_kv_token * (tokens cached by the admitted requests)
              + prefill_per_token * (context tokens admitted at that step)

(the step model of App. finite concurrency).  As in the paper's calibrated
rollout estimate (eq:calibrated-rollout-speedup), the costs come from
measurements, here of this library's kernels in the calling process:

  * attention: ctx_decode_attn_run at the student's shape, timed over several
    batches and context lengths, each point cycling distinct caches that
    together exceed the 256 MB on-die cache; a least-squares line gives
    seconds per call = a + b * KV tokens, and a step costs layers * (a + b * tokens);
  * weight streaming: the student's bf16 parameters read once per step at the
    read ceiling measured by ctx_hbm_read;
  * prefill: 2 x parameters flops per admitted context token at the
    matrix-core rate of this library's causal prefill kernel
    (ctx_prefill_attn_run), measured on a burst of new tokens over cached history.

Only device memory and streams come from PyTorch; every timed kernel is one of
this library's.
"""
from __future__ import annotations

import math

import numpy as np

from . import binding
from . import workloads as wl

# Qwen3-1.7B, the student of the rollout-efficiency study: 28 layers, 16 query
# and 8 KV heads of 128, about 1.72e9 bf16 parameters streamed once per decode step
STUDENT_LAYERS, STUDENT_HQ, STUDENT_HKV, STUDENT_PARAMS = 28, 16, 8, 1.72e9

# (batch, context tokens) points of the attention fit
POINTS_FULL = ((16, 2048), (64, 2048), (64, 4096), (128, 3072), (256, 2048), (256, 4096))
POINTS_REDUCED = ((16, 2048), (64, 4096), (256, 2048))
ROTATION_BYTES = 1 << 30  # distinct caches per point: at least this many bytes in rotation
PROBE_WORKGROUPS_PER_CU = 16  # grid of the streaming probes (a sweep of 2..64 per CU moved the rate by ~1%)


def _events(torch):
    return torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)


def measure_hbm(torch, dev, gib: float = 4.0, reps: int = 8, copy: bool = False, nontemporal: bool = True,
                workgroups: int | None = None) -> dict:
    """Streaming rate of ctx_hbm_read (copy=False) or ctx_hbm_copy over a
    buffer of `gib` GiB: GB/s of bytes moved (a copy moves each byte twice),
    median and best of `reps` timed launches after one untimed one."""
    if workgroups is None:
        workgroups = PROBE_WORKGROUPS_PER_CU * torch.cuda.get_device_properties(dev).multi_processor_count
    n = int(gib * 2**30) // 16 * 16
    src = torch.empty(n, dtype=torch.uint8, device=dev)
    src.view(torch.int32).fill_(0x3F80_1234)
    dst = torch.empty(n, dtype=torch.uint8, device=dev) if copy else None
    sink = torch.empty(workgroups * binding.CTX_HBM_SINK_BYTES_PER_WORKGROUP, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)

    def launch():
        if copy:
            binding.ctx_hbm_copy(src, dst, workgroups, nontemporal, stream)
        else:
            binding.ctx_hbm_read(src, sink, workgroups, nontemporal, stream)

    launch()
    torch.cuda.synchronize(dev)
    times = []
    for _ in range(reps):
        e0, e1 = _events(torch)
        e0.record(stream)
        launch()
        e1.record(stream)
        e1.synchronize()
        times.append(e0.elapsed_time(e1) / 1e3)
    moved = n * (2 if copy else 1)
    rates = sorted(moved / t / 1e9 for t in times)
    del src, dst, sink
    return {"gbs": round(float(np.median(rates)), 1), "best_gbs": round(rates[-1], 1), "bytes": moved,
            "reps": reps, "workgroups": workgroups, "nontemporal": nontemporal,
            "kernel": "ctx_hbm_copy" if copy else "ctx_hbm_read"}


def measure_mfma(torch, dev, shape: int = binding.CTX_MFMA_16X16X32, waves_per_simd: int = 2,
                 iterations: int = 4096, reps: int = 5) -> dict:
    """bf16 matrix-core rate of ctx_mfma_bf16 (TFLOP/s, median and best of
    `reps` timed launches after one untimed one), with `waves_per_simd`
    four-wave workgroups per compute unit."""
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    workgroups = cus * waves_per_simd
    sink = torch.empty(workgroups * binding.CTX_HBM_SINK_BYTES_PER_WORKGROUP, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    binding.ctx_mfma_bf16(shape, workgroups, iterations, sink, stream)
    torch.cuda.synchronize(dev)
    rates = []
    for _ in range(reps):
        e0, e1 = _events(torch)
        e0.record(stream)
        flops = binding.ctx_mfma_bf16(shape, workgroups, iterations, sink, stream)
        e1.record(stream)
        e1.synchronize()
        rates.append(flops / (e0.elapsed_time(e1) / 1e3) / 1e12)
    rates.sort()
    return {"tflops": round(float(np.median(rates)), 1), "best_tflops": round(rates[-1], 1),
            "shape": "16x16x32" if shape == binding.CTX_MFMA_16X16X32 else "32x32x16",
            "waves_per_simd": waves_per_simd, "kernel": "ctx_mfma_bf16"}


def calibrate_attention(torch, dev, points=POINTS_FULL, reps: int = 40) -> dict:
    """Seconds per ctx_decode_attn_run call at the student's shape for each
    (batch, context) point, every point cycling distinct K/V caches of at
    least ROTATION_BYTES in total; least-squares fit a + b * KV tokens."""
    pts = []
    total_bytes, total_s, calls = 0, 0.0, 0
    stream = torch.cuda.current_stream(dev)
    for batch, ctx in points:
        lens = np.full(batch, ctx, np.int32)
        layout = wl.make_layout(lens, 1)
        layer_bytes = layout.num_rows * STUDENT_HKV * 128 * 2 * 2
        nbuf = max(2, math.ceil(ROTATION_BYTES / layer_bytes))
        w = wl.Workload("calibration", 0, 1, batch, STUDENT_HQ, STUDENT_HKV, 1, "uniform", ctx, ctx)
        caches = []
        for i in range(nbuf):
            k = torch.empty((layout.num_rows, STUDENT_HKV, 128), dtype=torch.bfloat16, device=dev)
            v = torch.empty_like(k)
            wl.fill_kv_device(k, v, w, 1000 * batch + i, seed=7)
            caches.append((k, v))
        q = torch.empty((batch, STUDENT_HQ, 128), dtype=torch.bfloat16, device=dev)
        wl.fill_normal_bf16_device(q, 7, batch, ctx, 0)
        out = torch.empty((batch, STUDENT_HQ, 128), dtype=torch.float32, device=dev)
        offs = torch.from_numpy(layout.offsets).to(dev)
        tl = torch.from_numpy(lens).to(dev)
        with binding.DecodeAttention(STUDENT_HQ, STUDENT_HKV, batch, ctx) as attn:
            for i in range(nbuf):
                attn.run(q, *caches[i], offs, tl, w.scale, out, stream=stream)
            torch.cuda.synchronize(dev)
            e0, e1 = _events(torch)
            e0.record(stream)
            for i in range(reps):
                attn.run(q, *caches[i % nbuf], offs, tl, w.scale, out, stream=stream)
            e1.record(stream)
            e1.synchronize()
            sec = e0.elapsed_time(e1) / 1e3 / reps
        pts.append({"batch": batch, "context": ctx, "kv_tokens": batch * ctx, "seconds": sec, "buffers": nbuf})
        from_bytes = _decode_bytes(lens)
        total_bytes += from_bytes * reps
        total_s += sec * reps
        calls += reps
        del caches, q, out
    x = np.array([p["kv_tokens"] for p in pts], np.float64)
    y = np.array([p["seconds"] for p in pts], np.float64)
    b, a = np.polyfit(x, y, 1)
    torch.cuda.empty_cache()
    return {"per_call_s": float(a), "per_kv_token_s": float(b), "points": pts,
            "achieved_gbs": total_bytes / total_s / 1e9, "avg_call_us": total_s / calls * 1e6,
            "bytes_per_call": total_bytes / calls}


def _decode_bytes(lens: np.ndarray) -> int:
    """Algorithmic bytes of one decode call at the student's shape (K and V
    read once, q read, fp32 out written, offsets and lengths)."""
    b = len(lens)
    return int(lens.astype(np.int64).sum()) * STUDENT_HKV * 128 * 4 + b * STUDENT_HQ * 128 * 6 + 8 * b


def measure_prefill_rate(torch, dev, batch: int = 64, history: int = 4096, new: int = 256, reps: int = 6) -> dict:
    """TFLOP/s of ctx_prefill_attn_run (bf16 softmax weights) for `batch`
    sequences each prefilling `new` tokens over `history` cached ones, at the
    student's heads."""
    lens = np.full(batch, history + new, np.int32)
    nq = np.full(batch, new, np.int32)
    layout = wl.make_layout(lens, 1)
    w = wl.Workload("prefill-calibration", 0, 1, batch, STUDENT_HQ, STUDENT_HKV, 1, "uniform", 1, 2)
    k = torch.empty((layout.num_rows, STUDENT_HKV, 128), dtype=torch.bfloat16, device=dev)
    v = torch.empty_like(k)
    wl.fill_kv_device(k, v, w, 0, seed=11)
    q = torch.empty((batch * new, STUDENT_HQ, 128), dtype=torch.bfloat16, device=dev)
    wl.fill_normal_bf16_device(q, 11, batch, new, 0)
    out = torch.empty((batch * new, STUDENT_HQ, 128), dtype=torch.float32, device=dev)
    i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(dev)  # noqa: E731
    qs = np.arange(batch, dtype=np.int32) * new
    stream = torch.cuda.current_stream(dev)
    with binding.DecodeAttention(STUDENT_HQ, STUDENT_HKV, batch, history + new) as attn:
        args = (q, k, v, i32(layout.offsets), i32(lens), i32(qs), i32(nq), new, w.scale, out)
        attn.prefill(*args, stream=stream)
        torch.cuda.synchronize(dev)
        e0, e1 = _events(torch)
        e0.record(stream)
        for _ in range(reps):
            attn.prefill(*args, stream=stream)
        e1.record(stream)
        e1.synchronize()
        sec = e0.elapsed_time(e1) / 1e3 / reps
    positions = batch * (new * history + new * (new + 1) // 2)
    flops = positions * 4 * 128 * STUDENT_HQ
    del k, v, q, out
    torch.cuda.empty_cache()
    return {"tflops": flops / sec / 1e12, "seconds": sec, "flops": flops, "batch": batch, "history": history,
            "new": new, "kernel": "ctx_prefill_attn_run (bf16 softmax weights)"}


def calibrate_engine(torch, dev, reduced: bool = False) -> dict:
    """Engine parameters for ctx_rollout_simulate_engine from this process's
    measurements, with where each one comes from."""
    att = calibrate_attention(torch, dev, POINTS_REDUCED if reduced else POINTS_FULL, reps=20 if reduced else 40)
    read = measure_hbm(torch, dev, gib=2.0 if reduced else 4.0, reps=4 if reduced else 8)
    pf = measure_prefill_rate(torch, dev, batch=16 if reduced else 64, reps=3 if reduced else 6)
    weight_s = STUDENT_PARAMS * 2 / (read["gbs"] * 1e9)
    engine = {
        "step_base": weight_s + STUDENT_LAYERS * att["per_call_s"],
        "step_per_kv_token": STUDENT_LAYERS * att["per_kv_token_s"],
        "prefill_per_token": 2 * STUDENT_PARAMS / (pf["tflops"] * 1e12),
    }
    sources = {
        "step_base": (f"{STUDENT_PARAMS:.3g} bf16 parameters at the measured read ceiling "
                      f"({read['gbs']:.0f} GB/s, {read['kernel']}) + {STUDENT_LAYERS} x the fitted per-call "
                      f"attention cost ({att['per_call_s'] * 1e6:.2f} us)"),
        "step_per_kv_token": (f"{STUDENT_LAYERS} x the fitted per-KV-token attention cost "
                              f"({att['per_kv_token_s'] * 1e12:.3f} ps/token, ctx_decode_attn_run at "
                              f"{STUDENT_HQ}/{STUDENT_HKV} heads, {len(att['points'])} points)"),
        "prefill_per_token": (f"2 x {STUDENT_PARAMS:.3g} flops per token at the measured prefill rate "
                              f"({pf['tflops']:.0f} TFLOP/s, {pf['kernel']})"),
    }
    return {"engine": engine, "sources": sources, "attention": att, "read_ceiling": read, "prefill": pf}
