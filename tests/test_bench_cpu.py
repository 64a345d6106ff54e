"""Host-side parts of bench.py: the algorithmic byte count the reported GB/s
divides by, and the refusal of more than one GPU (no GPU needed)."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2609_36608_amd import workloads as wl  # noqa: E402


def test_algorithmic_bytes_by_hand():
    # 2 sequences of 3 and 5 tokens, 4 query heads over 2 KV heads, D = 128:
    # K and V: 8 tokens x 2 heads x 128 x 2 B x 2 = 8192; q (bf16) and out (fp32):
    # 2 x 4 x 128 x (2 + 4) = 6144; offsets and lengths: 2 x 8 = 16
    w = wl.Workload("byhand", 0, 1, 2, 4, 2, 1, "uniform", 1, 8)
    assert bench.algorithmic_bytes(np.array([3, 5], np.int32), w) == 8192 + 6144 + 16
    # bf16 out: 2 x 4 x 128 x (2 + 2)
    assert bench.algorithmic_bytes(np.array([3, 5], np.int32), w, out_bytes=2) == 8192 + 4096 + 16


def test_algorithmic_bytes_long_batch_step0():
    # the long-horizon batch: every K/V byte of every token once, 36 layers per step
    w = wl.WORKLOADS["long_ragged"]
    lens = wl.workload_layout(w).lens_at(0)
    kv = int(lens.sum()) * 8 * 128 * 4
    assert bench.algorithmic_bytes(lens, w) == kv + 32 * 32 * 128 * 6 + 32 * 8


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_cpu_baseline_reports_threads_single_thread_and_model():
    # the oracle baseline on the tiny batch: the multi-thread and one-thread rates
    # over the same sample, the thread counts used, and the host CPU's model
    w = wl.WORKLOADS["tiny"]
    r = bench.cpu_baseline(w, wl.workload_layout(w), 0.2, 2, single_thread_s=0.1)
    assert r["kind"] == "oracle" and r["cores"] == 2 and r["unit"] == "GB/s" and r["value"] > 0
    assert r["single_thread"]["cores"] == 1 and r["single_thread"]["value"] > 0
    assert r["single_thread"]["runs"] >= 1
    assert isinstance(r["cpu_model"], str)


def test_roofline_traffic_is_bytes_per_launch_from_a_current_profile():
    """`traffic` is a plain byte count, taken from a committed counter summary
    only while the kernel source still hashes to the one it records."""
    import glob
    import hashlib

    paths = glob.glob(os.path.join(ROOT, "profiles", "*hbm_traffic*.md"))
    assert paths
    for path in paths:
        fields = dict(line.strip().split(": ", 1) for line in open(path)
                      if line.startswith(("kernel", "workload", "traffic_bytes")) and ": " in line)
        src = fields.get("kernel_source", "paper_2609_36608_amd/csrc/ctx_decode_attn.hip")
        current = hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest()
        got = bench.traffic_fields(fields["workload"], fields.get("kernel", "decode_split_kernel"))
        if current == fields["kernel_source_sha256"]:
            assert got["traffic"] == int(fields["traffic_bytes_per_launch"])
            assert isinstance(got["traffic"], int)
            assert got["traffic_detail"]["source"] == os.path.relpath(path, ROOT)
        else:
            assert got == {"traffic": None, "traffic_detail": None}
    assert bench.traffic_fields("no_such_workload") == {"traffic": None, "traffic_detail": None}
