"""Build libctx_decode_attn.so (HIP, gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "ctx_decode_attn.hip")
SRCS = [SRC, os.path.join(PKG, "csrc", "ctx_prefill_attn.hip"), os.path.join(PKG, "csrc", "ctx_opd_loss.hip"),
        os.path.join(PKG, "csrc", "ctx_rollout_sim.cpp")]
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libctx_decode_attn.so")
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc"),
                 shutil.which("hipcc") or ""):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def compile_flags() -> list[str]:
    return [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
            # no packed-fp32 VALU instructions in device code
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            # MFMA results in VGPRs: the kernels post-process them with VALU ops,
            # so AGPR destinations would only add copies
            "-mllvm", "-amdgpu-mfma-vgpr-form",
            "-I", INCLUDE]


def build(verbose: bool = False, extra: list[str] | None = None, out: str | None = None) -> str:
    out = out or LIB
    cmd = [hipcc(), *compile_flags(), *(extra or []), "-shared", "-o", out + ".tmp", *SRCS]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msgs = [l for l in (res.stdout + res.stderr).splitlines() if noise not in l]
    if msgs and (verbose or res.returncode):
        print("\n".join(msgs), file=sys.stderr, flush=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode})")
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
