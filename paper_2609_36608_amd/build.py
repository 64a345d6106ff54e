"""Build libctx_decode_attn.so (HIP, gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "ctx_decode_attn.hip")
SRCS = [SRC, os.path.join(PKG, "csrc", "ctx_prefill_attn.hip"), os.path.join(PKG, "csrc", "ctx_opd_loss.hip"),
        os.path.join(PKG, "csrc", "ctx_ceiling_probe.hip"), os.path.join(PKG, "csrc", "ctx_rollout_sim.cpp")]
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


# Extra device-compiler flags per source file.
FILE_FLAGS = {
    # The OPD row kernel holds a row's 16-byte chunks in a small array indexed
    # by the unrolled chunk loops.  Promoting that array to one vector value
    # made the instantiations for up to 8 chunks per thread spill hundreds of
    # VGPRs; kept as separate registers they need 44-64.
    "ctx_opd_loss.hip": ["-mllvm", "-disable-promote-alloca-to-vector"],
}
BUILD_DIR = os.path.join(PKG, "_build")
_NOISE = "is not a recognized feature for this target"


def _run(cmd: list[str], verbose: bool) -> None:
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [l for l in (res.stdout + res.stderr).splitlines() if _NOISE not in l]
    if msgs and (verbose or res.returncode):
        print("\n".join(msgs), file=sys.stderr, flush=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}): {' '.join(cmd[-3:])}")


def build(verbose: bool = False, extra: list[str] | None = None, out: str | None = None) -> str:
    """Compile every source to an object (in parallel, each with its own extra
    flags), then link the shared library `out` (default: the in-tree library)."""
    out = out or LIB
    os.makedirs(BUILD_DIR, exist_ok=True)
    objdir = tempfile.mkdtemp(dir=BUILD_DIR)
    try:
        def compile_one(src: str) -> str:
            obj = os.path.join(objdir, os.path.basename(src) + ".o")
            _run([hipcc(), *compile_flags(), *FILE_FLAGS.get(os.path.basename(src), []), *(extra or []),
                  "-c", src, "-o", obj], verbose)
            return obj

        with ThreadPoolExecutor(max_workers=len(SRCS)) as pool:
            objs = list(pool.map(compile_one, SRCS))
        _run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", out + ".tmp", *objs], verbose)
    finally:
        shutil.rmtree(objdir, ignore_errors=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
