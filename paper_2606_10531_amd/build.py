"""Build liblcvq.so (all HIP sources, gfx950) in-tree with hipcc."""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "liblcvq.so")
SOURCES = ["lcvq_api.hip", "lcvq_prep.hip", "lcvq_gemm.hip", "lcvq_f32.hip", "lcvq_adam.hip", "lcvq_packed.hip", "lcvq_encode.hip"]
ARCH = "gfx950"
# Packed fp32 instructions are kept out of every kernel; the host pass warns
# that it does not know the feature, which is harmless.
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-Wno-unused-result"]


# The products' epilogues issue matrix-core instructions through the compiler's
# builtins, accumulating in vector registers (the accumulator registers hold the
# main loop's results): select the vector-register form for them.
PER_FILE_FLAGS = {"lcvq_gemm.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=true"]}


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build liblcvq.so)")


def _run(cmd):
    p = subprocess.run(cmd, capture_output=True, text=True)
    if p.returncode != 0:
        raise RuntimeError("command failed: " + " ".join(cmd) + "\n" + p.stdout + p.stderr)
    return p


def build(verbose: bool = False) -> str:
    """Compile every HIP source and link liblcvq.so; returns its path."""
    cc = hipcc()
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    jobs = []
    for s in SOURCES:
        obj = os.path.join(objdir, s.replace(".hip", ".o"))
        jobs.append((obj, [cc, *FLAGS, *PER_FILE_FLAGS.get(s, []), "-c", os.path.join(CSRC, s), "-o", obj]))
    with cf.ThreadPoolExecutor(max_workers=min(len(jobs), 8)) as ex:
        for obj, p in zip([j[0] for j in jobs], ex.map(_run, [j[1] for j in jobs])):
            if verbose:
                print(obj, p.stderr.strip()[-400:])
    tmp = LIB + ".tmp"
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *[j[0] for j in jobs]])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
