"""Build libboostcap.so (HIP for gfx950 + host C++) in-tree.

Usage: python -m paper_2609_13592_amd.build   (or build() from Python)
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.environ.get("BOOST_OUT_DIR") or os.path.join(HERE, "_lib")
LIB = os.path.join(OUT_DIR, "libboostcap.so")
ROOT = os.path.dirname(HERE)

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
EXTRA = os.environ.get("BOOST_EXTRA_FLAGS", "").split()
# -amdgpu-mfma-vgpr-form: MFMA accumulators stay in VGPRs (left to itself the
# register allocator moved the GEMM accumulators between AGPRs and VGPRs on
# every step, stalling each MFMA on those moves)
HIP_FLAGS = EXTRA + ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-mllvm", "-amdgpu-mfma-vgpr-form=1",
             "-Wall", "-Wno-unused-function", "-Wno-unused-command-line-argument",
             f"-I{ROOT}/include"]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", f"-I{ROOT}/include"]


def _sources():
    hip = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    cpp = sorted(f for f in os.listdir(CSRC) if f.endswith(".cpp"))
    return hip, cpp


def _compile(src: str, obj: str, is_hip: bool):
    if is_hip:
        cmd = [HIPCC, *HIP_FLAGS, "-x", "hip", "-c", src, "-o", obj]
    else:
        cmd = ["g++", *CXX_FLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature: harmless warning
    err = "\n".join(l for l in r.stderr.splitlines()
                    if "packed-fp32-ops" not in l and "not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stderr}")
    return err.strip()


def build(verbose: bool = False) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    obj_dir = os.path.join(OUT_DIR, "obj")
    os.makedirs(obj_dir, exist_ok=True)
    hip, cpp = _sources()
    jobs = []
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 4)) as ex:
        for f in hip:
            jobs.append(ex.submit(_compile, os.path.join(CSRC, f),
                                  os.path.join(obj_dir, f + ".o"), True))
        for f in cpp:
            jobs.append(ex.submit(_compile, os.path.join(CSRC, f),
                                  os.path.join(obj_dir, f + ".o"), False))
        for j in jobs:
            msg = j.result()
            if msg and verbose:
                print(msg, file=sys.stderr)
    objs = [os.path.join(obj_dir, f + ".o") for f in hip + cpp]
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
