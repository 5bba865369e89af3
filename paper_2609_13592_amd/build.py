"""Build libboostcap.so (HIP for gfx950 + host C++) in-tree.

Usage: python -m paper_2609_13592_amd.build   (or build() from Python)

       python -m paper_2609_13592_amd.build --sanitize
           host-code AddressSanitizer (+ UndefinedBehaviorSanitizer for the
           plain C++ files) build into _lib_sanitize/, for the CPU tests:
           BOOST_LIB=<that .so> LD_PRELOAD="<libasan.so> <libubsan.so>"
           ASAN_OPTIONS=detect_leaks=0 python -m pytest tests -m "not gpu".
           Device code is built as usual (no GPU sanitizer).
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


# host-only sanitizer flags: each -fsanitize= right after -Xarch_host on the
# hipcc lines, so device code is never built with it
SAN_HIP = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]
SAN_CXX = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-fno-omit-frame-pointer"]


def _compile(src: str, obj: str, is_hip: bool, sanitize: bool = False):
    if is_hip:
        cmd = [HIPCC, *HIP_FLAGS, *(SAN_HIP if sanitize else []), "-x", "hip", "-c", src,
               "-o", obj]
    else:
        cmd = ["g++", *CXX_FLAGS, *(SAN_CXX if sanitize else []), "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature: harmless warning
    err = "\n".join(l for l in r.stderr.splitlines()
                    if "packed-fp32-ops" not in l and "not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stderr}")
    return err.strip()


def build(verbose: bool = False, sanitize: bool = False) -> str:
    out_dir = os.path.join(HERE, "_lib_sanitize") if sanitize else OUT_DIR
    lib = os.path.join(out_dir, "libboostcap.so")
    os.makedirs(out_dir, exist_ok=True)
    obj_dir = os.path.join(out_dir, "obj")
    os.makedirs(obj_dir, exist_ok=True)
    hip, cpp = _sources()
    jobs = []
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 4)) as ex:
        for f in hip:
            jobs.append(ex.submit(_compile, os.path.join(CSRC, f),
                                  os.path.join(obj_dir, f + ".o"), True, sanitize))
        for f in cpp:
            jobs.append(ex.submit(_compile, os.path.join(CSRC, f),
                                  os.path.join(obj_dir, f + ".o"), False, sanitize))
        for j in jobs:
            msg = j.result()
            if msg and verbose:
                print(msg, file=sys.stderr)
    objs = [os.path.join(obj_dir, f + ".o") for f in hip + cpp]
    tmp = lib + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, *objs]
    if sanitize:
        cmd += ["-Xarch_host", "-fsanitize=address", "-lubsan"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stderr}")
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose=True, sanitize="--sanitize" in sys.argv[1:]))
