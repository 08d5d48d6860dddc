"""Build lib/libattnfuse.so from csrc/ with hipcc for gfx950.

Usage: python -m paper_2609_13612_amd.build [-j N]

Each translation unit compiles in its own hipcc process (they are independent
template-instantiation units), then one hipcc line links the shared library
in-tree so it travels with the source tree.
"""
import argparse
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "libattnfuse.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Packed fp32 VALU ops are disabled for every device compile.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", f"-I{INCLUDE}", f"-I{CSRC}",
          "-Wall", "-Wno-unused-function"]

SOURCES = ["api.cpp", "rope.hip", "fwd_bf16.hip", "fwd_fp32.hip", "bwd_bf16.hip", "bwd_dkdv.hip", "bwd_fp32.hip",
           "decode.hip"]
# Code-generation options of single translation units.  The dK/dV kernels
# run faster when the machine scheduler keeps its first schedule instead of
# re-scheduling high-register-pressure regions without memory-op clustering
# (same box, HIP-graph replays: 4.2 % at the Llama-3-8B shape, 4.0 % under a
# 1024-key window, 1.3 % at D = 64, 0.6 % with ALiBi; no instantiation
# spills).  The dQ kernels keep the default: with the option their ALiBi and
# window instantiations ran 5-10 % slower.
SOURCE_FLAGS = {"bwd_dkdv.hip": ["-mllvm", "-amdgpu-disable-unclustered-high-rp-reschedule=1"]}


def _compile(src):
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, "-c", os.path.join(CSRC, src), "-o", obj] + COMMON
    if src.endswith(".hip"):
        cmd += DEVICE_FLAGS + SOURCE_FLAGS.get(src, [])
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    return src, obj, res.returncode, err


def build(jobs=None, verbose=False):
    """Compile every source and link the library; raises RuntimeError on failure."""
    if shutil.which(HIPCC) is None and not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    jobs = jobs or min(len(SOURCES), os.cpu_count() or 4)
    objs = []
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        for src, obj, rc, err in ex.map(_compile, SOURCES):
            if rc != 0:
                raise RuntimeError(f"hipcc failed on {src}:\n{err}")
            if verbose and err.strip():
                print(f"[{src}]\n{err}", file=sys.stderr)
            objs.append(obj)
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("-j", type=int, default=None)
    ap.add_argument("-v", action="store_true")
    a = ap.parse_args()
    print(build(a.j, a.v))
