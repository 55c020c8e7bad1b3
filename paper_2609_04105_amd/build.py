"""Build libfp4attn.so (the HIP kernels and the C-ABI) in-tree with hipcc for gfx950.

Usage: python paper_2609_04105_amd/build.py [--jobs N]   (does not import the package)
"""
import argparse
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libfp4attn.so")
SOURCES = ["fwd_mxfp4_guard.hip", "fwd_mxfp4_causal.hip", "fwd_mxfp4_ex2.hip", "fwd_mxfp4.hip",
           "fwd_mxfp4_ex2_dense.hip", "fwd_mxfp4_fp8pv.hip", "fwd_bf16.hip", "api.hip", "quantize.hip", "mfma_stream.hip"]
# The attention kernels never rely on NaN ordering in fmax; without this flag the
# compiler canonicalizes every fmax operand with an extra v_max_f32.
EXTRA = {f: ["-fno-honor-nans"] for f in ("fwd_mxfp4.hip", "fwd_mxfp4_ex2.hip", "fwd_mxfp4_ex2_dense.hip",
                                          "fwd_mxfp4_guard.hip", "fwd_mxfp4_causal.hip", "fwd_mxfp4_fp8pv.hip",
                                          "fwd_bf16.hip")}
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")
FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-function",
    # packed fp32 vector instructions stay disabled for every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _compile(src):
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *EXTRA.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err.strip():
        sys.stderr.write(err + "\n")
    return obj


def build(jobs=8, verbose=True):
    """Compile every HIP source for gfx950 and link the shared library (always rebuilds)."""
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=8)
    build(ap.parse_args().jobs)
