"""Builds libheadkv.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree,
and the measurement tool stream_probe (launch floor and streaming ceiling at
the attention kernel's launch shape; not part of the library)."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libheadkv.so")
PROBE = os.path.join(HERE, "stream_probe")
SOURCES = ["cache_kernels.hip", "attn_kernels.hip", "prefill_attn.hip", "scratch.hip",
           "headkv_abi.cpp"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wextra",
    # no packed fp32 instructions (v_pk_*_f32) in generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]

# per source: the attention kernels and the fused update + attention kernel
# take the arguments their first loads need as leading plain arguments,
# preloaded into scalar registers at wave launch (and so do the probe's
# kernels, which bound them)
PRELOAD = ["-mllvm", "-amdgpu-kernarg-preload-count=16"]
SOURCE_FLAGS = {"attn_kernels.hip": PRELOAD, "cache_kernels.hip": PRELOAD,
                "stream_probe.hip": PRELOAD}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; the HIP library cannot be built")


def build(verbose: bool = False) -> str:
    """Compile every source and link the shared library; returns its path."""
    out_dir = os.path.join(HERE, "_build")
    os.makedirs(out_dir, exist_ok=True)
    objs = []
    for src in SOURCES:
        obj = os.path.join(out_dir, src + ".o")
        cmd = [hipcc(), *HIPCC_FLAGS, *SOURCE_FLAGS.get(src, []), "-I",
               os.path.join(ROOT, "include"), "-c",
               os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        objs.append(obj)
    tmp = LIB + f".tmp{os.getpid()}"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    tmp = PROBE + f".tmp{os.getpid()}"
    cmd = [hipcc(), *HIPCC_FLAGS, *SOURCE_FLAGS["stream_probe.hip"],
           os.path.join(CSRC, "stream_probe.hip"), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, PROBE)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
