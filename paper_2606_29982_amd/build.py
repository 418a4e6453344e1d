"""Build the CAEE HIP library (libcaee.so) in-tree for gfx950 with hipcc."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libcaee.so")
SOURCES = ["api.hip", "route.hip", "ffn.hip", "ffn_fp8.hip", "ffn_gemm.hip", "offload.hip"]

# Packed-fp32 VALU ops are disabled on every HIP translation unit.
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wno-unused-command-line-argument"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False, out: str = LIB, defines=()) -> str:
    """Compile every HIP source into one shared library; returns its path.
    ``defines`` are extra -D options (tuning knobs of the kernels)."""
    objs = []
    t0 = time.time()
    procs = []
    for src in SOURCES:
        obj = out + "." + src.replace(".hip", ".o")
        cmd = [hipcc(), *HIP_FLAGS, *[f"-D{d}" for d in defines], "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
        objs.append(obj)
    for src, pr in procs:
        log, _ = pr.communicate()
        if pr.returncode != 0:
            sys.stderr.write(log.decode(errors="replace"))
            raise RuntimeError(f"hipcc failed on {src}")
        if verbose and log:
            sys.stderr.write(log.decode(errors="replace"))
    tmp = out + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    for o in objs:
        os.remove(o)
    if verbose:
        print(f"built {out} in {time.time() - t0:.1f}s", flush=True)
    return out


if __name__ == "__main__":
    build(verbose=True)
