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
SOURCES = ["api.hip", "route.hip", "ffn.hip", "ffn_fp8.hip", "ffn_gemm.hip", "ffn_prefill8.hip", "offload.hip"]

# Packed-fp32 VALU ops are disabled on every HIP translation unit.
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wno-unused-command-line-argument"]


# Host-side AddressSanitizer and UndefinedBehaviorSanitizer for a checking
# build of the host code (argument validation, workspace layout, the
# residency plan); each flag is scoped to the host pass, the device code is
# built as usual.
SANITIZE_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]


def asan_runtime() -> str:
    """The ASan runtime a process must preload to load the sanitized build."""
    clang = os.path.join(os.path.dirname(os.path.realpath(hipcc())), "..", "lib", "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang"
    out = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    return out.stdout.strip()


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False, out: str = LIB, defines=(), sanitize_host: bool = False) -> str:
    """Compile every HIP source into one shared library; returns its path.
    ``defines`` are extra -D options (tuning knobs of the kernels);
    ``sanitize_host`` builds the host code with ASan and UBSan (load it with
    the runtime of ``asan_runtime()`` preloaded)."""
    objs = []
    t0 = time.time()
    procs = []
    flags = HIP_FLAGS + (["-g", *SANITIZE_HOST] if sanitize_host else [])
    os.makedirs(os.path.dirname(out), exist_ok=True)
    for src in SOURCES:
        obj = out + "." + src.replace(".hip", ".o")
        cmd = [hipcc(), *flags, *[f"-D{d}" for d in defines], "-c", os.path.join(CSRC, src), "-o", obj]
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
    link = [*SANITIZE_HOST, "-shared-libasan"] if sanitize_host else []
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *link, *objs, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    for o in objs:
        os.remove(o)
    if verbose:
        print(f"built {out} in {time.time() - t0:.1f}s", flush=True)
    return out


if __name__ == "__main__":
    build(verbose=True)
