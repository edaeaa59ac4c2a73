"""Build libtandem.so (gfx950) in-tree with hipcc.

    python -m paper_2606_28166_amd.build

Every source under csrc/ is compiled with hipcc for gfx950 (packed fp32
instructions disabled) and linked into paper_2606_28166_amd/libtandem.so.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libtandem.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["tandem.cpp", "k_gemm.hip", "k_stream.hip", "k_attn.hip", "k_misc.hip", "k_grpo.hip"]


def hip_runtime_dir() -> str:
    """Directory of the HIP runtime the process uses.

    PyTorch-ROCm ships its own libamdhip64.so; a process must hold ONE HIP
    runtime, so the library links against that copy (same SONAME, found
    through an rpath) and shares torch's device context and streams.
    """
    import importlib.util
    spec = importlib.util.find_spec("torch")
    if spec is not None and spec.origin:
        d = os.path.join(os.path.dirname(spec.origin), "lib")
        if os.path.exists(os.path.join(d, "libamdhip64.so")):
            return d
    return "/opt/rocm/lib"

FLAGS = [
    "--offload-arch=gfx950", "-mcode-object-version=5", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    warn = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l and l.strip())
    if warn:
        print(warn, file=sys.stderr)
    return obj


def build(verbose: bool = True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(min(len(SOURCES), max(1, os.cpu_count() or 1))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    # The library's HIP runtime dependency (libamdhip64.so.7) resolves through
    # $ORIGIN/_hiprt, a link to the runtime PyTorch loads, so one process holds
    # one HIP runtime (device context, streams and allocations are shared).
    rtdir = os.path.join(PKG, "_hiprt")
    os.makedirs(rtdir, exist_ok=True)
    link = os.path.join(rtdir, "libamdhip64.so.7")
    target = os.path.join(hip_runtime_dir(), "libamdhip64.so")
    if not os.path.exists(target):
        target = "/opt/rocm/lib/libamdhip64.so.7"
    if os.path.islink(link) or os.path.exists(link):
        os.remove(link)
    os.symlink(target, link)
    cmd = ["g++", "-shared", "-fPIC", "-o", tmp, *objs, "-L/opt/rocm/lib", "-lamdhip64",
           "-Wl,--disable-new-dtags", "-Wl,-rpath,$ORIGIN/_hiprt", "-Wl,--no-undefined"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build()
