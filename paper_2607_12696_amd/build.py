"""Build libecospec_moe.so for gfx950 with hipcc (in-tree, no JIT cache).

    python -m paper_2607_12696_amd.build          # or build() from Python

Every HIP source is compiled for gfx950 only; packed-fp32 VALU ops are
disabled for all device code.  Objects go to _build/ next to the repo root.
"""
from __future__ import annotations

import hashlib
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libecospec_moe.so")
BUILD = os.path.join(ROOT, "_build")

SOURCES = ["route_topk.hip", "expert_union.hip", "expert_ffn.hip", "pack.hip", "router.hip", "noalloc.hip", "abi.cpp", "selector.cpp"]
ARCH = "gfx950"
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"-I{INCLUDE}", f"-I{CSRC}", "-Wall", "-Wno-unused-function"]


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return "hipcc"


def _compile(src: str, defines=(), build_dir=BUILD) -> str:
    path = os.path.join(CSRC, src)
    obj = os.path.join(build_dir, src + ".o")
    if src.endswith(".hip"):
        cmd = [_hipcc(), f"--offload-arch={ARCH}", "-x", "hip", *COMMON, *DEVICE_FLAGS, *defines, "-c", path, "-o", obj]
    else:
        cmd = [_hipcc(), *COMMON, "-D__HIP_PLATFORM_AMD__", "-c", path, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, defines=(), out: str = LIB) -> str:
    """Compile all sources and link the shared library; returns its path.

    ``defines`` (e.g. ["-DECOSPEC_PD_FP8=4"]) override the kernels' compile-time
    tuning knobs; ``out`` names the library file.
    """
    tag = hashlib.sha1(" ".join(defines).encode()).hexdigest()[:10]
    build_dir = BUILD if not defines else os.path.join(BUILD, "v" + tag)
    os.makedirs(build_dir, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda src: _compile(src, tuple(defines), build_dir), SOURCES))
    tmp = out + f".tmp{os.getpid()}"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    if verbose:
        print(f"built {out}")
    return out


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
