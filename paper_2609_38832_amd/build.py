"""Build libnamoh.so for gfx950 with hipcc (in-tree, no JIT cache).

    python -m paper_2609_38832_amd.build        # or __graft_entry__.build()

Each source compiles to an object under ``_build/`` in parallel, then one
shared library is linked next to this file.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libnamoh.so")
ARCH = "gfx950"

SOURCES = ["route.hip", "attn.hip", "decode.hip", "bwd.hip", "proj.hip", "api.cpp", "profile.cpp"]

COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Wall", "-Wno-unused-function",
    # keep the compiler from forming packed fp32 ops (v_pk_*_f32)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{os.path.join(ROOT, 'include')}",
]


def hipcc() -> str:
    p = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(p):
        raise RuntimeError("hipcc not found")
    return p


# Per-source flags.  The attention kernels never produce NaN (masked scores are
# -inf and are only ever compared or exponentiated), so max/min need no NaN
# quieting.
EXTRA = {"attn.hip": ["-fno-honor-nans", "-mno-amdgpu-ieee"]}


# Host-side AddressSanitizer and UndefinedBehaviorSanitizer (the C ABI's
# validation, workspace carving and launch set-up); device code is built as
# usual.  Used by the CPU tests only, never loaded on a GPU run.
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]
SAN_BUILD = os.path.join(BUILD, "sanitize")
SAN_LIB = os.path.join(SAN_BUILD, "libnamoh.so")


def _compile(src: str, out_dir: str = None, extra=()) -> str:
    out_dir = out_dir or BUILD
    obj = os.path.join(out_dir, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *COMMON, *EXTRA.get(src, []), *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".hip"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{r.stderr}")
    return obj


def build_library(verbose: bool = True, sanitize: bool = False) -> str:
    out_dir = SAN_BUILD if sanitize else BUILD
    lib = SAN_LIB if sanitize else LIB
    extra = SANITIZE if sanitize else []
    os.makedirs(out_dir, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(lambda src: _compile(src, out_dir, extra), SOURCES))
    tmp = lib + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *extra, "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stderr}")
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib}")
    return lib


if __name__ == "__main__":
    build_library()
    sys.exit(0)
