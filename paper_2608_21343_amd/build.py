"""Build libtbias.so in-tree: HIP sources for gfx950 with hipcc, host C++ with g++.

Usage: python -m paper_2608_21343_amd.build   (or build_library() from Python)
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
from pathlib import Path

PKG = Path(__file__).resolve().parent
CSRC = PKG / "csrc"
BUILD = PKG / "_build"
LIB = PKG / "libtbias.so"
ROCM = Path(os.environ.get("ROCM_PATH", "/opt/rocm"))

HIP_SOURCES = ["capi.hip", "greedy.hip", "greedy_seg.hip",
               "greedy_seg_1_8.hip", "greedy_seg_9_16.hip", "greedy_seg_17_24.hip",
               "greedy_seg_25_32.hip", "greedy_wide.hip", "beam.hip", "beam_wide_f32.hip", "beam_wide_bf16.hip",
               "beam_pipe_f32.hip", "beam_pipe_bf16.hip", "beam_fast_1_8.hip", "beam_fast_9_16.hip",
               "beam_fast_17_24.hip", "beam_fast_25_32.hip", "beam_stream_1_8.hip",
               "beam_stream_9_16.hip", "beam_stream_17_24.hip", "beam_stream_25_32.hip", "state.hip", "registry.hip"]
CXX_SOURCES = ["compiler.cpp", "variative.cpp", "cache.cpp", "errors.cpp"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # the selection contract needs plain IEEE adds/subs (no fused multiply-add)
    "-ffp-contract=off",
    # keep hipcc from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]
# per-file additions to HIPCC_FLAGS
HIP_EXTRA: dict = {}
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-ffp-contract=off", "-Wall", "-pthread"]


def _hipcc() -> str:
    p = ROCM / "bin" / "hipcc"
    return str(p) if p.exists() else (shutil.which("hipcc") or "hipcc")


def build_library(verbose: bool = False, poison: bool = False) -> Path:
    """Compile every source and link libtbias.so next to this file.

    poison=True builds the LDS-poisoning debug variant (every kernel fills its
    LDS with all bits set before use) as libtbias_poison.so, for the test
    that decodes through it. A failed build removes the library it would
    have replaced, so that nothing runs a stale build."""
    build_dir = BUILD if not poison else PKG / "_build_poison"
    out_lib = LIB if not poison else PKG / "libtbias_poison.so"
    extra = [] if not poison else ["-DTB_POISON_LDS"]
    build_dir.mkdir(exist_ok=True)
    hipcc = _hipcc()
    cxx = shutil.which("g++") or "g++"
    jobs = []
    objs = []
    for src in HIP_SOURCES:
        obj = build_dir / (src + ".o")
        objs.append(obj)
        jobs.append([hipcc, *HIPCC_FLAGS, *extra, *HIP_EXTRA.get(src, []), "-c", str(CSRC / src),
                     "-o", str(obj)])
    for src in CXX_SOURCES:
        obj = build_dir / (src + ".o")
        objs.append(obj)
        jobs.append([cxx, *CXX_FLAGS, "-c", str(CSRC / src), "-o", str(obj)])
    procs = []
    for cmd in jobs:
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
    failed = []
    for cmd, p in procs:
        out, _ = p.communicate()
        if p.returncode != 0:
            failed.append((cmd, out.decode(errors="replace")))
        elif verbose and out:
            print(out.decode(errors="replace"), flush=True)
    if failed:
        out_lib.unlink(missing_ok=True)
        msg = "\n".join(" ".join(c) + "\n" + o for c, o in failed)
        raise RuntimeError("libtbias build failed:\n" + msg)
    tmp = out_lib.with_suffix(".so.tmp")
    link = [hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", str(tmp),
            *map(str, objs), "-pthread"]
    if verbose:
        print(" ".join(link), flush=True)
    r = subprocess.run(link, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    if r.returncode != 0:
        out_lib.unlink(missing_ok=True)
        raise RuntimeError("libtbias link failed:\n" + r.stdout.decode(errors="replace"))
    os.replace(tmp, out_lib)
    return out_lib


if __name__ == "__main__":
    print(build_library(verbose="-v" in sys.argv, poison="--poison" in sys.argv))
