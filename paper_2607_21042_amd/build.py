"""Build libftts.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2607_21042_amd.build            # the library
    python -m paper_2607_21042_amd.build --trace    # also libftts_trace.so (below)

Each translation unit under csrc/ is compiled in parallel, then linked into
paper_2607_21042_amd/libftts.so next to this file.  `--trace` links a second
library, libftts_trace.so, whose persistent decode step stamps a per-phase
timeline (FTTS_MEGA_TRACE; read by `mega_timeline.py`); it is never loaded
unless a tool asks for it by path.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libftts.so")
TRACE_LIB = os.path.join(PKG, "libftts_trace.so")
ARCH = "gfx950"

# Packed-fp32 VALU ops are disabled on purpose: hipcc may otherwise emit them from
# plain float code.
HIPFLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
    "-I", INCLUDE, "-I", CSRC,
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def _headers():
    hs = [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hpp", ".h"))]
    return hs + [os.path.join(INCLUDE, f) for f in os.listdir(INCLUDE) if f.endswith(".h")]


def _stale(src: str, obj: str) -> bool:
    if not os.path.exists(obj):
        return True
    t = os.path.getmtime(obj)
    return any(os.path.getmtime(f) > t for f in [src, *_headers()])


def _compile(src: str, force: bool = True) -> str:
    obj = os.path.join(OBJDIR, os.path.basename(src)[:-4] + ".o")
    if not force and not _stale(src, obj):
        return obj
    cmd = [hipcc(), *HIPFLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        if os.path.exists(obj):
            os.remove(obj)
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, force: bool = True) -> str:
    """Compile every source and link libftts.so; returns the library path.
    With force=False, objects newer than their source and every header are reused."""
    os.makedirs(OBJDIR, exist_ok=True)
    srcs = sources()
    with ThreadPoolExecutor(min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda f: _compile(f, force), srcs))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


def build_trace(verbose: bool = False) -> str:
    """Link libftts_trace.so: the library's objects with the persistent step
    recompiled under FTTS_MEGA_TRACE."""
    build(verbose, force=False)
    tdir = os.path.join(OBJDIR, "trace")
    os.makedirs(tdir, exist_ok=True)
    src = os.path.join(CSRC, "decode_mega.hip")
    tobj = os.path.join(tdir, "decode_mega.o")
    r = subprocess.run([hipcc(), *HIPFLAGS, "-DFTTS_MEGA_TRACE", "-c", src, "-o", tobj], capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src} (trace):\n{r.stdout}\n{r.stderr}")
    objs = [os.path.join(OBJDIR, os.path.basename(f)[:-4] + ".o") for f in sources()
            if os.path.basename(f) != "decode_mega.hip"] + [tobj]
    tmp = TRACE_LIB + ".tmp"
    r = subprocess.run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed (trace):\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, TRACE_LIB)
    if verbose:
        print(f"built {TRACE_LIB}")
    return TRACE_LIB


if __name__ == "__main__":
    if "--trace" in sys.argv:
        build_trace(verbose=True)
    else:
        build(verbose=True, force="--incremental" not in sys.argv)
    sys.exit(0)
