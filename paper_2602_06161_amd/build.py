"""Build the COVER HIP library for gfx950 (in-tree, hipcc).

Produces ``paper_2602_06161_amd/lib/libcover.so`` from ``csrc/``.  Run as
``python -m paper_2602_06161_amd.build``; ``__graft_entry__.build()`` calls ``build()``.
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
OBJDIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "lib", "libcover.so")
# the same library with the attention kernel's phase timestamps compiled in (measurement only)
LIB_TIMING = os.path.join(PKG, "lib", "libcover_timing.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC") or shutil.which("hipcc") or "/opt/rocm/bin/hipcc"

COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # packed-fp32 VALU instructions stay off: plain fp32 ops only
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
    "-I", INCLUDE, "-I", CSRC,
]
# per-source extra flags
SOURCES = {
    "api.cpp": ["-x", "hip"],
    "cover_attn.hip": [],
    "cover_attn_w4.hip": [],
    "cover_attn_rect.hip": [],
    "cover_debug.hip": [],
    "cover_decode.hip": [],
    "cover_select.hip": ["-ffp-contract=off"],  # the selection is bit-exact fp64
    "cover_stats.hip": [],
    "cover_sample.hip": [],
}


# sources compiled a second time, with these flags, for LIB_TIMING
TIMING = {"cover_attn_w4.hip": ["-DCOVER_ATTN_TIMING=1"], "cover_attn_rect.hip": ["-DCOVER_RECT_TIMING=1"]}
# sources of LIB_TIMING only (the MFMA-counter calibration kernel)
TIMING_ONLY = {"cover_calib.hip": []}


def _compile(src: str, timing: bool = False) -> str:
    obj = os.path.join(OBJDIR, src + (".timing.o" if timing else ".o"))
    flags = SOURCES[src] if src in SOURCES else TIMING_ONLY[src]
    extra = TIMING.get(src, []) if timing else []
    cmd = [HIPCC, *COMMON, *flags, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = True) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    os.makedirs(os.path.dirname(LIB), exist_ok=True)
    jobs = ([(src, False) for src in SOURCES] + [(src, True) for src in TIMING]
            + [(src, True) for src in TIMING_ONLY])
    with ThreadPoolExecutor(max_workers=len(jobs)) as ex:
        built = dict(zip(jobs, ex.map(lambda j: _compile(*j), jobs)))
    plain = [built[(src, False)] for src in SOURCES]
    timed = [built[(src, src in TIMING)] for src in SOURCES] + [built[(src, True)] for src in TIMING_ONLY]
    for lib, objs in ((LIB, plain), (LIB_TIMING, timed)):
        tmp = lib + ".tmp"
        cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
        os.replace(tmp, lib)
        if verbose:
            print(f"built {lib}", file=sys.stderr)
    return LIB


if __name__ == "__main__":
    build()
