"""Compile the gfx950 HIP library ``libshiftadd.so`` in-tree with hipcc.

Each source is compiled to an object in parallel, then the objects are linked
into the shared library.

    python -m paper_2406_05981_amd.build
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = [os.path.join(HERE, "csrc", "shiftadd.hip"), os.path.join(HERE, "csrc", "bcq.hip"),
           os.path.join(HERE, "csrc", "alloc.hip")]
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libshiftadd.so")
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def compile_flags(extra=()) -> list:
    return [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
            "-ffp-contract=off",
            # packed fp32 VALU ops stay off: plain fp32 adds only
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", INCLUDE, *extra]


def command(out: str = LIB, extra=()) -> list:
    """One hipcc command building the whole library from all sources."""
    return [hipcc(), *compile_flags(extra), "-shared", "-o", out, *SOURCES]


def build(verbose: bool = False) -> str:
    tag = f".tmp{os.getpid()}"
    objs = [os.path.join(HERE, os.path.basename(src) + tag + ".o") for src in SOURCES]
    cmds = [[hipcc(), *compile_flags(), "-c", "-o", obj, src] for src, obj in zip(SOURCES, objs)]
    try:
        with concurrent.futures.ThreadPoolExecutor(max_workers=len(cmds)) as ex:
            futs = []
            for cmd in cmds:
                if verbose:
                    print(" ".join(cmd), flush=True)
                futs.append(ex.submit(subprocess.run, cmd, check=True))
            for f in futs:
                f.result()
        tmp = LIB + tag
        link = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-o", tmp, *objs]
        if verbose:
            print(" ".join(link), flush=True)
        subprocess.run(link, check=True)
        os.replace(tmp, LIB)
    finally:
        for obj in objs:
            if os.path.exists(obj):
                os.remove(obj)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
