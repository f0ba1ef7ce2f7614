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


def sanitized_flags() -> list:
    """Host code under AddressSanitizer and UndefinedBehaviorSanitizer (each
    -fsanitize= applies to the host pass only; device code is built as usual)."""
    return ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host",
            "-fno-omit-frame-pointer", "-shared-libsan"]


def build_sanitized(out: str, verbose: bool = False) -> str:
    """The library with its host code (validation, plans, the allocation fits and
    dynamic programme) under ASan and UBSan, for the CPU tests; a process
    loading it must preload clang's ASan runtime (``asan_runtime()``) and set
    ``SHIFTADD_LIB`` to ``out``."""
    tag = f".tmp{os.getpid()}"
    objs = [out + "." + os.path.basename(src) + tag + ".o" for src in SOURCES]
    flags = compile_flags(sanitized_flags())
    cmds = [[hipcc(), *flags, "-c", "-o", obj, src] for src, obj in zip(SOURCES, objs)]
    try:
        with concurrent.futures.ThreadPoolExecutor(max_workers=len(cmds)) as ex:
            for f in [ex.submit(subprocess.run, cmd, check=True) for cmd in cmds]:
                f.result()
        tmp = out + tag
        subprocess.run([hipcc(), f"--offload-arch={ARCH}", "-shared", *sanitized_flags(), "-o",
                        tmp, *objs], check=True)
        os.replace(tmp, out)
    finally:
        for obj in objs:
            if os.path.exists(obj):
                os.remove(obj)
    return out


def asan_runtime() -> str:
    """Path of the clang ASan runtime the sanitized library links against."""
    out = subprocess.run([hipcc(), "--print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True).stdout.strip()
    if out and os.path.isabs(out) and os.path.exists(out):
        return out
    import glob
    found = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not found:
        raise RuntimeError("clang ASan runtime not found")
    return found[-1]


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
