"""Build libffsl.so (HIP, gfx950) in-tree with hipcc."""
from __future__ import annotations

import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libffsl.so")
ARCH = os.environ.get("FFSL_OFFLOAD_ARCH", "gfx950")

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared",
    "--offload-arch=" + ARCH,
    # keep the compiler from forming packed-fp32 VALU ops
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fvisibility=hidden",
    "-Wall", "-Wno-unused-function",
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def headers():
    return sorted(glob.glob(os.path.join(CSRC, "*.h"))) + [os.path.join(ROOT, "include", "ffsl.h")]


def build(force: bool = True, verbose: bool = False) -> str:
    """Compile every HIP source into paper_2411_03171_amd/libffsl.so."""
    srcs = sources()
    if not force and os.path.exists(LIB):
        newest = max(os.path.getmtime(p) for p in srcs + headers())
        if os.path.getmtime(LIB) >= newest:
            return LIB
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tmp = LIB + ".tmp%d" % os.getpid()
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    compile_flags = [f for f in HIPCC_FLAGS if f != "-shared"]
    jobs = []
    for src in srcs:
        obj = os.path.join(objdir, os.path.basename(src)[:-4] + ".o")
        jobs.append((src, obj, [hipcc] + compile_flags + ["-I", os.path.join(ROOT, "include"), "-c", "-o", obj, src]))
    # one compiler process per source, a few at a time
    workers = max(1, min(len(jobs), int(os.environ.get("MAX_JOBS", "8")), os.cpu_count() or 1))
    pending = list(jobs)
    running = []
    while pending or running:
        while pending and len(running) < workers:
            src, obj, cmd = pending.pop(0)
            if verbose:
                print(" ".join(cmd), file=sys.stderr)
            running.append((src, subprocess.Popen(cmd)))
        src, proc = running.pop(0)
        if proc.wait() != 0:
            for _, other in running:
                other.wait()
            raise subprocess.CalledProcessError(proc.returncode, "hipcc " + src)
    link = [hipcc, "-shared", "-fPIC", "--offload-arch=" + ARCH, "-o", tmp] + [obj for _, obj, _ in jobs]
    if verbose:
        print(" ".join(link), file=sys.stderr)
    subprocess.check_call(link)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(force=True, verbose=True))
