"""Build libsnls.so (the HIP library) in-tree for gfx950.

Every .hip file under csrc/ is compiled with hipcc for gfx950 only; the
host-only argument checks (validate.cpp) with g++.  Packed fp32 VALU
instructions are disabled for all device code.  Usage:
``python -m paper_2309_16849_amd.build`` (or ``build()`` from Python).
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
OUT = os.path.join(HERE, "libsnls.so")
BUILD_DIR = os.path.join(HERE, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

HIP_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "-mcode-object-version=5",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-munsafe-fp-atomics", "-Wall", "-Wno-unused-function", "-I" + INCLUDE, "-I" + CSRC,
]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-I" + INCLUDE, "-I" + CSRC]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l and "target-feature" not in l)
    if r.returncode != 0:
        raise RuntimeError("command failed: %s\n%s" % (" ".join(cmd), out))
    return out


def build(verbose: bool = False, jobs: int = 8) -> str:
    """Compile every source and link libsnls.so; always rebuilds.  Returns the path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    hips = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    cpps = sorted(glob.glob(os.path.join(CSRC, "*.cpp")))
    jobs_list = []
    for src in hips:
        obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
        jobs_list.append([HIPCC] + HIP_FLAGS + ["-c", src, "-o", obj])
    for src in cpps:
        obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
        jobs_list.append(["g++"] + CXX_FLAGS + ["-c", src, "-o", obj])
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        for out in ex.map(_run, jobs_list):
            if verbose and out.strip():
                print(out)
    objs = [c[-1] for c in jobs_list]
    tmp = OUT + ".tmp%d" % os.getpid()
    _run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp] + objs)
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
