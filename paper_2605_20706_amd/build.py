"""Build the HIP libraries for gfx950 with hipcc (in-tree).

Run ``python -m paper_2605_20706_amd.build``. ``liblw.so`` (the product) is
every HIP source in ``csrc/``; ``libceiling.so`` (the streaming-ceiling
kernels the benchmark times beside it) is ``ceiling/ceiling.hip``. Both are
compiled for ``--offload-arch=gfx950`` only, with packed-FP32 instruction
selection disabled.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "liblw.so")
CEILING_LIB = os.path.join(HERE, "libceiling.so")
CEILING_SRC = os.path.join(HERE, "ceiling", "ceiling.hip")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

OBJ_DIR = os.path.join(ROOT, "_build")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    # export only the C ABI (LW_API in lw.h): internal symbols stay inside
    "-fvisibility=hidden", "-fvisibility-inlines-hidden",
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def _run(cmd, verbose, tmp):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 feature and says so: harmless.
    err = "\n".join(l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        if os.path.exists(tmp):
            os.remove(tmp)
        raise RuntimeError("hipcc failed:\n" + err)
    if verbose and err.strip():
        print(err, file=sys.stderr)


def _hipcc(srcs, out, verbose):
    """Each source compiled to an object (in parallel), then one shared link."""
    os.makedirs(OBJ_DIR, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]

    def obj(src):
        o = os.path.join(OBJ_DIR, os.path.basename(out) + "." + os.path.basename(src) + ".o")
        tmp = o + ".tmp%d" % os.getpid()
        _run([HIPCC] + FLAGS + inc + ["-c", src, "-o", tmp], verbose, tmp)
        os.replace(tmp, o)
        return o

    jobs = max(1, min(len(srcs), int(os.environ.get("MAX_JOBS", "0")) or (os.cpu_count() or 1), 16))
    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(obj, srcs))
    tmp = out + ".tmp%d" % os.getpid()
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + objs + ["-o", tmp], verbose, tmp)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    """Builds liblw.so and libceiling.so; returns the path of liblw.so. The
    kernel-selection table is generated from the committed sweep first."""
    from . import gen_select
    gen_select.write()
    _hipcc([CEILING_SRC], CEILING_LIB, verbose)
    return _hipcc(sources(), LIB, verbose)


if __name__ == "__main__":
    print(build(verbose=True))
