"""Build libsom.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_1905_09598_amd.build

Every HIP translation unit is compiled for gfx950 only, with packed-fp32
instructions disabled, and the objects are linked into
paper_1905_09598_amd/libsom.so next to this file.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libsom.so")
SOURCES = ["som_api.cpp", "som_train.hip", "som_train_pipe.hip", "som_train_pipe_stream.hip",
           "som_eval.hip", "som_util.hip", "som_pca.hip", "som_sparse.hip", "som_batch.hip",
           "som_stream.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP toolchain is required to build libsom")


def common_flags() -> list:
    return ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
            "-Wall", "-Wno-unused-result",
            # keep the compiler from emitting packed fp32 (v_pk_*_f32) math
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            f"-I{INCLUDE}", f"-I{CSRC}"]


# Translation units whose grid-exchange polls keep several loads in flight
# (som_device.h, poll_slots).  Left structured, the poll loop's uniform early
# exits are folded into the loop latch, and the merged path makes the
# compiler wait for every poll in flight at each check; skipping the
# structurization of uniform regions (their branches need no exec-mask
# bookkeeping) keeps the exits as real exits.  The streamed pipelined
# kernels (som_train_pipe_stream.hip) and the sparse kernel poll one load at
# a time and are built without it.
UNIFORM_EXIT_SOURCES = ("som_train.hip", "som_train_pipe.hip")


def unit_flags(src: str) -> list:
    if src in UNIFORM_EXIT_SOURCES:
        return ["-mllvm", "-structurizecfg-skip-uniform-regions=true"]
    return []


def _compile(src: str) -> str:
    os.makedirs(BUILD, exist_ok=True)
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = ([hipcc()] + common_flags() + unit_flags(src)
           + ["-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj])
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{err}")
    if err.strip():
        sys.stderr.write(err + "\n")
    return obj


def build(verbose: bool = True) -> str:
    with ThreadPoolExecutor(max_workers=min(5, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build()
