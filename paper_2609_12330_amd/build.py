"""Build the gfx950 HIP library ``lib/libef_attention.so`` in-tree with hipcc.

Every HIP source under ``csrc/`` is compiled for gfx950 only, with packed
fp32 instruction selection disabled, and linked into one shared library that
exports the C ABI of ``include/ef_attention.h``.

    python -m paper_2609_12330_amd.build [-v]
"""

from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(PKG, "_build")
LIB_DIR = os.path.join(PKG, "lib")
LIB_PATH = os.path.join(LIB_DIR, "libef_attention.so")
# Microbenchmarks of the measurement script (streaming read, bare matrix-core
# loop): a library of their own, so the attention library exports only its ABI.
MICRO_DIR = os.path.join(CSRC, "micro")
MICRO_LIB_PATH = os.path.join(LIB_DIR, "libef_micro.so")

ARCH = "gfx950"
HIP_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-function",
    # packed fp32 (v_pk_*_f32) selection off
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}",
    f"-I{CSRC}",
]


def hipcc() -> str:
    exe = os.environ.get("HIPCC") or shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(exe):
        raise RuntimeError(f"hipcc not found ({exe})")
    return exe


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 feature name; that warning is noise.
    err = "\n".join(line for line in res.stderr.splitlines()
                    if "packed-fp32-ops" not in line and "not a recognized feature" not in line)
    if res.returncode != 0:
        raise RuntimeError(f"command failed ({res.returncode}): {' '.join(cmd)}\n{err}")
    if verbose and err.strip():
        print(err, flush=True)


def _link(cc, objs, path, verbose):
    tmp = path + ".tmp"
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, path)


def build(verbose: bool = False) -> str:
    """Compile every csrc/*.hip for gfx950 and link lib/libef_attention.so (and the
    microbenchmarks of csrc/micro/ into lib/libef_micro.so); returns the first path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    os.makedirs(LIB_DIR, exist_ok=True)
    cc = hipcc()
    sources = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    micro = sorted(glob.glob(os.path.join(MICRO_DIR, "*.hip")))
    if not sources:
        raise RuntimeError("no HIP sources found")
    objs, micro_objs, jobs = [], [], []
    with cf.ThreadPoolExecutor(max_workers=min(8, len(sources) + len(micro))) as ex:
        for src in sources + micro:
            obj = os.path.join(BUILD_DIR, os.path.basename(src)[:-4] + ".o")
            (micro_objs if src in micro else objs).append(obj)
            jobs.append(ex.submit(_run, [cc, *HIP_FLAGS, "-c", src, "-o", obj], verbose))
        for j in jobs:
            j.result()
    _link(cc, objs, LIB_PATH, verbose)
    if micro_objs:
        _link(cc, micro_objs, MICRO_LIB_PATH, verbose)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
