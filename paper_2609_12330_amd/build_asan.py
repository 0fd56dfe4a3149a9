"""The attention library with AddressSanitizer on its host code, for checking the host-side
validation and workspace arithmetic on the CPU (the device code is built as usual).

    python -m paper_2609_12330_amd.build_asan OUT_DIR
    cp OUT_DIR/libef_attention.so paper_2609_12330_amd/lib/libef_attention.so
    LD_PRELOAD=<clang>/lib/linux/libclang_rt.asan-x86_64.so ASAN_OPTIONS=detect_leaks=0 \
        python -m pytest tests/test_abi.py
    python -m paper_2609_12330_amd.build        # the normal library again
"""

from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import sys

from paper_2609_12330_amd.build import ARCH, CSRC, HIP_FLAGS, _run, hipcc


def build_asan(out_dir: str, verbose: bool = False) -> str:
    """Builds the instrumented library into out_dir; returns its path."""
    os.makedirs(out_dir, exist_ok=True)
    cc = hipcc()
    asan = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = [f for f in HIP_FLAGS if f != "-O3"] + ["-O1", "-g", *asan]
    objs, jobs = [], []
    sources = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(sources))) as ex:
        for src in sources:
            obj = os.path.join(out_dir, os.path.basename(src)[:-4] + ".o")
            objs.append(obj)
            jobs.append(ex.submit(_run, [cc, *flags, "-c", src, "-o", obj], verbose))
        for j in jobs:
            j.result()
    path = os.path.join(out_dir, "libef_attention.so")
    tmp = path + ".tmp"
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-Xarch_host", "-fsanitize=address",
          *objs, "-o", tmp], verbose)
    os.replace(tmp, path)
    return path


if __name__ == "__main__":
    print(build_asan(sys.argv[1], verbose="-v" in sys.argv))
