"""Build libntc.so (HIP, gfx950) in-tree.

    python -m paper_2608_27888_amd.build

Every ``csrc/*.hip`` source is compiled to an object of its own, in parallel
(the decode kernels are split by shape family so that no one translation unit
dominates), then the objects are linked into one shared library.
"""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libntc.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 instructions stay off: plain fp32 arithmetic only
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA results in arch VGPRs: the epilogue reads them without AGPR copies
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
    "-Wall", "-Wno-unused-function",
]

# Flags of single sources.  Binning: its LDS atomics come from one lane, at a
# wave-uniform address; the compiler's atomic optimizer would wrap each in a
# wave reduction that costs more than the atomic (512-decoder frame: 74 -> 66 us
# without it).
SOURCE_FLAGS = {
    "ntc_bins.hip": ["-mllvm", "-amdgpu-atomic-optimizer-strategy=None"],
}


def sources():
    return sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))


def jobs() -> int:
    n = os.cpu_count() or 4
    for var in ("MAX_JOBS", "CMAKE_BUILD_PARALLEL_LEVEL"):
        v = os.environ.get(var, "")
        if v.isdigit() and int(v) > 0:
            n = min(n, int(v))
    return max(1, min(n, 16))


def build(verbose: bool = False) -> str:
    inc = ["-I", os.path.join(ROOT, "include")]
    objdir = tempfile.mkdtemp(prefix="ntc_build_")
    try:
        def compile_one(src):
            obj = os.path.join(objdir, os.path.basename(src) + ".o")
            extra = SOURCE_FLAGS.get(os.path.basename(src), [])
            cmd = [HIPCC, *FLAGS, *extra, *inc, "-c", "-o", obj, src]
            if verbose:
                print(" ".join(cmd), flush=True)
            subprocess.check_call(cmd)
            return obj

        srcs = sources()
        # largest sources first: they set the critical path
        srcs.sort(key=lambda s: -os.path.getsize(s))
        with ThreadPoolExecutor(max_workers=jobs()) as pool:
            objs = list(pool.map(compile_one, srcs))
        tmp = LIB + ".tmp%d" % os.getpid()
        cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *sorted(objs)]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.check_call(cmd)
        os.replace(tmp, LIB)
    finally:
        shutil.rmtree(objdir, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
