"""Build libturbomuon.so (gfx950) in-tree with hipcc.

    python -m paper_2512_04632_amd.build

The bf16 and fp32 kernel sets are compiled as two translation units in
parallel with the host planner, then linked into one shared library next to
this file.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "libturbomuon.so"
LIB_PATH = os.path.join(HERE, LIB_NAME)

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17",
    "-I", CSRC, "-I", INCLUDE,
    # keep hipcc from forming packed fp32 instructions on its own
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("build step failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    return r


def build(verbose: bool = False) -> str:
    """Compile every HIP source for gfx950 and link the shared library."""
    tmp = tempfile.mkdtemp(prefix="tm_build_")
    try:
        units = [
            (os.path.join(CSRC, "tm_kernels.hip"), ["-DTM_ELEM_BYTES=2"], "k_bf16.o"),
            (os.path.join(CSRC, "tm_kernels.hip"), ["-DTM_ELEM_BYTES=4"], "k_f32.o"),
            (os.path.join(CSRC, "tm_fast.hip"), [], "k_fast.o"),
            (os.path.join(CSRC, "tm_optim.hip"), [], "k_optim.o"),
            (os.path.join(CSRC, "tm_noalloc.hip"), [], "noalloc.o"),
            (os.path.join(CSRC, "tm_small.hip"), [], "k_small.o"),
            (os.path.join(CSRC, "tm_api.cpp"), [], "api.o"),
        ]
        cmds = [[HIPCC] + COMMON + extra + ["-c", src, "-o", os.path.join(tmp, obj)]
                for src, extra, obj in units]
        with ThreadPoolExecutor(max_workers=len(cmds)) as ex:
            for r, cmd in zip(ex.map(_run, cmds), cmds):
                if verbose:
                    print(" ".join(cmd))
        out_tmp = os.path.join(tmp, LIB_NAME)
        _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", out_tmp]
             + [os.path.join(tmp, u[2]) for u in units])
        shutil.move(out_tmp, LIB_PATH + ".tmp")
        os.replace(LIB_PATH + ".tmp", LIB_PATH)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
