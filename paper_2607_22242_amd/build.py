"""Compile the HIP library libsched.so for gfx950, in-tree.

    python -m paper_2607_22242_amd.build
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libsched.so")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
# (source, extra flags); the kernel instantiations are split by tool count so
# that they compile in parallel.
INST_PARTS = [(1, 12), (13, 17), (18, 21), (22, 25), (26, 29), (30, 32), (33, 36), (37, 40)]
UNITS = [("api.cpp", []), ("monitor.cpp", []), ("dispatch.hip", []), ("probe.hip", []),
         ("scratch.hip", [])] + [
    ("inst.hip", [f"-DINST_LO={lo}", f"-DINST_HI={hi}"]) for lo, hi in INST_PARTS]
ARCH = "gfx950"


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else "hipcc"


def compile_flags():
    return [
        f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
        # no packed FP32 instructions anywhere in device code
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        f"-I{INCLUDE}", f"-I{CSRC}",
    ]


def build(verbose: bool = False, jobs: int = 8) -> str:
    """Compile every unit to an object, link libsched.so; returns its path."""
    from concurrent.futures import ThreadPoolExecutor

    cmds, objs = [], []
    for i, (src, extra) in enumerate(UNITS):
        obj = os.path.join(CSRC, f"_unit{i}.o")
        cmds.append([hipcc()] + compile_flags() + extra +
                    ["-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)

    def run(cmd):
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.check_call(cmd)

    with ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        list(ex.map(run, cmds))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC"] + objs + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    for obj in objs:
        os.remove(obj)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
