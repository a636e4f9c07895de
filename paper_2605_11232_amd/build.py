"""Build libpa.so (HIP kernels for gfx950 + host C++) in-tree.

Usage: ``python -m paper_2605_11232_amd.build`` (or ``build()`` from Python).
Always recompiles.  The library is written next to this file.
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
LIB_PATH = os.path.join(HERE, "libpa.so")

HIP_SOURCES = ["attn_bf16.hip", "attn_f32.hip", "kv_append.hip", "stage.hip", "api.hip"]
HOST_SOURCES = ["pool.cpp", "plan.cpp", "batch.cpp", "step.cpp", "errors.cpp"]

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CXX = os.environ.get("CXX", "g++")  # host-only sources (no device code)
COMMON = ["-O3", "-std=c++17", "-fPIC", f"-I{INCLUDE}", f"-I{CSRC}", "-Wall"]
# Packed-fp32 VALU forms are kept out of the generated code.  MFMA results stay
# in ordinary VGPRs: with accumulation registers the compiler copied every
# output accumulator between register files on each iteration of the softmax
# loops.
HIP_FLAGS = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang",
             "-packed-fp32-ops", "-munsafe-fp-atomics", "-mllvm", "--amdgpu-mfma-vgpr-form"]


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(line for line in p.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in line)
    if p.returncode != 0:
        raise RuntimeError(f"command failed ({p.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False, jobs: int = 8, defines=(), out_path: str = LIB_PATH) -> str:
    """Compile every source and link libpa.so at ``out_path``; ``defines``
    are extra -D options for all sources (kernel and planner tuning knobs)."""
    tmp = tempfile.mkdtemp(prefix="pa_build_")
    try:
        cmds = []
        objs = []
        for s in HIP_SOURCES:
            o = os.path.join(tmp, s + ".o")
            cmds.append([HIPCC, *COMMON, *HIP_FLAGS, *[f"-D{d}" for d in defines], "-c",
                         os.path.join(CSRC, s), "-o", o])
            objs.append(o)
        for s in HOST_SOURCES:
            o = os.path.join(tmp, s + ".o")
            cmds.append([CXX, *COMMON, *[f"-D{d}" for d in defines], "-c",
                         os.path.join(CSRC, s), "-o", o])
            objs.append(o)
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            outs = list(ex.map(_run, cmds))
        if verbose:
            for o in outs:
                if o.strip():
                    print(o)
        tmp_lib = os.path.join(tmp, "libpa.so")
        _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp_lib])
        shutil.move(tmp_lib, out_path)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return out_path


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
