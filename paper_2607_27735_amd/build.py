"""Build the C-ABI library ``libsparsespec_l.so`` for gfx950 with hipcc.

Usage: ``python -m paper_2607_27735_amd.build`` (or ``build()`` from Python).
Always recompiles; objects go to ``_build/`` inside the package, the library
next to this file.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
LIB_NAME = "libsparsespec_l.so"
LIB_PATH = os.path.join(HERE, LIB_NAME)
ARCH = "gfx950"

HIP_SOURCES = ["verify.hip", "verify_fused.hip", "select.hip", "draft.hip", "logits.hip"]
CXX_SOURCES = ["api.cpp", "controller.cpp"]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else (shutil.which("hipcc") or path)


def _compile(src: str, obj: str, is_hip: bool) -> None:
    cmd = [hipcc(), "-c", "-fPIC", "-O3", "-std=c++17", "-Wall", "-I", INCLUDE, "-I", CSRC]
    if is_hip:
        # gfx950 only; packed fp32 arithmetic is kept out of the generated code.
        cmd += ["-x", "hip", f"--offload-arch={ARCH}",
                "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
    cmd += [src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")


def build(verbose: bool = False) -> str:
    out_dir = os.path.join(HERE, "_build")
    os.makedirs(out_dir, exist_ok=True)
    jobs = []
    for s in HIP_SOURCES:
        jobs.append((os.path.join(CSRC, s), os.path.join(out_dir, s + ".o"), True))
    for s in CXX_SOURCES:
        jobs.append((os.path.join(CSRC, s), os.path.join(out_dir, s + ".o"), False))
    with ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        list(ex.map(lambda j: _compile(*j), jobs))
    tmp = LIB_PATH + ".tmp%d" % os.getpid()
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *[j[1] for j in jobs], "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB_PATH)
    if verbose:
        print(f"built {LIB_PATH}")
    return LIB_PATH


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
