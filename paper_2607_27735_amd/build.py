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

HIP_SOURCES = ["verify.hip", "verify_fused.hip", "select.hip", "draft.hip", "logits.hip",
               "spec.hip", "status.hip", "static_scratch.hip"]
CXX_SOURCES = ["api.cpp", "controller.cpp"]


def source_id() -> str:
    """Hash of every source the library is built from (kernels, ABI, headers and
    the build script itself); the library reports it through ssl_build_id()."""
    import hashlib
    files = [os.path.join(CSRC, f) for f in sorted(os.listdir(CSRC))
             if f.endswith((".hip", ".cpp", ".h"))]
    files += [os.path.join(INCLUDE, f) for f in sorted(os.listdir(INCLUDE)) if f.endswith(".h")]
    files.append(os.path.abspath(__file__))
    h = hashlib.sha256()
    for f in files:
        h.update(os.path.basename(f).encode() + b"\0")
        with open(f, "rb") as fh:
            h.update(fh.read())
        h.update(b"\0")
    return h.hexdigest()[:16]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else (shutil.which("hipcc") or path)


def _compile(src: str, obj: str, is_hip: bool, build_id: str) -> None:
    cmd = [hipcc(), "-c", "-fPIC", "-O3", "-std=c++17", "-Wall", "-I", INCLUDE, "-I", CSRC,
           f'-DSSL_BUILD_ID="{build_id}"']
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
    bid = source_id()
    jobs = []
    for s in HIP_SOURCES:
        jobs.append((os.path.join(CSRC, s), os.path.join(out_dir, s + ".o"), True, bid))
    for s in CXX_SOURCES:
        jobs.append((os.path.join(CSRC, s), os.path.join(out_dir, s + ".o"), False, bid))
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
