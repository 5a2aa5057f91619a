"""Scratch memory of the built kernels (CPU: reads the library's own gfx950
code objects, built here from source, with the ROCm tools).

A kernel that copies its launch arguments to scratch (what the compiler does
when a device function that takes them by reference is called rather than
inlined), or keeps a large private array, still gives correct results but
runs slower: every workgroup first writes its ~2.5 KB argument block to
memory.  This pins that the kernels on the named workloads' paths use no
scratch at all, and that no kernel uses more than a few spill slots."""
import os
import re
import shutil
import subprocess

import pytest

LIB = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "paper_2607_27735_amd", "libsparsespec_l.so")
ROCM_LLVM = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm", "bin")
BUNDLER = os.path.join(ROCM_LLVM, "clang-offload-bundler")
READELF = os.path.join(ROCM_LLVM, "llvm-readelf")
MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"

# kernels that must use no scratch (demangled-name prefixes)
NO_SCRATCH = (
    "verify_fused_kernel<1,", "verify_fused_kernel<2,", "verify_fused_kernel<3,",
    "verify_pipe_kernel<1,", "verify_pipe_kernel<2,",
    "verify_stats_kernel", "verify_main_kernel", "verify_combine_kernel",
    "select_fused_kernel", "select_hist_kernel", "select_mark_kernel", "select_finish_kernel",
    "draft_kernel<0,", "draft_kernel<1,", "draft_materialize_kernel",
    "greedy_accept_kernel", "spec_",
)
MAX_SPILL_BYTES = 128


def _kernels(tmp_path):
    if not os.path.exists(LIB):
        pytest.skip("library not built")
    for tool in (BUNDLER, READELF):
        if not os.path.exists(tool):
            pytest.skip(f"{tool} not available")
    if not shutil.which("objcopy") or not shutil.which("c++filt"):
        pytest.skip("binutils not available")
    # objcopy with no output file rewrites its input in place, which would
    # change the pages of a library this process already has loaded: it works
    # on a copy.
    lib_copy = tmp_path / "lib.so"
    shutil.copyfile(LIB, lib_copy)
    fatbin = tmp_path / "fatbin.bin"
    subprocess.run(["objcopy", "--dump-section", f".hip_fatbin={fatbin}", str(lib_copy)], check=True)
    data = fatbin.read_bytes()
    starts = [m.start() for m in re.finditer(re.escape(MAGIC), data)]
    assert starts, "no offload bundles in the library"
    sizes = {}
    for i, st in enumerate(starts):
        end = starts[i + 1] if i + 1 < len(starts) else len(data)
        part, co = tmp_path / f"b{i}.bin", tmp_path / f"co{i}.o"
        part.write_bytes(data[st:end])
        subprocess.run([BUNDLER, "--unbundle", "--type=o", "--targets=hipv4-amdgcn-amd-amdhsa--gfx950",
                        f"--input={part}", f"--output={co}"], check=True, capture_output=True)
        notes = subprocess.run([READELF, "--notes", str(co)], check=True, capture_output=True,
                               text=True).stdout
        name = None
        for line in notes.splitlines():
            line = line.strip()
            if line.startswith(".name:"):
                name = line.split(":", 1)[1].strip()
            elif line.startswith(".private_segment_fixed_size:") and name:
                sizes[name] = int(line.split(":", 1)[1])
                name = None
    names = list(sizes)
    out = subprocess.run(["c++filt"], input="\n".join(names), capture_output=True, text=True,
                         check=True).stdout.splitlines()
    short = {}
    for n, d in zip(names, out):
        m = re.search(r"([A-Za-z_0-9]+_kernel(<[^>]*>)?)\(", d)
        short[m.group(1) if m else d] = sizes[n]
    return short


def test_kernels_use_no_scratch(tmp_path):
    k = _kernels(tmp_path)
    assert len(k) >= 60, f"only {len(k)} kernels found"
    hot = {n: v for n, v in k.items() if n.startswith(NO_SCRATCH)}
    assert len(hot) >= 40, f"only {len(hot)} hot kernels found"
    bad = {n: v for n, v in hot.items() if v}
    assert not bad, f"kernels with scratch memory: {bad}"
    big = {n: v for n, v in k.items() if v > MAX_SPILL_BYTES}
    assert not big, f"kernels with more than {MAX_SPILL_BYTES} B of scratch: {big}"
