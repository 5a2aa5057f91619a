"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

The library's host side (argument checks, plans, workspace layouts, the
controller) is rebuilt with g++ -fsanitize=address,undefined and linked with
the kernels' objects as they are built; the oracle is rebuilt the same way
with gcc.  A child process, with the sanitizer runtime preloaded, runs the
ABI, controller and oracle-pin tests against those builds.  A planted
out-of-bounds write in a throwaway C function shows that the set-up catches
one.  No GPU is used: the ABI tests stop every call before its first HIP call."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_27735_amd", "csrc")
BUILD = os.path.join(ROOT, "paper_2607_27735_amd", "_build")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
       "-fno-omit-frame-pointer", "-g", "-O1", "-fPIC"]


def _asan_runtime():
    if not shutil.which("gcc") or not shutil.which("g++"):
        return None
    p = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = p.stdout.strip()
    return path if p.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"


def _child_env(runtime):
    env = dict(os.environ)
    pre = env.get("LD_PRELOAD", "")
    env["LD_PRELOAD"] = runtime + (" " + pre if pre else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:exitcode=86"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1:exitcode=87"
    return env


@pytest.fixture(scope="module")
def san_builds(tmp_path_factory):
    runtime = _asan_runtime()
    if runtime is None:
        pytest.skip("gcc/g++ with AddressSanitizer not available")
    from paper_2607_27735_amd import build
    if not all(os.path.exists(os.path.join(BUILD, s + ".o")) for s in build.HIP_SOURCES):
        build.build()
    d = tmp_path_factory.mktemp("sanitize")
    bid = build.source_id()
    objs = []
    for src in build.CXX_SOURCES:
        o = str(d / (src + ".o"))
        _run(["g++", "-c", "-std=c++17", "-Wall", *SAN, "-D__HIP_PLATFORM_AMD__",
              f"-I{ROCM}/include", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
              f'-DSSL_BUILD_ID="{bid}"', os.path.join(CSRC, src), "-o", o])
        objs.append(o)
    lib = str(d / "libsparsespec_l_san.so")
    _run(["g++", "-shared", *SAN, *objs, *[os.path.join(BUILD, s + ".o") for s in build.HIP_SOURCES],
          f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib", "-o", lib])
    olib = str(d / "liboracle_san.so")
    _run(["gcc", "-shared", "-std=c11", "-Wall", "-fopenmp", *SAN,
          os.path.join(ROOT, "oracle", "oracle.c"), "-o", olib, "-lm"])
    return runtime, lib, olib, d


def test_a_planted_overflow_is_caught(san_builds):
    runtime, _, _, d = san_builds
    src = d / "planted.c"
    src.write_text("#include <stdlib.h>\n"
                   "int planted(int n) { int *a = malloc(sizeof(int) * n); a[n] = 1;"
                   " int r = a[0]; free(a); return r; }\n")
    so = str(d / "libplanted.so")
    _run(["gcc", "-shared", *SAN, str(src), "-o", so])
    code = f"import ctypes; ctypes.CDLL({so!r}).planted(4)"
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                       env=_child_env(runtime), timeout=120)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr, r.stderr[-2000:]


def test_host_code_and_oracle_under_sanitizers(san_builds):
    runtime, lib, olib, _ = san_builds
    code = "\n".join([
        "import sys",
        f"sys.path[:0] = [{ROOT!r}, {os.path.join(ROOT, 'tests')!r}]",
        "import oracle",
        f"oracle._lib = oracle.load({olib!r})",
        "from paper_2607_27735_amd import binding as B",
        f"B._lib = B.load({lib!r})",
        f"assert B.load()._name == {lib!r} and oracle.load()._name == {olib!r}",
        "import pytest",
        "sys.exit(pytest.main(['-q', '-x', '-p', 'no:cacheprovider', '-m', 'not gpu',",
        f"    {os.path.join(ROOT, 'tests', 'test_abi.py')!r},",
        f"    {os.path.join(ROOT, 'tests', 'test_controller.py')!r},",
        f"    {os.path.join(ROOT, 'tests', 'test_oracle_pins.py')!r}]))",
    ])
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                       env=_child_env(runtime), timeout=900, cwd=ROOT)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in r.stdout
