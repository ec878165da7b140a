"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only, no GPU calls).

The ABI layer (dit.hip: argument checks, model and workspace planning, routing,
interpolation weights) and the timing hook (prof.hip) are rebuilt with the
sanitizers on their host code only; the kernels' translation units are linked
unchanged from the regular build.  The host ABI tests then run against that
library in a child process with the ASan runtime preloaded: any heap overflow,
use after free or undefined behaviour in the host paths ends the child with an
error report instead of passing silently."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_17572_amd", "csrc")
BUILD = os.path.join(ROOT, "_build")
# the units rebuilt with the sanitizers; every other unit is linked from the
# regular build
HOST_UNITS = ("dit.hip", "prof.hip")
# sanitizers on the host side of each hipcc line only
SAN = "-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined".split()


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    return None


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def test_host_abi_under_asan_and_ubsan(tmp_path):
    hipcc, rt = _hipcc(), _asan_runtime()
    if not hipcc or not rt:
        pytest.skip("hipcc or the ASan runtime is not installed")
    units = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip") and f not in HOST_UNITS)
    objs = [os.path.join(BUILD, u + ".o") for u in units]
    if not all(os.path.exists(o) for o in objs):
        pytest.skip("the regular build's objects are missing (run paper_2607_17572_amd.build.build())")
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-fno-omit-frame-pointer", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
    san_objs = []
    for unit in HOST_UNITS:
        o = str(tmp_path / (unit + ".o"))
        r = subprocess.run([hipcc, *flags, *SAN, "-c", os.path.join(CSRC, unit), "-o", o],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        san_objs.append(o)
    so = str(tmp_path / "libjagg_san.so")
    r = subprocess.run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *san_objs, *objs, "-o", so],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]

    env = dict(os.environ)
    env["LD_PRELOAD"] = rt
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    code = ("import sys, pytest\n"
            "import paper_2607_17572_amd.api as api\n"
            f"api.LIB_PATH = {so!r}\n"
            "sys.exit(pytest.main(['-q', '-x', '-s', '-p', 'no:cacheprovider', '-m', 'not gpu', "
            f"{os.path.join(ROOT, 'tests', 'test_capi_host.py')!r}]))\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=600)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]
    assert r.returncode == 0, out[-6000:]
    assert " passed" in out
