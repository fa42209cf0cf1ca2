"""The C ABI's host-side argument checks under AddressSanitizer and
UndefinedBehaviorSanitizer (no GPU needed).

The library's sources are compiled with the sanitizers on the host side only
(each -fsanitize is preceded by -Xarch_host, so device code is unchanged) and
linked with tests/sanitize/abi_errors.cpp, which drives every entry point
through its refusal paths, including sizes at the extremes of their types. The
run must end with status 0 and no sanitizer report. The build is cached under
_build/asan by a hash of the sources.
"""

import glob
import hashlib
import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2605_06892_amd", "csrc")
DRIVER = os.path.join(ROOT, "tests", "sanitize", "abi_errors.cpp")
OUT = os.path.join(ROOT, "_build", "asan")
ROCM = "/opt/rocm"
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]


def _tools():
    hipcc = shutil.which("hipcc") or os.path.join(ROCM, "bin", "hipcc")
    clang = os.path.join(ROCM, "llvm", "bin", "clang++")
    if not (os.path.exists(hipcc) and os.path.exists(clang)):
        pytest.skip("ROCm compilers not found")
    return hipcc, clang


def _build():
    hipcc, clang = _tools()
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    h = hashlib.sha256()
    for f in srcs + sorted(glob.glob(os.path.join(CSRC, "*.h"))) + [DRIVER, os.path.join(ROOT, "include", "hsa_step.h")]:
        h.update(open(f, "rb").read())
    exe = os.path.join(OUT, "abi_errors_" + h.hexdigest()[:16])
    if os.path.exists(exe):
        return exe
    os.makedirs(OUT, exist_ok=True)
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-I", os.path.join(ROOT, "include"),
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"] + SAN

    def compile_one(src):
        obj = os.path.join(OUT, os.path.basename(src) + ".o")
        r = subprocess.run([hipcc, *flags, "-c", src, "-o", obj], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-4000:]
        return obj

    with ThreadPoolExecutor(min(8, len(srcs))) as ex:
        objs = list(ex.map(compile_one, srcs))
    drv = os.path.join(OUT, "abi_errors.o")
    r = subprocess.run([clang, "-O1", "-g", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                        "-I", os.path.join(ROCM, "include"), "-fsanitize=address,undefined",
                        "-fno-sanitize-recover=undefined", "-c", DRIVER, "-o", drv], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    r = subprocess.run([hipcc, "--offload-arch=gfx950", *SAN, "-o", exe + ".tmp", drv, *objs,
                        "-L", os.path.join(ROCM, "lib"), "-lamdhip64"], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    os.replace(exe + ".tmp", exe)
    return exe


def test_abi_error_paths_under_asan_ubsan():
    exe = _build()
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["HIP_VISIBLE_DEVICES"] = ""  # refusal paths only: no device may be touched
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    report = r.stdout + r.stderr
    assert "ERROR: AddressSanitizer" not in report, report[-4000:]
    assert "runtime error" not in report, report[-4000:]
    assert r.returncode == 0, report[-4000:]
    assert "abi error paths ok" in r.stdout
