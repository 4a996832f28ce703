"""CPU: the C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

api.cpp is built with the sanitizers on its host side (-Xarch_host), linked
with stubs of the kernel launchers (tests/host_check/stubs.cpp) and driven by
tests/host_check/host_check.c through every argument check, size computation,
launch decision and error path of include/hagdn.h.  Any out-of-bounds access
or undefined behaviour in the host code aborts the program.  Leak detection is
off: the HIP runtime keeps allocations until exit by design.
"""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang"
CLANGXX = "/opt/rocm/llvm/bin/clang++"
SAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all"]
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"]


def _need(tool):
    if not (os.path.exists(tool) or shutil.which(tool)):
        pytest.skip(f"{tool} not available")


def test_host_code_under_sanitizers(tmp_path):
    for t in (HIPCC, CLANG, CLANGXX):
        _need(t)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2609_32114_amd", "csrc")]
    hip = [HIPCC, "-x", "hip", "--offload-arch=gfx950", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           *SAN_HOST, *inc]
    steps = [
        hip + ["-c", os.path.join(ROOT, "paper_2609_32114_amd", "csrc", "api.cpp"), "-o", str(tmp_path / "api.o")],
        hip + ["-c", os.path.join(ROOT, "tests", "host_check", "stubs.cpp"), "-o", str(tmp_path / "stubs.o")],
        [CLANG, "-O1", "-g", *SAN, *inc, "-c", os.path.join(ROOT, "tests", "host_check", "host_check.c"),
         "-o", str(tmp_path / "hc.o")],
        [CLANGXX, *SAN, str(tmp_path / "hc.o"), str(tmp_path / "api.o"), str(tmp_path / "stubs.o"),
         "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", str(tmp_path / "host_check")],
    ]
    for cmd in steps:
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stderr}"
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(tmp_path / "host_check")], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0 and "host checks passed" in r.stdout, r.stdout + r.stderr
