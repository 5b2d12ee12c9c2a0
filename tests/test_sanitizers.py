"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only,
no device is touched).

* The oracle's C Householder QR (oracle/householder.c), built with gcc and
  both sanitizers, factors a few matrices (n = 1 .. 130, a zero and a
  repeated column) through tests/sanitize/householder_driver.c.
* The library's host code (argument validation, workspace layouts, the
  status, timing and test-hook entry points), built with the sanitizers on
  its host side only (each -fsanitize flag behind -Xarch_host; device code is
  unchanged), driven by tests/sanitize/abi_driver.cpp: every call fails
  validation or computes on the host, with the documented status codes.
The sanitizer build of the library goes to _build/ and is rebuilt only when a
source changes (the first build takes about a minute)."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
SAN_DIR = os.path.join(ROOT, "_build", "sanitize")
CLANG = "/opt/rocm/llvm/bin/clang++"


def _run(exe, **env_extra):
    env = dict(os.environ, **env_extra)
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    return out


def test_oracle_householder_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "householder_driver")
    subprocess.check_call(["gcc", "-std=c99", "-O1", "-g", "-fno-omit-frame-pointer", "-fopenmp",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                           os.path.join(HERE, "householder_driver.c"),
                           os.path.join(ROOT, "oracle", "householder.c"), "-o", exe, "-lm"])
    assert "ok" in _run(exe, ASAN_OPTIONS="detect_leaks=1")


@pytest.mark.skipif(not os.path.exists(CLANG), reason="ROCm clang++ not found")
def test_library_host_code_under_asan_and_ubsan(tmp_path):
    from paper_2607_20548_amd import build
    san = []
    for f in ("address", "undefined"):
        san += ["-Xarch_host", f"-fsanitize={f}"]
    san += ["-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
    lib = build.build(force=False, extra=san, out=os.path.join(SAN_DIR, "libsoap_sanitize.so"))
    exe = str(tmp_path / "abi_driver")
    subprocess.check_call([CLANG, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                           "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                           "-I", "/opt/rocm/include", os.path.join(HERE, "abi_driver.cpp"),
                           "-L", SAN_DIR, "-lsoap_sanitize", "-Wl,-rpath," + SAN_DIR,
                           "-L", "/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib",
                           "-o", exe])
    # the HIP runtime keeps its allocations until exit: no leak report
    out = _run(exe, ASAN_OPTIONS="detect_leaks=0")
    assert "ok (0 failures)" in out, out[-4000:]
