"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

* The CPU oracle (oracle/mpt_oracle.c) compiled with gcc -fsanitize=address,
  undefined into tests/c/oracle_sanitize.c, which drives every oracle
  function on the paper's pinned instances (Theorems 1, 4, 5 and 7, Section
  6.3) and checks the pins.
* The library's host code (validation, workspace layout, the context layer)
  compiled with the host pass instrumented (hipcc -Xarch_host -fsanitize=...,
  the device code as usual), driven by the C ABI test program's host checks.

Both builds go to a temporary directory; a sanitizer report fails the test.
"""
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2609_13692_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def run(cmd, env=None, timeout=600):
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=timeout, env=env)
    return r.returncode, r.stdout + r.stderr


def test_oracle_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_san")
    rc, out = run(["gcc", "-std=c11", "-O1", "-g", "-fopenmp", "-fno-omit-frame-pointer",
                   "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                   os.path.join(HERE, "c", "oracle_sanitize.c"), "-o", exe])
    assert rc == 0, out
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", OMP_NUM_THREADS="2")
    rc, out = run([exe], env=env)
    assert rc == 0, out
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out
    assert "all checks hold" in out


@pytest.mark.slow
def test_library_host_code_under_asan_and_ubsan(tmp_path):
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    lib = str(tmp_path / "libmpt.so")
    srcs = [os.path.join(CSRC, f) for f in ("mpt.hip", "ctx.hip", "greedy.hip", "layout.hip", "pinned.hip")]
    rc, out = run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-shared",
                   "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-fno-honor-nans", *san,
                   "-I", os.path.join(ROOT, "include"), *srcs, "-o", lib,
                   "-L", "/opt/rocm/lib", "-lrocprofiler-sdk-roctx", "-Wl,-rpath,/opt/rocm/lib"])
    assert rc == 0, out
    exe = str(tmp_path / "abi_test_san")
    rc, out = run([HIPCC, "-x", "c", "-std=c11", "-O1", "-g", "-D__HIP_PLATFORM_AMD__",
                   "-isystem", "/opt/rocm/include", "-I", os.path.join(ROOT, "include"), *san,
                   os.path.join(HERE, "c", "abi_test.c"), "-o", exe, "-L", str(tmp_path), "-lmpt",
                   "-L", "/opt/rocm/lib", "-lamdhip64", f"-Wl,-rpath,{tmp_path}"])
    assert rc == 0, out
    # the HIP runtime keeps allocations until exit: leak checking is off here
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0")
    rc, out = run([exe, "host"], env=env)
    assert rc == 0, out
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out
