"""Compile tests/c/abi_test.c as C11 with hipcc against the built libmpt.so."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "abi_test.c")
EXE = os.path.join(HERE, "abi_test")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build() -> str:
    tmp = EXE + ".tmp"
    cmd = [HIPCC, "-x", "c", "-std=c11", "-O1", "-Wall", "-Wextra", "-Werror", "-pedantic",
           "-D__HIP_PLATFORM_AMD__", "-isystem", "/opt/rocm/include", "-I", os.path.join(ROOT, "include"),
           SRC, "-o", tmp, "-L", os.path.join(ROOT, "paper_2609_13692_amd"), "-lmpt",
           "-L", "/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,$ORIGIN/../../paper_2609_13692_amd"]
    subprocess.check_call(cmd)
    os.replace(tmp, EXE)
    return EXE


if __name__ == "__main__":
    print(build())
