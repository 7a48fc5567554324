"""The C ABI from a C program (tests/c/abi_test.c, compiled as C11 by hipcc
and linked against libmpt.so): host-side argument checks without a GPU, and
on the GPU the context layer's whole path on the tiny workload, written out
by the C program and compared here with the CPU oracle."""
import os
import subprocess

import numpy as np
import pytest

import oracle
from paper_2609_13692_amd import workloads as wl

HERE = os.path.dirname(os.path.abspath(__file__))
EXE = os.path.join(HERE, "c", "abi_test")


def exe():
    if not os.path.exists(EXE):
        pytest.fail("tests/c/abi_test is not built (run __graft_entry__.build())")
    return EXE


def test_c_program_host_checks():
    r = subprocess.run([exe(), "host"], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr


def write_instance(inst, path):
    with open(path, "w") as f:
        f.write(f"{inst.m} {inst.n_chunks} {inst.nnz}\n")
        f.write(" ".join(str(int(x)) for x in inst.weights) + "\n")
        f.write(" ".join(str(int(x)) for x in inst.req_off) + "\n")
        f.write(" ".join(str(int(x)) for x in inst.req_chunks) + "\n")


@pytest.mark.gpu
@pytest.mark.parametrize("seed", [0, 3])
def test_c_program_solves_the_tiny_workload(tmp_path, seed):
    inst = wl.config(1, seed=seed)
    src, out = tmp_path / "in.txt", tmp_path / "out.txt"
    write_instance(inst, src)
    print(f"[gpu] abi_test run config 1 seed {seed}", flush=True)
    r = subprocess.run([exe(), "run", str(src), str(out)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    vals = np.array(out.read_text().split(), dtype=np.int64)
    n = 1 << inst.m
    ref = oracle.solve(inst)
    opt, sav = vals[0], vals[1]
    W, C, split, orders = vals[2:2 + n], vals[2 + n:2 + 2 * n], vals[2 + 2 * n:2 + 3 * n], vals[2 + 3 * n:]
    assert opt == ref["opt"] and sav == int(inst.weights[inst.req_chunks].sum()) - ref["opt"]
    assert np.array_equal(W, ref["W"])
    assert np.array_equal(C[1:], ref["C"][1:])
    assert np.array_equal(split, ref["split"].astype(np.int64))
    assert np.array_equal(orders, ref["orders"])
