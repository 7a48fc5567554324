"""The allocation-free solve (mpt_solve_exact_noalloc), whose scratch is a
device array inside the library, against the workspace solve
(mpt_solve_exact) on the same W, bit for bit: several calls in a row on one
device, each smaller than the one before, so each call runs on what the
previous one left in the shared array."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2609_13692_amd import mpt
from paper_2609_13692_amd import workloads as wl

pytestmark = pytest.mark.gpu


def built(inst):
    dev = torch.device("cuda")
    t = lambda a, dt: torch.as_tensor(a, dtype=dt).to(dev)
    n = 1 << inst.m
    W = torch.empty(n, dtype=torch.int64, device=dev)
    sig = torch.empty(max(1, inst.n_chunks), dtype=torch.int32, device=dev)
    ws = mpt.alloc_workspace(inst.m, inst.nnz, dev)
    mpt.mpt_build_weights(inst.m, inst.n_chunks, t(inst.weights, torch.int64), t(inst.req_off, torch.int64),
                          t(inst.req_chunks, torch.int32), sig, W, ws)
    return W, ws


def test_noalloc_solve_equals_the_workspace_solve():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    # m = 20 (the array's limit), then smaller packed-key instances, then the
    # plain kernels (m = 12), then m = 20 again with narrow and wide keys
    cases = [wl.config(3), wl.gen_retrieval(m=17, u=800, topics=20, k=8, seed=5),
             wl.gen_retrieval(m=14, u=300, topics=10, k=6, seed=6), wl.config(1), wl.config(2)]
    import dataclasses
    base = wl.config(3)
    cases.append(dataclasses.replace(base, weights=base.weights * 64, name=base.name + " x64"))
    for inst in cases:
        print(f"[gpu] noalloc {inst.name} m={inst.m}", flush=True)
        W, ws = built(inst)
        n = 1 << inst.m
        C_ref = torch.empty(n, dtype=torch.int64, device="cuda")
        S_ref = torch.empty(n, dtype=torch.int32, device="cuda")
        opt_ref = mpt.mpt_solve_exact(inst.m, W, C_ref, S_ref, ws)
        C = torch.full((n,), -7, dtype=torch.int64, device="cuda")
        S = torch.full((n,), -7, dtype=torch.int32, device="cuda")
        opt = mpt.mpt_solve_exact_noalloc(inst.m, W, C, S)
        torch.cuda.synchronize()
        assert opt == opt_ref, inst.name
        assert torch.equal(C, C_ref), inst.name
        assert torch.equal(S, S_ref), inst.name


def test_noalloc_rejects_m_above_its_limit():
    lib = mpt.load()
    P = ctypes.c_void_p
    dummy = P(4096)          # never dereferenced: the call fails its host checks
    assert lib.mpt_solve_exact_noalloc(mpt.MPT_NOALLOC_MAX_M + 1, dummy, dummy, dummy, None, None) == -1
    assert b"MPT_NOALLOC_MAX_M" in lib.mpt_last_error()
    assert lib.mpt_solve_exact_noalloc(0, dummy, dummy, dummy, None, None) == -1
    assert lib.mpt_solve_exact_noalloc(4, None, dummy, dummy, None, None) == -1
