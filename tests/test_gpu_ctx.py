"""GPU tests of the context layer (mpt_create ... mpt_copy_table): the three
phases on a context against the CPU oracle, the state machine, host and
device inputs, and identical tables under every level plan of the DP
(MPT_OPT_CHUNK_PAIRS), i.e. results that do not depend on how the cross
pairs are split over workgroups."""
import ctypes
import hashlib
import json
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2609_13692_amd import mpt
from paper_2609_13692_amd import workloads as wl

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    mpt.load()
    yield


def say(msg):
    print(msg, flush=True)


def digest(a, dtype):
    return hashlib.sha256(np.ascontiguousarray(a, dtype=dtype).tobytes()).hexdigest()


def tensors(inst, device):
    return (torch.as_tensor(inst.weights, dtype=torch.int64).to(device),
            torch.as_tensor(inst.req_off, dtype=torch.int64).to(device),
            torch.as_tensor(inst.req_chunks, dtype=torch.int32).to(device))


def ctx_solve(inst, chunk_pairs=0, device="cuda"):
    """Whole path on a fresh context; host copies of every table."""
    say(f"[gpu ctx] {inst.name} m={inst.m} nnz={inst.nnz} chunk_pairs={chunk_pairs} inputs on {device}")
    ctx = mpt.Context("cuda")
    if chunk_pairs:
        ctx.set_option(mpt.MPT_OPT_CHUNK_PAIRS, chunk_pairs)
    w, off, ch = tensors(inst, device)
    ctx.reserve(inst.m, inst.n_chunks, inst.nnz)
    ctx.build_weights(inst.m, inst.n_chunks, w, off, ch)
    opt, sav, split_host = ctx.solve_exact(want_split=True)
    orders = ctx.extract_orders()
    out = {"opt": opt, "savings": sav, "orders": orders, "split_host": split_host,
           "W": ctx.copy_table(mpt.MPT_TABLE_W), "C": ctx.copy_table(mpt.MPT_TABLE_C),
           "split": ctx.copy_table(mpt.MPT_TABLE_SPLIT), "sig": ctx.copy_table(mpt.MPT_TABLE_SIG),
           "orders_table": ctx.copy_table(mpt.MPT_TABLE_ORDERS)}
    ctx.close()
    return out


def assert_matches_oracle(inst, got, ref):
    assert got["opt"] == ref["opt"]
    assert got["savings"] == int(inst.weights[inst.req_chunks].sum()) - ref["opt"]
    assert np.array_equal(got["W"], ref["W"])
    assert got["C"][0] == mpt.MPT_COST_SENTINEL and np.array_equal(got["C"][1:], ref["C"][1:])
    assert np.array_equal(got["split"], ref["split"].astype(np.uint32))
    assert np.array_equal(got["split_host"], got["split"])
    assert np.array_equal(got["sig"], oracle.demand_sets(inst))
    assert np.array_equal(got["orders"], ref["orders"])
    assert np.array_equal(got["orders_table"], ref["orders"])


@pytest.mark.parametrize("idx", [1, 2, 3])
@pytest.mark.parametrize("where", ["cuda", "cpu"])
def test_context_against_the_oracle(idx, where):
    """Inputs from device or host memory give the oracle's tables."""
    inst = wl.config(idx)
    assert_matches_oracle(inst, ctx_solve(inst, device=where), oracle.solve(inst))


def test_context_on_the_largest_workload():
    with open(os.path.join(GOLDEN, "config_5.json")) as f:
        g = json.load(f)
    inst = wl.config(5)
    got = ctx_solve(inst)
    assert got["opt"] == g["opt"] and got["savings"] == g["savings"]
    assert digest(got["W"], "<i8") == g["W_sha256"]
    assert digest(got["C"][1:], "<i8") == g["C_sha256_from_1"]
    assert digest(got["split"], "<u4") == g["split_sha256"]
    assert got["orders"].tolist() == g["orders"]


# chunk sizes: 1 pair per workgroup (every level split to the limit), 2, 3, 5
# and 7 (chunk boundaries that cut the A_H order at odd places; narrow keys run
# pairs in sets of two on alternating buffers, so these end a chunk on a full
# set, after one pair of the second set, after one pair of a reused first set
# and after one pair of a reused second set) and 1 << 20 (every level in one
# chunk, rows finished in the cross-pair kernel)
PLANS = [1, 2, 3, 5, 7, 1 << 20]


@pytest.mark.parametrize("idx", [3, 4])
def test_tables_do_not_depend_on_the_level_plan(idx):
    with open(os.path.join(GOLDEN, f"config_{idx}.json")) as f:
        g = json.load(f)
    inst = wl.config(idx)
    for cp in PLANS:
        got = ctx_solve(inst, chunk_pairs=cp)
        assert got["opt"] == g["opt"], cp
        assert digest(got["C"][1:], "<i8") == g["C_sha256_from_1"], cp
        assert digest(got["split"], "<u4") == g["split_sha256"], cp
        assert got["orders"].tolist() == g["orders"], cp


def test_wide_keys_do_not_depend_on_the_level_plan():
    """The same on the 64-bit key paths: the m = 20 retrieval workload with
    weights x64 (doubles) and x2^17 (uint64), every level split to one pair
    per workgroup and every level in one chunk."""
    import dataclasses
    with open(os.path.join(GOLDEN, "config_3.json")) as f:
        g = json.load(f)
    base = wl.config(3)
    for scale in (64, 1 << 17):
        inst = dataclasses.replace(base, weights=base.weights * scale, name=f"{base.name} x{scale}")
        for cp in (1, 1 << 20):
            got = ctx_solve(inst, chunk_pairs=cp)
            assert got["opt"] == scale * g["opt"]
            assert not (got["C"][1:] % scale).any()
            assert digest(got["C"][1:] // scale, "<i8") == g["C_sha256_from_1"], (scale, cp)
            assert digest(got["split"], "<u4") == g["split_sha256"], (scale, cp)


def routed_W(inst, route):
    ctx = mpt.Context("cuda")
    ctx.set_option(mpt.MPT_OPT_WEIGHT_ROUTE, route)
    w, off, ch = tensors(inst, "cuda")
    ctx.reserve(inst.m, inst.n_chunks, inst.nnz)
    ctx.build_weights(inst.m, inst.n_chunks, w, off, ch)
    W = ctx.copy_table(mpt.MPT_TABLE_W)
    ctx.close()
    return W


# m below the 11-bit low pass, at it, one past it, and the high passes (the
# m - 11 high bits in passes of at most 7, as even as possible): one pass of
# 1 .. 5 bits in registers, of 6 or 7 bits through LDS tiles, and two passes
# of each kind and mixed (19: 4 + 4, 21: 5 + 5, 22: 6 + 5, 23: 6 + 6)
ROUTE_MS = [1, 4, 10, 11, 12, 13, 14, 15, 16, 17, 18, 19, 21, 22, 23]


@pytest.mark.parametrize("m", ROUTE_MS)
def test_both_weight_routes_give_the_oracle_table(m):
    """The list route and the dense route (scatter, then the zeta passes)
    on the same instances: requests of random sizes, chunks of random
    weights, some chunks held by no request, and a slice of chunks held by
    every request (S_x = all requests)."""
    rng = np.random.default_rng(100 + m)
    u = int(rng.integers(50, 4000))
    sets = []
    for i in range(m):
        k = int(rng.integers(0, u // 2 + 1))
        sets.append(sorted(set(rng.choice(u, size=k, replace=False).tolist()) | {0, 1}))
    w = rng.integers(1, 1 << 20, size=u + 7, dtype=np.int64)
    inst = wl.from_sets(sets, w, u + 7, name=f"routes m={m}")
    say(f"[gpu ctx] weight routes m={m} u={inst.n_chunks} nnz={inst.nnz}")
    ref = oracle.intersection_weights(inst)
    for route in (mpt.MPT_ROUTE_LIST, mpt.MPT_ROUTE_DENSE):
        assert np.array_equal(routed_W(inst, route), ref), route


def test_dense_route_with_repeated_demand_sets():
    """Many chunks with the same few S_x (hash slots shared within a
    workgroup) after a first stretch of chunks with nearly all-distinct S_x:
    the list keeps chunk order, so those slices fill the LDS table past its
    probe limit and the overflow goes to W directly."""
    rng = np.random.default_rng(7)
    m, u = 18, 300000
    # the first 40% of chunks in 3 .. m random requests, the others in 1 or 2
    k = np.where(np.arange(u) < 2 * u // 5, rng.integers(3, m + 1, size=u), rng.integers(1, 3, size=u))
    rank = rng.random((u, m)).argsort(1).argsort(1)
    held = rank < k[:, None]
    memb = [np.nonzero(held[:, i])[0].tolist() for i in range(m)]
    w = rng.integers(1, 1000, size=u, dtype=np.int64)
    inst = wl.from_sets(memb, w, u, name="repeated demand sets")
    say(f"[gpu ctx] dense route, repeated sets m={m} nnz={inst.nnz}")
    assert np.array_equal(routed_W(inst, mpt.MPT_ROUTE_DENSE), oracle.intersection_weights(inst))


def test_state_machine():
    """created -> built -> solved -> extracted, MPT_E_STATE out of order; a
    new build, a failed build, a new workspace or an option reset it."""
    inst = wl.config(1)
    ctx = mpt.Context("cuda")
    w, off, ch = tensors(inst, "cuda")

    def expect(code, fn, *a):
        with pytest.raises(mpt.MptError) as ei:
            fn(*a)
        assert ei.value.name == code, ei.value

    expect("MPT_E_WORKSPACE", ctx.build_weights, inst.m, inst.n_chunks, w, off, ch)   # no workspace yet
    ctx.reserve(inst.m, inst.n_chunks, inst.nnz)
    expect("MPT_E_STATE", ctx.solve_exact)
    expect("MPT_E_STATE", ctx.extract_orders)
    ctx.build_weights(inst.m, inst.n_chunks, w, off, ch)
    expect("MPT_E_STATE", ctx.extract_orders)
    expect("MPT_E_STATE", ctx.optimum)
    expect("MPT_E_STATE", ctx.copy_table, mpt.MPT_TABLE_C)
    assert np.array_equal(ctx.copy_table(mpt.MPT_TABLE_W), oracle.intersection_weights(inst))
    opt, sav, _ = ctx.solve_exact()
    assert ctx.optimum() == (opt, sav)
    expect("MPT_E_STATE", ctx.copy_table, mpt.MPT_TABLE_ORDERS)
    orders = ctx.extract_orders()
    ref = oracle.solve(inst)
    assert opt == ref["opt"] and np.array_equal(orders, ref["orders"])
    # extraction and solve may be repeated
    assert np.array_equal(ctx.extract_orders(), orders)
    assert ctx.solve_exact()[0] == opt
    # a failed build (a duplicate chunk) leaves no instance
    bad = ch.clone()
    bad[1] = bad[0]
    expect("MPT_E_DUP", ctx.build_weights, inst.m, inst.n_chunks, w, off, bad)
    expect("MPT_E_STATE", ctx.solve_exact)
    expect("MPT_E_STATE", ctx.copy_table, mpt.MPT_TABLE_W)
    # a workspace too small for the instance
    ctx.set_workspace(ctx.workspace[:1024])
    expect("MPT_E_WORKSPACE", ctx.build_weights, inst.m, inst.n_chunks, w, off, ch)
    ctx.set_workspace(ctx.workspace)
    ctx.build_weights(inst.m, inst.n_chunks, w, off, ch)
    ctx.set_option(mpt.MPT_OPT_CHUNK_PAIRS, 2)
    expect("MPT_E_STATE", ctx.solve_exact)
    expect("MPT_E_INVALID", ctx.set_option, 99, 1)
    expect("MPT_E_INVALID", ctx.set_option, mpt.MPT_OPT_WEIGHT_ROUTE, 3)
    expect("MPT_E_INVALID", ctx.set_option, mpt.MPT_OPT_CHUNK_PAIRS, -1)
    expect("MPT_E_INVALID", ctx.copy_table, 17)
    # table_device gives the table's address inside the workspace
    ctx.build_weights(inst.m, inst.n_chunks, w, off, ch)
    ptr, nb = ctx.table_device(mpt.MPT_TABLE_W)
    base = ctx.workspace.data_ptr()
    assert nb == 8 << inst.m and base <= ptr and ptr + nb <= base + ctx.workspace.numel()
    ctx.close()


def test_solve_and_extract_without_host_data():
    """A solve that returns nothing to the host and the extraction queue
    their work back to back; mpt_ctx_optimum then reads OPT_free."""
    inst = wl.config(3)
    ref = oracle.solve(inst)
    ctx = mpt.Context("cuda")
    w, off, ch = tensors(inst, "cuda")
    ctx.reserve(inst.m, inst.n_chunks, inst.nnz)
    ctx.build_weights(inst.m, inst.n_chunks, w, off, ch)
    assert ctx.solve_exact(want_cost=False) == (None, None, None)
    assert ctx.extract_orders(to_host=False) is None
    assert ctx.optimum() == (ref["opt"], int(inst.weights[inst.req_chunks].sum()) - ref["opt"])
    assert np.array_equal(ctx.copy_table(mpt.MPT_TABLE_ORDERS), ref["orders"])
    ctx.close()


def test_two_contexts_are_independent():
    a_inst, b_inst = wl.config(1), wl.config(1, seed=2)
    a, b = mpt.Context("cuda"), mpt.Context("cuda")
    ra = a.run(a_inst)
    rb = b.run(b_inst)
    assert ra["opt"] == oracle.solve(a_inst)["opt"] and rb["opt"] == oracle.solve(b_inst)["opt"]
    assert np.array_equal(a.copy_table(mpt.MPT_TABLE_SPLIT), oracle.solve(a_inst)["split"].astype(np.uint32))
    a.close()
    b.close()


def test_context_on_a_side_stream():
    """Work goes to the context's stream, which may be any stream of its
    device."""
    inst = wl.config(3)
    s = torch.cuda.Stream()
    ctx = mpt.Context("cuda", stream=s)
    r = ctx.run(inst)
    assert r["opt"] == json.load(open(os.path.join(GOLDEN, "config_3.json")))["opt"]
    ctx.close()
