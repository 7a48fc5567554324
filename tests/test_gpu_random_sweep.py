"""Seeded random sweep through the C ABI against the CPU oracle: the exact
DP (32-bit and 64-bit keys, several level plans), the greedy with its
layout and bound, global-order layouts, trie cost and DFS order of
shuffled layouts, and the W table's dense route. Integer results, compared
exactly. The shapes vary across the paths' thresholds: requests of up to
64 chunks and longer, DP instances past 2^20 total weight, and high zeta
passes of 1 to 7 bits."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_13692_amd import mpt
from paper_2609_13692_amd import workloads as wl

pytestmark = pytest.mark.gpu

SEED = 20260601


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    mpt.load()
    yield


def say(msg):
    print(msg, flush=True)


def tensors(inst):
    return (torch.as_tensor(inst.weights, dtype=torch.int64).cuda(),
            torch.as_tensor(inst.req_off, dtype=torch.int64).cuda(),
            torch.as_tensor(inst.req_chunks, dtype=torch.int32).cuda())


def rand_inst(rng, m_lo, m_hi, u_lo, u_hi, k_hi):
    m = int(rng.integers(m_lo, m_hi)); u = int(rng.integers(u_lo, u_hi))
    return wl.random_small(m=m, u=u, kmin=0, kmax=min(u, int(rng.integers(1, k_hi))),
                           wmax=int(rng.integers(1, 400)), seed=int(rng.integers(1 << 30)))


@pytest.mark.parametrize("case", range(12))
def test_dp_random(case):
    rng = np.random.default_rng((SEED, 1, case))
    inst = rand_inst(rng, 13, 19, 20, 3000, 60)
    if case % 3 == 2:   # past the 32-bit keys' range: doubles or uint64
        inst = wl.from_sets(inst.requests(), (inst.weights * (64 if case % 2 else 4096)).tolist(), inst.n_chunks)
    cp = [0, 1, 2, 3, 7, 20][case % 6]
    say(f"[gpu sweep] dp case {case} m={inst.m} nnz={inst.nnz} chunk_pairs={cp}")
    ctx = mpt.Context("cuda")
    if cp:
        ctx.set_option(mpt.MPT_OPT_CHUNK_PAIRS, cp)
    w, off, ch = tensors(inst)
    ctx.reserve(inst.m, inst.n_chunks, inst.nnz)
    ctx.build_weights(inst.m, inst.n_chunks, w, off, ch)
    opt, _, _ = ctx.solve_exact()
    orders = ctx.extract_orders()
    W, C = ctx.copy_table(mpt.MPT_TABLE_W), ctx.copy_table(mpt.MPT_TABLE_C)
    split = ctx.copy_table(mpt.MPT_TABLE_SPLIT)
    ctx.close()
    ref = oracle.solve(inst)
    assert opt == ref["opt"]
    assert np.array_equal(W, ref["W"])
    assert np.array_equal(C[1:], ref["C"][1:])
    assert np.array_equal(split, ref["split"].astype(np.uint32))
    assert np.array_equal(np.asarray(orders), np.asarray(ref["orders"]))


@pytest.mark.parametrize("case", range(8))
def test_greedy_random(case):
    rng = np.random.default_rng((SEED, 2, case))
    inst = rand_inst(rng, 20, 300, 30, 2000, 100)
    say(f"[gpu sweep] greedy case {case} m={inst.m} nnz={inst.nnz}")
    g = mpt.Greedy(inst)
    got = g.run()
    torch.cuda.synchronize()
    got.update(g.host())
    ref = oracle.greedy_solve(inst)
    for k in ("P", "merge_a", "merge_b", "gain", "parent", "orders"):
        assert np.array_equal(got[k], ref[k]), k
    assert got["mst"] == ref["mst"] and got["cost"] == ref["cost"] and got["lower_bound"] == ref["lower_bound"]


@pytest.mark.parametrize("case", range(8))
def test_layouts_random(case):
    rng = np.random.default_rng((SEED, 3, case))
    inst = rand_inst(rng, 50, 3000, 10, 400, 90)
    say(f"[gpu sweep] layouts case {case} m={inst.m} nnz={inst.nnz}")
    L = mpt.Layouts(inst)
    for kind, rank in ((mpt.MPT_ORDER_ID, oracle.id_rank(inst)), (mpt.MPT_ORDER_POPULARITY, oracle.popularity_rank(inst))):
        assert np.array_equal(L.global_order(kind).cpu().numpy(), oracle.global_order_layout(inst, rank)), kind
    lay = np.asarray(inst.req_chunks, dtype=np.int32).copy()
    for r in range(inst.m):
        a, b = inst.req_off[r], inst.req_off[r + 1]
        lay[a:b] = rng.permutation(lay[a:b])
    assert L.cost(L.seqs(lay)) == oracle.trie_cost(inst, lay)
    assert np.array_equal(L.dfs.cpu().numpy(), oracle.dfs_schedule(inst, lay))


# high zeta passes: 1, 3, 5 bits in registers; 6, 7 through LDS tiles;
# 4 + 4, 6 + 5, 6 + 6
DENSE_MS = [12, 14, 16, 17, 18, 19, 22, 23]


@pytest.mark.parametrize("case", range(len(DENSE_MS)))
def test_dense_route_random(case):
    rng = np.random.default_rng((SEED, 4, case))
    m = DENSE_MS[case]
    u = int(rng.integers(100, 5000))
    inst = wl.random_small(m=m, u=u, kmin=0, kmax=int(rng.integers(1, u)), wmax=int(rng.integers(1, 1000)),
                           seed=int(rng.integers(1 << 30)))
    say(f"[gpu sweep] dense route case {case} m={m} nnz={inst.nnz}")
    ctx = mpt.Context("cuda")
    ctx.set_option(mpt.MPT_OPT_WEIGHT_ROUTE, mpt.MPT_ROUTE_DENSE)
    w, off, ch = tensors(inst)
    ctx.reserve(inst.m, inst.n_chunks, inst.nnz)
    ctx.build_weights(inst.m, inst.n_chunks, w, off, ch)
    W = ctx.copy_table(mpt.MPT_TABLE_W)
    ctx.close()
    assert np.array_equal(W, oracle.intersection_weights(inst))
