"""GPU parity of the Section 6.2-6.3 calls (pair weights, agglomerative
hierarchy H_g with its layout, spanning-tree bound) through the C ABI
against the CPU oracle. Integer work, so every comparison is bit-exact:
the pair-weight matrix, the merge sequence (names and gains, under the
tie reading of the header), the node parents, the read-off orders, the
savings and the spanning-tree weight.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_13692_amd import mpt
from paper_2609_13692_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    mpt.load()
    yield


def say(msg):
    print(msg, flush=True)


def gpu_greedy(inst):
    say(f"[gpu greedy] {inst.name} m={inst.m} nnz={inst.nnz}")
    g = mpt.Greedy(inst)
    res = g.run()
    torch.cuda.synchronize()
    res.update(g.host())
    return res


def assert_same(inst, got, ref):
    m = inst.m
    assert np.array_equal(got["P"], ref["P"]), "pair weights differ"
    assert got["request_total"] == ref["request_total"]
    a, b, g = got["merge_a"], got["merge_b"], got["gain"]
    bad = np.nonzero((a != ref["merge_a"]) | (b != ref["merge_b"]) | (g != ref["gain"]))[0]
    assert bad.size == 0, f"merge {bad[:4]} differs: gpu {list(zip(a[bad[:4]], b[bad[:4]], g[bad[:4]]))} " \
                          f"oracle {list(zip(ref['merge_a'][bad[:4]], ref['merge_b'][bad[:4]], ref['gain'][bad[:4]]))}"
    assert np.array_equal(got["parent"], ref["parent"]), "node parents differ"
    assert got["savings"] == ref["savings"]
    assert np.array_equal(got["orders"], ref["orders"]), "orders differ"
    assert got["mst"] == ref["mst"]
    assert got["cost"] == ref["cost"] and got["lower_bound"] == ref["lower_bound"]
    assert got["parent"].size == 2 * m - 1


@pytest.mark.parametrize("n", [2, 3, 5, 16, 33, 64, 128])
def test_loo(n):
    """L_n: exactly optimal (Section 6.2), bound 2(n-1)."""
    inst = wl.gen_loo(n)
    got = gpu_greedy(inst)
    assert_same(inst, got, oracle.greedy_solve(inst))
    assert got["lower_bound"] == 2 * (n - 1)


def test_tightness_witness():
    inst = wl.from_sets([[0, 1, 2, 3], [1, 4], [2, 5, 7, 8], [4, 6]], [1] * 9, 9)
    got = gpu_greedy(inst)
    assert_same(inst, got, oracle.greedy_solve(inst))
    assert got["gain"].tolist() == [1, 0, 0]


@pytest.mark.parametrize("seed", range(16))
def test_random_small(seed):
    rng = np.random.default_rng(seed)
    m = int(rng.integers(1, 70))
    u = int(rng.integers(1, 60))
    inst = wl.random_small(m=m, u=u, kmin=0, kmax=min(u, 12), wmax=int(rng.choice([1, 3, 1000])), seed=1000 + seed)
    got = gpu_greedy(inst)
    assert_same(inst, got, oracle.greedy_solve(inst))


@pytest.mark.parametrize("name", ["trace_512", "trace_2048"])
def test_trace_shaped(name):
    inst = wl.trace_config(name)
    got = gpu_greedy(inst)
    ref = oracle.greedy_solve(inst)
    assert_same(inst, got, ref)
    # the Theorem 1 sandwich for the layout read off H_g
    assert oracle.trie_cost(inst, got["orders"]) <= got["cost"]
    assert got["lower_bound"] <= got["cost"]


@pytest.mark.parametrize("seed", [1, 2])
def test_trace_shaped_seeds(seed):
    inst = wl.trace_config("trace_512", seed=seed)
    got = gpu_greedy(inst)
    assert_same(inst, got, oracle.greedy_solve(inst))


def test_trace_4096_full():
    """The benchmark instance, whole outputs against the oracle."""
    inst = wl.trace_config("trace_4096")
    got = gpu_greedy(inst)
    ref = oracle.greedy_solve(inst)
    assert_same(inst, got, ref)
    gains = got["gain"]
    assert np.all(gains[:-1] >= gains[1:])                # Theorem 6 part (i)


def test_degenerate_families():
    cases = [
        wl.from_sets([[5, 2, 9]], [1] * 10, 10),                          # one request
        wl.from_sets([[], []], [], 0),                                     # empty universe
        wl.from_sets([[1, 0], [0, 1], [1, 0]], [4, 7], 2),                 # identical requests
        wl.from_sets([[], [3], [], [1, 2]], [1] * 4, 4),                   # empty and disjoint requests
        wl.from_sets([[0]] * 40, [1 << 32], 1),                            # heaviest weight, all equal
        wl.from_sets([[i] for i in range(50)], [1] * 50, 50),              # nothing shared at all
    ]
    for inst in cases:
        got = gpu_greedy(inst)
        assert_same(inst, got, oracle.greedy_solve(inst))


def test_many_ties():
    """Unit weights with heavy overlap: long runs of equal merge values,
    decided by the tie reading alone."""
    rng = np.random.default_rng(7)
    sets = [sorted(rng.choice(6, size=int(rng.integers(1, 6)), replace=False).tolist()) for _ in range(300)]
    inst = wl.from_sets(sets, [1] * 6, 6)
    got = gpu_greedy(inst)
    assert_same(inst, got, oracle.greedy_solve(inst))


def test_error_codes():
    good = wl.from_sets([[0, 1], [1, 2]], [1, 1, 1], 3)
    g = mpt.Greedy(good)
    # chunk id out of range
    g.req_chunks[0] = 7
    with pytest.raises(mpt.MptError) as e:
        g.pair_weights()
    assert e.value.status == -2
    # repeated chunk inside a request
    g.req_chunks[0] = 1
    with pytest.raises(mpt.MptError) as e:
        g.hierarchy()
    assert e.value.status == -3
    # bad weight
    g.req_chunks[0] = 0
    g.chunk_w[2] = 0
    with pytest.raises(mpt.MptError) as e:
        g.pair_weights()
    assert e.value.status == -4
    # offsets that are not CSR
    g.chunk_w[2] = 1
    g.req_off[1] = 5
    with pytest.raises(mpt.MptError) as e:
        g.hierarchy()
    assert e.value.status == -1
    # and the instance is fine again once repaired
    g.req_off[1] = 2
    res = g.run()
    assert res["savings"] == 1 and res["mst"] == 1


def test_determinism():
    inst = wl.trace_config("trace_512", seed=5)
    a = gpu_greedy(inst)
    b = gpu_greedy(inst)
    for k in ("P", "merge_a", "merge_b", "gain", "parent", "orders"):
        assert np.array_equal(a[k], b[k]), k


# --- shapes that stress the merge rounds -----------------------------------

@pytest.mark.parametrize("seed", range(24))
def test_rounds_give_the_sequential_merges(seed):
    """Unit or small weights over a small pool: many equal merge values
    within a round and across rounds, so the sequence differs from the
    order the rounds find the merges in and rests on the pair order alone."""
    rng = np.random.default_rng(500 + seed)
    m = int(rng.integers(5, 160))
    u = int(rng.integers(4, 40))
    sets = [rng.choice(u, size=int(rng.integers(0, u // 2 + 1)), replace=False).tolist() for _ in range(m)]
    w = rng.integers(1, 1 + int(rng.choice([1, 2, 6])), size=u)
    inst = wl.from_sets(sets, w.tolist(), u, name=f"ties seed {seed}")
    got = gpu_greedy(inst)
    assert_same(inst, got, oracle.greedy_solve(inst))


def test_cluster_state_in_global_memory():
    """m = 6000 requests: more clusters than one workgroup could hold state
    for; rounds of thousands of merges and rescans."""
    inst = wl.gen_retrieval(m=6000, u=18000, topics=188, k=8, seed=3)
    got = gpu_greedy(inst)
    assert_same(inst, got, oracle.greedy_solve(inst))


def test_long_intersections():
    """Requests of 1500-4000 chunks around a shared core of 2500: long
    signature intersections in the merges and in the new rows."""
    rng = np.random.default_rng(11)
    u = 9000
    core = rng.choice(u, size=2500, replace=False)
    rest = np.setdiff1d(np.arange(u), core)
    sets = []
    for _ in range(40):
        keep = core[rng.random(core.size) < rng.uniform(0.85, 1.0)]
        extra = rng.choice(rest, size=int(rng.integers(0, 1500)), replace=False)
        sets.append(np.concatenate([keep, extra]).tolist())
    w = rng.integers(1, 200, size=u)
    inst = wl.from_sets(sets, w.tolist(), u)
    got = gpu_greedy(inst)
    assert_same(inst, got, oracle.greedy_solve(inst))


def test_many_candidate_columns():
    """m = 3000 requests that all hold one common chunk: every merge has
    positive values against every other cluster, so every new row is
    recomputed in full."""
    base = wl.gen_retrieval(m=3000, u=9000, topics=94, k=8, seed=4)
    sets = [r + [9000] for r in base.requests()]
    w = np.concatenate([base.weights, [5]])
    inst = wl.from_sets(sets, w.tolist(), 9001)
    got = gpu_greedy(inst)
    assert_same(inst, got, oracle.greedy_solve(inst))


def test_largest_m_properties():
    """m = 16384, the largest the calls take. The cubic oracle is out of
    reach, so: pair weights and spanning-tree bound against the oracle,
    the first merge against the maximum of P (ties to the smallest pair),
    merge values non-increasing (Theorem 6 part (i)), the savings equal to
    the sum of the merge values and to Eq. 3 on the returned hierarchy, and
    the layout equal to the one read off that hierarchy."""
    inst = wl.gen_retrieval(m=16384, u=49152, topics=512, k=8, seed=6)
    got = gpu_greedy(inst)
    m = inst.m
    P = oracle.pair_weights(inst)
    assert np.array_equal(got["P"], P)
    assert got["mst"] == oracle.max_spanning_tree(P)
    off = P.copy()
    np.fill_diagonal(off, -1)
    best = off.max()
    i, j = np.argwhere(off == best)[0]                       # row-major: smallest (i, j), i < j
    assert (got["merge_a"][0], got["merge_b"][0], got["gain"][0]) == (i, j, best)
    g = got["gain"]
    assert np.all(g[:-1] >= g[1:]) and g[-1] >= 0
    assert got["savings"] == int(g.sum()) == oracle.tree_savings(inst, got["parent"])
    assert got["cost"] == int(np.trace(P)) - got["savings"]
    assert np.array_equal(got["orders"], oracle.tree_orders(inst, got["parent"]))
    parent = got["parent"]
    assert parent.size == 2 * m - 1 and parent[-1] == -1
    assert np.all(np.bincount(parent[:-1], minlength=2 * m - 1)[m:] == 2)


@pytest.mark.parametrize("n", [64, 65])
def test_list_lengths_at_the_short_path_limit(n):
    """Requests of up to 64 chunks have their lists ranked inside each
    request, longer ones go through the key sort: both sides of the limit,
    and a repeated chunk detected on each."""
    rng = np.random.default_rng(n)
    sets = [rng.permutation(n + 10)[:n].tolist() for _ in range(6)] + [list(range(3))]
    inst = wl.from_sets(sets, rng.integers(1, 50, size=n + 10).tolist(), n + 10)
    assert_same(inst, gpu_greedy(inst), oracle.greedy_solve(inst))
    g = mpt.Greedy(inst)
    g.req_chunks[1] = g.req_chunks[0]
    with pytest.raises(mpt.MptError) as e:
        g.hierarchy()
    assert e.value.status == -3
