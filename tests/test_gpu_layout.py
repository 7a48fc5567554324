"""GPU parity of the Section 7-8 calls (global-order layouts, trie cost and
DFS order, radix-cache simulation) through the C ABI against the CPU
oracle. Integer work: layouts, orders and billed weights are compared
exactly.
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


def max_request(inst):
    w = inst.weights
    return max(int(w[np.asarray(r, dtype=np.int64)].sum()) if r else 0 for r in inst.requests())


def test_global_orders_match_oracle():
    # (requests of up to 64 chunks are ordered inside each request, longer
    # ones by a key sort: both occur below)
    for inst in (wl.config(1), wl.gen_loo(9), wl.random_small(m=40, u=70, kmin=0, kmax=12, wmax=9, seed=3),
                 wl.random_small(m=20, u=400, kmin=40, kmax=120, wmax=9, seed=4),
                 wl.random_small(m=30, u=200, kmin=60, kmax=64, wmax=9, seed=6),
                 wl.trace_config("trace_512"), wl.trace_config("trace_4096")):
        say(f"[gpu layout] global orders {inst.name} m={inst.m}")
        L = mpt.Layouts(inst)
        for kind, rank in ((mpt.MPT_ORDER_ID, oracle.id_rank(inst)), (mpt.MPT_ORDER_POPULARITY, oracle.popularity_rank(inst))):
            got = L.global_order(kind).cpu().numpy()
            assert np.array_equal(got, oracle.global_order_layout(inst, rank)), kind


def layouts(inst):
    out = {"relevance": np.asarray(inst.req_chunks, dtype=np.int32),
           "popularity": oracle.global_order_layout(inst, oracle.popularity_rank(inst)),
           "greedy": oracle.greedy_solve(inst)["orders"]}
    rng = np.random.default_rng(inst.m + 1)
    rnd = np.asarray(inst.req_chunks, dtype=np.int32).copy()
    for i in range(inst.m):
        a, b = inst.req_off[i], inst.req_off[i + 1]
        rnd[a:b] = rng.permutation(rnd[a:b])
    out["random"] = rnd
    return out


@pytest.mark.parametrize("name", ["small", "trace_512", "trace_2048"])
def test_trie_cost_and_dfs_order(name):
    inst = wl.random_small(m=30, u=25, kmin=0, kmax=8, wmax=50, seed=5) if name == "small" else wl.trace_config(name)
    L = mpt.Layouts(inst)
    for lname, lay in layouts(inst).items():
        say(f"[gpu layout] cost {inst.name} {lname}")
        got = L.cost(L.seqs(lay))
        assert got == oracle.trie_cost(inst, lay), lname
        assert np.array_equal(L.dfs.cpu().numpy(), oracle.dfs_schedule(inst, lay)), lname


def cache_grid(inst):
    mx = max(1, max_request(inst))
    windows, caps = [], []
    for W in (1, 3, 16, 128, 0):
        for f in (0.0, 0.5, 1.0, 4.0, 64.0):
            windows.append(W)
            caps.append(int(f * mx))
    return windows, caps


@pytest.mark.parametrize("name", ["small", "trace_512"])
def test_cache_simulation_matches_oracle(name):
    inst = wl.random_small(m=25, u=20, kmin=0, kmax=7, wmax=20, seed=9) if name == "small" else wl.trace_config(name)
    windows, caps = cache_grid(inst)
    L = mpt.Layouts(inst, n_configs=len(windows))
    for lname, lay in layouts(inst).items():
        say(f"[gpu cache] {inst.name} {lname} {len(windows)} configurations")
        got, tc = L.simulate(L.seqs(lay), windows, caps)
        assert tc == oracle.trie_cost(inst, lay)
        for W, C, g in zip(windows, caps, got):
            assert g == oracle.lru_cache_cost(inst, lay, oracle.window_schedule(inst, lay, W), C), (lname, W, C)


def test_cache_configurations_in_any_order():
    """Configurations whose windows name the same schedule (0, -1, m and
    past m are all the whole stream) interleaved with others and with
    capacities in no order: every bill against the oracle's simulator."""
    inst = wl.random_small(m=40, u=30, kmin=1, kmax=9, wmax=50, seed=17)
    lay = oracle.greedy_solve(inst)["orders"]
    mx = max_request(inst)
    m = inst.m
    windows = [5, -1, 0, m + 5, m, 5, 1, 7, 1, 0, 13, -7]
    caps = [mx, 3 * mx, 0, mx // 2, 1 << 40, 2 * mx, mx, 5 * mx, 0, mx, 7, 4 * mx]
    L = mpt.Layouts(inst, n_configs=len(windows))
    got, tc = L.simulate(L.seqs(lay), windows, caps)
    assert tc == oracle.trie_cost(inst, lay)
    for W, C, g in zip(windows, caps, got):
        assert g == oracle.lru_cache_cost(inst, lay, oracle.window_schedule(inst, lay, W), C), (W, C)


def test_theorem7_on_gpu():
    """Theorem 7: in DFS order, one request's worth of capacity bills exactly
    the trie cost, for every layout; arrival order at that capacity does not."""
    inst = wl.trace_config("trace_2048")
    mx = max_request(inst)
    L = mpt.Layouts(inst, n_configs=4)
    for lname, lay in layouts(inst).items():
        say(f"[gpu cache] theorem 7 {inst.name} {lname}")
        got, tc = L.simulate(L.seqs(lay), [0, 0, 0, 1], [mx, 2 * mx, 1 << 60, mx])
        assert got[0] == got[1] == got[2] == tc, lname
        assert got[3] >= tc


def test_trace_4096_sampled_configurations():
    """The benchmark family at m = 4096: the greedy layout's bill for a few
    configurations against the oracle, and the whole grid's invariants
    (non-increasing in capacity, at least the trie cost, at most the sum of
    the request weights)."""
    inst = wl.trace_config("trace_4096")
    lay = oracle.greedy_solve(inst)["orders"]
    mx = max_request(inst)
    total = int(sum(int(inst.weights[np.asarray(r, dtype=np.int64)].sum()) for r in inst.requests()))
    windows, caps = [], []
    for W in (1, 128, 512, 2048, 0):
        for f in (1, 4, 16, 64, 256, 1024):
            windows.append(W)
            caps.append(f * mx)
    L = mpt.Layouts(inst, n_configs=len(windows))
    got, tc = L.simulate(L.seqs(lay), windows, caps)
    g = np.array(got).reshape(5, 6)
    assert np.all(g[:, :-1] >= g[:, 1:]) and np.all(g >= tc) and np.all(g <= total)
    assert np.all(g[4] == tc)                                   # whole-stream DFS order: Theorem 7
    for r, c in ((0, 0), (1, 2), (3, 0)):
        W, C = windows[r * 6 + c], caps[r * 6 + c]
        assert g[r, c] == oracle.lru_cache_cost(inst, lay, oracle.window_schedule(inst, lay, W), C)


def test_degenerate_inputs():
    cases = [
        wl.from_sets([[5, 2, 9]], [1] * 10, 10),
        wl.from_sets([[], []], [], 0),
        wl.from_sets([[1, 0], [0, 1], [1, 0]], [4, 7], 2),
        wl.from_sets([[], [3], [], [1, 2]], [1] * 4, 4),
        wl.from_sets([[0]] * 40, [1 << 32], 1),
    ]
    for inst in cases:
        L = mpt.Layouts(inst, n_configs=3)
        lay = np.asarray(inst.req_chunks, dtype=np.int32)
        seqs = L.seqs(lay)
        assert L.cost(seqs) == oracle.trie_cost(inst, lay)
        mx = max_request(inst)
        got, tc = L.simulate(seqs, [1, 0, 2], [0, mx, 1])
        for W, C, gv in zip([1, 0, 2], [0, mx, 1], got):
            assert gv == oracle.lru_cache_cost(inst, lay, oracle.window_schedule(inst, lay, W), C)


def test_error_codes():
    inst = wl.from_sets([[0, 1], [1, 2]], [1, 1, 1], 3)
    L = mpt.Layouts(inst, n_configs=1)
    bad = L.seqs(np.array([0, 7, 1, 2], dtype=np.int32))
    with pytest.raises(mpt.MptError) as e:
        L.cost(bad)
    assert e.value.status == -2
    with pytest.raises(mpt.MptError) as e:
        L.simulate(L.seqs(inst.req_chunks), [1], [-1])
    assert e.value.status == -1
    L.chunk_w[1] = 0
    with pytest.raises(mpt.MptError) as e:
        L.cost(L.seqs(inst.req_chunks))
    assert e.value.status == -4
    L.chunk_w[1] = 1
    assert L.cost(L.seqs(inst.req_chunks)) == 4


def test_cache_simulation_at_m_8192():
    """m = 8192 requests: a trie of more than 36K nodes and access logs of
    65K entries (256 sorted blocks per schedule, reuse distances across
    many of them). Sampled configurations against the oracle, the whole
    grid against the invariants."""
    inst = wl.gen_retrieval(m=8192, u=24576, topics=256, k=8, seed=2)
    lay = np.asarray(inst.req_chunks, dtype=np.int32)
    unit = wl.from_sets(inst.requests(), [1] * inst.n_chunks, inst.n_chunks)
    assert oracle.trie_cost(unit, lay) > 36 * 1024                # trie nodes
    mx = max_request(inst)
    total = int(sum(int(inst.weights[np.asarray(r, dtype=np.int64)].sum()) for r in inst.requests()))
    windows = [1, 1, 512, 512, 0, 0]
    caps = [mx, 16 * mx, mx, 16 * mx, mx, 16 * mx]
    L = mpt.Layouts(inst, n_configs=len(windows))
    say(f"[gpu cache] {inst.name} m={inst.m} {len(windows)} configurations")
    got, tc = L.simulate(L.seqs(lay), windows, caps)
    assert tc == oracle.trie_cost(inst, lay)
    assert got[4] == got[5] == tc                                   # Theorem 7
    for W, C, g in zip(windows, caps, got):
        assert tc <= g <= total
    assert got[0] >= got[1] and got[2] >= got[3]
    for k in (0, 3):
        W, C = windows[k], caps[k]
        assert got[k] == oracle.lru_cache_cost(inst, lay, oracle.window_schedule(inst, lay, W), C), (W, C)


def order_edge_instance(m, seed):
    """Requests whose sequences stress the lexicographic request order: a
    common first 8 chunks with tails that differ late, prefixes at length
    8 and below, duplicates (ordered by index), empty requests, and random
    sequences over a small alphabet (long shared prefixes)."""
    rng = np.random.default_rng(seed)
    base = [int(x) for x in rng.permutation(40)[:8]]
    fixed = [base + [50, 51, 52, 53], base + [50, 51, 52, 54], base + [50, 51], base, base[:7] + [60],
             base + [50, 51, 52, 53], [], [3], [3, 1], [1], base[:3], base[:3] + [61], [], base]
    sets = []
    while len(sets) < m:
        if rng.random() < 0.4:
            sets.append(list(fixed[int(rng.integers(len(fixed)))]))
        else:
            n = int(rng.integers(0, 17))
            head = base[:int(rng.integers(0, 9))] if rng.random() < 0.6 else []
            rest = [int(x) for x in rng.permutation(np.arange(40, 64))[:max(0, n - len(head))]]
            sets.append(head + rest)
    return wl.from_sets(sets, [int(x) for x in rng.integers(1, 9, 64)], 64)


@pytest.mark.parametrize("m", [300, 4096, 17000])
def test_request_order_edge_cases(m):
    """The request order behind the trie cost and the DFS order, on ties,
    prefixes and sequences equal on their first 8 chunks: up to 16384
    requests it comes from all-pairs ranks, above from the bitonic sort."""
    inst = order_edge_instance(m, seed=m)
    lay = np.asarray(inst.req_chunks, dtype=np.int32)
    L = mpt.Layouts(inst)
    say(f"[gpu layout] request order m={m}")
    assert L.cost(L.seqs(lay)) == oracle.trie_cost(inst, lay)
    assert np.array_equal(L.dfs.cpu().numpy(), oracle.dfs_schedule(inst, lay))
