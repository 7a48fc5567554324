"""Pins of the oracle's Section 7-8 functions: global-order layouts, the DFS
and windowed schedules, and the LRU-leaf radix cache.

Checked against Theorem 7, the capacity extremes (nothing kept: every
request pays in full; unbounded: the trie cost of Eq. 1), hand-worked
traces, a second simulator written on Python dictionaries, library sorts,
and the global-order values of Theorems 4-5.
"""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import brute
from paper_2609_13692_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def seq_list(inst, seqs):
    off = inst.req_off
    return [seqs[off[i]:off[i + 1]].tolist() for i in range(inst.m)]


def max_request(inst):
    w = inst.weights
    return max(int(w[np.asarray(r, dtype=np.int64)].sum()) if r else 0 for r in inst.requests())


def dict_lru(seqs, w, order, capacity):
    """The radix cache on Python dictionaries: nodes are prefixes (tuples);
    a node is evictable when no cached node extends it; the evicted one is
    the evictable node touched longest ago."""
    cached = {}            # prefix -> last time touched
    used = 0
    cost = 0
    for t, i in enumerate(order):
        s = seqs[i]
        for d in range(1, len(s) + 1):
            p = tuple(s[:d])
            if p not in cached:
                cost += int(w[s[d - 1]])
                used += int(w[s[d - 1]])
            cached[p] = t
        while used > capacity:
            leaves = [p for p in cached if not any(len(q) == len(p) + 1 and q[:-1] == p for q in cached)]
            p = min(leaves, key=lambda q: cached[q])
            used -= int(w[p[-1]])
            del cached[p]
    return cost


def layouts(inst):
    """Several layouts of one family: relevance (input) order, chunk-id and
    popularity global orders, the exact and the greedy read-offs, and a
    random permutation of every request."""
    out = {"relevance": np.asarray(inst.req_chunks, dtype=np.int32),
           "id": oracle.global_order_layout(inst, oracle.id_rank(inst)),
           "popularity": oracle.global_order_layout(inst, oracle.popularity_rank(inst)),
           "greedy": oracle.greedy_solve(inst)["orders"]}
    if inst.m <= 12:
        out["exact"] = oracle.solve(inst)["orders"]
    rng = np.random.default_rng(inst.m)
    rnd = np.asarray(inst.req_chunks, dtype=np.int32).copy()
    for i in range(inst.m):
        a, b = inst.req_off[i], inst.req_off[i + 1]
        rnd[a:b] = rng.permutation(rnd[a:b])
    out["random"] = rnd
    return out


def test_hand_traces():
    # [a,b], [a,c] with w = 1, 2, 3
    inst = wl.from_sets([[0, 1], [0, 2]], [1, 2, 3], 3)
    lay = np.array([0, 1, 0, 2], dtype=np.int32)
    order = np.array([0, 1], dtype=np.int32)
    assert oracle.lru_cache_cost(inst, lay, order, 3) == 6
    assert oracle.lru_cache_cost(inst, lay, order, 2) == 6
    assert oracle.lru_cache_cost(inst, lay, order, 0) == 7
    # [a,b], [c], [a,d], unit weights. Capacity 2: c's request evicts the
    # leaf b, a stays and is a hit for [a,d] (4 in all). Capacity 1: after
    # [a,b] only a is left, c's request evicts a, so [a,d] pays for a again
    # (5 in all).
    inst = wl.from_sets([[0, 1], [2], [0, 3]], [1, 1, 1, 1], 4)
    lay = np.array([0, 1, 2, 0, 3], dtype=np.int32)
    order = np.array([0, 1, 2], dtype=np.int32)
    assert oracle.lru_cache_cost(inst, lay, order, 2) == 4
    assert oracle.lru_cache_cost(inst, lay, order, 1) == 5
    assert oracle.lru_cache_cost(inst, lay, order, 100) == 4 == oracle.trie_cost(inst, lay)


@pytest.mark.parametrize("seed", range(10))
def test_cache_against_dict_simulator(seed):
    rng = np.random.default_rng(seed)
    inst = wl.random_small(m=int(rng.integers(2, 9)), u=int(rng.integers(3, 8)), kmin=0, kmax=5,
                           wmax=int(rng.choice([1, 4])), seed=40 + seed)
    for name, lay in layouts(inst).items():
        seqs = seq_list(inst, lay)
        for _ in range(3):
            order = rng.permutation(inst.m).astype(np.int32)
            cap = int(rng.integers(0, max_request(inst) * 2 + 2))
            assert oracle.lru_cache_cost(inst, lay, order, cap) == dict_lru(seqs, inst.weights, order, cap), name


@pytest.mark.parametrize("idx", ["small", "trace"])
def test_theorem7_one_request_cache_in_dfs_order(idx):
    """Theorem 7: served in DFS order, a radix cache with LRU-leaf eviction
    and capacity max_i w(R_i) pays exactly the unbounded-cache cost (the trie
    cost), for any layout."""
    insts = [wl.random_small(m=10, u=14, kmin=1, kmax=8, wmax=30, seed=s) for s in range(4)] if idx == "small" \
        else [wl.trace_config("trace_512")]
    for inst in insts:
        cap = max_request(inst)
        for name, lay in layouts(inst).items():
            tc = oracle.trie_cost(inst, lay)
            d = oracle.dfs_schedule(inst, lay)
            assert oracle.lru_cache_cost(inst, lay, d, cap) == tc, name
            assert oracle.lru_cache_cost(inst, lay, d, 10 * cap) == tc
            assert oracle.lru_cache_cost(inst, lay, np.arange(inst.m, dtype=np.int32), 1 << 60) == tc


def test_capacity_extremes_and_monotone():
    inst = wl.trace_config("trace_512", seed=3)
    lay = oracle.greedy_solve(inst)["orders"]
    total = int(sum(int(inst.weights[np.asarray(r, dtype=np.int64)].sum()) for r in inst.requests()))
    arrival = np.arange(inst.m, dtype=np.int32)
    assert oracle.lru_cache_cost(inst, lay, arrival, 0) == total
    cap = max_request(inst)
    costs = [oracle.lru_cache_cost(inst, lay, arrival, c) for c in (0, cap // 2, cap, 4 * cap, 64 * cap, 1 << 60)]
    assert all(costs[i] >= costs[i + 1] for i in range(len(costs) - 1))
    assert costs[-1] == oracle.trie_cost(inst, lay)


def test_schedules_match_library_sorts():
    inst = wl.trace_config("trace_512", seed=4)
    lay = oracle.greedy_solve(inst)["orders"]
    seqs = seq_list(inst, lay)
    d = oracle.dfs_schedule(inst, lay)
    assert d.tolist() == sorted(range(inst.m), key=lambda i: (seqs[i], i))
    for W in (1, 7, 64, 500, 0):
        got = oracle.window_schedule(inst, lay, W).tolist()
        Wd = inst.m if W <= 0 else W
        want = []
        for s in range(0, inst.m, Wd):
            want += sorted(range(s, min(inst.m, s + Wd)), key=lambda i: (seqs[i], i))
        assert got == want, W
    assert oracle.window_schedule(inst, lay, 1).tolist() == list(range(inst.m))


def test_global_orders():
    p = json.load(open(os.path.join(GOLDEN, "paper_values.json")))
    # Theorem 4: every global order of K4(3) costs 9
    k4 = wl.from_sets([[0, 1, 2], [0, 1, 3], [0, 2, 3], [1, 2, 3]], [1] * 4, 4)
    assert oracle.trie_cost(k4, oracle.global_order_layout(k4, oracle.id_rank(k4))) == p["k4_3uniform"]["opt_glob"]
    # Theorem 5: every global order of L_n costs (n-1)(n+2)/2
    for n in (4, 9, 20):
        inst = wl.gen_loo(n)
        for rank in (oracle.id_rank(inst), oracle.popularity_rank(inst), np.arange(n)[::-1].astype(np.int32)):
            assert oracle.trie_cost(inst, oracle.global_order_layout(inst, rank)) == (n - 1) * (n + 2) // 2
    # popularity rank and layouts against Python sorts and the brute-force evaluator
    inst = wl.random_small(m=9, u=25, kmin=1, kmax=9, wmax=20, seed=8)
    cnt = np.zeros(inst.n_chunks, dtype=np.int64)
    for r in inst.requests():
        cnt[r] += 1
    order = sorted(range(inst.n_chunks), key=lambda x: (-cnt[x], x))
    rank = oracle.popularity_rank(inst)
    assert [int(rank[x]) for x in order] == list(range(inst.n_chunks))
    for r in (rank, oracle.id_rank(inst)):
        lay = oracle.global_order_layout(inst, r)
        for i, s in enumerate(seq_list(inst, lay)):
            assert s == sorted(inst.requests()[i], key=lambda x: r[x])
        assert oracle.trie_cost(inst, lay) == brute.global_order_cost(inst, [int(x) for x in np.argsort(r)])
