"""Pins of the oracle's Section 6.2-6.3 functions: the agglomerative
hierarchy H_g, the layout read off it, and the spanning-tree lower bound.

They are checked against values the paper prints (tests/golden), closed
forms, the exact DP of Section 3.1 (itself pinned in test_oracle_pins.py),
a library spanning tree and brute force on tiny inputs.
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle
from oracle import brute
from paper_2609_13692_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def paper():
    with open(os.path.join(GOLDEN, "paper_values.json")) as f:
        return json.load(f)


def digits(sets):
    return [[int(c) for c in s] for s in sets]


def split_to_parent(m, split):
    """Explicit parent array (leaf i = node i, internal nodes m, m+1, ...) of
    the hierarchy encoded by a split table."""
    full = (1 << m) - 1
    parent = np.full(2 * m - 1, -1, dtype=np.int32)
    ids = {}
    nxt = m

    def node_id(mask):
        nonlocal nxt
        if mask & (mask - 1) == 0:
            return mask.bit_length() - 1
        if mask not in ids:
            ids[mask] = nxt
            nxt += 1
        return ids[mask]

    stack = [full]
    while stack:
        B = stack.pop()
        if B & (B - 1) == 0:
            continue
        A = int(split[B])
        for child in (A, B ^ A):
            parent[node_id(child)] = node_id(B)
            stack.append(child)
    return parent


def brute_greedy(inst):
    """The merge rule of Section 6.2 on Python sets: largest shared weight,
    ties to the lexicographically smallest pair of names (a cluster is named
    by its smallest request), the merged cluster keeps the smaller name."""
    w = inst.weights
    sig = {i: frozenset(r) for i, r in enumerate(inst.requests())}
    merges = []
    while len(sig) > 1:
        names = sorted(sig)
        best = None
        for a, b in itertools.combinations(names, 2):
            v = sum(int(w[x]) for x in sig[a] & sig[b])
            if best is None or v > best[0]:
                best = (v, a, b)
        v, a, b = best
        merges.append((a, b, v))
        sig[a] = sig[a] & sig[b]
        del sig[b]
    return merges


def check_layout(inst, res):
    orders = res["orders"]
    off = inst.req_off
    for i in range(inst.m):
        assert sorted(orders[off[i]:off[i + 1]].tolist()) == sorted(inst.req_chunks[off[i]:off[i + 1]].tolist())
    seqs = [orders[off[i]:off[i + 1]].tolist() for i in range(inst.m)]
    return brute.trie_cost(seqs, inst.weights)


def test_agglomerative_exact_on_loo():
    """Section 6.2: on L_n the greedy is exactly optimal (printed values for
    n = 16, 32, 64, 128), which is the Theorem 5 closed form."""
    for n, cost in paper()["agglomerative_on_loo"]["rows"]:
        inst = wl.gen_loo(n)
        r = oracle.greedy_solve(inst)
        assert r["cost"] == cost == brute.loo_opt_free(n)
        assert r["request_total"] == n * (n - 1)


def test_agglomerative_tightness_witness():
    """Section 6.3, tightness: on {0123},{14},{2578},{46} the greedy can take
    saving 1 against the optimal 2. Under the tie reading it does: (0,1)
    first (value 1), after which every pair shares nothing."""
    p = paper()["greedy_tightness_witness"]
    inst = wl.from_sets(digits(p["requests"]), [1] * 9, 9)
    r = oracle.greedy_solve(inst)
    assert r["merge_a"].tolist() == [0, 0, 0]
    assert r["merge_b"].tolist() == [1, 2, 3]
    assert r["gain"].tolist() == [1, 0, 0]
    assert 2 * r["savings"] == p["optimal_savings"]
    assert r["cost"] == p["opt_free_derived"] + 1
    assert check_layout(inst, r) == 11


@pytest.mark.parametrize("seed", range(12))
def test_agglomerative_theorem6_against_exact(seed):
    """Theorem 6 against the exact DP: SAV* / 2 <= SAV(H_g) <= SAV*, the
    merge values never increase (part i), the per-threshold inequality
    A(theta) <= 2 G(theta) (part ii), the savings recounted from the nodes
    (Eq. 3), and the Theorem 1 sandwich for the layout read off H_g."""
    rng = np.random.default_rng(seed)
    m = int(rng.integers(3, 11))
    inst = wl.random_small(m=m, u=int(rng.integers(6, 24)), kmin=1, kmax=8, wmax=int(rng.choice([1, 5, 40])),
                           seed=500 + seed)
    g = oracle.greedy_solve(inst)
    ex = oracle.solve(inst)
    assert g["savings"] <= ex["savings"] <= 2 * g["savings"]
    assert g["cost"] >= ex["opt"]
    gains = g["gain"].tolist()
    assert all(gains[t] >= gains[t + 1] for t in range(len(gains) - 1))
    # part (ii): internal nodes of the optimal hierarchy and their w(I(v))
    full = (1 << m) - 1
    vals, stack = [], [full]
    while stack:
        B = stack.pop()
        if B & (B - 1) == 0:
            continue
        vals.append(int(ex["W"][B]))
        A = int(ex["split"][B])
        stack += [A, B ^ A]
    for theta in sorted(set(vals + gains)):
        if theta <= 0:
            continue
        assert sum(v >= theta for v in vals) <= 2 * sum(x >= theta for x in gains)
    assert oracle.tree_savings(inst, g["parent"]) == g["savings"]
    trie = check_layout(inst, g)
    assert trie == oracle.trie_cost(inst, g["orders"])
    assert ex["opt"] <= trie <= g["cost"]


@pytest.mark.parametrize("seed", range(6))
def test_agglomerative_merge_sequence_brute_force(seed):
    inst = wl.random_small(m=7, u=12, kmin=1, kmax=7, wmax=3, seed=900 + seed)
    g = oracle.greedy(inst)
    got = list(zip(g["merge_a"].tolist(), g["merge_b"].tolist(), g["gain"].tolist()))
    assert got == brute_greedy(inst)


def test_pair_weights_match_w_table():
    """P[i][j] = W({i, j}) and P[i][i] = W({i}), with W from the per-chunk
    subset enumeration (a separate route to the same definition)."""
    for inst in (wl.config(1), wl.random_small(m=10, u=30, kmin=0, kmax=12, wmax=50, seed=3)):
        P = oracle.pair_weights(inst)
        W = oracle.intersection_weights(inst)
        for i in range(inst.m):
            assert P[i, i] == W[1 << i]
            for j in range(inst.m):
                if i != j:
                    assert P[i, j] == W[(1 << i) | (1 << j)]


def test_spanning_tree_bound_loo_closed_form():
    """On L_n every pair shares n - 2 chunks, so the maximum spanning tree
    weighs (n-1)(n-2) and the bound is n(n-1) - (n-1)(n-2) = 2(n-1)."""
    for n in range(2, 41):
        r = oracle.greedy_solve(wl.gen_loo(n))
        assert r["mst"] == (n - 1) * (n - 2)
        assert r["lower_bound"] == 2 * (n - 1)
        assert r["lower_bound"] <= brute.loo_opt_free(n)


def test_spanning_tree_matches_scipy():
    from scipy.sparse.csgraph import minimum_spanning_tree
    for seed in range(5):
        inst = wl.random_small(m=14, u=40, kmin=1, kmax=15, wmax=60, seed=40 + seed)
        P = oracle.pair_weights(inst)
        big = int(P.max()) + 1
        D = (big - P).astype(np.float64)
        np.fill_diagonal(D, 0.0)
        t = minimum_spanning_tree(D)
        mst = (inst.m - 1) * big - int(round(t.sum()))
        assert oracle.max_spanning_tree(P) == mst


@pytest.mark.parametrize("seed", range(8))
def test_spanning_tree_bound_below_opt(seed):
    """Section 6.3: OPT_free >= sum_i w(R_i) - MST, and so is every
    hierarchy's cost."""
    inst = wl.random_small(m=9, u=20, kmin=1, kmax=9, wmax=30, seed=700 + seed)
    g = oracle.greedy_solve(inst)
    ex = oracle.solve(inst, with_orders=False)
    assert g["lower_bound"] <= ex["opt"] <= g["cost"]


@pytest.mark.parametrize("seed", range(6))
def test_tree_orders_match_split_orders(seed):
    """The explicit-tree read-off agrees with the split-table read-off on the
    optimal hierarchy (both are the Theorem 1 construction)."""
    inst = wl.random_small(m=8, u=18, kmin=0, kmax=9, wmax=20, seed=300 + seed)
    ex = oracle.solve(inst)
    parent = split_to_parent(inst.m, ex["split"])
    assert np.array_equal(oracle.tree_orders(inst, parent), ex["orders"])
    assert oracle.tree_savings(inst, parent) == ex["savings"]


def test_degenerate_families():
    # one request: no merge, the layout is the sorted request
    inst = wl.from_sets([[5, 2, 9]], [1] * 10, 10)
    r = oracle.greedy_solve(inst)
    assert r["savings"] == 0 and r["cost"] == 3 and r["orders"].tolist() == [2, 5, 9]
    assert r["mst"] == 0 and r["lower_bound"] == 3
    # identical requests: one merge chain of full value
    inst = wl.from_sets([[1, 0], [0, 1], [1, 0]], [4, 7], 2)
    r = oracle.greedy_solve(inst)
    assert r["gain"].tolist() == [11, 11] and r["cost"] == 11
    # empty requests and disjoint requests: every gain is 0
    inst = wl.from_sets([[], [3], [], [1, 2]], [1] * 4, 4)
    r = oracle.greedy_solve(inst)
    assert r["gain"].tolist() == [0, 0, 0]
    assert r["merge_a"].tolist() == [0, 0, 0] and r["merge_b"].tolist() == [1, 2, 3]
