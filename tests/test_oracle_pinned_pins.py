"""Pins of the oracle's Section 7.1 construction (top-t pinned at the end in
relevance order, most relevant last; the rest laid out by the exact DP or
the greedy over the distinct free sets).

Checked against: t = 0 (the unconstrained optimum), t at least every request
size (every request is its reversed relevance order), brute force over all
free permutations where no pinned chunk occurs in any free set (then no
trie node can be shared across the boundary and the construction is
optimal), and the bounds OPT_free <= pinned optimum <= construction.
"""
import itertools

import numpy as np
import pytest

import oracle
from oracle import brute
from paper_2609_13692_amd import workloads as wl


def seqs_of(inst, flat):
    off = inst.req_off
    return [flat[off[i]:off[i + 1]].tolist() for i in range(inst.m)]


def brute_pinned(inst, t):
    """Least trie cost over every permutation of every free part, with the
    pinned suffixes fixed."""
    reqs = inst.requests()
    parts = []
    for r in reqs:
        tp = min(t, len(r))
        parts.append((r[tp:], list(reversed(r[:tp]))))
    best = None
    for perms in itertools.product(*[itertools.permutations(f) for f, _ in parts]):
        c = brute.trie_cost([list(p) + s for p, (_, s) in zip(perms, parts)], inst.weights)
        best = c if best is None or c < best else best
    return best


def test_t0_is_the_unconstrained_optimum():
    for seed in range(4):
        inst = wl.random_small(m=9, u=18, kmin=1, kmax=7, wmax=25, seed=60 + seed)
        r = oracle.pinned_layout(inst, 0, "exact")
        assert r["cost"] == oracle.solve(inst, with_orders=False)["opt"]


def test_everything_pinned():
    inst = wl.random_small(m=8, u=15, kmin=0, kmax=6, wmax=9, seed=3)
    for method in ("exact", "greedy"):
        r = oracle.pinned_layout(inst, 6, method)
        assert r["n_distinct"] == 1
        want = [list(reversed(q)) for q in inst.requests()]
        assert seqs_of(inst, r["orders"]) == want
        assert r["cost"] == brute.trie_cost(want, inst.weights)


@pytest.mark.parametrize("seed", range(8))
def test_layout_shape(seed):
    inst = wl.random_small(m=12, u=20, kmin=0, kmax=8, wmax=30, seed=90 + seed)
    for t in (1, 2, 3):
        for method in ("exact", "greedy"):
            r = oracle.pinned_layout(inst, t, method)
            for q, s in zip(inst.requests(), seqs_of(inst, r["orders"])):
                tp = min(t, len(q))
                assert sorted(s) == sorted(q)
                assert s[len(s) - tp:] == list(reversed(q[:tp]))
            assert r["cost"] == brute.trie_cost(seqs_of(inst, r["orders"]), inst.weights)
            assert r["cost"] >= oracle.solve(inst, with_orders=False)["opt"]


@pytest.mark.parametrize("seed", range(10))
def test_optimal_when_pinned_chunks_are_never_free(seed):
    """Pinned chunks drawn from their own pool: the free trie and the suffix
    tries cannot share a node, identical free sets are given one sequence,
    so the exact construction reaches the brute-force pinned optimum."""
    rng = np.random.default_rng(seed)
    t = int(rng.integers(1, 3))
    m = int(rng.integers(2, 5))
    pin_pool, free_pool = list(range(4)), list(range(4, 9))
    sets = []
    for _ in range(m):
        pins = rng.choice(pin_pool, size=t, replace=False).tolist()
        free = rng.choice(free_pool, size=int(rng.integers(0, 4)), replace=False).tolist()
        sets.append(pins + free)
    w = rng.integers(1, 6, size=9)
    inst = wl.from_sets(sets, w, 9)
    assert oracle.pinned_layout(inst, t, "exact")["cost"] == brute_pinned(inst, t)


@pytest.mark.parametrize("seed", range(6))
def test_bounds_against_brute_force(seed):
    inst = wl.random_small(m=4, u=6, kmin=1, kmax=4, wmax=4, seed=120 + seed)
    opt = oracle.solve(inst, with_orders=False)["opt"]
    for t in (1, 2):
        best = brute_pinned(inst, t)
        assert opt <= best <= oracle.pinned_layout(inst, t, "exact")["cost"]
