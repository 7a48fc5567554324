"""CPU oracle for the exact MPT solver -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. The product path (``libmpt.so`` and its
binding) never imports, links or runs anything here, and nothing here uses
the product path.

* :mod:`oracle.mpt_oracle` (C, built into ``libmpt_oracle.so``): W table,
  exact DP, layout read-off, trie cost and hierarchy cost, written from the
  paper's definitions (Section 2 Eq. 1, Section 3 Thm 1 Eqs. 2-3, Section 3.1);
  pair weights, the agglomerative hierarchy, its layout and savings, and the
  spanning-tree bound for any m (Sections 6.2-6.3, Theorem 6); global-order
  layouts, DFS and windowed schedules, and the LRU-leaf radix cache
  (Sections 7-8, Theorem 7); the pinned variant (Section 7.1) as a
  composition of those, in Python.
* :mod:`oracle.brute` (pure Python, tiny inputs only): brute force over
  permutations, over hierarchies and over global orders, vertex cover, and the
  closed forms of Section 5 -- the pins that check the C oracle.

Input instances come from :mod:`paper_2609_13692_amd.workloads`, which only
draws numbers; any object with ``n_chunks``, ``weights``, ``req_off``,
``req_chunks`` works.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mpt_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libmpt_oracle.so")
_lib = None


def build() -> str:
    """Compile the C oracle in place (gcc, OpenMP). Returns the library path."""
    tmp = _LIB_PATH + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-shared", "-fPIC",
                           _SRC, "-o", tmp])
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i32, i64 = ctypes.c_int, ctypes.c_int64
    lib.oracle_demand_sets.argtypes = [i32, i64, P, P, P]
    lib.oracle_intersection_weights.argtypes = [i32, i64, P, P, P, P]
    lib.oracle_exact_dp.argtypes = [i32, P, P, P, i32]
    lib.oracle_cost_table.argtypes = [i32, P, P, P]
    lib.oracle_orders.argtypes = [i32, i64, P, P, P, P]
    lib.oracle_trie_cost.argtypes = [i32, i64, P, P, P]
    lib.oracle_trie_cost.restype = i64
    lib.oracle_hierarchy_cost.argtypes = [i32, i64, P, P, P, P]
    lib.oracle_hierarchy_cost.restype = i64
    lib.oracle_max_threads.restype = i32
    lib.oracle_pair_weights.argtypes = [i32, i64, P, P, P, P, i32]
    lib.oracle_greedy.argtypes = [i32, i64, P, P, P, P, P, P, P, i32]
    lib.oracle_greedy.restype = i64
    lib.oracle_tree_orders.argtypes = [i32, i64, P, P, i32, P, P]
    lib.oracle_tree_savings.argtypes = [i32, i64, P, P, P, i32, P]
    lib.oracle_tree_savings.restype = i64
    lib.oracle_max_spanning_tree.argtypes = [i32, P]
    lib.oracle_max_spanning_tree.restype = i64
    lib.oracle_global_order_layout.argtypes = [i32, i64, P, P, P, P]
    lib.oracle_popularity_rank.argtypes = [i32, i64, P, P, P]
    lib.oracle_dfs_schedule.argtypes = [i32, P, P, P]
    lib.oracle_window_schedule.argtypes = [i32, P, P, i64, P]
    lib.oracle_lru_cache_cost.argtypes = [i32, i64, P, P, P, P, i64]
    lib.oracle_lru_cache_cost.restype = i64
    _lib = lib
    return lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


class OracleError(RuntimeError):
    pass


def _check(rc: int, what: str) -> None:
    if rc < 0:
        raise OracleError(f"{what} failed with status {rc}")


def _arrays(inst):
    w = np.ascontiguousarray(inst.weights, dtype=np.int64)
    off = np.ascontiguousarray(inst.req_off, dtype=np.int64)
    ch = np.ascontiguousarray(inst.req_chunks, dtype=np.int32)
    if ch.size == 0:
        ch = np.zeros(1, dtype=np.int32)   # valid pointer for an all-empty family
    return w, off, ch


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def demand_sets(inst) -> np.ndarray:
    """S_x as uint32 masks, one per chunk (Section 3)."""
    lib = _load()
    w, off, ch = _arrays(inst)
    sx = np.zeros(max(1, inst.n_chunks), dtype=np.uint32)
    _check(lib.oracle_demand_sets(inst.m, inst.n_chunks, _p(off), _p(ch), _p(sx)), "demand_sets")
    return sx[:inst.n_chunks]


def intersection_weights(inst) -> np.ndarray:
    """W(B) = w(I(B)) for all 2^m subsets B; I(empty) = U."""
    lib = _load()
    w, off, ch = _arrays(inst)
    W = np.empty(1 << inst.m, dtype=np.int64)
    _check(lib.oracle_intersection_weights(inst.m, inst.n_chunks, _p(w), _p(off), _p(ch), _p(W)),
           "intersection_weights")
    return W


def exact_dp(m: int, W: np.ndarray, threads: int = 0) -> tuple[np.ndarray, np.ndarray]:
    """Savings table M and split table of the Section 3.1 recurrence."""
    lib = _load()
    W = np.ascontiguousarray(W, dtype=np.int64)
    M = np.empty(1 << m, dtype=np.int64)
    split = np.empty(1 << m, dtype=np.uint32)
    if threads <= 0:
        threads = max_threads()
    _check(lib.oracle_exact_dp(m, _p(W), _p(M), _p(split), threads), "exact_dp")
    return M, split


def cost_table(m: int, W: np.ndarray, M: np.ndarray) -> np.ndarray:
    """C(B) = sum_{i in B} w(R_i) - M(B) (Eq. 3 applied to each sub-instance)."""
    lib = _load()
    C = np.empty(1 << m, dtype=np.int64)
    _check(lib.oracle_cost_table(m, _p(np.ascontiguousarray(W)), _p(np.ascontiguousarray(M)), _p(C)),
           "cost_table")
    return C


def orders(inst, split: np.ndarray) -> np.ndarray:
    """pi_i for every request, CSR with the instance's req_off."""
    lib = _load()
    w, off, ch = _arrays(inst)
    out = np.full(max(1, inst.nnz), -1, dtype=np.int32)
    sp = np.ascontiguousarray(split, dtype=np.uint32)
    _check(lib.oracle_orders(inst.m, inst.n_chunks, _p(off), _p(ch), _p(sp), _p(out)), "orders")
    return out[:inst.nnz]


def trie_cost(inst, seqs: np.ndarray) -> int:
    """Eq. (1) for the layout seqs (CSR with the instance's req_off)."""
    lib = _load()
    w, off, _ = _arrays(inst)
    s = np.ascontiguousarray(seqs, dtype=np.int32)
    if s.size == 0:
        s = np.zeros(1, dtype=np.int32)
    c = int(lib.oracle_trie_cost(inst.m, inst.n_chunks, _p(w), _p(off), _p(s)))
    _check(c, "trie_cost")
    return c


def hierarchy_cost(inst, split: np.ndarray) -> int:
    """Eq. (2) for the hierarchy encoded by split: sum_x w(x) t_x(H)."""
    lib = _load()
    w, off, ch = _arrays(inst)
    sp = np.ascontiguousarray(split, dtype=np.uint32)
    c = int(lib.oracle_hierarchy_cost(inst.m, inst.n_chunks, _p(w), _p(off), _p(ch), _p(sp)))
    _check(c, "hierarchy_cost")
    return c


def solve(inst, threads: int = 0, with_orders: bool = True) -> dict:
    """Full oracle run: W, M, C, split, OPT, savings and (optionally) orders."""
    W = intersection_weights(inst)
    M, split = exact_dp(inst.m, W, threads)
    C = cost_table(inst.m, W, M)
    full = (1 << inst.m) - 1
    res = {"W": W, "M": M, "C": C, "split": split,
           "opt": int(C[full]), "savings": int(M[full])}
    if with_orders:
        res["orders"] = orders(inst, split)
    return res


# --- Sections 6.2-6.3: agglomerative hierarchy and spanning-tree bound -----

def pair_weights(inst, threads: int = 0) -> np.ndarray:
    """P[i, j] = w(R_i ∩ R_j) for all requests (diagonal: w(R_i))."""
    lib = _load()
    w, off, ch = _arrays(inst)
    P = np.empty((inst.m, inst.m), dtype=np.int64)
    _check(lib.oracle_pair_weights(inst.m, inst.n_chunks, _p(w), _p(off), _p(ch), _p(P), threads),
           "pair_weights")
    return P


def greedy(inst, threads: int = 0) -> dict:
    """Agglomerative hierarchy H_g (Section 6.2, Theorem 6): merges (a_t, b_t)
    with gains g_t, node parents (leaf i = node i, step t = node m + t) and
    SAV(H_g)."""
    lib = _load()
    m = inst.m
    w, off, ch = _arrays(inst)
    a = np.full(max(1, m - 1), -1, dtype=np.int32)
    b = np.full(max(1, m - 1), -1, dtype=np.int32)
    g = np.full(max(1, m - 1), -1, dtype=np.int64)
    parent = np.full(2 * m - 1, -2, dtype=np.int32)
    sav = int(lib.oracle_greedy(m, inst.n_chunks, _p(w), _p(off), _p(ch), _p(a), _p(b), _p(g), _p(parent),
                                threads))
    _check(sav, "greedy")
    return {"merge_a": a[:m - 1], "merge_b": b[:m - 1], "gain": g[:m - 1], "parent": parent, "savings": sav}


def tree_orders(inst, parent: np.ndarray) -> np.ndarray:
    """Layout read off an explicit hierarchy (proof of Theorem 1), CSR with
    the instance's req_off."""
    lib = _load()
    w, off, ch = _arrays(inst)
    par = np.ascontiguousarray(parent, dtype=np.int32)
    out = np.full(max(1, inst.nnz), -1, dtype=np.int32)
    _check(lib.oracle_tree_orders(inst.m, inst.n_chunks, _p(off), _p(ch), int(par.size), _p(par), _p(out)),
           "tree_orders")
    return out[:inst.nnz]


def tree_savings(inst, parent: np.ndarray) -> int:
    """SAV(H) = sum over internal nodes of w(I(v)) (Eq. 3) for an explicit
    hierarchy."""
    lib = _load()
    w, off, ch = _arrays(inst)
    par = np.ascontiguousarray(parent, dtype=np.int32)
    s = int(lib.oracle_tree_savings(inst.m, inst.n_chunks, _p(w), _p(off), _p(ch), int(par.size), _p(par)))
    _check(s, "tree_savings")
    return s


def max_spanning_tree(P: np.ndarray) -> int:
    """Weight of a maximum spanning tree of the complete graph with edge
    weights P (Prim)."""
    lib = _load()
    P = np.ascontiguousarray(P, dtype=np.int64)
    v = int(lib.oracle_max_spanning_tree(int(P.shape[0]), _p(P)))
    _check(v, "max_spanning_tree")
    return v


def greedy_solve(inst, threads: int = 0) -> dict:
    """H_g, its layout, and the spanning-tree bound of Sections 6.2-6.3."""
    P = pair_weights(inst, threads)
    total = int(np.trace(P))
    res = greedy(inst, threads)
    res["orders"] = tree_orders(inst, res["parent"])
    res["cost"] = total - res["savings"]
    res["request_total"] = total
    res["mst"] = max_spanning_tree(P)
    res["lower_bound"] = total - res["mst"]
    res["P"] = P
    return res


# --- Sections 7-8: layouts, schedules and the radix cache -----------------

def global_order_layout(inst, rank: np.ndarray) -> np.ndarray:
    """Every request sorted by rank[chunk] ascending (a global order)."""
    lib = _load()
    w, off, ch = _arrays(inst)
    r = np.ascontiguousarray(rank, dtype=np.int32)
    out = np.full(max(1, inst.nnz), -1, dtype=np.int32)
    _check(lib.oracle_global_order_layout(inst.m, inst.n_chunks, _p(off), _p(ch), _p(r), _p(out)),
           "global_order_layout")
    return out[:inst.nnz]


def popularity_rank(inst) -> np.ndarray:
    """rank[x] of the popularity order: demand descending, id ascending."""
    lib = _load()
    w, off, ch = _arrays(inst)
    r = np.empty(max(1, inst.n_chunks), dtype=np.int32)
    _check(lib.oracle_popularity_rank(inst.m, inst.n_chunks, _p(off), _p(ch), _p(r)), "popularity_rank")
    return r[:inst.n_chunks]


def id_rank(inst) -> np.ndarray:
    """rank[x] = x: the chunk-id order."""
    return np.arange(inst.n_chunks, dtype=np.int32)


def _seq_arrays(inst, seqs):
    off = np.ascontiguousarray(inst.req_off, dtype=np.int64)
    s = np.ascontiguousarray(seqs, dtype=np.int32)
    if s.size == 0:
        s = np.zeros(1, dtype=np.int32)
    return off, s


def dfs_schedule(inst, seqs: np.ndarray) -> np.ndarray:
    """Requests in the DFS order of the layout's trie (Theorem 7)."""
    lib = _load()
    off, s = _seq_arrays(inst, seqs)
    order = np.empty(inst.m, dtype=np.int32)
    _check(lib.oracle_dfs_schedule(inst.m, _p(off), _p(s), _p(order)), "dfs_schedule")
    return order


def window_schedule(inst, seqs: np.ndarray, window: int) -> np.ndarray:
    """Arrival order with every window of `window` requests served in DFS
    order (window <= 0: the whole stream)."""
    lib = _load()
    off, s = _seq_arrays(inst, seqs)
    order = np.empty(inst.m, dtype=np.int32)
    _check(lib.oracle_window_schedule(inst.m, _p(off), _p(s), int(window), _p(order)), "window_schedule")
    return order


def lru_cache_cost(inst, seqs: np.ndarray, order: np.ndarray, capacity: int) -> int:
    """Prefill bill of serving the layout in `order` through a radix cache of
    weight `capacity` with LRU-leaf eviction (Section 8)."""
    lib = _load()
    w, _, _ = _arrays(inst)
    off, s = _seq_arrays(inst, seqs)
    o = np.ascontiguousarray(order, dtype=np.int32)
    c = int(lib.oracle_lru_cache_cost(inst.m, inst.n_chunks, _p(w), _p(off), _p(s), _p(o), int(capacity)))
    _check(c, "lru_cache_cost")
    return c


# --- Section 7.1: the pinned variant ----------------------------------------

def pinned_split(inst, t: int):
    """Every request's top-t chunks in relevance (input) order are pinned at
    the end, most relevant last; the rest is free. Returns the distinct free
    sets (ascending lists, in order of their first request), each request's
    distinct-set index, and the pinned suffixes."""
    t = max(0, int(t))
    reqs = inst.requests()
    index = {}
    sets = []
    dmap = []
    suffix = []
    for r in reqs:
        tp = min(t, len(r))
        free = tuple(sorted(r[tp:]))
        if free not in index:
            index[free] = len(sets)
            sets.append(list(free))
        dmap.append(index[free])
        suffix.append(list(reversed(r[:tp])))
    return sets, dmap, suffix


def pinned_layout(inst, t: int, method: str = "exact") -> dict:
    """Section 7.1's constraint: the free parts are laid out by the exact DP
    (Section 3.1) or the agglomerative greedy (Section 6.2) over the distinct
    free sets, every request takes its set's free sequence and appends its
    pinned suffix. Returns the layout (CSR with the request offsets) and its
    trie cost (Eq. 1)."""
    from paper_2609_13692_amd import workloads as wl
    sets, dmap, suffix = pinned_split(inst, t)
    sub = wl.from_sets(sets, inst.weights, inst.n_chunks)
    if method == "exact":
        lay = solve(sub)["orders"]
    elif method == "greedy":
        lay = tree_orders(sub, greedy(sub)["parent"])
    else:
        raise ValueError(method)
    free_seq = [lay[sub.req_off[d]:sub.req_off[d + 1]].tolist() for d in range(sub.m)]
    out = []
    for i in range(inst.m):
        out += free_seq[dmap[i]] + suffix[i]
    seqs = np.asarray(out, dtype=np.int32)
    return {"orders": seqs, "cost": trie_cost(inst, seqs), "n_distinct": sub.m, "dmap": np.asarray(dmap)}
