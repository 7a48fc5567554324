"""Brute-force checkers for tiny MPT instances -- TEST INFRASTRUCTURE ONLY.

Pure Python, exponential, meant for a handful of requests. Each function
restates a definition of the paper directly, with no shared code with the C
oracle, so that agreement between the two pins the oracle:

* :func:`trie_cost`            Eq. (1), with a dict-of-dicts trie;
* :func:`opt_free_permutations` OPT_free as the minimum of Eq. (1) over every
                               choice of one permutation per request (Section 2);
* :func:`opt_free_hierarchies` min over all binary hierarchies H of
                               sum_x w(x) t_x(H) (Thm 1, Eq. 2);
* :func:`opt_glob_orders`      OPT_glob: every request sorted by one linear
                               order on the chunks (Section 2);
* :func:`intersection_weights` w(I(B)) by explicit set intersection;
* :func:`vertex_cover_number`  tau(G) by enumeration (Prop. 2);
* :func:`min_external_path_length` the classical recursion behind Eq. (6);
* :func:`loo_opt_free`, :func:`loo_opt_glob` the closed forms of Eq. (5).
"""
from __future__ import annotations

import itertools
import math
from typing import Iterator, Sequence


def _sets(inst) -> list[list[int]]:
    return inst.requests()


def trie_cost(seqs: Sequence[Sequence[int]], w: Sequence[int]) -> int:
    """Eq. (1): total weight of the non-root nodes of the trie of seqs."""
    root: dict = {}
    cost = 0
    for s in seqs:
        node = root
        for x in s:
            if x not in node:
                node[x] = {}
                cost += int(w[x])
            node = node[x]
    return cost


def opt_free_permutations(inst) -> int:
    """Minimum of Eq. (1) over all prod_i |R_i|! layouts."""
    sets = _sets(inst)
    w = inst.weights
    best = None
    for layout in itertools.product(*[itertools.permutations(s) for s in sets]):
        c = trie_cost(layout, w)
        if best is None or c < best:
            best = c
    return 0 if best is None else best


def hierarchies(leaves: tuple[int, ...]) -> Iterator[list[tuple[int, int]]]:
    """Every binary hierarchy on the given leaves, as a list of
    (cluster mask, parent mask) pairs, root first with parent 0."""
    def rec(items: tuple[int, ...]) -> Iterator[list[int]]:
        # yields the list of cluster masks of one hierarchy on items, in
        # pre-order; the first entry is the cluster of all items
        mask = 0
        for i in items:
            mask |= 1 << i
        if len(items) == 1:
            yield [mask]
            return
        first, rest = items[0], items[1:]
        n = len(rest)
        for pick in range(0, (1 << n) - 1):      # rest subsets that stay with `first`, not all
            left = (first,) + tuple(rest[j] for j in range(n) if (pick >> j) & 1)
            right = tuple(rest[j] for j in range(n) if not (pick >> j) & 1)
            for hl in rec(left):
                for hr in rec(right):
                    yield [mask] + hl + hr

    def with_parents(clusters: list[int]) -> list[tuple[int, int]]:
        out = []
        for c in clusters:
            # parent = smallest strict superset among the clusters (laminar)
            par = 0
            for d in clusters:
                if d != c and (c & d) == c and (par == 0 or bin(d).count("1") < bin(par).count("1")):
                    par = d
            out.append((c, par))
        return out

    for h in rec(tuple(leaves)):
        yield with_parents(h)


def t_x(h: list[tuple[int, int]], sx: int) -> int:
    """Number of maximal clusters of h contained in sx."""
    return sum(1 for c, par in h if (c & ~sx) == 0 and (par == 0 or (par & ~sx) != 0))


def demand_masks(inst) -> list[int]:
    sx = [0] * inst.n_chunks
    for i, s in enumerate(_sets(inst)):
        for x in s:
            sx[x] |= 1 << i
    return sx


def opt_free_hierarchies(inst) -> int:
    """Eq. (2): min over binary hierarchies on the requests of sum_x w(x) t_x(H)."""
    sx = demand_masks(inst)
    w = inst.weights
    best = None
    for h in hierarchies(tuple(range(inst.m))):
        c = sum(int(w[x]) * t_x(h, sx[x]) for x in range(inst.n_chunks) if sx[x])
        if best is None or c < best:
            best = c
    return best


def opt_glob_orders(inst) -> tuple[int, list[int]]:
    """OPT_glob: minimum trie cost when every request is sorted by one linear
    order on the requested chunks. Returns (cost, a best order)."""
    sets = _sets(inst)
    used = sorted({x for s in sets for x in s})
    best, best_order = None, used
    for order in itertools.permutations(used):
        rank = {x: r for r, x in enumerate(order)}
        c = trie_cost([sorted(s, key=rank.__getitem__) for s in sets], inst.weights)
        if best is None or c < best:
            best, best_order = c, list(order)
    return (0 if best is None else best), best_order


def global_order_cost(inst, order: Sequence[int]) -> int:
    """Trie cost of the layout induced by one linear order on the chunks."""
    rank = {x: r for r, x in enumerate(order)}
    return trie_cost([sorted(s, key=rank.__getitem__) for s in _sets(inst)], inst.weights)


def intersection_weights(inst) -> list[int]:
    """w(I(B)) for every subset B, with I(empty) = U, by set intersection."""
    sets = [set(s) for s in _sets(inst)]
    universe = set(range(inst.n_chunks))
    out = []
    for b in range(1 << inst.m):
        inter = set(universe)
        for i in range(inst.m):
            if (b >> i) & 1:
                inter &= sets[i]
        out.append(sum(int(inst.weights[x]) for x in inter))
    return out


def vertex_cover_number(n_vertices: int, edges: Sequence[Sequence[int]]) -> int:
    """tau(G): size of a smallest vertex set meeting every edge."""
    for size in range(n_vertices + 1):
        for cover in itertools.combinations(range(n_vertices), size):
            cs = set(cover)
            if all(a in cs or b in cs for a, b in edges):
                return size
    return n_vertices


def min_external_path_length(n: int) -> int:
    """Minimum over binary trees with n leaves of the sum of leaf depths,
    by the recursion E(1) = 0, E(n) = n + min_k E(k) + E(n - k)."""
    E = [0, 0]
    for k in range(2, n + 1):
        E.append(k + min(E[j] + E[k - j] for j in range(1, k)))
    return E[n]


def loo_opt_free(n: int) -> int:
    """Eq. (5), free value: n*ceil(log2 n) - 2^ceil(log2 n) + n."""
    c = math.ceil(math.log2(n)) if n > 1 else 0
    return n * c - (1 << c) + n


def loo_opt_glob(n: int) -> int:
    """Eq. (5), global value: (n - 1)(n + 2) / 2."""
    return (n - 1) * (n + 2) // 2
