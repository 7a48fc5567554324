"""Seeded synthetic MPT instances.

This module only draws inputs: it holds none of the solver's arithmetic, so
both the HIP path and the CPU oracle may consume what it produces.

An instance of the Minimum Prefix Trie with Free Permutations problem
(Section 2 of the paper) is a universe of ``n_chunks`` chunks with positive
integer weights (token counts) and ``m`` requests, each a set of chunk ids.
Requests are stored in CSR form: request ``i`` is
``req_chunks[req_off[i]:req_off[i+1]]``.

Generators
----------
* :func:`gen_tiny`       uniform random requests of exactly ``k`` chunks.
* :func:`gen_loo`        the leave-one-out family L_n of Section 5.
* :func:`gen_retrieval`  retrieval-shaped requests: Zipf over topics, Zipf
                         popularity inside a topic, 20% cross-topic slots,
                         log-normal passage lengths. This stands in for the
                         BM25 retrieval traces over BEIR corpora that the
                         paper evaluates on (Section 7), which are not
                         available here.
* :func:`from_sets`      any explicit family (the paper's worked examples).
* :func:`config`         the five benchmark workloads by index.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Sequence

import numpy as np

__all__ = [
    "Instance", "from_sets", "gen_tiny", "gen_loo", "gen_retrieval",
    "gen_two_chunk_graph", "config", "CONFIGS", "random_small",
]


@dataclasses.dataclass(frozen=True)
class Instance:
    """One MPT instance in CSR form (all arrays are host numpy arrays)."""

    n_chunks: int
    weights: np.ndarray      # int64[n_chunks], every entry > 0
    req_off: np.ndarray      # int64[m + 1], req_off[0] == 0, non-decreasing
    req_chunks: np.ndarray   # int32[req_off[m]], chunk ids in [0, n_chunks)
    name: str = ""

    @property
    def m(self) -> int:
        return int(self.req_off.shape[0] - 1)

    @property
    def nnz(self) -> int:
        return int(self.req_off[-1])

    def requests(self) -> list[list[int]]:
        off = self.req_off
        return [self.req_chunks[off[i]:off[i + 1]].tolist() for i in range(self.m)]

    def sha256(self) -> str:
        h = hashlib.sha256()
        h.update(np.int64(self.n_chunks).tobytes())
        h.update(np.ascontiguousarray(self.weights, dtype="<i8").tobytes())
        h.update(np.ascontiguousarray(self.req_off, dtype="<i8").tobytes())
        h.update(np.ascontiguousarray(self.req_chunks, dtype="<i4").tobytes())
        return h.hexdigest()

    def stats(self) -> dict:
        """Overlap statistics of the kind Section 7 reports for real traces."""
        ids = self.req_chunks.astype(np.int64)
        used, counts = np.unique(ids, return_counts=True)
        return {
            "m": self.m,
            "n_chunks": self.n_chunks,
            "slots": int(ids.size),
            "distinct_used": int(used.size),
            "dedup": float(ids.size / max(1, used.size)),
            "mean_demand": float(counts.mean()) if counts.size else 0.0,
            "shared_frac": float((counts > 1).mean()) if counts.size else 0.0,
            "max_demand": int(counts.max()) if counts.size else 0,
        }


def from_sets(sets: Sequence[Sequence[int]], weights: Sequence[int] | None = None,
              n_chunks: int | None = None, name: str = "") -> Instance:
    """Build an instance from explicit request sets (order inside a set kept)."""
    if n_chunks is None:
        n_chunks = 1 + max((max(s) for s in sets if len(s)), default=-1)
    if weights is None:
        weights = [1] * n_chunks
    w = np.asarray(weights, dtype=np.int64)
    if w.shape != (n_chunks,):
        raise ValueError("weights must have one entry per chunk")
    off = np.zeros(len(sets) + 1, dtype=np.int64)
    off[1:] = np.cumsum([len(s) for s in sets])
    flat = np.asarray([c for s in sets for c in s], dtype=np.int32)
    return Instance(int(n_chunks), w, off, flat, name)


def gen_tiny(m: int = 12, u: int = 64, k: int = 4, wmax: int = 32, seed: int = 0) -> Instance:
    """Uniform random instance: weights U{1..wmax}, each request k distinct
    chunks drawn uniformly without replacement."""
    rng = np.random.default_rng(np.random.PCG64(seed))
    w = rng.integers(1, wmax + 1, size=u, dtype=np.int64)
    sets = [rng.choice(u, size=k, replace=False).tolist() for _ in range(m)]
    return from_sets(sets, w, u, f"tiny(m={m},u={u},k={k},seed={seed})")


def gen_loo(n: int) -> Instance:
    """Leave-one-out family L_n (Section 5): universe [n], R_i = [n] minus i,
    unit weights."""
    sets = [[x for x in range(n) if x != i] for i in range(n)]
    return from_sets(sets, [1] * n, n, f"loo(n={n})")


def _zipf_probs(n: int, s: float) -> np.ndarray:
    p = 1.0 / np.power(np.arange(1, n + 1, dtype=np.float64), s)
    return p / p.sum()


def gen_retrieval(m: int, u: int, topics: int, k: int, seed: int = 0,
                  s: float = 1.1, cross_frac: float = 0.2,
                  mu: float = float(np.log(180.0)), sigma: float = 0.5,
                  wmin: int = 60, wmax: int = 600) -> Instance:
    """Retrieval-shaped requests.

    * passage p belongs to topic floor(p * topics / u) (contiguous blocks);
    * passage lengths are drawn once, before any request:
      clip(rint(exp(N(mu, sigma))), wmin, wmax) tokens;
    * each request draws a topic t ~ Zipf(s) over topic ids, then
      k - round(cross_frac * k) passages of t by Zipf(s) over the local rank,
      and round(cross_frac * k) cross-topic passages, each from a topic
      t' ~ Zipf(s) redrawn while t' == t, again by in-topic Zipf(s);
    * a request never repeats a passage (duplicates are redrawn).
    """
    rng = np.random.default_rng(np.random.PCG64(seed))
    if k > u:
        raise ValueError("k must not exceed u")
    w = np.clip(np.rint(np.exp(rng.normal(mu, sigma, size=u))), wmin, wmax).astype(np.int64)
    # start[t] = first passage p with floor(p * topics / u) == t, i.e. ceil(t * u / topics)
    start = np.array([-(-t * u // topics) for t in range(topics + 1)], dtype=np.int64)
    sizes = np.diff(start)
    topic_p = _zipf_probs(topics, s)
    local_p = {int(n): _zipf_probs(int(n), s) for n in np.unique(sizes)}
    n_cross = int(round(cross_frac * k))
    sets = []
    for _ in range(m):
        t = int(rng.choice(topics, p=topic_p))
        chosen: list[int] = []
        taken: set[int] = set()

        def draw_from(topic: int) -> None:
            n = int(sizes[topic])
            while True:
                p = int(start[topic] + rng.choice(n, p=local_p[n]))
                if p not in taken:
                    taken.add(p)
                    chosen.append(p)
                    return

        if k - n_cross > sizes[t]:
            raise ValueError("topic too small for the in-topic draws")
        for _ in range(k - n_cross):
            draw_from(t)
        for _ in range(n_cross):
            t2 = t
            while t2 == t:
                t2 = int(rng.choice(topics, p=topic_p))
            draw_from(t2)
        sets.append(chosen)
    return from_sets(sets, w, u, f"retrieval(m={m},u={u},T={topics},k={k},seed={seed})")


def gen_two_chunk_graph(n_vertices: int, m: int, seed: int = 0) -> Instance:
    """m distinct edges of a random simple graph as two-chunk requests with
    unit weights (the setting of Proposition 2)."""
    rng = np.random.default_rng(np.random.PCG64(seed))
    all_edges = [(a, b) for a in range(n_vertices) for b in range(a + 1, n_vertices)]
    if m > len(all_edges):
        raise ValueError("too many edges")
    pick = rng.choice(len(all_edges), size=m, replace=False)
    sets = []
    for e in pick:
        a, b = all_edges[int(e)]
        sets.append([a, b] if rng.integers(2) else [b, a])
    return from_sets(sets, [1] * n_vertices, n_vertices, f"graph(n={n_vertices},m={m},seed={seed})")


def random_small(m: int, u: int, kmin: int, kmax: int, wmax: int, seed: int,
                 allow_empty: bool = False) -> Instance:
    """Random requests of varying size for sweeps (kmin may be 0)."""
    rng = np.random.default_rng(np.random.PCG64(seed))
    w = rng.integers(1, wmax + 1, size=u, dtype=np.int64)
    sets = []
    for _ in range(m):
        k = int(rng.integers(kmin, kmax + 1))
        if k == 0 and not allow_empty:
            k = 1
        sets.append(rng.choice(u, size=min(k, u), replace=False).tolist())
    return from_sets(sets, w, u, f"random(m={m},u={u},k={kmin}..{kmax},seed={seed})")


# The five benchmark workloads (sizes as named in the workload descriptions).
CONFIGS = {
    1: dict(kind="tiny", m=12, u=64, k=4, wmax=32, seed=0),
    2: dict(kind="loo", n=20),
    3: dict(kind="retrieval", m=20, u=2000, topics=50, k=10, seed=0),
    4: dict(kind="retrieval", m=24, u=5000, topics=80, k=20, seed=0),
    5: dict(kind="retrieval", m=25, u=10000, topics=100, k=50, seed=0),
}


def config(idx: int, seed: int | None = None) -> Instance:
    """Benchmark workload ``idx`` (1..5); ``seed`` overrides the canonical 0."""
    c = dict(CONFIGS[idx])
    kind = c.pop("kind")
    if seed is not None and "seed" in c:
        c["seed"] = seed
    if kind == "tiny":
        return gen_tiny(**c)
    if kind == "loo":
        return gen_loo(**c)
    return gen_retrieval(**c)


# Request families for the Section 6.2-6.3 heuristic and bound, far past the
# exact solver's reach: retrieval traces of thousands of queries with a small
# top-k over a passage pool a few times larger (the shape of the paper's
# Section 7 traces, e.g. about 3000 queries, k = 8, a few thousand passages).
TRACE_CONFIGS = {
    "trace_512": dict(m=512, u=1536, topics=16, k=8, seed=0),
    "trace_2048": dict(m=2048, u=6144, topics=64, k=8, seed=0),
    "trace_4096": dict(m=4096, u=12288, topics=128, k=8, seed=0),
}


def gen_long_lists(m: int = 25, u: int = 1 << 20, k: int = 90000, wmax: int = 999, seed: int = 12) -> Instance:
    """Long requests over a large pool: each of the m requests holds k
    distinct chunks drawn uniformly from u, weights U{1..wmax} drawn after
    the sets. At the defaults most chunks are held by one to three requests
    (the same few demand sets over and over) and the list of held chunks is
    about 0.9 u long: the shape for which W is built by the dense route."""
    rng = np.random.default_rng(seed)
    sets = [rng.choice(u, size=k, replace=False).tolist() for _ in range(m)]
    w = rng.integers(1, wmax + 1, size=u, dtype=np.int64)
    return from_sets(sets, w, u, f"long_lists(m={m},u={u},k={k},seed={seed})")


def trace_config(name: str, seed: int | None = None) -> Instance:
    c = dict(TRACE_CONFIGS[name])
    if seed is not None:
        c["seed"] = seed
    return gen_retrieval(**c)
