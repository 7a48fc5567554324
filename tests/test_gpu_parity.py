"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Integer work throughout, so every comparison is bit-exact: the W table, the
cost table C (entries 1 .. 2^m-1; C[0] is the documented sentinel), the
tie-broken split table, the demand sets and the read-off orders.
"""
import hashlib
import json
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import brute
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


def gpu_run(inst):
    say(f"[gpu] {inst.name} m={inst.m} nnz={inst.nnz}")
    got = mpt.solve(inst)
    torch.cuda.synchronize()
    return got


def gpu_run_labelled(inst):
    """gpu_run, plus the set of launch labels the library recorded (they
    name the key width of the DP's cross-pair launches: rb_cross_u32 for
    32-bit keys, rb_cross_f64 for exact-integer doubles, rb_cross_u64 for
    uint64; dp_* for the plain kernels)."""
    mpt.profile_begin()
    try:
        got = gpu_run(inst)
    finally:
        prof = mpt.profile_end()
    return got, set(prof)


def cross_labels(labels):
    return {k for k in labels if k.startswith("rb_cross")}


def assert_same(inst, got, ref):
    assert got["opt"] == ref["opt"]
    assert np.array_equal(got["W"], ref["W"]), "W table differs"
    assert got["C"][0] == mpt.MPT_COST_SENTINEL
    bad = np.nonzero(got["C"][1:] != ref["C"][1:])[0]
    assert bad.size == 0, f"C differs at {bad[:8] + 1}"
    bad = np.nonzero(got["split"] != ref["split"])[0]
    assert bad.size == 0, f"split differs at {bad[:8]}"
    assert np.array_equal(got["sig"], oracle.demand_sets(inst))
    assert np.array_equal(got["orders"], ref["orders"]), "orders differ"


def digest(a, dtype):
    return hashlib.sha256(np.ascontiguousarray(a, dtype=dtype).tobytes()).hexdigest()


# --- the five benchmark workloads ------------------------------------------------

@pytest.mark.parametrize("idx", [1, 2, 3])
def test_config_against_live_oracle(idx):
    inst = wl.config(idx)
    got = gpu_run(inst)
    assert_same(inst, got, oracle.solve(inst))


@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
def test_config_full_tables_against_golden(idx):
    """Full tables at the benchmark sizes against digests the oracle wrote."""
    with open(os.path.join(GOLDEN, f"config_{idx}.json")) as f:
        g = json.load(f)
    inst = wl.config(idx)
    assert inst.sha256() == g["instance_sha256"], "workload generator drifted"
    got = gpu_run(inst)
    assert got["opt"] == g["opt"]
    for s, w, c, sp in g["sample"]:
        assert (got["W"][s], got["C"][s], got["split"][s]) == (w, c, sp), s
    assert digest(got["W"], "<i8") == g["W_sha256"]
    assert digest(got["C"][1:], "<i8") == g["C_sha256_from_1"]
    assert digest(got["split"], "<u4") == g["split_sha256"]
    assert got["orders"].tolist() == g["orders"]
    # Thm 1 sandwich on the GPU's own output: its layout's trie costs OPT
    assert oracle.trie_cost(inst, got["orders"]) == got["opt"]
    assert oracle.hierarchy_cost(inst, got["split"]) == got["opt"]


# Scaling every chunk weight by s scales every W and every cost by s and keeps
# every tie, so the split table and the orders do not change. Scaled copies
# of the largest workloads push sum_i w(R_i) past the 32-bit key limit and
# run the 64-bit key paths at full size, checked against the same oracle
# digests: config 5 x 64 (total 1.6e7 < 2^26: exact-integer doubles),
# config 5 x 4096 (1.0e9: uint64 keys) and config 4 x 4096 (4.0e8 >= 2^27:
# uint64 keys), each with split levels of up to 256 chunks.
SCALED = [(5, 64, "rb_cross_f64"), (5, 4096, "rb_cross_u64"), (4, 4096, "rb_cross_u64")]


@pytest.mark.parametrize("idx,scale,label", SCALED, ids=lambda v: str(v))
def test_scaled_config_takes_the_wide_keys(idx, scale, label):
    import dataclasses
    with open(os.path.join(GOLDEN, f"config_{idx}.json")) as f:
        g = json.load(f)
    base = wl.config(idx)
    assert base.sha256() == g["instance_sha256"], "workload generator drifted"
    inst = dataclasses.replace(base, weights=base.weights * scale, name=f"{base.name} x{scale}")
    total = int(inst.weights[inst.req_chunks].sum())
    assert total >= (1 << 20) - 1
    got, labels = gpu_run_labelled(inst)
    assert cross_labels(labels) == {label}
    assert "rb_reduce" in labels                         # split levels ran
    assert got["opt"] == scale * g["opt"]
    W, C = got["W"], got["C"][1:]
    assert not (W % scale).any() and not (C % scale).any()
    assert digest(W // scale, "<i8") == g["W_sha256"]
    assert digest(C // scale, "<i8") == g["C_sha256_from_1"]
    assert digest(got["split"], "<u4") == g["split_sha256"]
    assert got["orders"].tolist() == g["orders"]
    for s_, w, c, sp in g["sample"]:
        assert (W[s_], got["C"][s_], got["split"][s_]) == (scale * w, scale * c if s_ else got["C"][0], sp), s_


def test_config5_sampled_sub_instances():
    """C(S) at the largest workload equals the oracle's optimum of the
    sub-instance {R_i : i in S}, for sampled S of up to 14 requests."""
    inst = wl.config(5)
    got = gpu_run(inst)
    sets = inst.requests()
    rng = np.random.default_rng(3)
    for trial in range(24):
        k = int(rng.integers(1, 15))
        members = sorted(rng.choice(inst.m, size=k, replace=False).tolist())
        s = sum(1 << i for i in members)
        sub = wl.from_sets([sets[i] for i in members], inst.weights, inst.n_chunks)
        assert got["C"][s] == oracle.solve(sub, with_orders=False)["opt"], members


@pytest.mark.timeout(600)
def test_m27_retrieval_sampled():
    """A retrieval-shaped instance at m = 27 (the level plan runs tails of
    shorter chunks in seven levels, three of them behind a split head;
    2^27-entry tables): the split hierarchy's
    Eq. (2) cost and the orders' trie cost equal OPT; C(S) equals the
    oracle's optimum of the sub-instance for sampled S of up to 14 requests;
    and at sampled S of up to 16 requests the tables satisfy the recurrence
    under the tie rule, C(S) = C(A) + C(S \\ A) - W(S) for the stored A, which
    is the least A (lowbit(S) in A, A a proper subset) reaching the minimum."""
    inst = wl.gen_retrieval(m=27, u=10000, topics=100, k=50, seed=7)
    got = gpu_run(inst)
    W, C, split = got["W"], got["C"], got["split"]
    opt = int(got["opt"])
    assert oracle.hierarchy_cost(inst, split) == opt
    assert oracle.trie_cost(inst, got["orders"][:inst.nnz]) == opt
    sets = inst.requests()
    rng = np.random.default_rng(27)
    for trial in range(16):
        k = int(rng.integers(1, 15))
        members = sorted(rng.choice(inst.m, size=k, replace=False).tolist())
        s_ = sum(1 << i for i in members)
        sub = wl.from_sets([sets[i] for i in members], inst.weights, inst.n_chunks)
        assert C[s_] == oracle.solve(sub, with_orders=False)["opt"], members
    for trial in range(40):
        k = int(rng.integers(2, 17))
        members = rng.choice(inst.m, size=k, replace=False)
        s_ = int(sum(1 << int(i) for i in members))
        low = s_ & -s_
        bits = [1 << int(i) for i in sorted(members)]
        # every submask of S, as numpy integers: A = sum of the chosen bits
        idx = np.arange(1 << k, dtype=np.int64)
        subs = np.zeros(1 << k, dtype=np.int64)
        for j, b in enumerate(bits):
            subs |= ((idx >> j) & 1) * b
        cand = subs[((subs & low) != 0) & (subs != s_)]
        costs = C[cand] + C[s_ ^ cand] - W[s_]
        best = costs.min()
        assert C[s_] == best, members
        assert int(split[s_]) == int(cand[costs == best].min()), members
# --- sweeps over shapes and seeds ---------------------------------------------------

SWEEP = [
    # (m, u, kmin, kmax, wmax)
    (1, 5, 0, 5, 9), (2, 4, 1, 4, 9), (3, 6, 0, 6, 50), (5, 8, 1, 5, 20),
    (6, 12, 2, 6, 7), (7, 30, 1, 9, 100), (8, 20, 0, 12, 1000), (9, 40, 3, 10, 3),
    (10, 64, 4, 4, 32), (11, 16, 5, 12, 1), (12, 200, 1, 20, 600), (13, 50, 2, 30, 64),
    (14, 100, 5, 25, 1 << 20), (15, 300, 10, 40, 600), (16, 64, 8, 32, 5),
    (17, 500, 5, 15, 600), (18, 2000, 10, 10, 600),
]


@pytest.mark.parametrize("shape", SWEEP, ids=lambda s: f"m{s[0]}")
def test_random_sweep(shape):
    m, u, kmin, kmax, wmax = shape
    for seed in range(3 if m <= 14 else 1):
        inst = wl.random_small(m, u, kmin, kmax, wmax, seed=1000 * m + seed, allow_empty=True)
        got = gpu_run(inst)
        assert_same(inst, got, oracle.solve(inst))


@pytest.mark.parametrize("seed", range(1, 11))
def test_retrieval_shape_seeds(seed):
    inst = wl.gen_retrieval(m=16, u=2000, topics=50, k=10, seed=seed)
    got = gpu_run(inst)
    assert_same(inst, got, oracle.solve(inst))


@pytest.mark.parametrize("seed", range(1, 51))
def test_tiny_shape_seeds(seed):
    """Config 1's shape (m = 12, k = 4 of 64 chunks, w ~ U{1..32}), seeds
    1..50: the plain path, whole tables and orders."""
    inst = wl.config(1, seed=seed)
    got = gpu_run(inst)
    assert_same(inst, got, oracle.solve(inst))


@pytest.mark.parametrize("seed", range(1, 51))
def test_config3_shape_seeds(seed):
    """Config 3's shape (m = 20 retrieval requests, k = 10 of 2000 passages in
    50 topics), seeds 1..50: the row-blocked path, whole tables and orders."""
    inst = wl.config(3, seed=seed)
    got = gpu_run(inst)
    assert_same(inst, got, oracle.solve(inst))


# --- the paper's pins through the HIP path -----------------------------------------

def test_k4_3uniform_on_gpu():
    inst = wl.from_sets([[0, 1, 2], [0, 1, 3], [0, 2, 3], [1, 2, 3]], [1] * 4, 4)
    got = gpu_run(inst)
    assert got["opt"] == 8
    layout = ["".join("abcd"[x] for x in got["orders"][3 * i:3 * i + 3]) for i in range(4)]
    assert layout == ["abc", "abd", "cda", "cdb"]


def test_leave_one_out_closed_form_on_gpu():
    for n in range(1, 21):
        got = gpu_run(wl.gen_loo(n))
        assert got["opt"] == brute.loo_opt_free(n), n
    n = 16
    got = gpu_run(wl.gen_loo(n))
    pc = np.array([bin(s).count("1") for s in range(1 << n)])
    E = np.array([0] + [brute.loo_opt_free(s) for s in range(1, n + 1)])
    assert np.array_equal(got["C"][1:], ((n - pc) + E[pc])[1:])
    assert np.array_equal(got["W"][1:], (n - pc)[1:]) and got["W"][0] == n


def test_vertex_cover_on_gpu():
    for seed in range(6):
        inst = wl.gen_two_chunk_graph(7, 9, seed)
        got = gpu_run(inst)
        assert got["opt"] == brute.vertex_cover_number(7, inst.requests()) + inst.m


def test_worst_ratio_and_witness_on_gpu():
    inst = wl.from_sets([[int(c) for c in s] for s in
                         ["0145", "0236", "1236", "1245", "1345", "1456", "2346", "2356"]], [1] * 7, 7)
    assert gpu_run(inst)["opt"] == 14
    inst = wl.from_sets([[0, 1, 2, 3], [1, 4], [2, 5, 7, 8], [4, 6]], [1] * 9, 9)
    assert gpu_run(inst)["opt"] == 10


# --- edge cases ----------------------------------------------------------------------

def test_single_request():
    inst = wl.from_sets([[5, 2, 9, 0]], [3] * 10, 10)
    got = gpu_run(inst)
    assert got["opt"] == 12
    assert got["orders"].tolist() == [0, 2, 5, 9]
    assert_same(inst, got, oracle.solve(inst))


def test_empty_and_identical_requests():
    inst = wl.from_sets([[], [1, 2, 3], [3, 2, 1], [], [1, 2, 3], [4]], [5, 6, 7, 8, 9], 5)
    got = gpu_run(inst)
    assert_same(inst, got, oracle.solve(inst))
    assert got["opt"] == 6 + 7 + 8 + 9


def test_all_requests_empty_and_empty_universe():
    inst = wl.from_sets([[], [], []], [4, 4], 2)
    got = gpu_run(inst)
    assert got["opt"] == 0 and got["W"][0] == 8
    assert_same(inst, got, oracle.solve(inst))
    inst = wl.from_sets([[], []], [], 0)
    got = gpu_run(inst)
    assert got["opt"] == 0 and got["W"].tolist() == [0, 0, 0, 0]


def test_large_weights():
    rng = np.random.default_rng(5)
    w = rng.integers(1 << 31, (1 << 32) + 1, size=400, dtype=np.int64)
    sets = [rng.choice(400, size=int(rng.integers(50, 300)), replace=False).tolist() for _ in range(14)]
    inst = wl.from_sets(sets, w, 400)
    got = gpu_run(inst)
    assert_same(inst, got, oracle.solve(inst))


@pytest.mark.parametrize("excess", [-1, 0])
def test_double_keys_at_their_limit(excess):
    """Costs are packed into doubles while sum_i w(R_i) < 2^(51-m) and into
    uint64 from there on. Private chunks (weights <= 2^32, spread over the
    requests) set the total to 2^(51-m) + excess, so the largest keys either
    path ever holds are exercised (m = 14, row-blocked kernels)."""
    m = 14
    rng = np.random.default_rng(31 + excess)
    n = 300
    target = (1 << (51 - m)) + excess
    w = list(rng.integers(1 << 26, 1 << 28, size=n, dtype=np.int64))
    sets = [rng.choice(n, size=int(rng.integers(10, 40)), replace=False).tolist() for _ in range(m)]
    left = target - int(sum(sum(w[x] for x in s) for s in sets))
    assert left > 0
    i = 0
    while left > 0:
        piece = min(left, (1 << 32) - int(rng.integers(0, 1 << 20)))
        w.append(piece)
        sets[i % m].append(len(w) - 1)
        left -= piece
        i += 1
    w = np.array(w, dtype=np.int64)
    inst = wl.from_sets(sets, w, len(w))
    assert int(sum(w[s].sum() for s in sets)) == target
    got, labels = gpu_run_labelled(inst)
    assert cross_labels(labels) == ({"rb_cross_f64"} if excess < 0 else {"rb_cross_u64"})
    assert_same(inst, got, oracle.solve(inst))


@pytest.mark.parametrize("excess", [-1, 0])
def test_narrow_keys_at_their_limit(excess):
    """Cross pairs run on 32-bit keys (cost << 12 | in-row part of A) while
    sum_i w(R_i) < 2^20 - 1, and on doubles from there on. The total is set
    to 2^20 - 1 + excess with mostly private chunks, so the top-level
    candidates reach the largest narrow keys (m = 16: levels of up to 7
    cross pairs per row)."""
    m = 16
    rng = np.random.default_rng(41 + excess)
    n = 120
    target = (1 << 20) - 1 + excess
    w = list(rng.integers(1, 64, size=n, dtype=np.int64))
    sets = [rng.choice(n, size=int(rng.integers(4, 12)), replace=False).tolist() for _ in range(m)]
    left = target - int(sum(sum(w[x] for x in s) for s in sets))
    assert left > 0
    for i in range(m):
        piece = left // (m - i)
        w.append(piece)
        sets[i].append(len(w) - 1)
        left -= piece
    w = np.array(w, dtype=np.int64)
    inst = wl.from_sets(sets, w, len(w))
    assert int(sum(w[s].sum() for s in sets)) == target
    got, labels = gpu_run_labelled(inst)
    assert cross_labels(labels) == ({"rb_cross_u32"} if excess < 0 else {"rb_cross_f64"})
    assert_same(inst, got, oracle.solve(inst))


def test_wide_keys_on_the_retrieval_shape():
    """The retrieval-shaped m = 20 workload with every weight times 64:
    sum_i w(R_i) passes 2^20 - 1, so the 64-bit kernels run (levels split
    into up to 127 chunks, reduce and finishing passes). Against the oracle,
    and against the narrow path on the unscaled instance: scaling every
    weight by 64 scales every cost by 64 and keeps every tie, so C is 64
    times the narrow C and split is the same."""
    import dataclasses
    base = wl.config(3)
    inst = dataclasses.replace(base, weights=base.weights * 64, name=base.name + " x64")
    assert int(inst.weights[inst.req_chunks].sum()) >= (1 << 20) - 1
    got, labels = gpu_run_labelled(inst)
    assert cross_labels(labels) == {"rb_cross_f64"}
    assert_same(inst, got, oracle.solve(inst))
    narrow = gpu_run(base)
    assert np.array_equal(got["C"][1:], 64 * narrow["C"][1:])
    assert np.array_equal(got["split"], narrow["split"])
    assert np.array_equal(got["orders"], narrow["orders"])


@pytest.mark.parametrize("seed", [1, 2])
def test_narrow_keys_with_many_ties(seed):
    """Unit weights over a small universe: many bipartitions tie on cost and
    on the in-row part of A, differing only in the row part A_H, which the
    narrow path keeps beside each best key (m = 18, up to 31 cross pairs per
    row, split over chunks)."""
    rng = np.random.default_rng(700 + seed)
    sets = [rng.choice(10, size=int(rng.integers(2, 6)), replace=False).tolist() for _ in range(18)]
    inst = wl.from_sets(sets, np.ones(10, dtype=np.int64), 10)
    got, labels = gpu_run_labelled(inst)
    assert cross_labels(labels) == {"rb_cross_u32"}
    assert_same(inst, got, oracle.solve(inst))


def test_costs_too_large_to_pack_take_the_plain_kernels():
    """With sum_i w(R_i) >= 2^(61-m) the packed-key kernels are not used;
    the result must not change."""
    rng = np.random.default_rng(9)
    w = rng.integers(1 << 31, (1 << 32) + 1, size=3000, dtype=np.int64)
    sets = [rng.choice(3000, size=60, replace=False).tolist() for _ in range(20)]
    inst = wl.from_sets(sets, w, 3000)
    assert int(sum(w[s].sum() for s in sets)) >= 1 << (61 - 20)
    got = gpu_run(inst)
    assert_same(inst, got, oracle.solve(inst))


def test_max_m_weight_table():
    """W at MPT_MAX_M = 30 (an 8 GiB table) for L_30: W(S) = 30 - |S|."""
    n = mpt.MPT_MAX_M
    inst = wl.gen_loo(n)
    say(f"[gpu] build only, {inst.name}")
    prob = mpt.Problem(inst)
    prob.build()
    idx = torch.arange(1 << n, device="cuda", dtype=torch.int64)
    pc = torch.zeros_like(idx)
    for b in range(n):
        pc += (idx >> b) & 1
    expect = n - pc
    expect[0] = n
    assert torch.equal(prob.W, expect)
    del prob, idx, pc, expect
    torch.cuda.empty_cache()


def test_max_m_full_solve():
    """Whole path at MPT_MAX_M = 30 (2^30-entry tables, 1.0e14 bipartitions)
    on L_30, where every entry has a closed form: C(S) = (n - |S|) + E(|S|)
    with E the Eq. (5) free value; the split table encodes a hierarchy whose
    Eq. (2) cost and read-off trie cost are both OPT."""
    n = mpt.MPT_MAX_M
    inst = wl.gen_loo(n)
    say(f"[gpu] full solve, {inst.name}")
    prob = mpt.Problem(inst)
    opt = prob.run()
    torch.cuda.synchronize()
    c = (n - 1).bit_length()                               # ceil(log2 n)
    assert opt == brute.loo_opt_free(n) == n * c - (1 << c) + n    # Eq. (5): 148 at n = 30
    E = torch.tensor([0] + [brute.loo_opt_free(s) for s in range(1, n + 1)], dtype=torch.int64, device="cuda")
    for lo in range(0, 1 << n, 1 << 26):                 # in slices to bound temporaries
        idx = torch.arange(lo, lo + (1 << 26), device="cuda", dtype=torch.int64)
        pc = torch.zeros_like(idx)
        for b in range(n):
            pc += (idx >> b) & 1
        expect = (n - pc) + E[pc]
        if lo == 0:
            expect[0] = mpt.MPT_COST_SENTINEL
        assert torch.equal(prob.C[lo:lo + (1 << 26)], expect), lo
        del idx, pc, expect
    split = prob.split.cpu().numpy().view("uint32")
    assert oracle.hierarchy_cost(inst, split) == opt
    orders = prob.orders.cpu().numpy()[:inst.nnz]
    assert oracle.trie_cost(inst, orders) == opt
    del prob
    torch.cuda.empty_cache()


@pytest.mark.parametrize("m", [13, 17])
def test_unaligned_tables(m):
    """The solve's W, C and split may start anywhere a whole element does
    (the build's W output must be 16-byte aligned): offset views, 8- and
    4-byte aligned but not 16, give the same tables as the oracle."""
    inst = wl.gen_retrieval(m=m, u=600, topics=20, k=6, seed=41 + m)
    say(f"[gpu] unaligned tables m={m}")
    dev = torch.device("cuda")
    n = 1 << m
    t = lambda a, dt: torch.as_tensor(a, dtype=dt, device=dev)
    W_built = torch.empty(n, dtype=torch.int64, device=dev)
    W = torch.empty(n + 1, dtype=torch.int64, device=dev)[1:]
    C = torch.empty(n + 1, dtype=torch.int64, device=dev)[1:]
    split = torch.empty(n + 3, dtype=torch.int32, device=dev)[3:]
    sig = torch.empty(max(1, inst.n_chunks), dtype=torch.int32, device=dev)
    ws = mpt.alloc_workspace(m, inst.nnz, dev)
    assert W.data_ptr() % 16 and C.data_ptr() % 16 and split.data_ptr() % 16
    mpt.mpt_build_weights(m, inst.n_chunks, t(inst.weights, torch.int64), t(inst.req_off, torch.int64),
                          t(inst.req_chunks, torch.int32), sig, W_built, ws)
    W.copy_(W_built)
    opt = mpt.mpt_solve_exact(m, W, C, split, ws)
    torch.cuda.synchronize()
    ref = oracle.solve(inst)
    assert opt == ref["opt"]
    assert np.array_equal(W.cpu().numpy(), ref["W"])
    Cg = C.cpu().numpy()
    assert Cg[0] == mpt.MPT_COST_SENTINEL and np.array_equal(Cg[1:], ref["C"][1:])
    assert np.array_equal(split.cpu().numpy().view(np.uint32), ref["split"].astype(np.uint32))


def test_determinism_and_reuse():
    inst = wl.config(3)
    prob = mpt.Problem(inst)
    a = prob.run()
    t1 = prob.host_tables()
    b = prob.run()
    t2 = prob.host_tables()
    assert a == b
    for k in t1:
        assert np.array_equal(t1[k], t2[k]), k


@pytest.mark.parametrize("case", ["range", "dup", "weight", "offsets", "workspace"])
def test_errors_are_reported(case):
    inst = wl.config(1)
    prob = mpt.Problem(inst)
    expect = {"range": "MPT_E_RANGE", "dup": "MPT_E_DUP", "weight": "MPT_E_WEIGHT",
              "offsets": "MPT_E_INVALID", "workspace": "MPT_E_WORKSPACE"}[case]
    if case == "range":
        prob.req_chunks[3] = inst.n_chunks
    elif case == "dup":
        prob.req_chunks[1] = prob.req_chunks[0]
    elif case == "weight":
        prob.chunk_w[7] = 0
    elif case == "offsets":
        prob.req_off[2] = prob.req_off[3] + 1
    else:
        prob.workspace = prob.workspace[:128]
    with pytest.raises(mpt.MptError) as ei:
        prob.build()
    assert ei.value.name == expect
    # the library stays usable after an error
    prob2 = mpt.Problem(inst)
    assert prob2.run() == oracle.solve(inst, with_orders=False)["opt"]


def test_weight_table_dense_route_for_long_lists():
    """25 requests of 90000 chunks over 2^20: 8192 tiles x 2.25M slots is
    past the tile kernel's list scan, so W is built by scatter plus a dense
    superset zeta; it must equal the oracle's table."""
    inst = wl.gen_long_lists()
    say(f"[gpu] dense W route m={inst.m} nnz={inst.nnz}")
    prob = mpt.Problem(inst)
    mpt.profile_begin()
    prob.build()
    torch.cuda.synchronize()
    prof = mpt.profile_end()
    assert "weights_dense" in prof and "weights_tile" not in prof
    assert np.array_equal(prob.W.cpu().numpy(), oracle.intersection_weights(inst))


def test_long_requests():
    """Requests of thousands of chunks: every table and the orders against
    the oracle (the orders come from one sort of (request, depth, id) keys)."""
    rng = np.random.default_rng(21)
    u = 30000
    sets = [rng.choice(u, size=int(rng.integers(6000, 12000)), replace=False).tolist() for _ in range(8)]
    w = rng.integers(1, 300, size=u, dtype=np.int64)
    inst = wl.from_sets(sets, w, u)
    got = gpu_run(inst)
    assert_same(inst, got, oracle.solve(inst))
