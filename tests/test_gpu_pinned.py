"""GPU parity of the Section 7.1 pinned variant through the C ABI (split,
exact or greedy layout of the distinct free sets, assemble, trie cost)
against the oracle's construction: layouts and costs compared exactly."""
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


def check(inst, t, method):
    print(f"[gpu pinned] {inst.name} m={inst.m} t={t} {method}", flush=True)
    got = mpt.pinned_layout(inst, t, method)
    ref = oracle.pinned_layout(inst, t, method)
    assert got["n_distinct"] == ref["n_distinct"]
    assert np.array_equal(got["dmap"].cpu().numpy(), ref["dmap"])
    assert np.array_equal(got["orders"].cpu().numpy(), ref["orders"])
    assert got["cost"] == ref["cost"]
    return got


@pytest.mark.parametrize("idx", [1, 3])
def test_configs_exact_and_greedy(idx):
    inst = wl.config(idx)
    for t in (0, 1, 2, 3, 100):
        for method in ("exact", "greedy"):
            check(inst, t, method)


@pytest.mark.parametrize("seed", range(6))
def test_random_families(seed):
    rng = np.random.default_rng(seed)
    inst = wl.random_small(m=int(rng.integers(1, 26)), u=int(rng.integers(2, 30)), kmin=0, kmax=8,
                           wmax=int(rng.choice([1, 20])), seed=300 + seed)
    for t in (1, 2):
        for method in ("exact", "greedy"):
            check(inst, t, method)


def test_trace_shaped_greedy():
    inst = wl.trace_config("trace_2048")
    for t in (0, 1, 2, 3):
        check(inst, t, "greedy")


def test_errors():
    inst = wl.config(1)
    with pytest.raises(mpt.MptError) as e:
        mpt.pinned_layout(inst, -1)
    assert e.value.status == -1
    big = wl.random_small(m=40, u=200, kmin=5, kmax=9, wmax=5, seed=1)
    with pytest.raises(mpt.MptError):
        mpt.pinned_layout(big, 1, "exact")          # 40 distinct free sets: beyond the exact solver
