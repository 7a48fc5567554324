"""Write tests/golden/config_<k>.json from the CPU oracle alone.

Each file records, for one benchmark workload, the instance hash, the optimum,
the savings, SHA-256 digests of the full W, C and split tables and of the
read-off orders, the orders themselves and a fixed sample of table entries.
GPU parity tests compare the HIP path's full tables against these digests at
sizes where running the oracle inside a test would take minutes.

Usage: python tests/golden/make_golden.py 3 4 5   (calls only oracle/)
"""
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2609_13692_amd import workloads as wl  # noqa: E402


def digest(a: np.ndarray, dtype: str) -> str:
    return hashlib.sha256(np.ascontiguousarray(a, dtype=dtype).tobytes()).hexdigest()


def main(idxs):
    for idx in idxs:
        inst = wl.config(idx)
        t0 = time.time()
        res = oracle.solve(inst)
        dt = time.time() - t0
        m = inst.m
        rng = np.random.default_rng(12345)
        sample = np.unique(np.concatenate([
            rng.integers(1, 1 << m, size=512),
            np.array([(1 << m) - 1, 1, 1 << (m - 1), (1 << m) - 2], dtype=np.int64)]))
        out = {
            "config": idx,
            "name": inst.name,
            "instance_sha256": inst.sha256(),
            "m": m,
            "opt": res["opt"],
            "savings": res["savings"],
            "W_sha256": digest(res["W"], "<i8"),
            "C_sha256_from_1": digest(res["C"][1:], "<i8"),
            "split_sha256": digest(res["split"], "<u4"),
            "orders_sha256": digest(res["orders"], "<i4"),
            "orders": res["orders"].tolist(),
            "sample": [[int(s), int(res["W"][s]), int(res["C"][s]), int(res["split"][s])] for s in sample],
            "oracle_seconds": round(dt, 2),
            "oracle_threads": oracle.max_threads(),
        }
        path = os.path.join(os.path.dirname(os.path.abspath(__file__)), f"config_{idx}.json")
        with open(path, "w") as f:
            json.dump(out, f, indent=1)
        print(f"config {idx}: m={m} opt={res['opt']} oracle {dt:.1f}s -> {path}", flush=True)


if __name__ == "__main__":
    main([int(a) for a in sys.argv[1:]] or [1, 2, 3, 4, 5])
