"""ctypes binding of libmpt.so (the C ABI in include/mpt.h).

Argument marshalling only: each function checks tensor dtypes, devices and
sizes, then passes raw device pointers and the current HIP stream to the
library. Every step of the computation runs in the library's HIP kernels.
PyTorch only provides device memory and streams. If libmpt.so is missing
the binding raises; it never falls back to another implementation.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmpt.so")

MPT_MAX_M = 30
MPT_COST_SENTINEL = 1 << 62
MPT_GREEDY_MAX_M = 16384
MPT_LAYOUT_MAX_M = 1 << 24
MPT_CACHE_MAX_CONFIGS = 256
MPT_ORDER_ID = 0
MPT_ORDER_POPULARITY = 1
MPT_TABLE_W, MPT_TABLE_SIG, MPT_TABLE_C, MPT_TABLE_SPLIT, MPT_TABLE_ORDERS = 0, 1, 2, 3, 4
MPT_OPT_CHUNK_PAIRS = 1
MPT_OPT_WEIGHT_ROUTE = 2
MPT_ROUTE_AUTO, MPT_ROUTE_LIST, MPT_ROUTE_DENSE = 0, 1, 2
MPT_NOALLOC_MAX_M = 20

_STATUS = {
    0: "MPT_OK", -1: "MPT_E_INVALID", -2: "MPT_E_RANGE", -3: "MPT_E_DUP",
    -4: "MPT_E_WEIGHT", -5: "MPT_E_OVERFLOW", -6: "MPT_E_WORKSPACE", -7: "MPT_E_STATE",
    -8: "MPT_E_DEVICE", -9: "MPT_E_INTERNAL",
}
EXPORTED = ("mpt_workspace_bytes", "mpt_build_weights", "mpt_solve_exact", "mpt_extract_orders",
            "mpt_status_string", "mpt_last_error", "mpt_profile_begin", "mpt_profile_end",
            "mpt_greedy_workspace_bytes", "mpt_pair_weights", "mpt_greedy_hierarchy",
            "mpt_spanning_tree_bound", "mpt_layout_workspace_bytes", "mpt_global_order_layout",
            "mpt_layout_cost", "mpt_cache_simulate", "mpt_pinned_workspace_bytes", "mpt_pinned_split",
            "mpt_pinned_assemble", "mpt_create", "mpt_destroy", "mpt_set_option", "mpt_ctx_workspace_bytes",
            "mpt_set_workspace", "mpt_ctx_build_weights", "mpt_ctx_solve_exact", "mpt_ctx_extract_orders",
            "mpt_copy_table", "mpt_table_device", "mpt_solve_exact_noalloc", "mpt_ctx_optimum",
            "mpt_profile_begin_prefix")


class MptError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        self.name = _STATUS.get(status, str(status))
        super().__init__(f"{where}: {self.name}: {detail}")


class ProfileRow(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_char * 48), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double), ("work", ctypes.c_double)]


_lib = None


def load() -> ctypes.CDLL:
    """Load libmpt.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(hipcc --offload-arch=gfx950); there is no fallback")
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
    lib.mpt_workspace_bytes.argtypes = [i32, i64]
    lib.mpt_workspace_bytes.restype = sz
    lib.mpt_build_weights.argtypes = [i32, i64, i64, P, P, P, P, P, P, sz, P]
    lib.mpt_build_weights.restype = i32
    lib.mpt_solve_exact.argtypes = [i32, P, P, P, P, P, sz, P]
    lib.mpt_solve_exact.restype = i32
    lib.mpt_extract_orders.argtypes = [i32, i64, i64, P, P, P, P, P, P, sz, P]
    lib.mpt_extract_orders.restype = i32
    lib.mpt_status_string.argtypes = [i32]
    lib.mpt_status_string.restype = ctypes.c_char_p
    lib.mpt_last_error.argtypes = []
    lib.mpt_last_error.restype = ctypes.c_char_p
    lib.mpt_profile_begin.argtypes = []
    lib.mpt_profile_begin.restype = i32
    lib.mpt_profile_begin_prefix.argtypes = [ctypes.c_char_p]
    lib.mpt_profile_begin_prefix.restype = i32
    lib.mpt_profile_end.argtypes = [ctypes.POINTER(ProfileRow), i32]
    lib.mpt_profile_end.restype = i32
    lib.mpt_greedy_workspace_bytes.argtypes = [i32, i64, i64]
    lib.mpt_greedy_workspace_bytes.restype = sz
    lib.mpt_pair_weights.argtypes = [i32, i64, i64, P, P, P, P, P, P, sz, P]
    lib.mpt_pair_weights.restype = i32
    lib.mpt_greedy_hierarchy.argtypes = [i32, i64, i64, P, P, P, P, P, P, P, P, P, P, sz, P]
    lib.mpt_greedy_hierarchy.restype = i32
    lib.mpt_spanning_tree_bound.argtypes = [i32, P, P, P, sz, P]
    lib.mpt_spanning_tree_bound.restype = i32
    lib.mpt_layout_workspace_bytes.argtypes = [i32, i64, i64, i32]
    lib.mpt_layout_workspace_bytes.restype = sz
    lib.mpt_global_order_layout.argtypes = [i32, i64, i64, P, P, i32, P, P, sz, P]
    lib.mpt_global_order_layout.restype = i32
    lib.mpt_layout_cost.argtypes = [i32, i64, i64, P, P, P, P, P, P, sz, P]
    lib.mpt_layout_cost.restype = i32
    lib.mpt_cache_simulate.argtypes = [i32, i64, i64, P, P, P, i32, P, P, P, P, P, sz, P]
    lib.mpt_cache_simulate.restype = i32
    lib.mpt_pinned_workspace_bytes.argtypes = [i32, i64]
    lib.mpt_pinned_workspace_bytes.restype = sz
    lib.mpt_pinned_split.argtypes = [i32, i64, i64, P, P, i32, P, P, P, P, P, sz, P]
    lib.mpt_pinned_split.restype = i32
    lib.mpt_pinned_assemble.argtypes = [i32, i64, P, P, i32, P, i32, P, P, P, P, sz, P]
    lib.mpt_pinned_assemble.restype = i32
    lib.mpt_solve_exact_noalloc.argtypes = [i32, P, P, P, P, P]
    lib.mpt_solve_exact_noalloc.restype = i32
    lib.mpt_create.argtypes = [ctypes.POINTER(P), i32, P]
    lib.mpt_create.restype = i32
    lib.mpt_destroy.argtypes = [P]
    lib.mpt_destroy.restype = None
    lib.mpt_set_option.argtypes = [P, i32, i64]
    lib.mpt_set_option.restype = i32
    lib.mpt_ctx_workspace_bytes.argtypes = [P, i32, i64, i64]
    lib.mpt_ctx_workspace_bytes.restype = sz
    lib.mpt_set_workspace.argtypes = [P, P, sz]
    lib.mpt_set_workspace.restype = i32
    lib.mpt_ctx_build_weights.argtypes = [P, i32, i64, i64, P, P, P]
    lib.mpt_ctx_build_weights.restype = i32
    lib.mpt_ctx_solve_exact.argtypes = [P, P, P, P]
    lib.mpt_ctx_solve_exact.restype = i32
    lib.mpt_ctx_optimum.argtypes = [P, P, P]
    lib.mpt_ctx_optimum.restype = i32
    lib.mpt_ctx_extract_orders.argtypes = [P, P]
    lib.mpt_ctx_extract_orders.restype = i32
    lib.mpt_copy_table.argtypes = [P, i32, P, sz]
    lib.mpt_copy_table.restype = i32
    lib.mpt_table_device.argtypes = [P, i32, ctypes.POINTER(P), ctypes.POINTER(sz)]
    lib.mpt_table_device.restype = i32
    _lib = lib
    return lib


def _check(rc: int, where: str) -> None:
    if rc != 0:
        raise MptError(rc, where, load().mpt_last_error().decode())


def _ptr(t: torch.Tensor | None, dtype: torch.dtype, n: int, name: str) -> int | None:
    if t is None:
        if n > 0:
            raise ValueError(f"{name} is required")
        return None
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() < n:
        raise ValueError(f"{name} has {t.numel()} elements, needs {n}")
    return t.data_ptr() if t.numel() else None


def _stream(stream) -> int | None:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream or None


def mpt_workspace_bytes(m: int, nnz: int) -> int:
    return int(load().mpt_workspace_bytes(m, nnz))


def alloc_workspace(m: int, nnz: int, device="cuda") -> torch.Tensor:
    """A uint8 device tensor big enough (and 256-byte aligned) for all calls."""
    n = mpt_workspace_bytes(m, nnz)
    if n == 0:
        raise MptError(-1, "mpt_workspace_bytes", f"invalid m={m} or nnz={nnz}")
    return torch.empty(n, dtype=torch.uint8, device=device)


def mpt_build_weights(m, n_chunks, chunk_w, req_off, req_chunks, sig, W, workspace, stream=None):
    """W(B) = w(I(B)) for all subsets and S_x per chunk (see include/mpt.h)."""
    nnz = int(req_chunks.numel()) if req_chunks is not None else 0
    rc = load().mpt_build_weights(
        m, n_chunks, nnz,
        _ptr(chunk_w, torch.int64, n_chunks, "chunk_w"),
        _ptr(req_off, torch.int64, m + 1, "req_off"),
        _ptr(req_chunks, torch.int32, nnz, "req_chunks") if nnz else None,
        _ptr(sig, torch.int32, n_chunks, "sig"),
        _ptr(W, torch.int64, 1 << m, "W"),
        _ptr(workspace, torch.uint8, 1, "workspace"), workspace.numel(), _stream(stream))
    _check(rc, "mpt_build_weights")


def mpt_solve_exact(m, W, C, split, workspace, stream=None, want_cost=True):
    """Section 3.1 DP; returns OPT_free (synchronising) or None."""
    out = ctypes.c_int64(0)
    rc = load().mpt_solve_exact(
        m, _ptr(W, torch.int64, 1 << m, "W"), _ptr(C, torch.int64, 1 << m, "C"),
        _ptr(split, torch.int32, 1 << m, "split"),
        ctypes.addressof(out) if want_cost else None,
        _ptr(workspace, torch.uint8, 1, "workspace"), workspace.numel(), _stream(stream))
    _check(rc, "mpt_solve_exact")
    return int(out.value) if want_cost else None


def mpt_solve_exact_noalloc(m, W, C, split, stream=None, want_cost=True):
    """mpt_solve_exact on the library's own scratch array (m <= 20)."""
    out = ctypes.c_int64(0)
    rc = load().mpt_solve_exact_noalloc(
        m, _ptr(W, torch.int64, 1 << m, "W"), _ptr(C, torch.int64, 1 << m, "C"),
        _ptr(split, torch.int32, 1 << m, "split"), ctypes.addressof(out) if want_cost else None, _stream(stream))
    _check(rc, "mpt_solve_exact_noalloc")
    return int(out.value) if want_cost else None


def mpt_extract_orders(m, n_chunks, req_off, req_chunks, sig, split, order_chunks, workspace, stream=None):
    """pi_i for every request into order_chunks (CSR with req_off)."""
    nnz = int(req_chunks.numel()) if req_chunks is not None else 0
    rc = load().mpt_extract_orders(
        m, n_chunks, nnz,
        _ptr(req_off, torch.int64, m + 1, "req_off"),
        _ptr(req_chunks, torch.int32, nnz, "req_chunks") if nnz else None,
        _ptr(sig, torch.int32, n_chunks, "sig") if nnz else None,
        _ptr(split, torch.int32, 1 << m, "split"),
        _ptr(order_chunks, torch.int32, nnz, "order_chunks") if nnz else None,
        _ptr(workspace, torch.uint8, 1, "workspace"), workspace.numel(), _stream(stream))
    _check(rc, "mpt_extract_orders")


def profile_begin(prefix: str = "") -> None:
    """Start recording launch times (only labels starting with prefix)."""
    _check(load().mpt_profile_begin_prefix(prefix.encode()), "mpt_profile_begin_prefix")


def profile_end(max_rows: int = 64) -> dict:
    """{kernel: {"launches", "total_ms", "work"}} for the launches since
    profile_begin()."""
    rows = (ProfileRow * max_rows)()
    n = load().mpt_profile_end(rows, max_rows)
    if n < 0:
        _check(n, "mpt_profile_end")
    return {rows[i].kernel.decode(): {"launches": rows[i].launches, "total_ms": rows[i].total_ms,
                                      "work": rows[i].work} for i in range(min(n, max_rows))}


# --- Sections 6.2-6.3: agglomerative hierarchy and spanning-tree bound ------

def mpt_greedy_workspace_bytes(m: int, n_chunks: int, nnz: int) -> int:
    return int(load().mpt_greedy_workspace_bytes(m, n_chunks, nnz))


def alloc_greedy_workspace(m: int, n_chunks: int, nnz: int, device="cuda") -> torch.Tensor:
    n = mpt_greedy_workspace_bytes(m, n_chunks, nnz)
    if n == 0:
        raise MptError(-1, "mpt_greedy_workspace_bytes", f"invalid m={m}, n_chunks={n_chunks} or nnz={nnz}")
    return torch.empty(n, dtype=torch.uint8, device=device)


def mpt_pair_weights(m, n_chunks, chunk_w, req_off, req_chunks, P, workspace, stream=None) -> int:
    """P[i, j] = w(R_i ∩ R_j) (see include/mpt.h); returns sum_i w(R_i)."""
    nnz = int(req_chunks.numel()) if req_chunks is not None else 0
    total = ctypes.c_int64(0)
    rc = load().mpt_pair_weights(
        m, n_chunks, nnz,
        _ptr(chunk_w, torch.int64, n_chunks, "chunk_w"),
        _ptr(req_off, torch.int64, m + 1, "req_off"),
        _ptr(req_chunks, torch.int32, nnz, "req_chunks") if nnz else None,
        _ptr(P, torch.int64, m * m, "P"), ctypes.addressof(total),
        _ptr(workspace, torch.uint8, 1, "workspace"), workspace.numel(), _stream(stream))
    _check(rc, "mpt_pair_weights")
    return int(total.value)


def mpt_greedy_hierarchy(m, n_chunks, chunk_w, req_off, req_chunks, merge_a, merge_b, gain, node_parent,
                         order_chunks, workspace, stream=None, want_savings=True):
    """Agglomerative hierarchy H_g and (if order_chunks is given) its layout;
    returns SAV(H_g) or None."""
    nnz = int(req_chunks.numel()) if req_chunks is not None else 0
    out = ctypes.c_int64(0)
    rc = load().mpt_greedy_hierarchy(
        m, n_chunks, nnz,
        _ptr(chunk_w, torch.int64, n_chunks, "chunk_w"),
        _ptr(req_off, torch.int64, m + 1, "req_off"),
        _ptr(req_chunks, torch.int32, nnz, "req_chunks") if nnz else None,
        _ptr(merge_a, torch.int32, m - 1, "merge_a"), _ptr(merge_b, torch.int32, m - 1, "merge_b"),
        _ptr(gain, torch.int64, m - 1, "gain"), _ptr(node_parent, torch.int32, 2 * m - 1, "node_parent"),
        _ptr(order_chunks, torch.int32, nnz, "order_chunks") if (order_chunks is not None and nnz) else None,
        ctypes.addressof(out) if want_savings else None,
        _ptr(workspace, torch.uint8, 1, "workspace"), workspace.numel(), _stream(stream))
    _check(rc, "mpt_greedy_hierarchy")
    return int(out.value) if want_savings else None


def mpt_spanning_tree_bound(m, P, workspace, stream=None) -> int:
    """Weight of a maximum spanning tree of the pair weights P."""
    out = ctypes.c_int64(0)
    rc = load().mpt_spanning_tree_bound(
        m, _ptr(P, torch.int64, m * m, "P"), ctypes.addressof(out),
        _ptr(workspace, torch.uint8, 1, "workspace"), workspace.numel(), _stream(stream))
    _check(rc, "mpt_spanning_tree_bound")
    return int(out.value)


class Greedy:
    """Device-resident instance plus the outputs of the Section 6.2-6.3 calls."""

    def __init__(self, inst, device="cuda"):
        if not 1 <= inst.m <= MPT_GREEDY_MAX_M:
            raise MptError(-1, "Greedy", f"m = {inst.m} outside [1, {MPT_GREEDY_MAX_M}]")
        self.m = inst.m
        self.n_chunks = inst.n_chunks
        self.nnz = inst.nnz
        dev = torch.device(device)
        self.chunk_w = torch.as_tensor(inst.weights, dtype=torch.int64).to(dev)
        self.req_off = torch.as_tensor(inst.req_off, dtype=torch.int64).to(dev)
        self.req_chunks = torch.as_tensor(inst.req_chunks, dtype=torch.int32).to(dev)
        m = self.m
        self.P = torch.empty(m * m, dtype=torch.int64, device=dev)
        self.merge_a = torch.empty(max(1, m - 1), dtype=torch.int32, device=dev)
        self.merge_b = torch.empty(max(1, m - 1), dtype=torch.int32, device=dev)
        self.gain = torch.empty(max(1, m - 1), dtype=torch.int64, device=dev)
        self.node_parent = torch.empty(2 * m - 1, dtype=torch.int32, device=dev)
        self.orders = torch.empty(max(1, self.nnz), dtype=torch.int32, device=dev)
        self.workspace = alloc_greedy_workspace(m, self.n_chunks, self.nnz, dev)

    def pair_weights(self, stream=None) -> int:
        return mpt_pair_weights(self.m, self.n_chunks, self.chunk_w, self.req_off, self.req_chunks, self.P,
                                self.workspace, stream)

    def hierarchy(self, stream=None, with_orders=True) -> int:
        return mpt_greedy_hierarchy(self.m, self.n_chunks, self.chunk_w, self.req_off, self.req_chunks,
                                    self.merge_a, self.merge_b, self.gain, self.node_parent,
                                    self.orders if with_orders else None, self.workspace, stream)

    def spanning_tree(self, stream=None) -> int:
        return mpt_spanning_tree_bound(self.m, self.P, self.workspace, stream)

    def run(self, stream=None) -> dict:
        """Pair weights, H_g with its layout, and the spanning-tree bound."""
        total = self.pair_weights(stream)
        sav = self.hierarchy(stream)
        mst = self.spanning_tree(stream)
        return {"savings": sav, "mst": mst, "request_total": total, "cost": total - sav,
                "lower_bound": total - mst}

    def host(self) -> dict:
        m = self.m
        return {"P": self.P.view(m, m).cpu().numpy(),
                "merge_a": self.merge_a.cpu().numpy()[:m - 1], "merge_b": self.merge_b.cpu().numpy()[:m - 1],
                "gain": self.gain.cpu().numpy()[:m - 1], "parent": self.node_parent.cpu().numpy(),
                "orders": self.orders.cpu().numpy()[:self.nnz]}


# --- Sections 7-8: layouts, serving schedules and the radix cache ---------

def mpt_layout_workspace_bytes(m: int, n_chunks: int, nnz: int, n_configs: int = 0) -> int:
    return int(load().mpt_layout_workspace_bytes(m, n_chunks, nnz, n_configs))


def alloc_layout_workspace(m, n_chunks, nnz, n_configs=0, device="cuda") -> torch.Tensor:
    n = mpt_layout_workspace_bytes(m, n_chunks, nnz, n_configs)
    if n == 0:
        raise MptError(-1, "mpt_layout_workspace_bytes", f"invalid sizes m={m} n_chunks={n_chunks} nnz={nnz}")
    return torch.empty(n, dtype=torch.uint8, device=device)


def mpt_global_order_layout(m, n_chunks, req_off, req_chunks, order_kind, seqs, workspace, stream=None):
    nnz = int(req_chunks.numel()) if req_chunks is not None else 0
    rc = load().mpt_global_order_layout(
        m, n_chunks, nnz, _ptr(req_off, torch.int64, m + 1, "req_off"),
        _ptr(req_chunks, torch.int32, nnz, "req_chunks") if nnz else None, int(order_kind),
        _ptr(seqs, torch.int32, nnz, "seqs") if nnz else None,
        _ptr(workspace, torch.uint8, 1, "workspace"), workspace.numel(), _stream(stream))
    _check(rc, "mpt_global_order_layout")


def mpt_layout_cost(m, n_chunks, chunk_w, seq_off, seqs, dfs_order, workspace, stream=None) -> int:
    """Trie cost of the layout; the DFS order into dfs_order if given."""
    nnz = int(seqs.numel()) if seqs is not None else 0
    out = ctypes.c_int64(0)
    rc = load().mpt_layout_cost(
        m, n_chunks, nnz, _ptr(chunk_w, torch.int64, n_chunks, "chunk_w"),
        _ptr(seq_off, torch.int64, m + 1, "seq_off"), _ptr(seqs, torch.int32, nnz, "seqs") if nnz else None,
        _ptr(dfs_order, torch.int32, m, "dfs_order") if dfs_order is not None else None,
        ctypes.addressof(out), _ptr(workspace, torch.uint8, 1, "workspace"), workspace.numel(), _stream(stream))
    _check(rc, "mpt_layout_cost")
    return int(out.value)


def mpt_cache_simulate(m, n_chunks, chunk_w, seq_off, seqs, windows, capacities, workspace, stream=None):
    """Billed weight of every (window, capacity) configuration, and the
    unbounded-cache bill (the trie cost)."""
    nnz = int(seqs.numel()) if seqs is not None else 0
    n = len(windows)
    if len(capacities) != n:
        raise ValueError("windows and capacities differ in length")
    win = (ctypes.c_int64 * n)(*[int(x) for x in windows])
    cap = (ctypes.c_int64 * n)(*[int(x) for x in capacities])
    out = (ctypes.c_int64 * n)()
    tc = ctypes.c_int64(0)
    rc = load().mpt_cache_simulate(
        m, n_chunks, nnz, _ptr(chunk_w, torch.int64, n_chunks, "chunk_w"),
        _ptr(seq_off, torch.int64, m + 1, "seq_off"), _ptr(seqs, torch.int32, nnz, "seqs") if nnz else None,
        n, win, cap, out, ctypes.addressof(tc),
        _ptr(workspace, torch.uint8, 1, "workspace"), workspace.numel(), _stream(stream))
    _check(rc, "mpt_cache_simulate")
    return [int(x) for x in out], int(tc.value)


class Layouts:
    """Device-resident instance for the Section 7-8 calls: global-order
    layouts, trie costs, DFS orders and radix-cache simulations of any layout
    of the instance (a layout = int32 sequences, CSR with the request
    offsets)."""

    def __init__(self, inst, n_configs=0, device="cuda"):
        self.m, self.n_chunks, self.nnz = inst.m, inst.n_chunks, inst.nnz
        dev = torch.device(device)
        self.chunk_w = torch.as_tensor(inst.weights, dtype=torch.int64).to(dev)
        self.req_off = torch.as_tensor(inst.req_off, dtype=torch.int64).to(dev)
        self.req_chunks = torch.as_tensor(inst.req_chunks, dtype=torch.int32).to(dev)
        self.dfs = torch.empty(self.m, dtype=torch.int32, device=dev)
        self.workspace = alloc_layout_workspace(self.m, self.n_chunks, self.nnz, n_configs, dev)

    def seqs(self, layout) -> torch.Tensor:
        return torch.as_tensor(layout, dtype=torch.int32).to(self.req_off.device).contiguous()

    def global_order(self, kind, stream=None) -> torch.Tensor:
        out = torch.empty(max(1, self.nnz), dtype=torch.int32, device=self.req_off.device)
        mpt_global_order_layout(self.m, self.n_chunks, self.req_off, self.req_chunks, kind, out, self.workspace, stream)
        return out[:self.nnz]

    def cost(self, seqs, stream=None) -> int:
        return mpt_layout_cost(self.m, self.n_chunks, self.chunk_w, self.req_off, seqs, self.dfs, self.workspace,
                               stream)

    def simulate(self, seqs, windows, capacities, stream=None):
        return mpt_cache_simulate(self.m, self.n_chunks, self.chunk_w, self.req_off, seqs, windows, capacities,
                                  self.workspace, stream)


# --- Section 7.1: the pinned variant ---------------------------------------

def pinned_layout(inst, t: int, method: str = "exact", device="cuda", stream=None) -> dict:
    """Top-t of every request pinned at its end (most relevant last), the
    free parts laid out by the exact DP or the greedy over the distinct free
    sets (see include/mpt.h). Returns the layout (device tensor, CSR with the
    request offsets), its trie cost and the distinct-set count."""
    from types import SimpleNamespace
    lib = load()
    dev = torch.device(device)
    m, nnz = inst.m, inst.nnz
    chunk_w = torch.as_tensor(inst.weights, dtype=torch.int64).to(dev)
    req_off = torch.as_tensor(inst.req_off, dtype=torch.int64).to(dev)
    req_chunks = torch.as_tensor(inst.req_chunks, dtype=torch.int32).to(dev)
    nbytes = int(lib.mpt_pinned_workspace_bytes(m, nnz))
    if nbytes == 0:
        raise MptError(-1, "mpt_pinned_workspace_bytes", f"invalid m={m} or nnz={nnz}")
    ws = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    dmap = torch.empty(m, dtype=torch.int32, device=dev)
    free_off = torch.empty(m + 1, dtype=torch.int64, device=dev)
    free_chunks = torch.empty(max(1, nnz), dtype=torch.int32, device=dev)
    nd = ctypes.c_int(0)
    rc = lib.mpt_pinned_split(m, inst.n_chunks, nnz, req_off.data_ptr(), req_chunks.data_ptr() if nnz else None,
                              int(t), dmap.data_ptr(), free_off.data_ptr(), free_chunks.data_ptr(),
                              ctypes.addressof(nd), ws.data_ptr(), ws.numel(), _stream(stream))
    _check(rc, "mpt_pinned_split")
    n_d = int(nd.value)
    nnz_f = int(free_off[n_d].item())
    sub = SimpleNamespace(m=n_d, n_chunks=inst.n_chunks, nnz=nnz_f, weights=chunk_w,
                          req_off=free_off[:n_d + 1], req_chunks=free_chunks[:nnz_f])
    if method == "exact":
        prob = Problem(sub, device)
        prob.run(stream)
        free_layout = prob.orders
    elif method == "greedy":
        g = Greedy(sub, device)
        g.hierarchy(stream)
        free_layout = g.orders
    else:
        raise ValueError(method)
    seqs = torch.empty(max(1, nnz), dtype=torch.int32, device=dev)
    rc = lib.mpt_pinned_assemble(m, nnz, req_off.data_ptr(), req_chunks.data_ptr() if nnz else None, int(t),
                                 dmap.data_ptr(), n_d, free_off.data_ptr(), free_layout.data_ptr(),
                                 seqs.data_ptr(), ws.data_ptr(), ws.numel(), _stream(stream))
    _check(rc, "mpt_pinned_assemble")
    L = Layouts(inst, 0, device)
    cost = L.cost(seqs[:nnz], stream)
    return {"orders": seqs[:nnz], "cost": cost, "n_distinct": n_d, "dmap": dmap}


class Problem:
    """Device-resident instance plus the output tables of one solve.

    Holds the caller-side allocations (torch tensors) that the C ABI expects:
    inputs uploaded once, W / C / split / orders / sig outputs, workspace.
    """

    def __init__(self, inst, device="cuda"):
        if not 1 <= inst.m <= MPT_MAX_M:
            raise MptError(-1, "Problem", f"m = {inst.m} outside [1, {MPT_MAX_M}] (the tables hold 2^m entries)")
        self.m = inst.m
        self.n_chunks = inst.n_chunks
        self.nnz = inst.nnz
        dev = torch.device(device)
        self.chunk_w = torch.as_tensor(inst.weights, dtype=torch.int64).to(dev)
        self.req_off = torch.as_tensor(inst.req_off, dtype=torch.int64).to(dev)
        self.req_chunks = torch.as_tensor(inst.req_chunks, dtype=torch.int32).to(dev)
        n = 1 << self.m
        self.sig = torch.empty(max(1, self.n_chunks), dtype=torch.int32, device=dev)
        self.W = torch.empty(n, dtype=torch.int64, device=dev)
        self.C = torch.empty(n, dtype=torch.int64, device=dev)
        self.split = torch.empty(n, dtype=torch.int32, device=dev)
        self.orders = torch.empty(max(1, self.nnz), dtype=torch.int32, device=dev)
        self.workspace = alloc_workspace(self.m, self.nnz, dev)

    def build(self, stream=None):
        mpt_build_weights(self.m, self.n_chunks, self.chunk_w, self.req_off, self.req_chunks,
                          self.sig, self.W, self.workspace, stream)

    def solve(self, stream=None, want_cost=True):
        return mpt_solve_exact(self.m, self.W, self.C, self.split, self.workspace, stream, want_cost)

    def extract(self, stream=None):
        mpt_extract_orders(self.m, self.n_chunks, self.req_off, self.req_chunks, self.sig, self.split,
                           self.orders, self.workspace, stream)

    def run(self, stream=None) -> int:
        """Whole hot path: W table, DP, orders. Returns OPT_free."""
        self.build(stream)
        opt = self.solve(stream)
        self.extract(stream)
        return opt

    def host_tables(self) -> dict:
        """Copies of the device tables as numpy arrays (uint32 views of masks)."""
        return {
            "W": self.W.cpu().numpy(),
            "C": self.C.cpu().numpy(),
            "split": self.split.cpu().numpy().view("uint32"),
            "sig": self.sig.cpu().numpy().view("uint32")[:self.n_chunks],
            "orders": self.orders.cpu().numpy()[:self.nnz],
        }


def solve(inst, device="cuda") -> dict:
    """One full run on the GPU; returns host copies of every output."""
    prob = Problem(inst, device)
    opt = prob.run()
    out = prob.host_tables()
    out["opt"] = opt
    return out


# --- the context layer ------------------------------------------------------

def _any_ptr(t, dtype, n: int, name: str):
    """Pointer to a contiguous tensor in host or device memory (the context
    build copies its inputs with hipMemcpyDefault)."""
    if t is None:
        if n > 0:
            raise ValueError(f"{name} is required")
        return None
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() < n:
        raise ValueError(f"{name} has {t.numel()} elements, needs {n}")
    return t.data_ptr() if t.numel() else None


class Context:
    """An mpt_ctx (include/mpt.h): one instance on one device, its phases in
    order, over a workspace tensor that this object allocates with torch and
    keeps alive."""

    _DTYPES = {MPT_TABLE_W: "int64", MPT_TABLE_SIG: "uint32", MPT_TABLE_C: "int64",
               MPT_TABLE_SPLIT: "uint32", MPT_TABLE_ORDERS: "int32"}

    def __init__(self, device="cuda", stream=None):
        lib = load()
        self.device = torch.device(device)
        idx = self.device.index if self.device.index is not None else torch.cuda.current_device()
        if stream is None:
            stream = torch.cuda.current_stream(idx)
        self.stream = stream
        h = ctypes.c_void_p()
        _check(lib.mpt_create(ctypes.byref(h), idx, stream.cuda_stream or None), "mpt_create")
        self._h = h
        self.workspace = None

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            load().mpt_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_option(self, option: int, value: int) -> None:
        _check(load().mpt_set_option(self._h, option, value), "mpt_set_option")

    def workspace_bytes(self, m: int, n_chunks: int, nnz: int) -> int:
        return int(load().mpt_ctx_workspace_bytes(self._h, m, n_chunks, nnz))

    def reserve(self, m: int, n_chunks: int, nnz: int) -> None:
        """Allocates (with torch) and attaches a workspace for these sizes,
        unless the attached one is already large enough."""
        need = self.workspace_bytes(m, n_chunks, nnz)
        if need == 0:
            raise MptError(-1, "mpt_ctx_workspace_bytes", f"invalid sizes m={m} n_chunks={n_chunks} nnz={nnz}")
        if self.workspace is None or self.workspace.numel() < need:
            self.workspace = None
            self.workspace = torch.empty(need, dtype=torch.uint8, device=self.device)
        self.set_workspace(self.workspace)

    def set_workspace(self, ws) -> None:
        ptr = _ptr(ws, torch.uint8, 1, "workspace") if ws is not None else None
        _check(load().mpt_set_workspace(self._h, ptr, ws.numel() if ws is not None else 0), "mpt_set_workspace")

    def build_weights(self, m, n_chunks, chunk_w, req_off, req_chunks) -> None:
        nnz = int(req_chunks.numel()) if req_chunks is not None else 0
        _check(load().mpt_ctx_build_weights(
            self._h, m, n_chunks, nnz, _any_ptr(chunk_w, torch.int64, n_chunks, "chunk_w"),
            _any_ptr(req_off, torch.int64, m + 1, "req_off"),
            _any_ptr(req_chunks, torch.int32, nnz, "req_chunks") if nnz else None), "mpt_ctx_build_weights")
        self._sizes = (m, n_chunks, nnz)

    def solve_exact(self, want_cost=True, want_split=False):
        """Returns (OPT_free, savings, split) with None for what was not asked."""
        import numpy as np
        opt, sav = ctypes.c_int64(0), ctypes.c_int64(0)
        split = None
        if want_split:
            n = self._table_len(MPT_TABLE_W)
            split = np.empty(n, dtype=np.uint32)
        _check(load().mpt_ctx_solve_exact(
            self._h, ctypes.addressof(opt) if want_cost else None, ctypes.addressof(sav) if want_cost else None,
            split.ctypes.data if split is not None else None), "mpt_ctx_solve_exact")
        return (int(opt.value) if want_cost else None, int(sav.value) if want_cost else None, split)

    def optimum(self):
        """(OPT_free, savings) of the last solve (one synchronisation)."""
        opt, sav = ctypes.c_int64(0), ctypes.c_int64(0)
        _check(load().mpt_ctx_optimum(self._h, ctypes.addressof(opt), ctypes.addressof(sav)), "mpt_ctx_optimum")
        return int(opt.value), int(sav.value)

    def extract_orders(self, to_host=True):
        import numpy as np
        out = None
        if to_host:
            out = np.empty(max(1, self._table_len(MPT_TABLE_ORDERS)), dtype=np.int32)
        _check(load().mpt_ctx_extract_orders(self._h, out.ctypes.data if out is not None else None),
               "mpt_ctx_extract_orders")
        return out[:self._nnz] if out is not None else None

    def copy_table(self, which: int):
        import numpy as np
        n = self._table_len(which)
        out = np.empty(max(1, n), dtype=self._DTYPES.get(which, "uint8"))   # unknown: the library says so
        _check(load().mpt_copy_table(self._h, which, out.ctypes.data, out.nbytes), "mpt_copy_table")
        return out[:n]

    def table_device(self, which: int):
        """(device address, bytes) of a table inside the workspace."""
        p, nb = ctypes.c_void_p(), ctypes.c_size_t(0)
        _check(load().mpt_table_device(self._h, which, ctypes.byref(p), ctypes.byref(nb)), "mpt_table_device")
        return int(p.value or 0), int(nb.value)

    # sizes of the last build, kept on the Python side for output buffers
    _sizes = (0, 0, 0)

    def _table_len(self, which):
        m, u, nnz = self._sizes
        return {MPT_TABLE_W: 1 << m, MPT_TABLE_C: 1 << m, MPT_TABLE_SPLIT: 1 << m, MPT_TABLE_SIG: u,
                MPT_TABLE_ORDERS: nnz}.get(which, 1)

    @property
    def _nnz(self):
        return self._sizes[2]

    def run(self, inst_or_tensors) -> dict:
        """Build, solve and extract one instance (a workloads instance or a
        (m, n_chunks, chunk_w, req_off, req_chunks) tuple of tensors); returns
        OPT_free, the savings and the orders (host)."""
        if isinstance(inst_or_tensors, tuple):
            m, u, chunk_w, req_off, req_chunks = inst_or_tensors
        else:
            inst = inst_or_tensors
            m, u = inst.m, inst.n_chunks
            chunk_w = torch.as_tensor(inst.weights, dtype=torch.int64)
            req_off = torch.as_tensor(inst.req_off, dtype=torch.int64)
            req_chunks = torch.as_tensor(inst.req_chunks, dtype=torch.int32)
        nnz = int(req_chunks.numel())
        self.reserve(m, u, nnz)
        self.build_weights(m, u, chunk_w, req_off, req_chunks)
        opt, sav, _ = self.solve_exact()
        orders = self.extract_orders()
        return {"opt": opt, "savings": sav, "orders": orders}
