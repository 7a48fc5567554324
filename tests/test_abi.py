"""The C ABI without a GPU: the library loads, exports every entry point the
header declares, sizes its workspace, and rejects bad arguments before any
HIP call."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mpt.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mpt_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_2609_13692_amd import mpt
    if not os.path.exists(mpt.LIB_PATH):
        pytest.fail("libmpt.so is not built (run __graft_entry__.build())")
    return mpt.load()


def test_header_declares_the_three_phases():
    names = declared_functions()
    for n in ("mpt_build_weights", "mpt_solve_exact", "mpt_extract_orders", "mpt_workspace_bytes"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    from paper_2609_13692_amd import mpt
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert set(declared_functions()) == set(mpt.EXPORTED)


def test_workspace_sizes(lib):
    from paper_2609_13692_amd import mpt
    assert mpt.mpt_workspace_bytes(0, 10) == 0
    assert mpt.mpt_workspace_bytes(mpt.MPT_MAX_M + 1, 10) == 0
    assert mpt.mpt_workspace_bytes(5, -1) == 0
    for m in (1, 12, 20, 25, 28, mpt.MPT_MAX_M):
        a = mpt.mpt_workspace_bytes(m, 0)
        b = mpt.mpt_workspace_bytes(m, 10000)
        assert a >= 256 and b >= a and b % 256 == 0
        assert b >= 256 + 12 * 10000


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4, -5, -6, -7, -8, -9):
        assert lib.mpt_status_string(code) != b"unknown status"
    assert lib.mpt_status_string(-77) == b"unknown status"


def test_host_side_validation_before_any_device_call(lib):
    P = ctypes.c_void_p
    dummy = P(4096)          # never dereferenced: every call below fails its host checks
    ws = P(256 * 16)
    # m out of range
    assert lib.mpt_build_weights(0, 1, 0, dummy, dummy, None, dummy, dummy, ws, 1 << 20, None) == -1
    assert b"m = 0" in lib.mpt_last_error()
    assert lib.mpt_solve_exact(31, dummy, dummy, dummy, None, ws, 1 << 20, None) == -1
    # NULL tables
    assert lib.mpt_solve_exact(4, None, dummy, dummy, None, ws, 1 << 20, None) == -1
    # workspace missing, misaligned, too small
    assert lib.mpt_solve_exact(4, dummy, dummy, dummy, None, None, 1 << 20, None) == -6
    assert lib.mpt_solve_exact(4, dummy, dummy, dummy, None, P(256 * 16 + 8), 1 << 20, None) == -6
    assert lib.mpt_solve_exact(4, dummy, dummy, dummy, None, ws, 16, None) == -6
    assert b"needs" in lib.mpt_last_error()
    # negative sizes
    assert lib.mpt_build_weights(3, -1, 0, dummy, dummy, None, dummy, dummy, ws, 1 << 20, None) == -1
    assert lib.mpt_extract_orders(3, 5, -2, dummy, dummy, dummy, dummy, dummy, ws, 1 << 20, None) == -1
    # missing request arrays when nnz > 0
    assert lib.mpt_build_weights(3, 5, 4, dummy, dummy, None, dummy, dummy, ws, 1 << 20, None) == -1


def test_header_declares_the_context_layer():
    """The calls and codes of the context layer: create / destroy, the
    workspace, the three phases on a context, table read-out, the state
    error and the internal error."""
    names = declared_functions()
    for n in ("mpt_create", "mpt_destroy", "mpt_set_workspace", "mpt_ctx_workspace_bytes", "mpt_set_option",
              "mpt_ctx_build_weights", "mpt_ctx_solve_exact", "mpt_ctx_extract_orders", "mpt_copy_table",
              "mpt_table_device", "mpt_status_string", "mpt_last_error"):
        assert n in names, n
    text = open(HEADER).read()
    for code, val in (("MPT_E_STATE", -7), ("MPT_E_INTERNAL", -9), ("MPT_E_DEVICE", -8)):
        assert re.search(rf"\b{code} = {val}\b", text), code
    assert re.search(r"#define MPT_MAX_M 30\b", text)


def test_context_host_side_validation(lib):
    """Context calls that must fail before any device work: NULL contexts,
    bad options, sizes out of range, phases out of order."""
    from paper_2609_13692_amd import mpt
    P = ctypes.c_void_p
    dummy = P(4096)
    assert lib.mpt_set_option(None, mpt.MPT_OPT_CHUNK_PAIRS, 1) == -1
    assert lib.mpt_set_workspace(None, None, 0) == -1
    assert lib.mpt_ctx_build_weights(None, 4, 1, 0, dummy, dummy, None) == -1
    assert lib.mpt_ctx_solve_exact(None, None, None, None) == -1
    assert lib.mpt_ctx_extract_orders(None, None) == -1
    assert lib.mpt_copy_table(None, 0, dummy, 8) == -1
    lib.mpt_destroy(None)                                     # NULL-safe
    assert lib.mpt_create(None, 0, None) == -1
    assert mpt.mpt_workspace_bytes(4, 0) > 0
    assert lib.mpt_ctx_workspace_bytes(None, 0, 1, 1) == 0
    assert lib.mpt_ctx_workspace_bytes(None, mpt.MPT_MAX_M + 1, 1, 1) == 0
    assert lib.mpt_ctx_workspace_bytes(None, 4, -1, 1) == 0
    a = lib.mpt_ctx_workspace_bytes(None, 20, 2000, 200)
    # the context's workspace holds W, C and split besides the phases' own
    assert a >= (20 << 20) + mpt.mpt_workspace_bytes(20, 200)


def test_context_creation_without_a_gpu(lib):
    """With no GPU present, mpt_create reports the device error (or an
    invalid device) and hands back no context."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    h = ctypes.c_void_p(1234)
    rc = lib.mpt_create(ctypes.byref(h), 0, None)
    assert rc in (-1, -8) and not h.value


def test_binding_refuses_host_tensors(lib):
    import torch
    from paper_2609_13692_amd import mpt
    W = torch.zeros(16, dtype=torch.int64)
    with pytest.raises(ValueError):
        mpt._ptr(W, torch.int64, 16, "W")
    with pytest.raises(TypeError):
        mpt._ptr(W.to(torch.int32), torch.int64, 16, "W")


def test_oracle_is_not_imported_by_the_product():
    """The product sources never reference the oracle."""
    pkg = os.path.join(ROOT, "paper_2609_13692_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in text and "from oracle" not in text, f
                assert "mpt_oracle" not in text, f


def test_greedy_workspace_and_host_validation(lib):
    from paper_2609_13692_amd import mpt
    P = ctypes.c_void_p
    dummy = P(4096)
    ws = P(256 * 16)
    assert mpt.mpt_greedy_workspace_bytes(0, 1, 1) == 0
    assert mpt.mpt_greedy_workspace_bytes(mpt.MPT_GREEDY_MAX_M + 1, 1, 1) == 0
    assert mpt.mpt_greedy_workspace_bytes(5, -1, 1) == 0
    for m, u, nnz in ((1, 0, 0), (100, 1000, 800), (4096, 12288, 32768)):
        a = mpt.mpt_greedy_workspace_bytes(m, u, nnz)
        assert a >= 8 * m * m + 8 * nnz and a % 256 == 0
    # m out of range, NULL outputs, workspace missing / misaligned / small
    assert lib.mpt_pair_weights(0, 1, 0, dummy, dummy, None, dummy, None, ws, 1 << 30, None) == -1
    assert lib.mpt_pair_weights(3, 5, 0, dummy, dummy, None, None, None, ws, 1 << 30, None) == -1
    assert lib.mpt_greedy_hierarchy(4, 5, 3, dummy, dummy, dummy, dummy, dummy, dummy, None, None, None,
                                    ws, 1 << 30, None) == -1
    assert lib.mpt_greedy_hierarchy(4, 5, 3, dummy, dummy, dummy, dummy, dummy, dummy, dummy, None, None,
                                    None, 1 << 30, None) == -6
    assert lib.mpt_greedy_hierarchy(4, 5, 3, dummy, dummy, dummy, dummy, dummy, dummy, dummy, None, None,
                                    ws, 64, None) == -6
    assert b"needs" in lib.mpt_last_error()
    assert lib.mpt_spanning_tree_bound(mpt.MPT_GREEDY_MAX_M + 1, dummy, dummy, ws, 1 << 20, None) == -1
    assert lib.mpt_spanning_tree_bound(4, dummy, dummy, P(256 * 16 + 8), 1 << 20, None) == -6
    assert lib.mpt_spanning_tree_bound(4, None, dummy, ws, 1 << 20, None) == -1


def test_layout_workspace_and_host_validation(lib):
    from paper_2609_13692_amd import mpt
    P = ctypes.c_void_p
    dummy = P(4096)
    ws = P(256 * 16)
    assert mpt.mpt_layout_workspace_bytes(0, 1, 1) == 0
    assert mpt.mpt_layout_workspace_bytes(4, 5, 3, mpt.MPT_CACHE_MAX_CONFIGS + 1) == 0
    a = mpt.mpt_layout_workspace_bytes(4096, 12288, 32768, 0)
    b = mpt.mpt_layout_workspace_bytes(4096, 12288, 32768, 30)
    assert a % 256 == 0 and b > a + 30 * 4 * 32768
    # bad order kind, NULL outputs, missing workspace, bad configuration count
    assert lib.mpt_global_order_layout(3, 5, 0, dummy, None, 7, None, ws, 1 << 30, None) == -1
    assert lib.mpt_layout_cost(3, 5, 4, dummy, dummy, dummy, None, None, ws, 1 << 30, None) == -1
    assert lib.mpt_layout_cost(3, 5, 4, dummy, dummy, dummy, None, dummy, None, 1 << 30, None) == -6
    win = (ctypes.c_int64 * 1)(1)
    cap = (ctypes.c_int64 * 1)(-5)
    out = (ctypes.c_int64 * 1)()
    assert lib.mpt_cache_simulate(3, 5, 4, dummy, dummy, dummy, 0, win, cap, out, None, ws, 1 << 30, None) == -1
    assert lib.mpt_cache_simulate(3, 5, 4, dummy, dummy, dummy, 1, win, cap, out, None, ws, 1 << 30, None) == -1
    assert b"negative" in lib.mpt_last_error()
