"""Host-side tests of the C ABI (no GPU needed): the shared library loads and exports
every function include/erc.h declares, the binding declares the same set, graph
validation returns the documented status codes, and the work plan covers every stored
entry exactly once (erc_debug_check_plan)."""
import ctypes
import os
import re

import numpy as np
import pytest

import gen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "erc.h")

E = pytest.importorskip("paper_2609_27209_amd")
from paper_2609_27209_amd import _abi  # noqa: E402


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(?:erc_status|const char\s*\*)\s*(erc_\w+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = ctypes.CDLL(_abi.LIB_PATH)
    names = declared_functions()
    assert len(names) >= 19
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(_abi.exported_names()) == names


def _desc(g, dtype="f32", w=None):
    return E._desc(g.rowptr, g.col, g.w if w is None else w, dtype)


def _status(fn, *args):
    try:
        fn(*args)
        return _abi.ERC_OK
    except _abi.ErcError as e:
        return e.status


def test_validate_accepts_and_counts_edges():
    for g in [gen.path_graph(5), gen.make_graph("er2k"), gen.make_graph("sbm20k"),
              gen.from_edges(6, [0, 2], [1, 3])]:
        d, keep = _desc(g)
        assert _abi.erc_validate(d) == g.m
        assert _abi.erc_graph_bytes(d) > 0


def _raw_desc(n, rowptr, col, w=None, wdt=_abi.ERC_F32, sdt=_abi.ERC_F32):
    rowptr = np.ascontiguousarray(rowptr, np.int64)
    col = np.ascontiguousarray(col, np.int32)
    keep = [rowptr, col]
    wp = None
    if w is not None:
        w = np.ascontiguousarray(w)
        keep.append(w)
        wp = w.ctypes.data
    d = _abi.erc_graph_desc(n=n, rowptr=rowptr.ctypes.data, col=col.ctypes.data, w=wp,
                            w_dtype=wdt, solve_dtype=sdt)
    return d, keep


@pytest.mark.parametrize("case,expect", [
    ("asymmetric", _abi.ERC_E_INVALID_GRAPH),
    ("self_loop", _abi.ERC_E_INVALID_GRAPH),
    ("unsorted", _abi.ERC_E_INVALID_GRAPH),
    ("duplicate", _abi.ERC_E_INVALID_GRAPH),
    ("out_of_range", _abi.ERC_E_INVALID_GRAPH),
    ("rowptr_decreasing", _abi.ERC_E_INVALID_GRAPH),
    ("rowptr_start", _abi.ERC_E_INVALID_GRAPH),
    ("negative_weight", _abi.ERC_E_INVALID_GRAPH),
    ("nan_weight", _abi.ERC_E_INVALID_GRAPH),
    ("asymmetric_weight", _abi.ERC_E_INVALID_GRAPH),
    ("zero_nodes", _abi.ERC_E_INVALID_ARG),
    ("n_at_limit", _abi.ERC_E_INVALID_ARG),
    ("nnz_at_limit", _abi.ERC_E_INVALID_GRAPH),
    ("bad_solve_dtype", _abi.ERC_E_INVALID_ARG),
    ("bad_weight_dtype", _abi.ERC_E_INVALID_ARG),
])
def test_validate_rejects(case, expect):
    # base graph: path 0-1-2 (rows 0:[1] 1:[0,2] 2:[1])
    n, rp, col, w = 3, [0, 1, 3, 4], [1, 0, 2, 1], np.array([1.0, 1.0, 2.0, 2.0], np.float32)
    if case == "asymmetric":
        rp, col, w = [0, 1, 2, 2], [1, 2], w[:2]
    elif case == "self_loop":
        rp, col, w = [0, 2, 4, 5], [0, 1, 0, 2, 1], np.ones(5, np.float32)
    elif case == "unsorted":
        col = [1, 2, 0, 1]
    elif case == "duplicate":
        rp, col, w = [0, 2, 4, 5], [1, 1, 0, 0, 1], np.ones(5, np.float32)
    elif case == "out_of_range":
        col = [1, 0, 3, 1]
    elif case == "rowptr_decreasing":
        rp = [0, 3, 1, 4]
    elif case == "rowptr_start":
        rp = [1, 1, 3, 4]
    elif case == "negative_weight":
        w = np.array([-1.0, -1.0, 2.0, 2.0], np.float32)
    elif case == "nan_weight":
        w = np.array([np.nan, np.nan, 2.0, 2.0], np.float32)
    elif case == "asymmetric_weight":
        w = np.array([1.0, 1.5, 2.0, 2.0], np.float32)
    elif case == "zero_nodes":
        n, rp, col, w = 0, [0], [0], None
    elif case == "n_at_limit":
        # n = 2^31 is refused before rowptr is read
        n, rp, col, w = 1 << 31, [0], [0], None
    elif case == "nnz_at_limit":
        # rowptr[n] = 2^31 is refused before col is read
        n, rp, col, w = 1, [0, 1 << 31], [0], None
    d, keep = _raw_desc(n, rp, col, w,
                        sdt=7 if case == "bad_solve_dtype" else _abi.ERC_F32,
                        wdt=7 if case == "bad_weight_dtype" else _abi.ERC_F32)
    assert _status(_abi.erc_validate, d) == expect
    assert _abi.erc_last_error() != ""


def test_validate_fp64_weights_and_status_strings():
    g = gen.erdos_renyi(50, 0.1, 2, weighted=True)
    d, keep = _raw_desc(g.n, g.rowptr, g.col, g.w.astype(np.float64), wdt=_abi.ERC_F64,
                        sdt=_abi.ERC_F64)
    assert _abi.erc_validate(d) == g.m
    assert _abi.erc_status_string(_abi.ERC_OK) == "ok"
    assert _abi.erc_status_string(_abi.ERC_E_NOT_CONVERGED) == "not converged"
    assert _abi.erc_status_string(_abi.ERC_E_HOST) == "host allocation or thread failure"


@pytest.mark.parametrize("name", ["er2k", "sbm20k", "cl170k"])
def test_work_plan_covers_every_entry(name):
    g = gen.make_graph(name)
    d, keep = _desc(g)
    _abi.erc_debug_check_plan(d)


def test_work_plan_hub_and_isolated_cases():
    # a 20k-leaf star (a row split over several blocks), isolated nodes, a two-node graph
    # ... and a 1.2M-node path, which has enough rows per wave for the larger SpMM grid
    for g in [gen.star_graph(20001), gen.from_edges(10, [0, 1], [1, 2]),
              gen.from_edges(2, [0], [1]), gen.chung_lu(5000, 2.1, 3.0, 60000, seed=4),
              gen.path_graph(1_200_001)]:
        d, keep = _desc(g, "f64")
        _abi.erc_debug_check_plan(d)


def test_product_path_has_no_cpu_fallback(monkeypatch):
    # a missing library is an ImportError, not a silent CPU path
    monkeypatch.setattr(_abi, "_lib", None)
    with pytest.raises(ImportError):
        _abi.load(os.path.join(ROOT, "no_such_dir", "liberc.so"))
