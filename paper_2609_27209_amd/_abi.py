"""ctypes declarations of the C ABI in include/erc.h (argument marshalling only).

Every function here has the name of the C entry point it calls.  Status codes other
than ERC_OK raise ``ErcError`` (``ErcNotConverged`` for ERC_E_NOT_CONVERGED, which
carries the solve info).  The shared library must have been built (``build.py``);
there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, byref, c_char_p, c_double, c_float, c_int, c_int32, c_int64, c_size_t, c_uint32, c_uint64, c_void_p

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liberc.so")

ERC_OK = 0
ERC_E_INVALID_ARG = 1
ERC_E_INVALID_GRAPH = 2
ERC_E_WORKSPACE = 3
ERC_E_DEVICE = 4
ERC_E_NOT_CONVERGED = 5
ERC_E_NUMERIC = 6
ERC_E_STATE = 7
ERC_E_HOST = 8

ERC_F32 = 0
ERC_F64 = 1
ERC_NODES = 0
ERC_EDGES = 1
ERC_ACCUMULATE = 1
ERC_PROFILE_SPMM = 2
ERC_JACOBI = 4
ERC_NO_GRAPH = 8
ERC_EARLY_STOP = 16


class erc_graph_desc(ctypes.Structure):
    _fields_ = [("n", c_int64), ("rowptr", c_void_p), ("col", c_void_p), ("w", c_void_p),
                ("w_dtype", c_int), ("solve_dtype", c_int)]


class erc_solve_params(ctypes.Structure):
    _fields_ = [("K_total", c_int32), ("k_block", c_int32), ("col_begin", c_int32),
                ("col_end", c_int32), ("delta", c_double), ("tol", c_double),
                ("max_iter", c_int32), ("check_every", c_int32), ("seed", c_uint64),
                ("flags", c_uint32)]


class erc_solve_info(ctypes.Structure):
    _fields_ = [("blocks", c_int32), ("iters_max", c_int32), ("cols_unconverged", c_int32),
                ("breakdowns", c_int32), ("iters_total", c_int64), ("launches", c_int64),
                ("nonpositive", c_int64), ("max_final_relres", c_double), ("ms_rhs", c_float),
                ("ms_cg", c_float), ("ms_accum", c_float), ("ms_total", c_float),
                ("ms_spmm", c_float), ("spmm_timed", c_int64), ("spmm_full", c_int64),
                ("bytes_model", c_double)]

    def as_dict(self) -> dict:
        return {name: getattr(self, name) for name, _ in self._fields_}


class ErcError(RuntimeError):
    def __init__(self, status: int, message: str, info=None):
        super().__init__(f"{_status_name(status)}: {message}")
        self.status = status
        self.info = info


class ErcNotConverged(ErcError):
    pass


_NAMES = {0: "ERC_OK", 1: "ERC_E_INVALID_ARG", 2: "ERC_E_INVALID_GRAPH", 3: "ERC_E_WORKSPACE",
          4: "ERC_E_DEVICE", 5: "ERC_E_NOT_CONVERGED", 6: "ERC_E_NUMERIC", 7: "ERC_E_STATE",
          8: "ERC_E_HOST"}


def _status_name(s: int) -> str:
    return _NAMES.get(int(s), f"status {s}")


# (name, argtypes) of every exported entry point of include/erc.h
_SIGNATURES = {
    "erc_validate": [POINTER(erc_graph_desc), POINTER(c_int64)],
    "erc_graph_bytes": [POINTER(erc_graph_desc), POINTER(c_size_t)],
    "erc_create": [POINTER(erc_graph_desc), c_void_p, c_size_t, c_void_p, POINTER(c_void_p)],
    "erc_num_nodes": [c_void_p, POINTER(c_int64)],
    "erc_num_edges": [c_void_p, POINTER(c_int64)],
    "erc_edge_endpoints": [c_void_p, c_void_p, c_void_p, c_void_p],
    "erc_destroy": [c_void_p],
    "erc_workspace_bytes": [c_void_p, c_int32, POINTER(c_size_t)],
    "erc_resistance": [c_void_p, POINTER(erc_solve_params), c_void_p, c_size_t, c_void_p,
                       POINTER(erc_solve_info), c_void_p],
    "erc_curvature": [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p],
    "erc_sampling_scratch_bytes": [c_void_p, POINTER(c_size_t)],
    "erc_sampling_probs": [c_void_p, c_void_p, c_double, c_void_p, c_size_t, c_void_p, c_void_p,
                           c_void_p],
    "erc_sampling_probs_static": [c_void_p, c_void_p, c_double, c_void_p, c_void_p, c_void_p],
    "erc_draw_scratch_bytes": [c_void_p, c_int, POINTER(c_size_t)],
    "erc_draw": [c_void_p, c_int, c_void_p, c_int64, c_uint64, c_void_p, c_size_t, c_void_p,
                 c_void_p],
    "erc_subgraph_scratch_bytes": [c_void_p, POINTER(c_size_t)],
    "erc_subgraph": [c_void_p, c_int, c_void_p, c_int64, c_void_p, c_size_t, c_void_p, c_void_p,
                     c_void_p, c_void_p, POINTER(c_int64), c_void_p],
    "erc_probe_out_bytes": [c_int64, c_int32, POINTER(c_size_t)],
    "erc_probe_gather": [c_void_p, c_int64, c_void_p, c_int64, c_int32, c_void_p, c_void_p],
    "erc_probe_gather_sliced": [c_void_p, c_int64, c_void_p, c_int64, c_int32, c_int32, c_void_p,
                                c_void_p],
    "erc_status_string": [c_int],
    "erc_last_error": [],
    "erc_debug_check_plan": [POINTER(erc_graph_desc)],
    "erc_debug_edge_ids": [c_void_p, c_void_p, c_void_p],
    "erc_debug_rhs": [c_void_p, c_int32, c_int32, c_int32, c_uint64, c_void_p, c_void_p, c_size_t,
                      c_void_p],
    "erc_debug_spmm": [c_void_p, c_double, c_int32, c_void_p, c_void_p, c_void_p, c_size_t,
                       c_void_p],
    "erc_debug_solve_block": [c_void_p, POINTER(erc_solve_params), c_int32, c_int32, c_void_p,
                              c_size_t, c_void_p, POINTER(c_int32), c_void_p],
}

_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the shared library once; raises ImportError if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2609_27209_amd.build` "
                          "(there is no CPU fallback)")
    lib = ctypes.CDLL(path)
    for name, args in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = c_char_p if name in ("erc_status_string", "erc_last_error") else c_int
    _lib = lib
    return lib


def exported_names():
    return list(_SIGNATURES)


def _check(status: int, info=None) -> int:
    if status == ERC_OK:
        return status
    msg = load().erc_last_error().decode(errors="replace")
    cls = ErcNotConverged if status == ERC_E_NOT_CONVERGED else ErcError
    raise cls(status, msg, info)


# ---- thin wrappers, one per entry point ----------------------------------------------

def erc_validate(desc: erc_graph_desc) -> int:
    m = c_int64(0)
    _check(load().erc_validate(byref(desc), byref(m)))
    return m.value


def erc_graph_bytes(desc: erc_graph_desc) -> int:
    b = c_size_t(0)
    _check(load().erc_graph_bytes(byref(desc), byref(b)))
    return b.value


def erc_create(desc: erc_graph_desc, dev_mem: int, nbytes: int, stream: int) -> int:
    h = c_void_p(0)
    _check(load().erc_create(byref(desc), c_void_p(dev_mem), nbytes, c_void_p(stream), byref(h)))
    return h.value


def erc_num_nodes(h: int) -> int:
    n = c_int64(0)
    _check(load().erc_num_nodes(c_void_p(h), byref(n)))
    return n.value


def erc_num_edges(h: int) -> int:
    m = c_int64(0)
    _check(load().erc_num_edges(c_void_p(h), byref(m)))
    return m.value


def erc_edge_endpoints(h: int, u_dev: int, v_dev: int, stream: int) -> None:
    _check(load().erc_edge_endpoints(c_void_p(h), c_void_p(u_dev), c_void_p(v_dev), c_void_p(stream)))


def erc_destroy(h: int) -> None:
    _check(load().erc_destroy(c_void_p(h)))


def erc_workspace_bytes(h: int, k_block: int) -> int:
    b = c_size_t(0)
    _check(load().erc_workspace_bytes(c_void_p(h), k_block, byref(b)))
    return b.value


def erc_resistance(h: int, params: erc_solve_params, ws: int, ws_bytes: int, R_dev: int,
                   stream: int, raise_not_converged: bool = True) -> erc_solve_info:
    info = erc_solve_info()
    st = load().erc_resistance(c_void_p(h), byref(params), c_void_p(ws), ws_bytes, c_void_p(R_dev),
                               byref(info), c_void_p(stream))
    if st == ERC_E_NOT_CONVERGED and not raise_not_converged:
        return info
    _check(st, info)
    return info


def erc_curvature(h: int, R_dev: int, p_dev: int, kappa_dev: int, stream: int) -> None:
    _check(load().erc_curvature(c_void_p(h), c_void_p(R_dev), c_void_p(p_dev), c_void_p(kappa_dev),
                                c_void_p(stream)))


def erc_sampling_scratch_bytes(h: int) -> int:
    b = c_size_t(0)
    _check(load().erc_sampling_scratch_bytes(c_void_p(h), byref(b)))
    return b.value


def erc_sampling_probs(h: int, kappa_dev: int, eta: float, scratch: int, scratch_bytes: int,
                       pn_dev: int, pe_dev: int, stream: int) -> None:
    _check(load().erc_sampling_probs(c_void_p(h), c_void_p(kappa_dev), eta, c_void_p(scratch),
                                     scratch_bytes, c_void_p(pn_dev), c_void_p(pe_dev),
                                     c_void_p(stream)))


def erc_sampling_probs_static(h: int, kappa_dev: int, eta: float, pn_dev: int, pe_dev: int,
                              stream: int) -> None:
    _check(load().erc_sampling_probs_static(c_void_p(h), c_void_p(kappa_dev), eta,
                                            c_void_p(pn_dev), c_void_p(pe_dev), c_void_p(stream)))


def erc_probe_out_bytes(count: int, row_bytes: int) -> int:
    b = c_size_t(0)
    _check(load().erc_probe_out_bytes(count, row_bytes, byref(b)))
    return b.value


def erc_probe_gather(idx_dev: int, count: int, table_dev: int, rows: int, row_bytes: int,
                     out_dev: int, stream: int) -> None:
    _check(load().erc_probe_gather(c_void_p(idx_dev), count, c_void_p(table_dev), rows, row_bytes,
                                   c_void_p(out_dev), c_void_p(stream)))


def erc_probe_gather_sliced(idx_dev: int, count: int, table_dev: int, rows: int, row_bytes: int,
                            slices: int, out_dev: int, stream: int) -> None:
    _check(load().erc_probe_gather_sliced(c_void_p(idx_dev), count, c_void_p(table_dev), rows,
                                          row_bytes, slices, c_void_p(out_dev),
                                          c_void_p(stream)))


def erc_draw_scratch_bytes(h: int, items: int) -> int:
    b = c_size_t(0)
    _check(load().erc_draw_scratch_bytes(c_void_p(h), items, byref(b)))
    return b.value


def erc_draw(h: int, items: int, prob_dev: int, draws: int, seed: int, scratch: int,
             scratch_bytes: int, idx_dev: int, stream: int) -> None:
    _check(load().erc_draw(c_void_p(h), items, c_void_p(prob_dev), draws, seed,
                           c_void_p(scratch), scratch_bytes, c_void_p(idx_dev), c_void_p(stream)))


def erc_subgraph_scratch_bytes(h: int) -> int:
    b = c_size_t(0)
    _check(load().erc_subgraph_scratch_bytes(c_void_p(h), byref(b)))
    return b.value


def erc_subgraph(h: int, items: int, idx_dev: int, count: int, scratch: int, scratch_bytes: int,
                 nodes_dev: int, edges_dev: int, u_dev: int, v_dev: int, stream: int):
    counts = (c_int64 * 2)()
    _check(load().erc_subgraph(c_void_p(h), items, c_void_p(idx_dev), count, c_void_p(scratch),
                               scratch_bytes, c_void_p(nodes_dev), c_void_p(edges_dev),
                               c_void_p(u_dev), c_void_p(v_dev), counts, c_void_p(stream)))
    return int(counts[0]), int(counts[1])


def erc_status_string(status: int) -> str:
    return load().erc_status_string(status).decode()


def erc_last_error() -> str:
    return load().erc_last_error().decode(errors="replace")


def erc_debug_check_plan(desc: erc_graph_desc) -> None:
    _check(load().erc_debug_check_plan(byref(desc)))


def erc_debug_edge_ids(h: int, eid_dev: int, stream: int) -> None:
    _check(load().erc_debug_edge_ids(c_void_p(h), c_void_p(eid_dev), c_void_p(stream)))


def erc_debug_rhs(h: int, K: int, col0: int, ncols: int, seed: int, Y_dev: int, ws: int,
                  ws_bytes: int, stream: int) -> None:
    _check(load().erc_debug_rhs(c_void_p(h), K, col0, ncols, seed, c_void_p(Y_dev), c_void_p(ws),
                                ws_bytes, c_void_p(stream)))


def erc_debug_spmm(h: int, delta: float, ncols: int, X_dev: int, Y_dev: int, ws: int,
                   ws_bytes: int, stream: int) -> None:
    _check(load().erc_debug_spmm(c_void_p(h), delta, ncols, c_void_p(X_dev), c_void_p(Y_dev),
                                 c_void_p(ws), ws_bytes, c_void_p(stream)))


def erc_debug_solve_block(h: int, params: erc_solve_params, col0: int, ncols: int, ws: int,
                          ws_bytes: int, Z_dev: int, stream: int, raise_not_converged=True):
    iters = (c_int32 * ncols)()
    st = load().erc_debug_solve_block(c_void_p(h), byref(params), col0, ncols, c_void_p(ws),
                                      ws_bytes, c_void_p(Z_dev), iters, c_void_p(stream))
    if not (st == ERC_E_NOT_CONVERGED and not raise_not_converged):
        _check(st)
    return list(iters), st
