"""MI355X resistance-curvature library: Python binding of the C ABI in include/erc.h.

PyTorch provides device memory and the current stream; every step of the computation
runs in the HIP kernels of ``liberc.so``.  If the library is not built, importing the
binding raises ImportError: there is no CPU fallback.

    import paper_2609_27209_amd as erc
    g = erc.Graph(rowptr, col, w, solve_dtype="f32")      # numpy CSR on the host
    R, info = g.resistance(K=256, k_block=64, delta=1e-4, tol=1e-5, seed=105)
    p, kappa = g.curvature(R)
    pn, pe = g.sampling_probs(kappa, eta=1e-12)
"""
from __future__ import annotations

import numpy as np

from . import _abi
from ._abi import (  # noqa: F401
    ERC_ACCUMULATE, ERC_F32, ERC_F64, ERC_PROFILE_SPMM, ErcError, ErcNotConverged,
    erc_solve_info, erc_solve_params,
)

__all__ = ["Graph", "ErcError", "ErcNotConverged", "resistance_curvature", "load_library"]


def load_library():
    return _abi.load()


def _torch():
    import torch

    if not torch.cuda.is_available():
        raise RuntimeError("no GPU visible: the library runs only on an MI355X (gfx950)")
    return torch


def _dtype_code(name: str) -> int:
    return {"f32": ERC_F32, "f64": ERC_F64}[name]


def _desc(rowptr, col, w, solve_dtype):
    rowptr = np.ascontiguousarray(rowptr, dtype=np.int64)
    col = np.ascontiguousarray(col, dtype=np.int32)
    keep = [rowptr, col]
    wptr, wcode = None, ERC_F32
    if w is not None:
        w = np.ascontiguousarray(w)
        if w.dtype == np.float32:
            wcode = ERC_F32
        else:
            w = w.astype(np.float64, copy=False)
            wcode = ERC_F64
        keep.append(w)
        wptr = w.ctypes.data
    d = _abi.erc_graph_desc(n=rowptr.size - 1, rowptr=rowptr.ctypes.data, col=col.ctypes.data,
                            w=wptr, w_dtype=wcode, solve_dtype=_dtype_code(solve_dtype))
    return d, keep


def _items(items) -> int:
    if items in ("nodes", _abi.ERC_NODES):
        return _abi.ERC_NODES
    if items in ("edges", _abi.ERC_EDGES):
        return _abi.ERC_EDGES
    raise ValueError(f"items must be 'nodes' or 'edges', not {items!r}")


def validate(rowptr, col, w=None, solve_dtype="f32") -> int:
    """Host-only check of a CSR graph; returns the number of undirected edges."""
    d, _keep = _desc(rowptr, col, w, solve_dtype)
    return _abi.erc_validate(d)


class Graph:
    """A graph copied to the GPU by erc_create, with torch-allocated buffers."""

    def __init__(self, rowptr, col, w=None, solve_dtype: str = "f32", device=None):
        torch = _torch()
        _abi.load()
        self.torch = torch
        self.device = torch.device("cuda" if device is None else device)
        self.solve_dtype = solve_dtype
        self.vdtype = torch.float32 if solve_dtype == "f32" else torch.float64
        d, keep = _desc(rowptr, col, w, solve_dtype)
        nbytes = _abi.erc_graph_bytes(d)
        self._gmem = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        assert self._gmem.data_ptr() % 256 == 0
        with torch.cuda.device(self.device):
            self.handle = _abi.erc_create(d, self._gmem.data_ptr(), nbytes, self._stream())
        del keep
        self.n = _abi.erc_num_nodes(self.handle)
        self.m = _abi.erc_num_edges(self.handle)
        self.nnz = int(np.asarray(rowptr)[-1])
        self._ws = {}
        self._scratch = None
        self._scratches = {}

    def _stream(self) -> int:
        return self.torch.cuda.current_stream(self.device).cuda_stream

    def close(self):
        if getattr(self, "handle", None):
            _abi.erc_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace(self, k_block: int):
        nb = _abi.erc_workspace_bytes(self.handle, k_block)
        ws = self._ws.get(nb)
        if ws is None:
            ws = self.torch.empty(nb, dtype=self.torch.uint8, device=self.device)
            self._ws = {nb: ws}
        return ws

    @staticmethod
    def params(K, k_block, delta, tol, max_iter=10000, seed=0, col_begin=0, col_end=None,
               accumulate=False, check_every=0, profile=False, precond="none", graph=True,
               early_stop=False):
        if precond not in ("none", "jacobi"):
            raise ValueError(f"precond must be 'none' or 'jacobi', not {precond!r}")
        flags = ((ERC_ACCUMULATE if accumulate else 0) | (ERC_PROFILE_SPMM if profile else 0)
                 | (_abi.ERC_JACOBI if precond == "jacobi" else 0)
                 | (0 if graph else _abi.ERC_NO_GRAPH)
                 | (_abi.ERC_EARLY_STOP if early_stop else 0))
        return _abi.erc_solve_params(
            K_total=K, k_block=k_block, col_begin=col_begin, col_end=K if col_end is None else col_end,
            delta=delta, tol=tol, max_iter=max_iter, check_every=check_every, seed=seed,
            flags=flags)

    def resistance(self, K, k_block, delta, tol, max_iter=10000, seed=0, col_begin=0, col_end=None,
                   out=None, accumulate=False, check_every=0, raise_not_converged=True,
                   profile=False, precond="none", graph=True, early_stop=False):
        """R (torch fp64, m) over columns [col_begin, col_end) and the solve info dict.
        precond="jacobi" selects the Jacobi-preconditioned CG variant; graph=False
        enqueues every iteration as separate launches instead of replaying a captured
        group of iterations; early_stop=True enqueues the early stopping test after
        every update whatever the graph's size (ERC_EARLY_STOP)."""
        torch = self.torch
        R = out if out is not None else torch.empty(max(self.m, 1), dtype=torch.float64,
                                                    device=self.device)
        ws = self.workspace(k_block)
        prm = self.params(K, k_block, delta, tol, max_iter, seed, col_begin, col_end, accumulate,
                          check_every, profile, precond, graph, early_stop)
        info = _abi.erc_resistance(self.handle, prm, ws.data_ptr(), ws.numel(), R.data_ptr(),
                                   self._stream(), raise_not_converged)
        return R[: self.m], info.as_dict()

    def curvature(self, R):
        torch = self.torch
        p = torch.empty(self.n, dtype=torch.float64, device=self.device)
        kappa = torch.empty(max(self.m, 1), dtype=torch.float64, device=self.device)
        _abi.erc_curvature(self.handle, R.data_ptr(), p.data_ptr(), kappa.data_ptr(), self._stream())
        return p, kappa[: self.m]

    def sampling_probs(self, kappa, eta=1e-12):
        torch = self.torch
        if self._scratch is None:
            nb = _abi.erc_sampling_scratch_bytes(self.handle)
            self._scratch = torch.empty(nb, dtype=torch.uint8, device=self.device)
        pn = torch.empty(self.n, dtype=torch.float64, device=self.device)
        pe = torch.empty(max(self.m, 1), dtype=torch.float64, device=self.device)
        _abi.erc_sampling_probs(self.handle, kappa.data_ptr(), eta, self._scratch.data_ptr(),
                                self._scratch.numel(), pn.data_ptr(), pe.data_ptr(), self._stream())
        return pn, pe[: self.m]

    def _scratch_of(self, key, nbytes):
        buf = self._scratches.get(key)
        if buf is None or buf.numel() < nbytes:
            buf = self.torch.empty(max(nbytes, 256), dtype=self.torch.uint8, device=self.device)
            self._scratches[key] = buf
        return buf

    def draw(self, items, prob, draws, seed):
        """`draws` indices (torch int64) drawn from the node ("nodes") or edge ("edges")
        distribution `prob` (device fp64, as sampling_probs returns it)."""
        it = _items(items)
        prob = prob.to(self.device, self.torch.float64).contiguous()
        need = self.n if it == _abi.ERC_NODES else self.m
        if prob.numel() != need:
            raise ValueError(f"prob has {prob.numel()} entries, expected {need}")
        sc = self._scratch_of(("draw", it), _abi.erc_draw_scratch_bytes(self.handle, it))
        idx = self.torch.empty(max(draws, 1), dtype=self.torch.int64, device=self.device)
        _abi.erc_draw(self.handle, it, prob.data_ptr(), draws, seed, sc.data_ptr(), sc.numel(),
                      idx.data_ptr(), self._stream())
        return idx[:draws]

    def subgraph(self, items, idx):
        """Subgraph from drawn indices: induced on the drawn nodes ("nodes"), or the drawn
        edges and their endpoints ("edges").  Returns the kept node ids, the kept edge ids
        and the kept edges' endpoints renumbered to positions in the node list."""
        torch = self.torch
        it = _items(items)
        idx = idx.to(self.device, torch.int64).contiguous()
        sc = self._scratch_of("subgraph", _abi.erc_subgraph_scratch_bytes(self.handle))
        nodes = torch.empty(max(self.n, 1), dtype=torch.int32, device=self.device)
        edges = torch.empty(max(self.m, 1), dtype=torch.int64, device=self.device)
        u = torch.empty(max(self.m, 1), dtype=torch.int32, device=self.device)
        v = torch.empty(max(self.m, 1), dtype=torch.int32, device=self.device)
        ns, ms = _abi.erc_subgraph(self.handle, it, idx.data_ptr(), idx.numel(), sc.data_ptr(),
                                   sc.numel(), nodes.data_ptr(), edges.data_ptr(), u.data_ptr(),
                                   v.data_ptr(), self._stream())
        return {"nodes": nodes[:ns], "edges": edges[:ms], "u": u[:ms], "v": v[:ms]}

    def edge_endpoints(self):
        torch = self.torch
        u = torch.empty(max(self.m, 1), dtype=torch.int32, device=self.device)
        v = torch.empty(max(self.m, 1), dtype=torch.int32, device=self.device)
        _abi.erc_edge_endpoints(self.handle, u.data_ptr(), v.data_ptr(), self._stream())
        return u[: self.m], v[: self.m]

    # ---- test hooks ------------------------------------------------------------------
    def debug_edge_ids(self):
        e = self.torch.empty(max(self.nnz, 1), dtype=self.torch.int32, device=self.device)
        _abi.erc_debug_edge_ids(self.handle, e.data_ptr(), self._stream())
        return e[: self.nnz]

    def debug_rhs(self, K, col0, ncols, seed):
        Y = self.torch.empty((self.n, ncols), dtype=self.vdtype, device=self.device)
        ws = self.workspace(ncols)
        _abi.erc_debug_rhs(self.handle, K, col0, ncols, seed, Y.data_ptr(), ws.data_ptr(),
                           ws.numel(), self._stream())
        return Y

    def debug_spmm(self, delta, X):
        X = X.to(self.device, self.vdtype).contiguous()
        Y = self.torch.empty_like(X)
        ws = self.workspace(X.shape[1])
        _abi.erc_debug_spmm(self.handle, delta, X.shape[1], X.data_ptr(), Y.data_ptr(),
                            ws.data_ptr(), ws.numel(), self._stream())
        return Y

    def debug_solve_block(self, K, k_block, delta, tol, seed, col0, ncols, max_iter=10000,
                          raise_not_converged=True, precond="none"):
        Z = self.torch.empty((self.n, ncols), dtype=self.vdtype, device=self.device)
        ws = self.workspace(k_block)
        prm = self.params(K, k_block, delta, tol, max_iter, seed, precond=precond)
        iters, st = _abi.erc_debug_solve_block(self.handle, prm, col0, ncols, ws.data_ptr(),
                                               ws.numel(), Z.data_ptr(), self._stream(),
                                               raise_not_converged)
        return Z, iters, st


def resistance_curvature(rowptr, col, w, K, k_block, delta, tol, seed, solve_dtype="f32",
                         max_iter=10000, eta=1e-12):
    """Whole path on one GPU: R, p, kappa, node and edge sampling probabilities."""
    g = Graph(rowptr, col, w, solve_dtype)
    R, info = g.resistance(K, k_block, delta, tol, max_iter, seed)
    p, kappa = g.curvature(R)
    pn, pe = g.sampling_probs(kappa, eta)
    return {"R": R, "p": p, "kappa": kappa, "node_prob": pn, "edge_prob": pe, "info": info,
            "graph": g}
