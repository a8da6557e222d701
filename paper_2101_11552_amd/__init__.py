"""Python binding of libtfg.so, the MI355X (gfx950) graph map-reduce hot path.

Argument marshalling only: every function here takes torch tensors on a ROCm
device, allocates outputs and workspaces with torch, and calls the C entry
point of the same name in ``include/tfg.h`` on torch's current stream. All
computation happens in the HIP kernels of the library; there is no fallback.

Index tensors may be int32 or int64. Features, weights and scores are
float32. ``edge_index`` has shape [2, E] (row 0 sources, row 1 targets).
"""

from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "TfgError", "TfgIndexError", "TfgValueError", "Graph",
    "tfg_graph_bytes", "tfg_graph_create", "tfg_graph_create_transposed", "tfg_graph_csr",
    "tfg_edge_reorder", "tfg_graph_segments", "tfg_check",
    "tfg_gcn_norm",
    "tfg_aggregate_ws_bytes", "tfg_aggregate", "tfg_aggregate_noalloc", "tfg_aggregate_backward",
    "tfg_gat_edge_scores", "tfg_segment_softmax", "tfg_segment_softmax_backward",
    "tfg_segment_pool", "tfg_segment_pool_backward",
    "tfg_batch_graphs", "tfg_batch_graphs_totals", "tfg_propagate", "tfg_gat_aggregate",
    "tfg_edge_dot_scores", "tfg_gat_dot_aggregate",
    "tfg_gat_graph_scores", "tfg_segment_softmax_graph", "tfg_segment_softmax_graph_backward",
    "library_path", "load",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtfg.so")

TFG_OK, TFG_ERR_INVALID_ARG, TFG_ERR_INDEX_RANGE, TFG_ERR_UNSORTED = 0, 1, 2, 3
TFG_ERR_TOO_LARGE, TFG_ERR_WORKSPACE, TFG_ERR_HIP = 4, 5, 6
_REDUCE = {"sum": 0, "mean": 1, "max": 2}
_ORDER = {"coo": 0, "csr": 1, "csr_t": 2}

_lib = None


class TfgError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


class TfgIndexError(TfgError, IndexError):
    pass


class TfgValueError(TfgError, ValueError):
    pass


def library_path() -> str:
    return LIB_PATH


def load():
    """Loads libtfg.so (built by ``paper_2101_11552_amd.build``); raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run paper_2101_11552_amd/build.py "
                           "(or __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    i64, sz, p, i32 = ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int
    ci = ctypes.c_int
    sig = {
        "tfg_status_string": (ctypes.c_char_p, [ci]),
        "tfg_last_error": (ctypes.c_char_p, []),
        "tfg_abi_version": (ci, []),
        "tfg_graph_bytes": (ci, [i64, i64, i64, ci, ci, ctypes.POINTER(sz), ctypes.POINTER(sz)]),
        "tfg_graph_create": (ci, [p, ci, i64, i64, i64, ci, ci, p, sz, p, sz, p,
                                  ctypes.POINTER(p)]),
        "tfg_graph_csr": (ci, [p, p, p, p, p]),
        "tfg_graph_segments": (ci, [p, p, p]),
        "tfg_graph_info": (ci, [p] + [ctypes.POINTER(i64)] * 7),
        "tfg_check": (ci, [p, p]),
        "tfg_graph_destroy": (ci, [p]),
        "tfg_gcn_norm_ws_bytes": (sz, [i64, i64, ci, p]),
        "tfg_gcn_norm": (ci, [p, ci, i64, p, i64, ci, p, p, p, p, p, p, sz, p]),
        "tfg_aggregate_ws_bytes": (sz, [i64, i64, i64, i64, ci, p]),
        "tfg_aggregate": (ci, [p, ci, i64, p, i64, ci, p, i64, i64, i64, i64, ci, p, p, p, p,
                               sz, p]),
        "tfg_aggregate_noalloc": (ci, [p, ci, i64, p, i64, ci, p, i64, i64, i64, i64, ci, p, p,
                                       p, p]),
        "tfg_gat_edge_scores_ws_bytes": (sz, [i64, i64]),
        "tfg_gat_edge_scores": (ci, [p, ci, i64, p, i64, i64, i64, p, p, ctypes.c_float, p, p,
                                     sz, p]),
        "tfg_segment_softmax_ws_bytes": (sz, [i64, i64, i64, p]),
        "tfg_segment_softmax": (ci, [p, i64, i64, p, ci, i64, p, p, p, p, sz, p]),
        "tfg_segment_pool_ws_bytes": (sz, [i64, i64]),
        "tfg_segment_pool": (ci, [p, i64, i64, i64, p, ci, i64, ci, p, p, ci, p, sz, p]),
        "tfg_batch_graphs_ws_bytes": (sz, [i64]),
        "tfg_batch_graphs_totals": (ci, [i64, p, p, ci, p, sz, p, ctypes.POINTER(i64),
                                         ctypes.POINTER(i64)]),
        "tfg_propagate_ws_bytes": (sz, [p, i64, i64]),
        "tfg_gat_aggregate_ws_bytes": (sz, [p, i64, i64]),
        "tfg_gat_aggregate": (ci, [p, p, i64, i64, p, p, ctypes.c_float, p, p, p, sz, p]),
        "tfg_propagate": (ci, [p, p, ci, p, i64, i64, i64, ctypes.c_float, p, i64, p, p, sz, p]),
        "tfg_batch_graphs": (ci, [i64, p, p, p, ci, i64, i64, p, p, p, p, ci, p, sz, p]),
        "tfg_graph_create_transposed": (ci, [p, ci, i64, i64, i64, ci, ci, p, sz, p, sz, p,
                                             ctypes.POINTER(p)]),
        "tfg_aggregate_backward_ws_bytes": (sz, [p, p, i64, i64, ci, ci, ci]),
        "tfg_aggregate_backward": (ci, [p, p, p, i64, ci, p, i64, p, i64, ci, p, p, p, ci, p, sz,
                                        p]),
        "tfg_segment_softmax_backward_ws_bytes": (sz, [i64, i64, i64, p]),
        "tfg_segment_softmax_backward": (ci, [p, p, i64, i64, p, ci, i64, p, p, p, sz, p]),
        "tfg_edge_reorder_ws_bytes": (sz, [p, p, i64]),
        "tfg_edge_dot_scores": (ci, [p, p, p, i64, i64, ctypes.c_float, p, ci, p]),
        "tfg_segment_pool_backward": (ci, [p, i64, i64, p, ci, i64, ci, p, p, i64, ci, p, sz, p]),
        "tfg_gat_dot_aggregate_ws_bytes": (sz, [p, i64, i64]),
        "tfg_gat_dot_aggregate": (ci, [p, p, p, p, i64, i64, ctypes.c_float, p, p, p, sz, p]),
        "tfg_edge_reorder": (ci, [p, p, p, i64, p, p, sz, p]),
        "tfg_gat_graph_scores_ws_bytes": (sz, [p, i64]),
        "tfg_gat_graph_scores": (ci, [p, p, i64, i64, p, p, ctypes.c_float, p, ci, p, sz, p]),
        "tfg_segment_softmax_graph_ws_bytes": (sz, [p, i64]),
        "tfg_segment_softmax_graph": (ci, [p, p, i64, ci, p, p, sz, p]),
        "tfg_segment_softmax_graph_backward": (ci, [p, p, p, i64, ci, p, p, sz, p]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    del i32
    _lib = lib
    return lib


def _check(status: int):
    if status == TFG_OK:
        return
    lib = load()
    msg = f"{lib.tfg_status_string(status).decode()}: {lib.tfg_last_error().decode()}"
    if status == TFG_ERR_INDEX_RANGE:
        raise TfgIndexError(status, msg)
    if status in (TFG_ERR_INVALID_ARG, TFG_ERR_UNSORTED, TFG_ERR_TOO_LARGE, TFG_ERR_WORKSPACE):
        raise TfgValueError(status, msg)
    raise TfgError(status, msg)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _index_type(t: torch.Tensor) -> int:
    if t.dtype == torch.int32:
        return 0
    if t.dtype == torch.int64:
        return 1
    raise TypeError(f"index tensor must be int32 or int64, got {t.dtype}")


def _dev(t: torch.Tensor, what: str, device=None) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")
    if device is not None and t.device != torch.device(device):
        raise ValueError(f"{what} is on {t.device}, the call runs on {device}")
    return t


def _out(t: torch.Tensor, shape, dtype, device, what: str) -> torch.Tensor:
    """A caller-supplied output: on the call's device, of the right dtype,
    exactly `shape` and contiguous (the kernels write it densely by row)."""
    _dev(t, what, device)
    if t.dtype != dtype:
        raise TypeError(f"{what} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{what} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    return t


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


def _ws(ws: torch.Tensor | None, need: int, device, what: str = "ws") -> torch.Tensor:
    """The caller's workspace if it is a contiguous device buffer of at least
    `need` bytes on the call's device, else a new one."""
    if ws is not None:
        _dev(ws, what, device)
        if not ws.is_contiguous():
            raise ValueError(f"{what} must be contiguous")
        if _nbytes(ws) >= max(int(need), 1):
            return ws
    return _workspace(need, device)


def _edges(edge_index: torch.Tensor) -> torch.Tensor:
    _dev(edge_index, "edge_index")
    if edge_index.dim() != 2 or edge_index.shape[0] != 2:
        raise ValueError("edge_index must have shape [2, E]")
    return edge_index.contiguous()


def _f32(t: torch.Tensor | None, what: str, device=None) -> torch.Tensor | None:
    if t is None:
        return None
    _dev(t, what, device)
    if t.dtype != torch.float32:
        raise TypeError(f"{what} must be float32")
    return t.contiguous()


def _per_edge(t: torch.Tensor) -> torch.Tensor:
    """[E] or [E, H] per-edge values as [E, H] (also for E = 0)."""
    return t.reshape(t.shape[0], t.shape[1] if t.dim() > 1 else 1)


def _rows(x: torch.Tensor, what: str, device=None):
    """float32 2-D device tensor with unit column stride; returns (x, ldx)."""
    _dev(x, what, device)
    if x.dtype != torch.float32 or x.dim() != 2:
        raise TypeError(f"{what} must be a float32 matrix")
    if x.stride(1) != 1 or x.stride(0) < x.shape[1]:
        x = x.contiguous()
    return x, max(x.stride(0), x.shape[1])


def _workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


class Graph:
    """CSR-by-target form of one edge list (the handle of tfg_graph_create).

    Holds the device buffer the handle's arrays live in; ``E`` counts all
    edges, including the N self-loops appended when ``add_self_loops``."""

    def __init__(self, handle, buf, E_in, E, N, N_src, loops, device):
        self._h = handle
        self.buf = buf
        self.E_in, self.E, self.N, self.N_src, self.loops = E_in, E, N, N_src, loops
        self.device = device

    @property
    def handle(self):
        return self._h

    def info(self):
        vals = [ctypes.c_int64() for _ in range(7)]
        _check(load().tfg_graph_info(self._h, *[ctypes.byref(v) for v in vals]))
        keys = ("E", "N", "N_src", "src_parts", "n_chunks", "n_rows_split", "n_part_items")
        return dict(zip(keys, (v.value for v in vals)))

    def __del__(self):
        h, self._h = getattr(self, "_h", None), None
        if h is not None and _lib is not None:
            _lib.tfg_graph_destroy(h)


def tfg_graph_bytes(E: int, N: int, add_self_loops: bool = False, N_src: int | None = None,
                    src_parts: int = 0):
    b, s = ctypes.c_size_t(), ctypes.c_size_t()
    N_src = N if N_src is None else N_src
    _check(load().tfg_graph_bytes(E, N_src, N, int(add_self_loops), int(src_parts),
                                  ctypes.byref(b), ctypes.byref(s)))
    return b.value, s.value


def _create(fn, edge_index, N, N_src, add_self_loops, src_parts, buf, scratch, transposed):
    ei = _edges(edge_index)
    E = ei.shape[1]
    N_src = N if N_src is None else N_src
    rows, cols = (N_src, N) if transposed else (N, N_src)
    nb, ns = tfg_graph_bytes(E, rows, add_self_loops, cols, src_parts)
    dev = ei.device
    buf = _ws(buf, nb, dev, "buf")
    scratch = _ws(scratch, ns, dev, "scratch")
    h = ctypes.c_void_p()
    _check(fn(_ptr(ei), _index_type(ei), E, N_src, N, int(add_self_loops), int(src_parts),
              _ptr(buf), _nbytes(buf), _ptr(scratch), _nbytes(scratch), _stream(dev),
              ctypes.byref(h)))
    return Graph(h, buf, E, E + (rows if add_self_loops else 0), rows, cols,
                 bool(add_self_loops), dev)


def tfg_graph_create(edge_index: torch.Tensor, N: int, N_src: int | None = None,
                     add_self_loops: bool = False, src_parts: int = 0,
                     buf: torch.Tensor | None = None,
                     scratch: torch.Tensor | None = None) -> Graph:
    """COO -> CSR by (target, source part) (synchronises once; raises
    IndexError on a bad id). src_parts: 0 = chosen by the library, 1 = the
    plain stable CSR by target."""
    return _create(load().tfg_graph_create, edge_index, N, N_src, add_self_loops, src_parts, buf,
                   scratch, False)


def tfg_graph_create_transposed(edge_index: torch.Tensor, N: int, N_src: int | None = None,
                                add_self_loops: bool = False, src_parts: int = 0,
                                buf: torch.Tensor | None = None,
                                scratch: torch.Tensor | None = None) -> Graph:
    """The graph of the reversed edges (rows = the N_src sources, col = targets,
    perm = input edge ids) that carries the backward aggregation. N and N_src
    are those of the forward edge list; the handle's ``N`` is N_src."""
    return _create(load().tfg_graph_create_transposed, edge_index, N, N_src, add_self_loops,
                   src_parts, buf, scratch, True)


def tfg_graph_csr(g: Graph):
    """(rowptr [N+1], col [E], perm [E]) as int32 device tensors."""
    rowptr = torch.empty(g.N + 1, dtype=torch.int32, device=g.device)
    col = torch.empty(g.E, dtype=torch.int32, device=g.device)
    perm = torch.empty(g.E, dtype=torch.int32, device=g.device)
    _check(load().tfg_graph_csr(g.handle, _ptr(rowptr), _ptr(col), _ptr(perm), _stream(g.device)))
    return rowptr, col, perm


def tfg_edge_reorder(values: torch.Tensor, src: Graph | None = None,
                     dst: Graph | None = None) -> torch.Tensor:
    """A per-edge array [E'] or [E', H] moved from the order of ``src`` to the
    order of ``dst`` (None = the caller's COO edge order)."""
    lib = load()
    g = src if src is not None else dst
    if g is None:
        raise ValueError("at least one graph is needed")
    v = _f32(values, "values", g.device)
    H = v.numel() // max(g.E, 1) if g.E else 1
    if v.numel() != g.E * H:
        raise ValueError("values must hold E' * H entries")
    out = torch.empty_like(v)
    hs = src.handle if src is not None else None
    hd = dst.handle if dst is not None else None
    ws = _workspace(lib.tfg_edge_reorder_ws_bytes(hs, hd, H), v.device)
    _check(lib.tfg_edge_reorder(hs, hd, _ptr(v), H, _ptr(out), _ptr(ws), _nbytes(ws),
                                _stream(v.device)))
    return out


def tfg_graph_segments(g: Graph):
    """Start of every (target, source part) segment: int32 [N * src_parts + 1]."""
    parts = g.info()["src_parts"]
    seg = torch.empty(g.N * parts + 1, dtype=torch.int32, device=g.device)
    _check(load().tfg_graph_segments(g.handle, _ptr(seg), _stream(g.device)))
    return seg


def tfg_check(g: Graph):
    _check(load().tfg_check(g.handle, _stream(g.device)))


def tfg_gcn_norm(edge_index: torch.Tensor, N: int, edge_weight: torch.Tensor | None = None,
                 add_self_loops: bool = True, graph: Graph | None = None,
                 out_edge_index: bool = True, out_edge_weight: bool = True,
                 out_edge_weight_csr: bool | None = None, out_deg: bool = True,
                 ws: torch.Tensor | None = None):
    """GCN normalisation D^-1/2 (A + I) D^-1/2 per edge.

    Returns a dict with the requested outputs: ``edge_index`` [2, E'] int32,
    ``edge_weight`` [E'] (COO order), ``edge_weight_csr`` [E'] (CSR order of
    ``graph``; default: requested when a graph is given) and ``deg`` [N]."""
    lib = load()
    ei = _edges(edge_index)
    E = ei.shape[1]
    dev = ei.device
    w = _f32(edge_weight, "edge_weight", dev)
    if w is not None and w.numel() != E:
        raise ValueError(f"edge_weight must hold E = {E} values")
    if graph is not None and graph.device != dev:
        raise ValueError("graph and edge_index are on different devices")
    Ep = E + (N if add_self_loops else 0)
    if out_edge_weight_csr is None:
        out_edge_weight_csr = graph is not None
    res = {}
    if out_edge_index:
        res["edge_index"] = torch.empty((2, Ep), dtype=torch.int32, device=dev)
    if out_edge_weight:
        res["edge_weight"] = torch.empty(Ep, dtype=torch.float32, device=dev)
    if out_edge_weight_csr:
        res["edge_weight_csr"] = torch.empty(Ep, dtype=torch.float32, device=dev)
    if out_deg:
        res["deg"] = torch.empty(N, dtype=torch.float32, device=dev)
    h = graph.handle if graph is not None else None
    ws = _ws(ws, lib.tfg_gcn_norm_ws_bytes(E, N, int(add_self_loops), h), dev)
    _check(lib.tfg_gcn_norm(_ptr(ei), _index_type(ei), E, _ptr(w), N, int(add_self_loops), h,
                            _ptr(res.get("edge_index")), _ptr(res.get("edge_weight")),
                            _ptr(res.get("edge_weight_csr")), _ptr(res.get("deg")), _ptr(ws),
                            _nbytes(ws), _stream(dev)))
    return res


def tfg_aggregate_ws_bytes(E: int, N: int, F: int, reduce: str = "sum",
                           graph: Graph | None = None, N_src: int | None = None) -> int:
    N_src = N if N_src is None else N_src
    return load().tfg_aggregate_ws_bytes(E, N_src, N, F, _REDUCE[reduce],
                                         graph.handle if graph is not None else None)


def tfg_aggregate(edge_index: torch.Tensor | None, x: torch.Tensor, N: int, reduce: str = "sum",
                  edge_weight: torch.Tensor | None = None, heads: int = 1,
                  weight_order: str = "coo", graph: Graph | None = None,
                  out: torch.Tensor | None = None, argmax: torch.Tensor | None = None,
                  ws: torch.Tensor | None = None):
    """Message aggregation into N targets. Returns ``out`` [N, F] (and
    ``argmax`` [N, F] int32 edge ids for ``reduce="max"``). ``edge_index`` may
    be None when ``graph`` is given."""
    lib = load()
    if edge_index is None:
        if graph is None:
            raise ValueError("edge_index is needed without a graph")
        ei, E = None, graph.E
    else:
        ei = _edges(edge_index)
        E = ei.shape[1]
    x, ldx = _rows(x, "x")
    dev = x.device
    if ei is not None and ei.device != dev:
        raise ValueError("edge_index and x are on different devices")
    if graph is not None and graph.device != dev:
        raise ValueError("graph and x are on different devices")
    N_src, F = x.shape
    w = _f32(edge_weight, "edge_weight", dev)
    if w is not None and w.numel() != E * heads:
        raise ValueError(f"edge_weight must hold E * heads = {E * heads} values")
    red = _REDUCE[reduce]
    if out is None:
        out = torch.empty((N, F), dtype=torch.float32, device=dev)
    _out(out, (N, F), torch.float32, dev, "out")
    if red == 2:
        if argmax is None:
            argmax = torch.empty((N, F), dtype=torch.int32, device=dev)
        _out(argmax, (N, F), torch.int32, dev, "argmax")
    h = graph.handle if graph is not None else None
    ws = _ws(ws, lib.tfg_aggregate_ws_bytes(E, N_src, N, F, red, h), dev)
    _check(lib.tfg_aggregate(_ptr(ei), _index_type(ei) if ei is not None else 0, E, _ptr(w), heads,
                             _ORDER[weight_order],
                             _ptr(x), N_src, F, ldx, N, red, h, _ptr(out),
                             _ptr(argmax) if red == 2 else None, _ptr(ws), _nbytes(ws),
                             _stream(dev)))
    return (out, argmax) if red == 2 else out


def tfg_aggregate_noalloc(edge_index: torch.Tensor | None, x: torch.Tensor, N: int,
                          graph: Graph, reduce: str = "sum",
                          edge_weight: torch.Tensor | None = None, heads: int = 1,
                          weight_order: str = "coo", out: torch.Tensor | None = None,
                          argmax: torch.Tensor | None = None):
    """``tfg_aggregate`` on a cached graph through the entry point that
    allocates nothing: its partial rows live in the library's static device
    scratch (TFG_NOALLOC_SCRATCH_BYTES per GPU). Pass ``out`` (and ``argmax``
    for max) to keep the call free of allocations on this side too."""
    lib = load()
    if graph is None:
        raise ValueError("the no-allocation aggregation needs a graph handle")
    x, ldx = _rows(x, "x", graph.device)
    dev = x.device
    ei = None
    if edge_index is not None:
        ei = _edges(edge_index)
        _dev(ei, "edge_index", dev)
    N_src, F = x.shape
    w = _f32(edge_weight, "edge_weight", dev)
    if w is not None and w.numel() != graph.E * heads:
        raise ValueError(f"edge_weight must hold E * heads = {graph.E * heads} values")
    red = _REDUCE[reduce]
    if out is None:
        out = torch.empty((N, F), dtype=torch.float32, device=dev)
    _out(out, (N, F), torch.float32, dev, "out")
    if red == 2:
        if argmax is None:
            argmax = torch.empty((N, F), dtype=torch.int32, device=dev)
        _out(argmax, (N, F), torch.int32, dev, "argmax")
    _check(lib.tfg_aggregate_noalloc(_ptr(ei), _index_type(ei) if ei is not None else 0, graph.E,
                                     _ptr(w), heads, _ORDER[weight_order], _ptr(x), N_src, F,
                                     ldx, N, red, graph.handle, _ptr(out),
                                     _ptr(argmax) if red == 2 else None, _stream(dev)))
    return (out, argmax) if red == 2 else out


def tfg_aggregate_backward(graph: Graph, dy: torch.Tensor, reduce: str = "sum",
                           graph_t: Graph | None = None, x: torch.Tensor | None = None,
                           edge_weight: torch.Tensor | None = None, heads: int = 1,
                           weight_order: str = "coo", argmax: torch.Tensor | None = None,
                           want_dx: bool = True, want_dw: bool = False, dw_order: str = "coo",
                           ws: torch.Tensor | None = None):
    """Gradients of ``tfg_aggregate`` for dy = dL/d out [N, F]. Returns
    (dx [N_src, F] or None, dw [E', heads] or None); dx needs ``graph_t``
    (tfg_graph_create_transposed), dw needs ``x``, max needs the forward ``argmax``."""
    lib = load()
    dy = _f32(dy, "dy", graph.device).contiguous()
    dev = dy.device
    if dy.dim() != 2 or dy.shape[0] != graph.N:
        raise ValueError("dy must be [N, F]")
    F = dy.shape[1]
    if graph_t is not None and graph_t.device != dev:
        raise ValueError("graph_t is on another device")
    w = _f32(edge_weight, "edge_weight", dev)
    if w is not None and w.numel() != graph.E * heads:
        raise ValueError(f"edge_weight must hold E' * heads = {graph.E * heads} values")
    xx, ldx = (None, F)
    if x is not None:
        xx, ldx = _rows(x, "x", dev)
        if xx.shape != (graph.N_src, F):
            raise ValueError("x must be [N_src, F]")
    if argmax is not None and tuple(argmax.shape) != (graph.N, F):
        raise ValueError("argmax must be [N, F]")
    red = _REDUCE[reduce]
    am = None
    if argmax is not None:
        am = _dev(argmax, "argmax", dev).contiguous()
        if am.dtype != torch.int32:
            raise TypeError("argmax must be int32")
    dx = torch.empty((graph.N_src, F), dtype=torch.float32, device=dev) if want_dx else None
    dw = torch.empty((graph.E, heads), dtype=torch.float32, device=dev) if want_dw else None
    ht = graph_t.handle if graph_t is not None else None
    need = lib.tfg_aggregate_backward_ws_bytes(graph.handle, ht, F, heads, red,
                                               _ORDER[weight_order], int(w is not None))
    ws = _ws(ws, need, dev)
    _check(lib.tfg_aggregate_backward(graph.handle, ht, _ptr(w), heads, _ORDER[weight_order],
                                      _ptr(xx), ldx, _ptr(dy), F, red, _ptr(am), _ptr(dx),
                                      _ptr(dw), _ORDER[dw_order], _ptr(ws), _nbytes(ws),
                                      _stream(dev)))
    return dx, dw


def tfg_segment_softmax_backward(alpha: torch.Tensor, dalpha: torch.Tensor, seg: torch.Tensor,
                                 N: int, graph: Graph | None = None) -> torch.Tensor:
    """dL/d scores from alpha = segment softmax(scores) and dalpha = dL/d alpha ([E, H] or [E])."""
    lib = load()
    a = _f32(alpha, "alpha")
    shape = a.shape
    a2 = _per_edge(a)
    da = _f32(dalpha, "dalpha", a.device)
    if da.numel() != a2.numel():
        raise ValueError("dalpha must have the shape of alpha")
    da = da.reshape(a2.shape)
    E, H = a2.shape
    seg = _dev(seg, "seg", a.device).contiguous()
    if seg.numel() != E:
        raise ValueError("seg must hold one id per edge")
    dev = a.device
    ds = torch.empty_like(a2)
    h = graph.handle if graph is not None else None
    ws = _workspace(lib.tfg_segment_softmax_backward_ws_bytes(E, H, N, h), dev)
    _check(lib.tfg_segment_softmax_backward(_ptr(a2), _ptr(da), E, H, _ptr(seg), _index_type(seg),
                                            N, h, _ptr(ds), _ptr(ws), _nbytes(ws), _stream(dev)))
    return ds.reshape(shape)


def tfg_gat_edge_scores(edge_index: torch.Tensor, h: torch.Tensor, a_src: torch.Tensor,
                        a_dst: torch.Tensor, slope: float = 0.2, out: torch.Tensor | None = None):
    """LeakyReLU(a_src . h[src] + a_dst . h[tgt]) per edge and head -> [E, H]."""
    lib = load()
    ei = _edges(edge_index)
    E = ei.shape[1]
    h = _f32(h, "h", ei.device)
    N = h.shape[0]
    a_src, a_dst = _f32(a_src, "a_src", ei.device), _f32(a_dst, "a_dst", ei.device)
    H = a_src.shape[0]
    D = a_src.numel() // H
    if h.dim() != 2 or h.shape[1] != H * D or a_dst.shape != a_src.shape:
        raise ValueError("h must be [N, H*D] and a_src, a_dst [H, D]")
    if out is None:
        out = torch.empty((E, H), dtype=torch.float32, device=h.device)
    _out(out, (E, H), torch.float32, h.device, "out")
    ws = _workspace(lib.tfg_gat_edge_scores_ws_bytes(N, H), h.device)
    _check(lib.tfg_gat_edge_scores(_ptr(ei), _index_type(ei), E, _ptr(h), N, H, D, _ptr(a_src),
                                   _ptr(a_dst), float(slope), _ptr(out), _ptr(ws), _nbytes(ws),
                                   _stream(h.device)))
    return out


def tfg_segment_softmax(scores: torch.Tensor, seg: torch.Tensor, N: int,
                        graph: Graph | None = None, out_csr: bool = False):
    """Softmax of scores [E, H] (or [E]) over the segments given by seg [E].
    With ``out_csr`` (needs ``graph``) also returns the result in CSR order."""
    lib = load()
    s = _f32(scores, "scores")
    squeeze = s.dim() == 1
    s2 = _per_edge(s)
    E, H = s2.shape
    seg = _dev(seg, "seg", s.device).contiguous()
    if seg.numel() != E:
        raise ValueError("seg must hold one id per edge")
    dev = s.device
    if graph is not None and graph.device != dev:
        raise ValueError("graph and scores are on different devices")
    out = torch.empty_like(s2)
    oc = torch.empty_like(s2) if out_csr else None
    h = graph.handle if graph is not None else None
    ws = _workspace(lib.tfg_segment_softmax_ws_bytes(E, H, N, h), dev)
    _check(lib.tfg_segment_softmax(_ptr(s2), E, H, _ptr(seg), _index_type(seg), N, h, _ptr(out),
                                   _ptr(oc), _ptr(ws), _nbytes(ws), _stream(dev)))
    if squeeze:
        out = out.reshape(E)
        oc = oc.reshape(E) if oc is not None else None
    return (out, oc) if out_csr else out


def tfg_gat_graph_scores(graph: Graph, h: torch.Tensor, a_src: torch.Tensor, a_dst: torch.Tensor,
                         slope: float = 0.2, order: str = "csr", out: torch.Tensor | None = None,
                         ws: torch.Tensor | None = None) -> torch.Tensor:
    """The additive attention scores [E', H] of the graph's edges, in ``order``
    ("csr": the graph order, "coo": edge ids)."""
    lib = load()
    dev = graph.device
    h = _f32(h, "h", dev)
    a_src, a_dst = _f32(a_src, "a_src", dev), _f32(a_dst, "a_dst", dev)
    H = a_src.shape[0]
    D = a_src.numel() // H
    if h.dim() != 2 or h.shape != (graph.N, H * D) or a_dst.shape != a_src.shape:
        raise ValueError("h must be [N, H*D] and a_src, a_dst [H, D]")
    if out is None:
        out = torch.empty((graph.E, H), dtype=torch.float32, device=dev)
    _out(out, (graph.E, H), torch.float32, dev, "out")
    ws = _ws(ws, lib.tfg_gat_graph_scores_ws_bytes(graph.handle, H), dev)
    _check(lib.tfg_gat_graph_scores(graph.handle, _ptr(h), H, D, _ptr(a_src), _ptr(a_dst),
                                    float(slope), _ptr(out), _ORDER[order], _ptr(ws), _nbytes(ws),
                                    _stream(dev)))
    return out


def tfg_segment_softmax_graph(graph: Graph, scores: torch.Tensor, order: str = "csr",
                              out: torch.Tensor | None = None,
                              ws: torch.Tensor | None = None) -> torch.Tensor:
    """Softmax of scores [E', H] (or [E']) over the graph's targets, scores and
    result in ``order`` ("csr": the graph order, "coo": edge ids)."""
    lib = load()
    dev = graph.device
    s = _f32(scores, "scores", dev)
    s2 = _per_edge(s)
    E, H = s2.shape
    if E != graph.E:
        raise ValueError(f"scores must hold one row per edge of the graph ({graph.E})")
    if out is None:
        out = torch.empty_like(s2)
    _out(out, (E, H), torch.float32, dev, "out")
    ws = _ws(ws, lib.tfg_segment_softmax_graph_ws_bytes(graph.handle, H), dev)
    _check(lib.tfg_segment_softmax_graph(graph.handle, _ptr(s2), H, _ORDER[order], _ptr(out),
                                         _ptr(ws), _nbytes(ws), _stream(dev)))
    return out.reshape(s.shape)


def tfg_segment_softmax_graph_backward(graph: Graph, alpha: torch.Tensor, dalpha: torch.Tensor,
                                       order: str = "csr") -> torch.Tensor:
    """dL/d scores from alpha and dalpha ([E', H] or [E']) in ``order``."""
    lib = load()
    dev = graph.device
    a = _f32(alpha, "alpha", dev)
    a2 = _per_edge(a)
    da = _f32(dalpha, "dalpha", dev)
    if da.numel() != a2.numel():
        raise ValueError("dalpha must have the shape of alpha")
    da = da.reshape(a2.shape)
    E, H = a2.shape
    if E != graph.E:
        raise ValueError(f"alpha must hold one row per edge of the graph ({graph.E})")
    ds = torch.empty_like(a2)
    ws = _workspace(lib.tfg_segment_softmax_graph_ws_bytes(graph.handle, H), dev)
    _check(lib.tfg_segment_softmax_graph_backward(graph.handle, _ptr(a2), _ptr(da), H,
                                                  _ORDER[order], _ptr(ds), _ptr(ws), _nbytes(ws),
                                                  _stream(dev)))
    return ds.reshape(a.shape)


def tfg_segment_pool(x: torch.Tensor, graph_index: torch.Tensor, G: int, reduce: str = "sum",
                     validate: bool = True, out: torch.Tensor | None = None,
                     argmax: torch.Tensor | None = None, ws: torch.Tensor | None = None):
    """Pools node rows x [Nb, F] into G graphs by the sorted graph_index [Nb].
    Returns out [G, F] (and argmax node ids [G, F] for ``reduce="max"``)."""
    lib = load()
    x, ldx = _rows(x, "x")
    Nb, F = x.shape
    dev = x.device
    gi = _dev(graph_index, "graph_index", dev).contiguous()
    if gi.dim() != 1 or gi.shape[0] != Nb:
        raise ValueError("graph_index must hold one id per row of x")
    red = _REDUCE[reduce]
    if out is None:
        out = torch.empty((G, F), dtype=torch.float32, device=dev)
    _out(out, (G, F), torch.float32, dev, "out")
    arg = None
    if red == 2:
        arg = argmax if argmax is not None else torch.empty((G, F), dtype=torch.int32, device=dev)
        _out(arg, (G, F), torch.int32, dev, "argmax")
    ws = _ws(ws, lib.tfg_segment_pool_ws_bytes(Nb, G), dev)
    _check(lib.tfg_segment_pool(_ptr(x), Nb, F, ldx, _ptr(gi), _index_type(gi), G, red, _ptr(out),
                                _ptr(arg), int(validate), _ptr(ws), _nbytes(ws), _stream(dev)))
    return (out, arg) if red == 2 else out


def tfg_segment_pool_backward(dy: torch.Tensor, graph_index: torch.Tensor, reduce: str = "sum",
                              argmax: torch.Tensor | None = None, validate: bool = True,
                              out: torch.Tensor | None = None) -> torch.Tensor:
    """Gradient of ``tfg_segment_pool`` for dy = dL/d out [G, F]: dx [Nb, F]."""
    lib = load()
    dy = _f32(dy, "dy")
    if dy.dim() != 2:
        raise ValueError("dy must be [G, F]")
    G, F = dy.shape
    gi = _dev(graph_index, "graph_index", dy.device).contiguous()
    Nb = gi.shape[0]
    red = _REDUCE[reduce]
    am = None
    if argmax is not None:
        am = _dev(argmax, "argmax", dy.device).contiguous()
        if am.dtype != torch.int32 or am.shape != dy.shape:
            raise ValueError("argmax must be int32 [G, F]")
    dx = out if out is not None else torch.empty((Nb, F), dtype=torch.float32, device=dy.device)
    _out(dx, (Nb, F), torch.float32, dy.device, "out")
    ws = _workspace(lib.tfg_segment_pool_ws_bytes(Nb, G), dy.device)
    _check(lib.tfg_segment_pool_backward(_ptr(dy), G, F, _ptr(gi), _index_type(gi), Nb, red,
                                         _ptr(am), _ptr(dx), F, int(validate), _ptr(ws),
                                         _nbytes(ws), _stream(dy.device)))
    return dx


def tfg_batch_graphs_totals(node_counts: torch.Tensor, edge_counts: torch.Tensor):
    """(Nb, E): the node and edge totals of a batch, summed on the device."""
    lib = load()
    nc = _dev(node_counts, "node_counts").contiguous()
    ec = _dev(edge_counts, "edge_counts").contiguous()
    if nc.dtype != ec.dtype or nc.shape != ec.shape or nc.dim() != 1:
        raise ValueError("node_counts and edge_counts must be [G] of one index dtype")
    G = nc.shape[0]
    ws = _workspace(lib.tfg_batch_graphs_ws_bytes(G), nc.device)
    nb, eb = ctypes.c_int64(), ctypes.c_int64()
    _check(lib.tfg_batch_graphs_totals(G, _ptr(nc), _ptr(ec), _index_type(nc), _ptr(ws),
                                       _nbytes(ws), _stream(nc.device), ctypes.byref(nb),
                                       ctypes.byref(eb)))
    return nb.value, eb.value


def tfg_batch_graphs(node_counts: torch.Tensor, edge_counts: torch.Tensor,
                     local_edge_index: torch.Tensor, Nb: int | None = None,
                     validate: bool = True, out=None, ws: torch.Tensor | None = None):
    """BatchGraph of G graphs: (edge_index [2, E], graph_index [Nb], node_offsets [G+1],
    edge_offsets [G+1]). local_edge_index holds graph 0's edges, then graph 1's, ...,
    with ids local to their graph; Nb defaults to the node total, which
    tfg_batch_graphs_totals sums on the device (one wait on the stream)."""
    lib = load()
    ei = _edges(local_edge_index)
    dev = ei.device
    nc = _dev(node_counts, "node_counts", dev).contiguous()
    ec = _dev(edge_counts, "edge_counts", dev).contiguous()
    if nc.dtype != ei.dtype or ec.dtype != ei.dtype:
        raise TypeError("counts and edge_index must share one index dtype")
    if nc.dim() != 1 or nc.shape != ec.shape:
        raise ValueError("node_counts and edge_counts must be [G]")
    G, E = nc.shape[0], ei.shape[1]
    ws = _ws(ws, lib.tfg_batch_graphs_ws_bytes(G), dev)
    if Nb is None:
        nb, eb = ctypes.c_int64(), ctypes.c_int64()
        _check(lib.tfg_batch_graphs_totals(G, _ptr(nc), _ptr(ec), _index_type(ei), _ptr(ws),
                                           _nbytes(ws), _stream(dev), ctypes.byref(nb),
                                           ctypes.byref(eb)))
        Nb = nb.value
    if out is not None:  # (edge_index, graph_index, node_offsets, edge_offsets) from a prior call
        out_ei, gi, noff, eoff = out
    else:
        out_ei = torch.empty_like(ei)
        gi = torch.empty(Nb, dtype=ei.dtype, device=dev)
        noff = torch.empty(G + 1, dtype=torch.int32, device=dev)
        eoff = torch.empty(G + 1, dtype=torch.int32, device=dev)
    _out(out_ei, tuple(ei.shape), ei.dtype, dev, "out edge_index")
    _out(gi, (Nb,), ei.dtype, dev, "out graph_index")
    _out(noff, (G + 1,), torch.int32, dev, "out node_offsets")
    _out(eoff, (G + 1,), torch.int32, dev, "out edge_offsets")
    _check(lib.tfg_batch_graphs(G, _ptr(nc), _ptr(ec), _ptr(ei), _index_type(ei), E, Nb,
                                _ptr(out_ei), _ptr(gi), _ptr(noff), _ptr(eoff), int(validate),
                                _ptr(ws), _nbytes(ws), _stream(dev)))
    return out_ei, gi, noff, eoff


def tfg_propagate(graph: Graph, x: torch.Tensor, K: int, alpha: float = 0.0,
                  h: torch.Tensor | None = None, edge_weight: torch.Tensor | None = None,
                  weight_order: str = "csr", out: torch.Tensor | None = None,
                  ws: torch.Tensor | None = None):
    """K steps of Z <- (1 - alpha) A Z + alpha h from Z = x (SGC: alpha = 0;
    APPNP: h = x). edge_weight in graph order by default (tfg_gcn_norm's
    ``edge_weight_csr``)."""
    lib = load()
    x, ldx = _rows(x, "x", graph.device)
    N, F = x.shape
    if N != graph.N:
        raise ValueError("x must be [N, F]")
    w = _f32(edge_weight, "edge_weight", x.device)
    if w is not None and w.numel() != graph.E:
        raise ValueError(f"edge_weight must hold E' = {graph.E} values")
    ldh = 0
    if h is not None:
        h, ldh = _rows(h, "h", x.device)
        if h.shape != (N, F):
            raise ValueError("h must be [N, F]")
    if out is None:
        out = torch.empty((N, F), dtype=torch.float32, device=x.device)
    _out(out, (N, F), torch.float32, x.device, "out")
    ws = _ws(ws, lib.tfg_propagate_ws_bytes(graph.handle, F, K), x.device)
    _check(lib.tfg_propagate(graph.handle, _ptr(w), _ORDER[weight_order], _ptr(x), F, ldx, K,
                             float(alpha), _ptr(h), ldh, _ptr(out), _ptr(ws), _nbytes(ws),
                             _stream(x.device)))
    return out


def tfg_gat_aggregate(graph: Graph, h: torch.Tensor, a_src: torch.Tensor, a_dst: torch.Tensor,
                      slope: float = 0.2, want_alpha: bool = False,
                      out: torch.Tensor | None = None):
    """Fused attention layer after the projection: out [N, H*D] (and alpha
    [E', H] in the graph's edge order when ``want_alpha``)."""
    lib = load()
    h = _f32(h, "h", graph.device)
    a_src, a_dst = _f32(a_src, "a_src", h.device), _f32(a_dst, "a_dst", h.device)
    H = a_src.shape[0]
    D = a_src.numel() // H
    N = h.shape[0]
    if h.dim() != 2 or h.shape[1] != H * D or a_dst.shape != a_src.shape:
        raise ValueError("h must be [N, H*D] and a_src, a_dst [H, D]")
    if N != graph.N or graph.N_src != graph.N:
        raise ValueError("h must be [N, H*D] for a square graph")
    if out is None:
        out = torch.empty((N, H * D), dtype=torch.float32, device=h.device)
    _out(out, (N, H * D), torch.float32, h.device, "out")
    alpha = torch.empty((graph.E, H), dtype=torch.float32, device=h.device) if want_alpha else None
    ws = _workspace(lib.tfg_gat_aggregate_ws_bytes(graph.handle, H, D), h.device)
    _check(lib.tfg_gat_aggregate(graph.handle, _ptr(h), H, D, _ptr(a_src), _ptr(a_dst),
                                 float(slope), _ptr(out), _ptr(alpha), _ptr(ws), _nbytes(ws),
                                 _stream(h.device)))
    return (out, alpha) if want_alpha else out



def tfg_edge_dot_scores(graph: Graph, q: torch.Tensor, key: torch.Tensor, heads: int,
                        scale: float | None = None, order: str = "coo",
                        out: torch.Tensor | None = None) -> torch.Tensor:
    """Scaled dot-product scores [E', heads]: scale * <q[tgt], key[src]> per head
    (scale defaults to 1/sqrt(D))."""
    lib = load()
    q, key = _f32(q, "q", graph.device), _f32(key, "key", graph.device)
    if q.dim() != 2:
        raise ValueError("q must be [N, H*D]")
    F = q.shape[1]
    D = F // heads
    if q.shape[0] != graph.N or key.shape != (graph.N_src, F) or F % heads:
        raise ValueError("q must be [N, H*D] and key [N_src, H*D]")
    if scale is None:
        scale = 1.0 / (D ** 0.5)
    if out is None:
        out = torch.empty((graph.E, heads), dtype=torch.float32, device=q.device)
    _out(out, (graph.E, heads), torch.float32, q.device, "out")
    _check(lib.tfg_edge_dot_scores(graph.handle, _ptr(q), _ptr(key), heads, D, float(scale),
                                   _ptr(out), _ORDER[order], _stream(q.device)))
    return out


def tfg_gat_dot_aggregate(graph: Graph, q: torch.Tensor, key: torch.Tensor, v: torch.Tensor,
                          heads: int, scale: float | None = None, want_alpha: bool = False,
                          out: torch.Tensor | None = None):
    """Transformer-style attention layer in one sweep: out [N, H*D] (and alpha
    [E', H] in edge-id order with ``want_alpha``)."""
    lib = load()
    q, key, v = (_f32(q, "q", graph.device), _f32(key, "key", graph.device),
                 _f32(v, "v", graph.device))
    if q.dim() != 2:
        raise ValueError("q must be [N, H*D]")
    F = q.shape[1]
    D = F // heads
    if (q.shape[0] != graph.N or key.shape != (graph.N_src, F) or v.shape != key.shape
            or F % heads):
        raise ValueError("q must be [N, H*D], key and v [N_src, H*D]")
    if scale is None:
        scale = 1.0 / (D ** 0.5)
    dev = q.device
    if out is None:
        out = torch.empty((graph.N, F), dtype=torch.float32, device=dev)
    _out(out, (graph.N, F), torch.float32, dev, "out")
    alpha = torch.empty((graph.E, heads), dtype=torch.float32, device=dev) if want_alpha else None
    ws = _workspace(lib.tfg_gat_dot_aggregate_ws_bytes(graph.handle, heads, D), dev)
    _check(lib.tfg_gat_dot_aggregate(graph.handle, _ptr(q), _ptr(key), _ptr(v), heads, D,
                                     float(scale), _ptr(out), _ptr(alpha), _ptr(ws), _nbytes(ws),
                                     _stream(dev)))
    return (out, alpha) if want_alpha else out
