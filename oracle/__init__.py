"""Oracle for the aggregation / pooling hot path: numpy wrappers around the
plain C implementation in ``oracle.c``.

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by the
CPU-baseline leg of the benchmark. The library under test never imports it.

All index arrays are int64; features, weights and scores float32. Sums come
back in float64 (``out64``) together with the error scale ``scale`` (the sum
of the absolute values of the terms), max reductions in float32 with int64
argmax, CSR arrays in int64.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

SUM, MEAN, MAX = 0, 1, 2
REDUCE = {"sum": SUM, "mean": MEAN, "max": MAX}
OK, ERR_INVALID_ARG, ERR_INDEX_RANGE, ERR_UNSORTED = 0, 1, 2, 3

_lib = None


class OracleError(Exception):
    def __init__(self, code: int):
        super().__init__(f"oracle status {code}")
        self.code = code


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _lib = ctypes.CDLL(_build.LIB)
        i64, p = ctypes.c_int64, ctypes.c_void_p
        _lib.orc_check_edges.argtypes = [i64, p, p, i64, i64]
        _lib.orc_csr_by_target.argtypes = [i64, i64, p, p, p, p, p]
        _lib.orc_csr_by_target.restype = None
        _lib.orc_gcn_norm.argtypes = [i64, i64, p, p, p, ctypes.c_int, p, p, p, p]
        _lib.orc_gcn_norm.restype = i64
        _lib.orc_aggregate.argtypes = [i64, p, p, p, i64, p, i64, i64, i64, ctypes.c_int,
                                       p, p, p, p]
        _lib.orc_aggregate_rows.argtypes = [i64, p, p, p, i64, p, i64, i64, i64, ctypes.c_int,
                                            p, i64, p, p, p, p]
        _lib.orc_segment_softmax.argtypes = [i64, i64, p, p, i64, p, p]
        _lib.orc_aggregate_backward.argtypes = [i64, p, p, p, i64, p, i64, i64, i64, i64,
                                                ctypes.c_int, p, p, p, p]
        _lib.orc_segment_softmax_backward.argtypes = [i64, i64, p, p, p, i64, p]
        _lib.orc_segment_pool_backward.argtypes = [i64, i64, p, i64, ctypes.c_int, p, p, p]
        _lib.orc_dot_scores.argtypes = [i64, p, p, p, p, i64, i64, i64, i64, ctypes.c_double, p]
        _lib.orc_dot_layer.argtypes = [i64, p, p, p, p, p, i64, i64, i64, i64, ctypes.c_double,
                                       p, p, p]
        _lib.orc_propagate.argtypes = [i64, p, p, p, p, i64, i64, i64, i64, ctypes.c_double, p,
                                       p, p]
        _lib.orc_segment_pool.argtypes = [i64, i64, i64, p, p, i64, ctypes.c_int, p, p, p, p]
        _lib.orc_gat_scores.argtypes = [i64, p, p, p, i64, i64, i64, p, p, ctypes.c_float, p, p]
        _lib.orc_gat_layer.argtypes = [i64, p, p, p, i64, i64, i64, p, p, ctypes.c_float, p, p, p]
        _lib.orc_batch_offsets.argtypes = [i64, p, p]
        _lib.orc_batch_offsets.restype = None
        _lib.orc_batch_graphs.argtypes = [i64, p, p, p, p, p, p]
        _lib.orc_batch_graphs.restype = None
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _rows(x):
    """float32 2-D array whose rows are unit-stride (a leading-dimension view is kept)."""
    x = np.asarray(x, dtype=np.float32)
    assert x.ndim == 2
    if x.strides[1] != 4 or x.strides[0] % 4 or x.strides[0] < 4 * x.shape[1]:
        x = np.ascontiguousarray(x)
    return x, max(x.strides[0] // 4, x.shape[1])


def _i64(a):
    return np.ascontiguousarray(a, dtype=np.int64)


def _f32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


def _check(code):
    if code != OK:
        raise OracleError(code)


def check_edges(edge_index, n_src, n):
    ei = _i64(edge_index)
    return lib().orc_check_edges(ei.shape[1], _ptr(ei[0]), _ptr(ei[1]), n_src, n)


def csr_by_target(edge_index, n, n_src=None):
    """Stable counting sort by target: (rowptr [N+1], col [E], perm [E]), input
    order kept within a row."""
    ei = _i64(edge_index)
    E = ei.shape[1]
    n_src = n if n_src is None else n_src
    _check(check_edges(ei, n_src, n))
    rowptr = np.empty(n + 1, np.int64)
    col = np.empty(E, np.int64)
    perm = np.empty(E, np.int64)
    src, tgt = np.ascontiguousarray(ei[0]), np.ascontiguousarray(ei[1])
    lib().orc_csr_by_target(E, n, _ptr(src), _ptr(tgt), _ptr(rowptr), _ptr(col), _ptr(perm))
    return rowptr, col, perm


def gcn_norm(edge_index, n, edge_weight=None, add_self_loops=True):
    """A_hat = D^-1/2 (A + I) D^-1/2 per edge: (edge_index' [2,E'], w' [E'], deg [N])."""
    ei = _i64(edge_index)
    E = ei.shape[1]
    _check(check_edges(ei, n, n))
    Ep = E + (n if add_self_loops else 0)
    src, tgt = np.ascontiguousarray(ei[0]), np.ascontiguousarray(ei[1])
    out_ei = np.empty((2, Ep), np.int64)
    out_w = np.empty(Ep, np.float32)
    deg = np.empty(n, np.float32)
    w = _f32(edge_weight)
    got = lib().orc_gcn_norm(E, n, _ptr(src), _ptr(tgt), _ptr(w), int(bool(add_self_loops)),
                             _ptr(out_ei[0]), _ptr(out_ei[1]), _ptr(out_w), _ptr(deg))
    assert got == Ep
    return out_ei, out_w, deg


def aggregate(edge_index, x, n, reduce="sum", edge_weight=None, heads=1, rows=None):
    """Sum / mean -> (out64 [N,F] float64, scale [N,F]); max -> (out [N,F] float32, arg int64).
    With ``rows``, only those target rows are computed (outputs have len(rows) rows)."""
    ei = _i64(edge_index)
    x, ldx = _rows(x)
    n_src, F = x.shape
    _check(check_edges(ei, n_src, n))
    red = REDUCE[reduce]
    src, tgt = np.ascontiguousarray(ei[0]), np.ascontiguousarray(ei[1])
    w = _f32(edge_weight)
    if w is not None and w.size != ei.shape[1] * heads:
        raise ValueError("edge_weight must hold E * heads values")
    n_rows = n if rows is None else len(rows)
    out64 = np.zeros((n_rows, F), np.float64) if red != MAX else None
    scale = np.zeros((n_rows, F), np.float64) if red != MAX else None
    outf = np.zeros((n_rows, F), np.float32) if red == MAX else None
    arg = np.zeros((n_rows, F), np.int64) if red == MAX else None
    xp = x.ctypes.data_as(ctypes.c_void_p)
    if rows is None:
        code = lib().orc_aggregate(ei.shape[1], _ptr(src), _ptr(tgt), _ptr(w), heads, xp, ldx, F,
                                   n, red, _ptr(out64), _ptr(outf), _ptr(arg), _ptr(scale))
    else:
        slot = np.full(n, -1, np.int64)
        slot[np.asarray(rows, np.int64)] = np.arange(n_rows)
        code = lib().orc_aggregate_rows(ei.shape[1], _ptr(src), _ptr(tgt), _ptr(w), heads, xp, ldx,
                                        F, n, red, _ptr(slot), n_rows, _ptr(out64), _ptr(outf),
                                        _ptr(arg), _ptr(scale))
    _check(code)
    return (outf, arg) if red == MAX else (out64, scale)


def host_threads() -> int:
    """Host threads this process may use: OMP_NUM_THREADS when set (the
    machine's share for this job), else the CPUs of the affinity mask."""
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        return int(env)
    return len(os.sched_getaffinity(0))


def aggregate_by_row_ranges(edge_index, x, n, reduce="sum", edge_weight=None, heads=1,
                            threads=None):
    """``aggregate`` over all N targets, split over host threads by target
    range: thread i computes rows [n*i/T, n*(i+1)/T), scanning every edge in
    input order and skipping the other targets, so every row is reduced in the
    same order as in one thread and the result is bit-identical."""
    from concurrent.futures import ThreadPoolExecutor
    threads = max(1, min(threads or host_threads(), max(n, 1)))
    ei = _i64(edge_index)
    x, _ = _rows(x)
    bounds = [n * i // threads for i in range(threads + 1)]

    def part(i):
        rows = np.arange(bounds[i], bounds[i + 1], dtype=np.int64)
        return aggregate(ei, x, n, reduce, edge_weight=edge_weight, heads=heads, rows=rows)

    with ThreadPoolExecutor(threads) as pool:  # the C calls release the GIL
        parts = list(pool.map(part, range(threads)))
    return tuple(np.concatenate([p[j] for p in parts], axis=0) for j in range(2))


def propagate(edge_index, x, K, alpha=0.0, h=None, edge_weight=None):
    """Z_K of Z_{k+1} = (1 - alpha) A Z_k + alpha h, Z_0 = x: (out64 [N,F], scale [N,F])."""
    ei = _i64(edge_index)
    x, ldx = _rows(x)
    N, F = x.shape
    hh = None if h is None else np.ascontiguousarray(h, dtype=np.float32).reshape(N, F)
    src, tgt = np.ascontiguousarray(ei[0]), np.ascontiguousarray(ei[1])
    w = _f32(edge_weight)
    out64 = np.empty((N, F), np.float64)
    scale = np.empty((N, F), np.float64)
    _check(lib().orc_propagate(ei.shape[1], _ptr(src), _ptr(tgt), _ptr(w),
                               x.ctypes.data_as(ctypes.c_void_p), ldx, N, F, K, float(alpha),
                               _ptr(hh), _ptr(out64), _ptr(scale)))
    return out64, scale


def segment_pool_backward(dy, graph_index, G, reduce="sum", arg=None):
    """Gradient of ``segment_pool`` for dL/d out = dy [G, F]: dx [Nb, F] in float64."""
    dy = np.ascontiguousarray(dy, dtype=np.float32)
    gi = _i64(graph_index)
    if dy.shape[0] != G or (arg is not None and np.shape(arg) != dy.shape):
        raise ValueError("dy and arg must be [G, F]")
    a = None if arg is None else _i64(arg)
    dx = np.empty((gi.shape[0], dy.shape[1]), np.float64)
    _check(lib().orc_segment_pool_backward(gi.shape[0], dy.shape[1], _ptr(gi), G, REDUCE[reduce],
                                           _ptr(dy), _ptr(a), _ptr(dx)))
    return dx


def dot_scores(edge_index, q, key, heads, scale):
    """Scaled dot-product scores [E, H] in float64: scale * <q[tgt], key[src]> per head."""
    ei = _i64(edge_index)
    q = np.ascontiguousarray(q, dtype=np.float32)
    key = np.ascontiguousarray(key, dtype=np.float32)
    n, F = q.shape
    n_src = key.shape[0]
    if key.shape[1] != F or F % heads:
        raise ValueError("q and key must be [*, H*D]")
    E = ei.shape[1]
    src, tgt = np.ascontiguousarray(ei[0]), np.ascontiguousarray(ei[1])
    s = np.empty((E, heads), np.float64)
    _check(lib().orc_dot_scores(E, _ptr(src), _ptr(tgt), _ptr(q), _ptr(key), n, n_src, heads,
                                F // heads, float(scale), _ptr(s)))
    return s


def dot_layer(edge_index, q, key, v, heads, scale):
    """Transformer-style attention layer: (out64 [N, H*D], alpha64 [E, H], scale [N, H*D])."""
    ei = _i64(edge_index)
    q = np.ascontiguousarray(q, dtype=np.float32)
    key = np.ascontiguousarray(key, dtype=np.float32)
    v = np.ascontiguousarray(v, dtype=np.float32)
    n, F = q.shape
    n_src = key.shape[0]
    if key.shape[1] != F or v.shape != key.shape or F % heads:
        raise ValueError("q, key and v must be [*, H*D]")
    E = ei.shape[1]
    src, tgt = np.ascontiguousarray(ei[0]), np.ascontiguousarray(ei[1])
    out = np.empty((n, F), np.float64)
    alpha = np.empty((E, heads), np.float64)
    S = np.empty((n, F), np.float64)
    _check(lib().orc_dot_layer(E, _ptr(src), _ptr(tgt), _ptr(q), _ptr(key), _ptr(v), n, n_src,
                               heads, F // heads, float(scale), _ptr(out), _ptr(alpha), _ptr(S)))
    return out, alpha, S


def aggregate_backward(edge_index, x, n, dy, reduce="sum", edge_weight=None, heads=1, arg=None):
    """Gradients of ``aggregate`` for dL/d out = dy: (dx [N_src, F], dw [E, H]) in float64."""
    ei = _i64(edge_index)
    x, ldx = _rows(x)
    n_src, F = x.shape
    E = ei.shape[1]
    src, tgt = np.ascontiguousarray(ei[0]), np.ascontiguousarray(ei[1])
    w = _f32(edge_weight)
    if w is not None and w.size != E * heads:
        raise ValueError("edge_weight must hold E * heads values")
    dy = np.ascontiguousarray(dy, dtype=np.float32)
    if dy.shape != (n, F) or (arg is not None and np.shape(arg) != (n, F)):
        raise ValueError("dy and arg must be [N, F]")
    a = None if arg is None else _i64(arg)
    dx = np.empty((n_src, F), np.float64)
    dw = np.empty((E, heads), np.float64)
    _check(lib().orc_aggregate_backward(E, _ptr(src), _ptr(tgt), _ptr(w), heads,
                                        x.ctypes.data_as(ctypes.c_void_p), ldx, F, n_src, n,
                                        REDUCE[reduce], _ptr(dy), _ptr(a), _ptr(dx), _ptr(dw)))
    return dx, dw


def segment_softmax_backward(alpha, dalpha, seg, n):
    """dL/d scores for alpha = segment softmax(scores) and dL/d alpha = dalpha (float64)."""
    a = np.ascontiguousarray(alpha, dtype=np.float32)
    shape = a.shape
    a = a.reshape(a.shape[0], -1)
    da = np.ascontiguousarray(dalpha, dtype=np.float32).reshape(a.shape)
    seg = _i64(seg)
    if seg.shape != (a.shape[0],):
        raise ValueError("seg must hold one id per row")
    ds = np.empty(a.shape, np.float64)
    _check(lib().orc_segment_softmax_backward(a.shape[0], a.shape[1], _ptr(a), _ptr(da), _ptr(seg),
                                              n, _ptr(ds)))
    return ds.reshape(shape)


def segment_softmax(scores, seg, n):
    """Per-segment softmax of float32 scores [E,H] (or [E]) -> (out64, out32)."""
    s = np.ascontiguousarray(scores, dtype=np.float32)
    squeeze = s.ndim == 1
    s2 = s.reshape(s.shape[0], -1)
    E, H = s2.shape
    seg = _i64(seg)
    if seg.shape != (E,):
        raise ValueError("seg must hold one id per score row")
    out64 = np.empty((E, H), np.float64)
    outf = np.empty((E, H), np.float32)
    _check(lib().orc_segment_softmax(E, H, _ptr(s2), _ptr(seg), n, _ptr(out64), _ptr(outf)))
    if squeeze:
        return out64[:, 0], outf[:, 0]
    return out64, outf


def segment_pool(x, graph_index, G, reduce="sum"):
    """Pool node rows by a sorted graph index. Sum / mean -> (out64, scale);
    max -> (out float32, arg int64 node ids)."""
    x, ldx = _rows(x)
    Nb, F = x.shape
    gi = _i64(graph_index)
    red = REDUCE[reduce]
    out64 = np.zeros((G, F), np.float64) if red != MAX else None
    scale = np.zeros((G, F), np.float64) if red != MAX else None
    outf = np.zeros((G, F), np.float32) if red == MAX else None
    arg = np.zeros((G, F), np.int64) if red == MAX else None
    _check(lib().orc_segment_pool(Nb, F, ldx, x.ctypes.data_as(ctypes.c_void_p), _ptr(gi), G, red,
                                  _ptr(out64), _ptr(outf), _ptr(arg), _ptr(scale)))
    return (outf, arg) if red == MAX else (out64, scale)


def gat_scores(edge_index, h, a_src, a_dst, heads, slope=0.2):
    """LeakyReLU(a_src . h[src] + a_dst . h[tgt]) per (edge, head) -> (out64 [E,H], scale)."""
    ei = _i64(edge_index)
    h = np.ascontiguousarray(h, dtype=np.float32)
    N = h.shape[0]
    D = h.shape[1] // heads
    a_src = np.ascontiguousarray(a_src, dtype=np.float32).reshape(heads, D)
    a_dst = np.ascontiguousarray(a_dst, dtype=np.float32).reshape(heads, D)
    E = ei.shape[1]
    src, tgt = np.ascontiguousarray(ei[0]), np.ascontiguousarray(ei[1])
    out64 = np.empty((E, heads), np.float64)
    scale = np.empty((E, heads), np.float64)
    _check(lib().orc_gat_scores(E, _ptr(src), _ptr(tgt), _ptr(h), N, heads, D, _ptr(a_src),
                                _ptr(a_dst), float(slope), _ptr(out64), _ptr(scale)))
    return out64, scale


def gat_layer(edge_index, h, a_src, a_dst, heads, slope=0.2):
    """Attention layer after the projection: (out64 [N, H*D], alpha64 [E, H], scale [N, H*D])."""
    ei = _i64(edge_index)
    h = np.ascontiguousarray(h, dtype=np.float32)
    N = h.shape[0]
    D = h.shape[1] // heads
    a_src = np.ascontiguousarray(a_src, dtype=np.float32).reshape(heads, D)
    a_dst = np.ascontiguousarray(a_dst, dtype=np.float32).reshape(heads, D)
    E = ei.shape[1]
    src, tgt = np.ascontiguousarray(ei[0]), np.ascontiguousarray(ei[1])
    out64 = np.empty((N, heads * D), np.float64)
    alpha = np.empty((E, heads), np.float64)
    scale = np.empty((N, heads * D), np.float64)
    _check(lib().orc_gat_layer(E, _ptr(src), _ptr(tgt), _ptr(h), N, heads, D, _ptr(a_src),
                               _ptr(a_dst), float(slope), _ptr(out64), _ptr(alpha), _ptr(scale)))
    return out64, alpha, scale


def batch_offsets(sizes):
    sizes = _i64(sizes)
    off = np.empty(sizes.shape[0] + 1, np.int64)
    lib().orc_batch_offsets(sizes.shape[0], _ptr(sizes), _ptr(off))
    return off


def batch_graphs(sizes, graphs):
    """Combine local graphs into one BatchGraph: (edge_index [2,E], graph_index [Nb])."""
    sizes = _i64(sizes)
    counts = np.array([g.shape[1] for g in graphs], np.int64)
    flat = (np.concatenate([_i64(g).reshape(-1) for g in graphs]) if graphs
            else np.zeros(0, np.int64))
    E = int(counts.sum())
    out = np.empty((2, E), np.int64)
    gi = np.empty(int(sizes.sum()), np.int64)
    lib().orc_batch_graphs(sizes.shape[0], _ptr(sizes), _ptr(counts), _ptr(flat),
                           _ptr(out[0]), _ptr(out[1]), _ptr(gi))
    return out, gi
