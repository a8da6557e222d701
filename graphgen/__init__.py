"""Seeded synthetic graph inputs for the aggregation / pooling hot path.

This module only draws random inputs: node features, COO edge lists, attention
vectors and batched graph indices. It holds none of the method's arithmetic
(no normalisation, no sorting by target, no reductions); both the oracle and
the HIP library consume the arrays it returns.

Every generator takes an explicit integer seed and derives independent numpy
``default_rng`` streams from ``[seed, stream]``:

* stream 0 — graph structure (edges, node relabelling, edge-order shuffle)
* stream 1 — node features
* stream 2 — attention vectors

The five workloads mirror the shapes of the paper's evaluation graphs (the
paper's own datasets are not available here, so these stand in for their
sizes and degree structure):

* ``uniform_small`` — 2,708 nodes, 5,278 distinct undirected pairs (citation-graph
  sized), F = 64.
* ``uniform_medium`` — 19,717 nodes, 44,324 distinct undirected pairs, F = 128.
* ``attention_graph`` — 169,343 nodes, Barabási–Albert preferential attachment with
  m = 7 (directed new -> old), 8 heads x 16 dims.
* ``power_law`` — 232,965 nodes, Chung–Lu power law (gamma = 2), 114.6M directed
  edges, F = 128.
* ``graph_batch`` — 4,096 small graphs of 10..60 nodes, G(n, 0.1), batched into one
  disjoint graph with a sorted graph index, F = 64.

Edge lists are int64 arrays of shape [2, E]: row 0 holds source ids, row 1
target ids. Features are float32, row-major.
"""

from __future__ import annotations

import numpy as np

SEED_BASE = 1000  # workload k uses seed SEED_BASE + k


def rng_for(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(stream)])


def features(seed: int, n: int, f: int, stream: int = 1) -> np.ndarray:
    """x ~ N(0, 1), float32, shape [n, f]."""
    return rng_for(seed, stream).standard_normal((n, f), dtype=np.float32)


def _relabel_and_shuffle(rng: np.random.Generator, n: int, src: np.ndarray,
                         tgt: np.ndarray, dtype=np.int64) -> np.ndarray:
    """Random node relabelling plus a random edge order, so that neither node
    ids nor edge positions carry structure."""
    relabel = rng.permutation(n).astype(dtype)
    e = src.shape[0]
    order = np.arange(e, dtype=np.int32 if e < 2**31 else np.int64)
    rng.shuffle(order)
    ei = np.empty((2, e), dtype=dtype)
    ei[0] = relabel[src[order]]
    ei[1] = relabel[tgt[order]]
    return ei


def _inverse_cdf(cdf: np.ndarray, u: np.ndarray, table: np.ndarray) -> np.ndarray:
    """Smallest i with cdf[i] > u, found from a guide table (table[j] = smallest
    i with cdf[i] > j / len(table)) followed by a forward scan."""
    m = table.shape[0]
    idx = table[np.minimum((u * m).astype(np.int64), m - 1)]
    while True:
        short = np.nonzero(cdf[idx] <= u)[0]
        if short.size == 0:
            return idx
        idx[short] += 1


def uniform_pairs(seed: int, n: int, n_pairs: int) -> np.ndarray:
    """``n_pairs`` distinct unordered pairs {u, v}, u != v, drawn uniformly
    (repeats rejected), emitted in both directions: edge_index [2, 2*n_pairs]."""
    rng = rng_for(seed, 0)
    keys = np.empty(0, dtype=np.int64)
    while keys.shape[0] < n_pairs:
        m = 2 * (n_pairs - keys.shape[0]) + 64
        a = rng.integers(0, n, size=m, dtype=np.int64)
        b = rng.integers(0, n, size=m, dtype=np.int64)
        keep = a != b
        lo = np.minimum(a[keep], b[keep])
        hi = np.maximum(a[keep], b[keep])
        cand = np.concatenate([keys, lo * n + hi])
        _, first = np.unique(cand, return_index=True)
        keys = cand[np.sort(first)]  # first occurrence, in draw order
    keys = keys[:n_pairs]
    u, v = keys // n, keys % n
    src = np.concatenate([u, v])
    tgt = np.concatenate([v, u])
    return _relabel_and_shuffle(rng, n, src, tgt)


def barabasi_albert(seed: int, n: int, m: int) -> np.ndarray:
    """Preferential attachment: m isolated seed nodes; node m links to all of
    them; every later node v links to m distinct existing nodes drawn with
    probability proportional to their current degree (uniform draws from the
    list that repeats each node once per incident edge). Edges point from the
    new node to the old one: E = m * (n - m)."""
    rng = rng_for(seed, 0)
    E = m * (n - m)
    src = np.empty(E, dtype=np.int64)
    tgt = np.empty(E, dtype=np.int64)
    rep = np.empty(2 * E, dtype=np.int64)  # repeated-node list
    src[:m] = m
    tgt[:m] = np.arange(m)
    rep[:m] = np.arange(m)
    rep[m:2 * m] = m
    n_rep = 2 * m
    e = m
    for v in range(m + 1, n):
        chosen: list[int] = []
        while len(chosen) < m:
            draws = rep[rng.integers(0, n_rep, size=2 * m)]
            for d in draws.tolist():
                if d not in chosen:
                    chosen.append(d)
                    if len(chosen) == m:
                        break
        src[e:e + m] = v
        tgt[e:e + m] = chosen
        rep[n_rep:n_rep + m] = chosen
        rep[n_rep + m:n_rep + 2 * m] = v
        n_rep += 2 * m
        e += m
    return _relabel_and_shuffle(rng, n, src, tgt)


def chung_lu(seed: int, n: int, n_pairs: int, offset: float = 850.2,
             chunk: int = 1 << 24, dtype=np.int64) -> np.ndarray:
    """Chung–Lu power law with gamma = 2: node i has weight (i + offset)^-1;
    ``n_pairs`` endpoint pairs are drawn i.i.d. proportional to weight (self
    pairs redrawn), each emitted in both directions; duplicates are kept."""
    rng = rng_for(seed, 0)
    wt = 1.0 / (np.arange(n, dtype=np.float64) + offset)
    cdf = np.cumsum(wt)
    cdf /= cdf[-1]
    cdf[-1] = 2.0  # every u in [0, 1) lands at or before the last node
    table = np.searchsorted(cdf, np.arange(4 * n) / (4 * n), side="right").astype(np.int32)
    ab = np.empty(2 * n_pairs, dtype=np.int32)
    a, b = ab[:n_pairs], ab[n_pairs:]
    for lo in range(0, n_pairs, chunk):
        hi = min(n_pairs, lo + chunk)
        a[lo:hi] = _inverse_cdf(cdf, rng.random(hi - lo), table)
        b[lo:hi] = _inverse_cdf(cdf, rng.random(hi - lo), table)
    while True:
        bad = np.nonzero(a == b)[0]
        if bad.size == 0:
            break
        b[bad] = _inverse_cdf(cdf, rng.random(bad.size), table)
    ba = np.concatenate([b, a])  # reverse direction of every pair
    return _relabel_and_shuffle(rng, n, ab, ba, dtype)


def random_graph(seed: int, n: int, e: int, n_src: int | None = None,
                 hub: int | None = None, hub_edges: int = 0,
                 self_loops: bool = True) -> np.ndarray:
    """Unstructured test graph: ``e`` edges with uniform endpoints (duplicates
    and self-loops allowed unless ``self_loops`` is False), plus optionally
    ``hub_edges`` extra edges all pointing at target ``hub`` (a skewed row)."""
    rng = rng_for(seed, 0)
    n_src = n if n_src is None else n_src
    src = rng.integers(0, n_src, size=e, dtype=np.int64)
    tgt = rng.integers(0, n, size=e, dtype=np.int64)
    if not self_loops and n_src == n and n > 1:
        bad = src == tgt
        while bad.any():
            src[bad] = rng.integers(0, n_src, size=int(bad.sum()), dtype=np.int64)
            bad = src == tgt
    if hub is not None and hub_edges > 0:
        hs = rng.integers(0, n_src, size=hub_edges, dtype=np.int64)
        src = np.concatenate([src, hs])
        tgt = np.concatenate([tgt, np.full(hub_edges, hub, dtype=np.int64)])
        order = rng.permutation(src.shape[0])
        src, tgt = src[order], tgt[order]
    return np.stack([src, tgt])


def batch_of_small_graphs(seed: int, n_graphs: int, n_min: int, n_max: int,
                          p: float):
    """``n_graphs`` independent G(n, p) graphs with n ~ U{n_min..n_max}; every
    unordered pair i < j is kept with probability p and emitted in both
    directions. Returns (sizes [G], local edge lists: list of int64 [2, e_g])."""
    rng = rng_for(seed, 0)
    sizes = rng.integers(n_min, n_max + 1, size=n_graphs, dtype=np.int64)
    graphs = []
    for n in sizes.tolist():
        iu, ju = np.triu_indices(n, k=1)
        keep = rng.random(iu.shape[0]) < p
        i, j = iu[keep].astype(np.int64), ju[keep].astype(np.int64)
        graphs.append(np.stack([np.concatenate([i, j]), np.concatenate([j, i])]))
    return sizes, graphs


def stack_batch(sizes: np.ndarray, graphs: list[np.ndarray]):
    """Input preparation for a batch of disjoint graphs: node j of graph i gets
    global id j + (number of nodes in graphs 0..i-1); edge lists are shifted
    accordingly and stacked; graph_index[n] is the graph of node n (sorted)."""
    n_total = int(sizes.sum())
    graph_index = np.repeat(np.arange(sizes.shape[0], dtype=np.int64), sizes)
    start = 0
    parts = []
    for n, g in zip(sizes.tolist(), graphs):
        parts.append(g + start)
        start += n
    edge_index = np.concatenate(parts, axis=1) if parts else np.zeros((2, 0), np.int64)
    assert start == n_total
    return edge_index, graph_index


# ---------------------------------------------------------------------------
# The five workloads
# ---------------------------------------------------------------------------

def uniform_small():
    s = SEED_BASE + 1
    n = 2708
    return {"name": "uniform-2708", "N": n, "F": 64, "edge_index": uniform_pairs(s, n, 5278),
            "x": features(s, n, 64)}


def uniform_medium():
    s = SEED_BASE + 2
    n = 19717
    return {"name": "uniform-19717", "N": n, "F": 128, "edge_index": uniform_pairs(s, n, 44324),
            "x": features(s, n, 128)}


def attention_graph():
    s = SEED_BASE + 3
    n, heads, dims = 169343, 8, 16
    ra = rng_for(s, 2)
    return {"name": "ba-169343", "N": n, "H": heads, "D": dims,
            "edge_index": barabasi_albert(s, n, 7),
            "h": features(s, n, heads * dims),
            "a_src": ra.standard_normal((heads, dims), dtype=np.float32),
            "a_dst": ra.standard_normal((heads, dims), dtype=np.float32),
            "slope": 0.2}


def power_law(n_pairs: int = 57_300_000, dtype=np.int64):
    s = SEED_BASE + 4
    n = 232965
    return {"name": "powerlaw-232965", "N": n, "F": 128,
            "edge_index": chung_lu(s, n, n_pairs, dtype=dtype),
            "x": features(s, n, 128)}


def graph_batch():
    s = SEED_BASE + 5
    sizes, graphs = batch_of_small_graphs(s, 4096, 10, 60, 0.1)
    edge_index, graph_index = stack_batch(sizes, graphs)
    nb = int(sizes.sum())
    return {"name": "batch-4096", "N": nb, "F": 64, "G": 4096, "layers": 3,
            "sizes": sizes, "graphs": graphs, "edge_index": edge_index,
            "graph_index": graph_index, "x": features(s, nb, 64)}


WORKLOADS = {"uniform-2708": uniform_small, "uniform-19717": uniform_medium, "ba-169343": attention_graph,
             "powerlaw-232965": power_law, "batch-4096": graph_batch}
