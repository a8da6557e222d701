"""GPU parity of the backward calls (tfg_aggregate_backward, the transposed
graph, tfg_segment_softmax_backward) against the oracle's gradients, which
the CPU tests pin to finite differences of the forward oracle.

Bars: the transposed CSR bit-exact; dx and dw within the float32 summation
bound scaled by the size of the terms, |y - ref| / sum|terms| <= 1e-5, as for
the forward sums; the softmax gradient likewise, its terms being alpha * |dalpha|
and alpha * sum(alpha |dalpha|).
"""

import numpy as np
import pytest

import graphgen
from graph_order import expected_graph

from test_parity import TOL, assert_scaled, dev, host, same_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tfg():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no ROCm device")
    import paper_2101_11552_amd as lib
    lib.load()
    return lib


def with_loops(ei, n):
    return np.concatenate([ei, np.stack([np.arange(n), np.arange(n)])], axis=1)


@pytest.mark.parametrize("n,n_src,e,loops,parts,idx", [
    (3000, 3000, 40_000, False, 1, np.int32),
    (2000, 500, 30_001, False, 1, np.int64),   # rectangular: 2000 targets, 500 sources
    (4000, 4000, 90_000, True, 4, np.int32),   # loops, source parts of the transposed keys
])
def test_transposed_csr_bit_exact(tfg, orc, n, n_src, e, loops, parts, idx):
    ei = graphgen.random_graph(e, n, e, n_src=n_src)
    gt = tfg.tfg_graph_create_transposed(dev(ei.astype(idx)), n, N_src=n_src,
                                         add_self_loops=loops, src_parts=parts)
    assert gt.N == n_src and gt.N_src == n
    full = with_loops(ei, n) if loops else ei
    rowptr, col, perm = (host(t) for t in tfg.tfg_graph_csr(gt))
    r, c, p = expected_graph(orc, full[::-1], n_src, parts=parts, n_src=n)[:3]
    assert np.array_equal(rowptr, r) and np.array_equal(col, c) and np.array_equal(perm, p)


def _check_backward(tfg, orc, ei, n, n_src, F, reduce, w=None, heads=1, order="coo",
                    dw_order="coo", parts=1, loops=False, seed=0):
    import torch
    x = graphgen.features(seed + 1, n_src, F)
    dy = graphgen.features(seed + 2, n, F)
    full = with_loops(ei, n) if loops else ei
    E = full.shape[1]
    g = tfg.tfg_graph_create(dev(ei), n, N_src=n_src, add_self_loops=loops, src_parts=parts)
    gt = tfg.tfg_graph_create_transposed(dev(ei), n, N_src=n_src, add_self_loops=loops,
                                         src_parts=parts)
    w_dev = None
    if w is not None:
        w_dev = dev(w)
        if order == "csr":
            perm = host(tfg.tfg_graph_csr(g)[2])
            w_dev = dev(w.reshape(E, -1)[perm].reshape(w.shape))
    arg_dev, arg = None, None
    if reduce == "max":
        _, arg = orc.aggregate(full, x, n, "max", edge_weight=w, heads=heads)
        _, arg_dev = tfg.tfg_aggregate(None, dev(x), n, "max", edge_weight=w_dev, heads=heads,
                                       weight_order=order, graph=g)
        assert np.array_equal(host(arg_dev), arg), "forward argmax differs"
    dx, dw = tfg.tfg_aggregate_backward(g, dev(dy), reduce, graph_t=gt, x=dev(x),
                                        edge_weight=w_dev, heads=heads, weight_order=order,
                                        argmax=arg_dev, want_dx=True, want_dw=True,
                                        dw_order=dw_order)
    torch.cuda.synchronize()
    rdx, rdw = orc.aggregate_backward(full, x, n, dy, reduce, edge_weight=w, heads=heads, arg=arg)
    aw = None if w is None else np.abs(w)
    sdx, sdw = orc.aggregate_backward(full, np.abs(x), n, np.abs(dy), reduce, edge_weight=aw,
                                      heads=heads, arg=arg)
    wdx = assert_scaled(host(dx), rdx, sdx, what=f"dx {reduce}")
    hdw = host(dw)
    if dw_order == "csr":
        perm = host(tfg.tfg_graph_csr(g)[2])
        back = np.empty_like(hdw)
        back[perm] = hdw
        hdw = back
    wdw = assert_scaled(hdw, rdw, sdw, what=f"dw {reduce}")
    # reproducible bit for bit
    dx2, dw2 = tfg.tfg_aggregate_backward(g, dev(dy), reduce, graph_t=gt, x=dev(x),
                                          edge_weight=w_dev, heads=heads, weight_order=order,
                                          argmax=arg_dev, want_dx=True, want_dw=True,
                                          dw_order=dw_order)
    assert same_bits(host(dx), host(dx2)) and same_bits(host(dw), host(dw2))
    return wdx, wdw


@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
@pytest.mark.parametrize("F", [64, 33])
def test_backward_square(tfg, orc, reduce, F):
    n, e = 3000, 60_000
    # a target hub (long forward row) and, reversed, a source hub (long transposed row)
    a = graphgen.random_graph(11, n, e // 2, hub=7, hub_edges=3000)
    b = graphgen.random_graph(12, n, e // 2, hub=11, hub_edges=3000)[::-1]
    ei = np.ascontiguousarray(np.concatenate([a, b], axis=1))
    w = graphgen.rng_for(13, 1).uniform(-1.0, 2.0, ei.shape[1]).astype(np.float32)
    _check_backward(tfg, orc, ei, n, n, F, reduce, w=w, seed=F)


@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
def test_backward_rectangular_unweighted(tfg, orc, reduce):
    n, n_src, e = 1500, 700, 25_000
    ei = graphgen.random_graph(21, n, e, n_src=n_src)
    _check_backward(tfg, orc, ei, n, n_src, 16, reduce, seed=21)


@pytest.mark.parametrize("reduce", ["sum", "max"])
def test_backward_heads_csr_weights(tfg, orc, reduce):
    n, e, H, D = 2000, 30_000, 4, 16
    ei = graphgen.random_graph(31, n, e)
    w = graphgen.rng_for(31, 2).uniform(0.0, 1.0, (e + n, H)).astype(np.float32)
    _check_backward(tfg, orc, ei, n, n, H * D, reduce, w=w, heads=H, order="csr",
                    dw_order="csr", loops=True, seed=31)


@pytest.mark.parametrize("plan", ["0", "1"])
@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
def test_backward_source_parts(tfg, orc, monkeypatch, plan, reduce):
    # both graphs in 5 source parts, gathered by the row plan or the part plan
    monkeypatch.setenv("TFG_PART_PLAN", plan)
    n, e = 5000, 120_000
    ei = graphgen.random_graph(41, n, e, hub=3, hub_edges=4000)
    w = graphgen.rng_for(41, 2).uniform(-1.0, 1.0, ei.shape[1] + n).astype(np.float32)
    _check_backward(tfg, orc, ei, n, n, 32, reduce, w=w, parts=5, loops=True, seed=41)


def test_edge_reorder(tfg, orc):
    n, e, H = 3000, 40_000, 3
    ei = graphgen.random_graph(91, n, e, hub=4, hub_edges=2000)
    g = tfg.tfg_graph_create(dev(ei), n, add_self_loops=True)
    gt = tfg.tfg_graph_create_transposed(dev(ei), n, add_self_loops=True)
    full = with_loops(ei, n)
    v = graphgen.features(91, full.shape[1], H)
    p = orc.csr_by_target(full, n)[2]
    pt = orc.csr_by_target(full[::-1], n)[2]
    vg = tfg.tfg_edge_reorder(dev(v), dst=g)                 # COO -> graph order
    assert same_bits(host(vg), v[p])
    vt = tfg.tfg_edge_reorder(vg, src=g, dst=gt)              # graph -> transposed order
    assert same_bits(host(vt), v[pt])
    back = tfg.tfg_edge_reorder(vt, src=gt)                   # transposed -> COO order
    assert same_bits(host(back), v)


@pytest.mark.parametrize("idx", [np.int32, np.int64])
def test_edge_reorder_bucketed(tfg, orc, idx):
    # one value per edge on a graph of more than 2^20 edges: graph order ->
    # edge order runs through buckets of destinations (a ragged last bucket
    # and tile); every path back and forth gives the same bits
    import torch
    n, e = 200_003, 3_000_000
    ei = graphgen.random_graph(95, n, e, hub=7, hub_edges=40_000)
    g = tfg.tfg_graph_create(dev(ei.astype(idx)), n, add_self_loops=True)
    gt = tfg.tfg_graph_create_transposed(dev(ei.astype(idx)), n, add_self_loops=True)
    full = with_loops(ei, n)
    v = graphgen.features(95, full.shape[1], 1)[:, 0].copy()
    p = orc.csr_by_target(full, n)[2]
    pt = orc.csr_by_target(full[::-1], n)[2]
    vg = tfg.tfg_edge_reorder(dev(v), dst=g)
    assert same_bits(host(vg), v[p])
    back = tfg.tfg_edge_reorder(vg, src=g)                    # bucketed scatter
    assert same_bits(host(back), v)
    vt = tfg.tfg_edge_reorder(vg, src=g, dst=gt)              # bucketed scatter, then gather
    assert same_bits(host(vt), v[pt])
    # the backward with weights in the forward graph's order moves them to
    # edge order the same way: the same gradient as with weights in edge order
    dy = dev(graphgen.features(97, n, 16))
    a, _ = tfg.tfg_aggregate_backward(g, dy, "sum", graph_t=gt, edge_weight=dev(v))
    b, _ = tfg.tfg_aggregate_backward(g, dy, "sum", graph_t=gt, edge_weight=vg,
                                      weight_order="csr")
    torch.cuda.synchronize()
    assert same_bits(host(a), host(b))


@pytest.mark.parametrize("n,e", [
    (1 << 16, (1 << 20) - (1 << 16)),   # E' = 2^20: the smallest bucketed scatter
    (50_000, (1 << 21) - 50_000),       # E' = 2^21: whole tiles and buckets
    (50_001, (1 << 21) - 50_000),       # one edge more: a one-position tile and bucket
])
def test_edge_reorder_bucket_boundaries(tfg, orc, n, e):
    ei = graphgen.random_graph(n + 3, n, e)
    g = tfg.tfg_graph_create(dev(ei.astype(np.int32)), n, add_self_loops=True)
    full = with_loops(ei, n)
    v = graphgen.features(n + 3, full.shape[1], 1)[:, 0].copy()
    p = orc.csr_by_target(full, n)[2]
    back = tfg.tfg_edge_reorder(dev(v[p]), src=g)
    assert same_bits(host(back), v)


@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
def test_backward_transposed_order_weights(tfg, orc, reduce):
    # weights already in the transposed graph's order give the same gradients
    import torch
    n, e = 3000, 50_000
    ei = graphgen.random_graph(92, n, e, hub=6, hub_edges=2500)
    w = graphgen.rng_for(92, 2).uniform(-1.0, 1.0, ei.shape[1] + n).astype(np.float32)
    g = tfg.tfg_graph_create(dev(ei), n, add_self_loops=True)
    gt = tfg.tfg_graph_create_transposed(dev(ei), n, add_self_loops=True)
    x = dev(graphgen.features(93, n, 32))
    dy = dev(graphgen.features(94, n, 32))
    arg = tfg.tfg_aggregate(None, x, n, "max", edge_weight=dev(w), graph=g)[1] \
        if reduce == "max" else None
    wt = tfg.tfg_edge_reorder(dev(w), dst=gt)
    a, _ = tfg.tfg_aggregate_backward(g, dy, reduce, graph_t=gt, edge_weight=dev(w), argmax=arg)
    b, _ = tfg.tfg_aggregate_backward(g, dy, reduce, graph_t=gt, edge_weight=wt,
                                      weight_order="csr_t", argmax=arg)
    torch.cuda.synchronize()
    # the same products in the same order: the same bits
    assert same_bits(host(a), host(b))


def test_backward_wide_rows_fallback(tfg, orc):
    # 300 columns = 75 float4 vectors: the per-edge dot products take the simple kernel
    n, e = 400, 5000
    ei = graphgen.random_graph(51, n, e)
    w = graphgen.rng_for(51, 2).uniform(0.5, 1.5, e).astype(np.float32)
    _check_backward(tfg, orc, ei, n, n, 300, "mean", w=w, seed=51)
    _check_backward(tfg, orc, ei, n, n, 300, "max", w=w, seed=52)


def test_backward_gcn_chain(tfg, orc):
    # the GCN layer's aggregation with the normalised weights of tfg_gcn_norm
    n, e, F = 4000, 50_000, 64
    ei = graphgen.random_graph(61, n, e, hub=5, hub_edges=2000)
    g = tfg.tfg_graph_create(dev(ei), n, add_self_loops=True)
    gt = tfg.tfg_graph_create_transposed(dev(ei), n, add_self_loops=True)
    norm = tfg.tfg_gcn_norm(dev(ei), n, graph=g)
    w_coo = host(norm["edge_weight"])
    x = graphgen.features(61, n, F)
    dy = graphgen.features(62, n, F)
    dx, dw = tfg.tfg_aggregate_backward(g, dev(dy), "sum", graph_t=gt, x=dev(x),
                                        edge_weight=norm["edge_weight_csr"], weight_order="csr",
                                        want_dw=True)
    full = with_loops(ei, n)
    # tfg_gcn_norm's weights equal the oracle's bit for bit (test_gcn_norm_bit_exact)
    rdx, rdw = orc.aggregate_backward(full, x, n, dy, "sum", edge_weight=w_coo)
    sdx, sdw = orc.aggregate_backward(full, np.abs(x), n, np.abs(dy), "sum",
                                      edge_weight=np.abs(w_coo))
    assert_scaled(host(dx), rdx, sdx, what="dx")
    assert_scaled(host(dw)[:, 0], rdw[:, 0], sdw[:, 0], what="dw")


def test_backward_empty_and_isolated(tfg, orc):
    import torch
    # no edges: dx = 0, dw empty
    n = 50
    ei = np.zeros((2, 0), np.int64)
    g = tfg.tfg_graph_create(dev(ei), n)
    gt = tfg.tfg_graph_create_transposed(dev(ei), n)
    dy = dev(graphgen.features(71, n, 8))
    dx, dw = tfg.tfg_aggregate_backward(g, dy, "mean", graph_t=gt, x=dy, want_dw=True)
    torch.cuda.synchronize()
    assert np.all(host(dx) == 0) and dw.shape == (0, 1)
    # sources without out-edges get exactly 0
    ei = np.array([[0, 0, 2], [1, 3, 3]])
    _check_backward(tfg, orc, ei, 5, 5, 4, "sum")


def test_backward_argument_errors(tfg):
    n = 10
    ei = dev(np.array([[0, 1], [1, 2]]))
    g = tfg.tfg_graph_create(ei, n)
    gt = tfg.tfg_graph_create_transposed(ei, n)
    dy = dev(np.ones((n, 4), np.float32))
    with pytest.raises(ValueError):  # dx without the transposed graph
        tfg.tfg_aggregate_backward(g, dy, "sum")
    with pytest.raises(ValueError):  # max without the forward argmax
        tfg.tfg_aggregate_backward(g, dy, "max", graph_t=gt)
    with pytest.raises(ValueError):  # graphs swapped
        tfg.tfg_aggregate_backward(gt, dy[:n], "sum", graph_t=g)
    other = tfg.tfg_graph_create_transposed(dev(np.array([[0], [1]])), n)
    with pytest.raises(ValueError):  # gt of another edge list
        tfg.tfg_aggregate_backward(g, dy, "sum", graph_t=other)
    with pytest.raises(ValueError):  # dw without x
        tfg.tfg_aggregate_backward(g, dy, "sum", want_dx=False, want_dw=True)


@pytest.mark.parametrize("H,with_graph", [(1, True), (3, False), (8, True)])
def test_softmax_backward(tfg, orc, H, with_graph):
    import torch
    n, e = 3000, 50_000
    ei = graphgen.random_graph(81 + H, n, e, hub=9, hub_edges=5000)
    seg = ei[1]
    E = ei.shape[1]
    s = graphgen.features(81, E, H)
    da = graphgen.features(82, E, H)
    a64, a32 = orc.segment_softmax(s, seg, n)
    g = tfg.tfg_graph_create(dev(ei), n) if with_graph else None
    ds = tfg.tfg_segment_softmax_backward(dev(a32), dev(da), dev(seg), n, graph=g)
    torch.cuda.synchronize()
    ref = orc.segment_softmax_backward(a32, da, seg, n)
    # terms: alpha |dalpha| and alpha * sum over the segment of alpha |dalpha|
    dot = np.zeros((n, H))
    np.add.at(dot, seg, a32.astype(np.float64) * np.abs(da))
    S = a32 * (np.abs(da) + dot[seg])
    assert_scaled(host(ds), ref, S, what="dscores")


@pytest.mark.parametrize("reduce,idx", [("sum", np.int32), ("mean", np.int64), ("max", np.int32)])
def test_pool_backward(tfg, orc, reduce, idx):
    import torch
    sizes = graphgen.rng_for(95, 0).integers(0, 40, 300)  # some graphs without nodes
    gi = np.repeat(np.arange(300), sizes)
    Nb, F, G = gi.shape[0], 24, 300
    x = graphgen.features(95, Nb, F)
    dy = graphgen.features(96, G, F)
    arg_dev, arg = None, None
    if reduce == "max":
        _, arg_dev = tfg.tfg_segment_pool(dev(x), dev(gi.astype(idx)), G, "max")
        _, arg = orc.segment_pool(x, gi, G, "max")
        assert np.array_equal(host(arg_dev), arg)
    dx = tfg.tfg_segment_pool_backward(dev(dy), dev(gi.astype(idx)), reduce, argmax=arg_dev)
    torch.cuda.synchronize()
    ref = orc.segment_pool_backward(dy, gi, G, reduce, arg=arg)
    # sum and max copy dy exactly; mean divides once in float32 (dy / count)
    if reduce == "mean":
        cnt = np.bincount(gi, minlength=G)[gi][:, None]
        assert same_bits(host(dx), (dy[gi] / cnt.astype(np.float32)).astype(np.float32))
        np.testing.assert_allclose(host(dx), ref, rtol=1e-6)
    else:
        assert same_bits(host(dx), ref.astype(np.float32))


def test_pool_backward_rejects_bad_index(tfg):
    dy = dev(np.ones((3, 4), np.float32))
    with pytest.raises(ValueError):  # decreasing ids (TfgValueError for TFG_ERR_UNSORTED)
        tfg.tfg_segment_pool_backward(dy, dev(np.array([0, 2, 1], np.int32)))
    with pytest.raises(IndexError):
        tfg.tfg_segment_pool_backward(dy, dev(np.array([0, 1, 3], np.int32)))


def test_new_calls_on_empty_inputs(tfg):
    import torch
    n = 20
    ei = dev(np.zeros((2, 0), np.int64))
    g = tfg.tfg_graph_create(ei, n)
    gt = tfg.tfg_graph_create_transposed(ei, n)
    x = dev(graphgen.features(97, n, 16))
    # attention over a graph without edges: zero output, nothing to score
    out = tfg.tfg_gat_dot_aggregate(g, x, x, x, 4)
    s = tfg.tfg_edge_dot_scores(g, x, x, 4)
    # reordering an empty per-edge array, pooling gradient without nodes
    r = tfg.tfg_edge_reorder(torch.zeros((0, 2), device=x.device), src=g, dst=gt)
    dxp = tfg.tfg_segment_pool_backward(dev(np.ones((3, 4), np.float32)),
                                        dev(np.zeros(0, np.int32)))
    # F = 0 features
    dx0, _ = tfg.tfg_aggregate_backward(g, dev(np.zeros((n, 0), np.float32)), "sum", graph_t=gt)
    torch.cuda.synchronize()
    assert np.all(host(out) == 0) and s.shape == (0, 4) and r.shape == (0, 2)
    assert dxp.shape == (0, 4) and dx0.shape == (n, 0)


@pytest.mark.parametrize("seed", range(20))
def test_random_backward_configurations(tfg, orc, seed):
    """Seeded random backward cases: graph shape (square with or without
    loops, rectangular), hub rows on either side, source parts, reducer,
    heads, weight order and gradient order, against the oracle."""
    r = np.random.default_rng([9003, seed])
    n = int(r.integers(2, 2500))
    square = r.random() < 0.6
    n_src = n if square else int(r.integers(2, 2500))
    heads = int(r.choice([1, 1, 2, 4]))
    F = heads * int(r.choice([1, 4, 16, 32]))
    reduce = str(r.choice(["sum", "mean", "max"]))
    a = graphgen.random_graph(600 + seed, n, int(r.integers(1, 20_000)), n_src=n_src,
                              hub=0, hub_edges=int(r.choice([0, 2000])))
    loops = bool(square and r.random() < 0.5)
    E = a.shape[1] + (n if loops else 0)
    w = (graphgen.rng_for(700 + seed, 1).uniform(-1.0, 2.0, (E, heads) if heads > 1 else E)
         .astype(np.float32))
    order = str(r.choice(["coo", "csr"]))
    dw_order = str(r.choice(["coo", "csr"]))
    _check_backward(tfg, orc, a, n, n_src, F, reduce, w=w, heads=heads, order=order,
                    dw_order=dw_order, parts=int(r.choice([1, 2, 4])), loops=loops, seed=seed)
