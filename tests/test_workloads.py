"""GPU parity on the five workloads at full size, in the launch configuration
the benchmark uses (graph handle with self-loops, CSR-order weights).

Each stage is checked on its own: the oracle of a stage consumes the GPU's
output of the previous stage (bit-identical inputs), so every stage is gated
on its own error and argmax stays checkable bit for bit. The largest graph is
checked in full: the graph order, degrees and normalised weights bit for bit,
and every output row of the aggregation, of its gradients and of the first
propagation step against the oracle (threads split the oracle's rows or edges;
the results are bit-identical to one thread).
"""

import numpy as np
import pytest

import graphgen
from graph_order import expected_graph
from test_parity import assert_rel, assert_scaled, dev, host, same_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tfg():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no ROCm device")
    import paper_2101_11552_amd as lib
    lib.load()
    return lib


def gcn_layer_setup(tfg, orc, ei, n):
    g = tfg.tfg_graph_create(dev(ei.astype(np.int32)), n, add_self_loops=True)
    norm = tfg.tfg_gcn_norm(dev(ei.astype(np.int32)), n, graph=g)
    oei, ow, odeg = orc.gcn_norm(ei, n)
    assert np.array_equal(host(norm["edge_index"]), oei)
    assert same_bits(host(norm["deg"]), odeg)
    assert same_bits(host(norm["edge_weight"]), ow)
    return g, norm, oei, ow


@pytest.mark.parametrize("name", ["uniform-2708", "uniform-19717"])
def test_uniform_graphs(tfg, orc, name):
    c = graphgen.WORKLOADS[name]()
    ei, x, n = c["edge_index"], c["x"], c["N"]
    g, norm, oei, ow = gcn_layer_setup(tfg, orc, ei, n)
    xd = dev(x)
    kw = dict(edge_weight=norm["edge_weight_csr"], weight_order="csr", graph=g)
    y = tfg.tfg_aggregate(norm["edge_index"], xd, n, "sum", **kw)
    ref, S = orc.aggregate(oei, x, n, "sum", edge_weight=ow)
    assert_scaled(host(y), ref, S, what=f"{name} sum")
    if name == "uniform-19717":
        ym = tfg.tfg_aggregate(norm["edge_index"], xd, n, "mean", **kw)
        ref, S = orc.aggregate(oei, x, n, "mean", edge_weight=ow)
        assert_scaled(host(ym), ref, S, what="uniform-19717 mean")
        mx, arg = tfg.tfg_aggregate(norm["edge_index"], xd, n, "max", **kw)
        rmx, rarg = orc.aggregate(oei, x, n, "max", edge_weight=ow)
        assert same_bits(host(mx), rmx) and np.array_equal(host(arg), rarg)


def test_gat_attention(tfg, orc):
    c = graphgen.attention_graph()
    ei, h, n, H = c["edge_index"], c["h"], c["N"], c["H"]
    eid = dev(ei.astype(np.int32))
    g = tfg.tfg_graph_create(eid, n)  # no self-loops on this workload
    s = tfg.tfg_gat_edge_scores(eid, dev(h), dev(c["a_src"]), dev(c["a_dst"]), c["slope"])
    ref, S = orc.gat_scores(ei, h, c["a_src"], c["a_dst"], H, slope=np.float32(c["slope"]))
    assert_scaled(host(s), ref, S, what="attention scores")
    alpha, alpha_csr = tfg.tfg_segment_softmax(s, eid[1], n, graph=g, out_csr=True)
    s_h = host(s)
    a64, _ = orc.segment_softmax(s_h, ei[1], n)
    assert_rel(host(alpha), a64, what="attention softmax")
    y = tfg.tfg_aggregate(eid, dev(h), n, "sum", edge_weight=alpha_csr, heads=H,
                          weight_order="csr", graph=g)
    ref, S = orc.aggregate(ei, h, n, "sum", edge_weight=host(alpha), heads=H)
    assert_scaled(host(y), ref, S, what="attention per-head aggregation")
    empty = np.bincount(ei[1], minlength=n) == 0
    assert empty.mean() > 0.2 and np.all(host(y)[empty] == 0)
    # the same layer with scores and alpha kept in the graph order
    perm = expected_graph(orc, ei, n)[2]
    s_g = tfg.tfg_gat_graph_scores(g, dev(h), dev(c["a_src"]), dev(c["a_dst"]), c["slope"],
                                   order="csr")
    assert same_bits(host(s_g), s_h[perm])
    a_g = tfg.tfg_segment_softmax_graph(g, s_g, order="csr")
    assert same_bits(host(a_g), host(alpha_csr))
    assert_rel(host(a_g), a64[perm], what="attention softmax in graph order")
    y_g = tfg.tfg_aggregate(None, dev(h), n, "sum", edge_weight=a_g, heads=H, weight_order="csr",
                            graph=g)
    assert same_bits(host(y_g), host(y))


def test_batched_pooling(tfg, orc):
    c = graphgen.graph_batch()
    ei, x, n, G = c["edge_index"], c["x"], c["N"], c["G"]
    g, norm, oei, ow = gcn_layer_setup(tfg, orc, ei, n)
    kw = dict(edge_weight=norm["edge_weight_csr"], weight_order="csr", graph=g)
    hd = dev(x)
    scale = np.abs(x).astype(np.float32)
    for layer in range(c["layers"]):
        h_in = host(hd)
        hd = tfg.tfg_aggregate(norm["edge_index"], hd, n, "sum", **kw)
        ref, S = orc.aggregate(oei, h_in, n, "sum", edge_weight=ow)
        assert_scaled(host(hd), ref, S, what=f"batch layer {layer}")
        scale = orc.aggregate(oei, scale, n, "sum", edge_weight=np.abs(ow))[0].astype(np.float32)
    # the independent chain, against |A_hat|^3 |x|
    ind = x
    for _ in range(c["layers"]):
        ind = orc.aggregate(oei, ind, n, "sum", edge_weight=ow)[0].astype(np.float32)
    assert_scaled(host(hd), ind.astype(np.float64), scale.astype(np.float64) + 1e-30,
                  tol=4e-5, what="batch chained")
    gi = dev(c["graph_index"].astype(np.int32))
    h3 = host(hd)
    for red in ("sum", "mean"):
        p = tfg.tfg_segment_pool(hd, gi, G, red)
        ref, S = orc.segment_pool(h3, c["graph_index"], G, red)
        assert_scaled(host(p), ref, S, what=f"batch pool {red}")
    p, arg = tfg.tfg_segment_pool(hd, gi, G, "max")
    ref, rarg = orc.segment_pool(h3, c["graph_index"], G, "max")
    assert same_bits(host(p), ref) and np.array_equal(host(arg), rarg)


@pytest.fixture(scope="module")
def pl():
    return graphgen.power_law(dtype=np.int32)


@pytest.fixture(scope="module")
def pl_norm_ref(orc, pl):
    """The oracle's normalisation of the whole power-law graph: (edge_index'
    [2, E'] with the self-loops appended, w' [E'], deg [N])."""
    return orc.gcn_norm(pl["edge_index"], pl["N"])


@pytest.fixture(scope="module")
def pl_graph(tfg, pl):
    """The graph handle and normalisation in the launch configuration the
    benchmark times: self-loops, the library's source-part choice."""
    eid = dev(pl["edge_index"])
    n = pl["N"]
    g = tfg.tfg_graph_create(eid, n, add_self_loops=True)
    norm = tfg.tfg_gcn_norm(eid, n, graph=g)
    return eid, g, norm


@pytest.fixture(scope="module")
def pl_sum_ref(orc, pl, pl_norm_ref):
    """The oracle's sum aggregation A_hat x over every row (threads split the
    rows; bit-identical to one thread): (out64, scale)."""
    oei, ow, _ = pl_norm_ref
    return orc.aggregate_by_row_ranges(oei, pl["x"], pl["N"], "sum", edge_weight=ow)


@pytest.mark.timeout(900)
def test_power_law_plain_csr_bit_exact(tfg, orc, pl, pl_norm_ref):
    """One source part: the stable CSR by target (the paper's reduce key),
    every rowptr, col and perm entry against the oracle at full size."""
    n = pl["N"]
    oei = pl_norm_ref[0]
    g = tfg.tfg_graph_create(dev(pl["edge_index"]), n, add_self_loops=True, src_parts=1)
    assert g.info()["src_parts"] == 1 and g.info()["E"] == oei.shape[1]
    rowptr, col, perm = (host(t) for t in tfg.tfg_graph_csr(g))
    del g
    r, c, p = orc.csr_by_target(oei, n)
    assert np.array_equal(rowptr, r)
    assert np.array_equal(perm, p)
    assert np.array_equal(col, c)


@pytest.mark.timeout(900)
def test_power_law_graph_order_and_norm(tfg, orc, pl, pl_norm_ref, pl_graph):
    """The timed handle (several source parts): its order equals the oracle's
    plain CSR regrouped by source part inside each row, bit for bit; degrees
    and normalised weights (COO and graph order) bit-exact on the whole graph."""
    n = pl["N"]
    oei, ow, odeg = pl_norm_ref
    _, g, norm = pl_graph
    info = g.info()
    assert info["E"] == oei.shape[1] and info["n_rows_split"] > 0
    P = info["src_parts"]
    assert P > 1 and info["n_part_items"] > 0  # the part plan is the one timed
    rowptr, col, perm = (host(t) for t in tfg.tfg_graph_csr(g))
    r, c, p, seg = expected_graph(orc, oei, n, parts=P)
    assert np.array_equal(rowptr, r)
    assert np.array_equal(perm, p)
    assert np.array_equal(col, c)
    assert np.array_equal(host(tfg.tfg_graph_segments(g)), seg)
    del r, c, seg
    assert np.array_equal(host(norm["edge_index"]), oei)
    assert same_bits(host(norm["deg"]), odeg)
    assert same_bits(host(norm["edge_weight"]), ow)
    assert same_bits(host(norm["edge_weight_csr"]), ow[perm])


@pytest.mark.timeout(900)
def test_power_law_aggregate_every_row(tfg, pl, pl_graph, pl_sum_ref):
    """The timed aggregation (part plan, weights in graph order) on all
    232,965 x 128 outputs against the oracle; the row plan on the same graph
    likewise; the same call twice gives the same bits."""
    import os
    import torch
    n = pl["N"]
    _, g, norm = pl_graph
    ref, S = pl_sum_ref
    xd = dev(pl["x"])
    kw = dict(edge_weight=norm["edge_weight_csr"], weight_order="csr", graph=g)
    y = tfg.tfg_aggregate(None, xd, n, "sum", **kw)
    assert_scaled(host(y), ref, S, what="pl every row, part plan")
    y2 = tfg.tfg_aggregate(None, xd, n, "sum", **kw)
    assert torch.equal(y, y2)
    os.environ["TFG_PART_PLAN"] = "0"
    try:
        y3 = tfg.tfg_aggregate(None, xd, n, "sum", **kw)
    finally:
        del os.environ["TFG_PART_PLAN"]
    assert_scaled(host(y3), ref, S, what="pl every row, row plan")


@pytest.mark.timeout(900)
def test_power_law_sqrt_deg_fixed_point(tfg, pl, pl_graph):
    """A_hat sqrt(deg) = sqrt(deg) on every row, at F = 128 so that the
    gathered table (119 MB) takes the part plan, as timed."""
    import torch
    n = pl["N"]
    _, g, norm = pl_graph
    s = torch.sqrt(norm["deg"]).reshape(n, 1).repeat(1, pl["x"].shape[1]).contiguous()
    assert s.numel() * 4 >= 32 << 20
    ys = tfg.tfg_aggregate(None, s, n, "sum", edge_weight=norm["edge_weight_csr"],
                           weight_order="csr", graph=g)
    rel = (ys - s).abs() / s
    assert float(rel.max()) <= 1e-5


def test_power_law_int64_ids_match_int32(tfg, pl):
    """The 64-bit index kernels (loads of two registers per id in the sort's
    first pass and in the COO-order normalisation) at full size: the graph
    and the normalisation from int64 ids equal those from int32 ids bit for
    bit."""
    import torch
    ei, n = pl["edge_index"], pl["N"]
    outs = []
    for dt in (np.int32, np.int64):
        eid = dev(ei.astype(dt))
        g = tfg.tfg_graph_create(eid, n, add_self_loops=True)
        norm = tfg.tfg_gcn_norm(eid, n, graph=g)
        rowptr, col, perm = tfg.tfg_graph_csr(g)
        outs.append([rowptr, col, perm, tfg.tfg_graph_segments(g), norm["edge_index"],
                     norm["edge_weight"].view(torch.int32),
                     norm["edge_weight_csr"].view(torch.int32), norm["deg"].view(torch.int32)])
        del g, norm, eid
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def test_gat_attention_fused(tfg, orc):
    c = graphgen.attention_graph()
    ei, h, n, H = c["edge_index"], c["h"], c["N"], c["H"]
    g = tfg.tfg_graph_create(dev(ei.astype(np.int32)), n)
    out = tfg.tfg_gat_aggregate(g, dev(h), dev(c["a_src"]), dev(c["a_dst"]), c["slope"])
    ref, _, S = orc.gat_layer(ei, h, c["a_src"], c["a_dst"], H, slope=np.float32(c["slope"]))
    assert_scaled(host(out), ref, S, what="attention fused attention layer")


def _dw_by_edge_ranges(orc, edge_index, x, n, dy, threads):
    """The oracle's dw of a sum aggregation for every edge, and its error
    scale (the same dot products over |x| and |dy|), computed over ranges of
    edges in threads: an edge's gradient depends on that edge alone."""
    from concurrent.futures import ThreadPoolExecutor
    E = edge_index.shape[1]
    bounds = [E * i // threads for i in range(threads + 1)]
    ax, ady = np.abs(x), np.abs(dy)

    def chunk(i):
        sub = np.ascontiguousarray(edge_index[:, bounds[i]:bounds[i + 1]])
        d = orc.aggregate_backward(sub, x, n, dy, "sum")[1][:, 0]
        sc = orc.aggregate_backward(sub, ax, n, ady, "sum")[1][:, 0]
        return d, sc

    with ThreadPoolExecutor(threads) as pool:
        parts = list(pool.map(chunk, range(threads)))
    return np.concatenate([q[0] for q in parts]), np.concatenate([q[1] for q in parts])


@pytest.mark.timeout(900)
def test_power_law_backward_and_propagation_full_size(tfg, orc, pl, pl_norm_ref, pl_graph,
                                                       pl_sum_ref):
    """The backward aggregation and APPNP propagation at full size, as timed
    by the benchmark: dx over the transposed graph with the normalised
    weights in its order (every source row), dw in graph order (every
    position), APPNP K = 3 (the first step on every row; the K-step call
    equals three chained steps bit for bit)."""
    x, n = pl["x"], pl["N"]
    oei, ow, _ = pl_norm_ref
    eid, g, norm = pl_graph
    gt = tfg.tfg_graph_create_transposed(eid, n, add_self_loops=True)

    # the transposed graph: the oracle's plain CSR of the reversed edges,
    # regrouped by target part inside each source row
    P = gt.info()["src_parts"]
    trow, tcol, tperm = (host(t) for t in tfg.tfg_graph_csr(gt))
    r, c, p, _ = expected_graph(orc, oei[::-1], n, parts=P)
    assert np.array_equal(trow, r) and np.array_equal(tperm, p) and np.array_equal(tcol, c)
    del r, c, p, trow, tcol

    w_t = tfg.tfg_edge_reorder(norm["edge_weight_csr"], src=g, dst=gt)
    assert same_bits(host(w_t), ow[tperm])
    del tperm
    dy = graphgen.features(2004, n, x.shape[1])
    xd, dyd = dev(x), dev(dy)
    dx, _ = tfg.tfg_aggregate_backward(g, dyd, "sum", graph_t=gt, edge_weight=w_t,
                                       weight_order="csr_t")
    _, dw = tfg.tfg_aggregate_backward(g, dyd, "sum", x=xd, want_dx=False, want_dw=True,
                                       dw_order="csr")
    # dx of a sum aggregation is the aggregation over the reversed edges (pinned on the CPU)
    ref, S = orc.aggregate_by_row_ranges(oei[::-1], dy, n, "sum", edge_weight=ow)
    assert_scaled(host(dx), ref, S, what="pl dx, every source row")
    del ref, S, dx
    # dw: every graph position, each a dot product of a dy row and an x row
    perm = host(tfg.tfg_graph_csr(g)[2])
    ref_dw, S_dw = _dw_by_edge_ranges(orc, oei, x, n, dy, orc.host_threads())
    assert_scaled(host(dw)[:, 0], ref_dw[perm], S_dw[perm], what="pl dw, every position")
    del ref_dw, S_dw, dw, perm

    # APPNP, K = 3, alpha = 0.1
    alpha = 0.1
    w_csr = norm["edge_weight_csr"]
    z3 = tfg.tfg_propagate(g, xd, 3, alpha=alpha, h=xd, edge_weight=w_csr)
    z = xd
    for k in range(3):
        z = tfg.tfg_propagate(g, z, 1, alpha=alpha, h=xd, edge_weight=w_csr)
        if k == 0:
            z1 = host(z)
    assert same_bits(host(z3), host(z))
    agg, S = pl_sum_ref
    a32 = np.float64(np.float32(alpha))
    ref = (1 - a32) * agg + a32 * x
    S = (1 - a32) * S + a32 * np.abs(x)
    assert_scaled(z1, ref, S, what="pl APPNP first step, every row")


def test_transformer_attention_full_size(tfg, orc):
    """The Transformer-style attention layer (scaled dot-product scores) on the
    attention workload's graph, fused and as the unfused chain, as timed."""
    import torch
    c = graphgen.attention_graph()
    ei, n, H, D = c["edge_index"], c["N"], c["H"], c["D"]
    r = graphgen.rng_for(3003, 1)
    q, k, v = (r.standard_normal((n, H * D), dtype=np.float32) for _ in range(3))
    scale = 1.0 / np.sqrt(D)
    g = tfg.tfg_graph_create(dev(ei.astype(np.int32)), n)
    out = tfg.tfg_gat_dot_aggregate(g, dev(q), dev(k), dev(v), H, scale=scale)
    torch.cuda.synchronize()
    ref, _, S = orc.dot_layer(ei, q, k, v, H, np.float32(scale))
    assert_scaled(host(out), ref, S, what="attention fused dot attention")
    s = tfg.tfg_edge_dot_scores(g, dev(q), dev(k), H, scale=scale)
    rs = orc.dot_scores(ei, q, k, H, np.float32(scale))
    assert_scaled(host(s), rs, orc.dot_scores(ei, np.abs(q), np.abs(k), H, np.float32(scale)),
                  what="attention dot scores")
