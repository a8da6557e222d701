"""HIP graphs around the library's stream-ordered calls on a cached graph.

A serving loop or a training step calls the same sequence of kernels over
the same graph again and again: the normalisation's graph-order weights, the
layers' aggregations, the pools, the attention's scores and softmax. These
calls launch on the caller's stream and neither synchronise nor allocate
device memory in the library (the binding's torch allocations come from the
graph's private pool), so the sequence can be captured once as a HIP graph
and replayed. Every replay here is checked bit for bit against the same
calls run eagerly on the same inputs, with the inputs changed and other
eager work (and synchronisation) between the replays.
"""

import numpy as np
import pytest

import graphgen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tfg():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no ROCm device")
    import paper_2101_11552_amd as lib
    lib.load()
    return lib


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def bits(t):
    a = t.detach().cpu().numpy()
    return a.view(np.uint32) if a.dtype == np.float32 else a


def capture(fn):
    """(graph, static outputs) of fn() captured after two warm-up runs on a
    side stream."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    gr = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gr):
        out = fn()
    torch.cuda.synchronize()
    return gr, out


def check_replays(tfg, gr, out, fn, x_static, new_x, other):
    """Replays with new inputs, each against fn() run eagerly on the same
    inputs; `other` is unrelated eager library work run between them."""
    import torch
    for rep in range(4):
        x_static.copy_(new_x(rep))
        other()
        torch.cuda.synchronize()
        gr.replay()
        torch.cuda.synchronize()
        ref = fn()
        torch.cuda.synchronize()
        for a, b in zip(out, ref):
            assert np.array_equal(bits(a), bits(b)), f"replay {rep} differs from the eager calls"


def test_minibatch_forward_replays(tfg, orc):
    """Normalisation (graph-order weights), three sum aggregations and three
    pools over a cached BatchGraph, as one graph."""
    import torch
    sizes, graphs = graphgen.batch_of_small_graphs(61, 400, 10, 60, 0.1)
    ei, gi = graphgen.stack_batch(sizes, graphs)
    nb, G, F = int(sizes.sum()), sizes.shape[0], 64
    eid, gid = dev(ei.astype(np.int32)), dev(gi.astype(np.int32))
    g = tfg.tfg_graph_create(eid, nb, add_self_loops=True)
    x_static = dev(graphgen.features(62, nb, F))

    def fwd():
        w = tfg.tfg_gcn_norm(eid, nb, graph=g, out_edge_index=False, out_edge_weight=False,
                             out_deg=False)["edge_weight_csr"]
        h = x_static
        for _ in range(3):
            h = tfg.tfg_aggregate(None, h, nb, "sum", edge_weight=w, weight_order="csr", graph=g)
        s = tfg.tfg_segment_pool(h, gid, G, "sum", validate=False)
        m = tfg.tfg_segment_pool(h, gid, G, "mean", validate=False)
        mx, arg = tfg.tfg_segment_pool(h, gid, G, "max", validate=False)
        return [h, s, m, mx, arg]

    gr, out = capture(fwd)
    other_x = dev(graphgen.features(63, nb, F))
    check_replays(tfg, gr, out, fwd, x_static, lambda r: dev(graphgen.features(70 + r, nb, F)),
                  lambda: tfg.tfg_aggregate(eid, other_x, nb, "mean"))
    # the last replay's layers against the oracle (three chained layers, 4e-5)
    oei, ow, _ = orc.gcn_norm(ei, nb)
    hx = graphgen.features(73, nb, F)
    S = np.abs(hx).astype(np.float64)
    for _ in range(3):
        hx = orc.aggregate(oei, hx, nb, "sum", edge_weight=ow)[0].astype(np.float32)
        S = orc.aggregate(oei, S.astype(np.float32), nb, "sum", edge_weight=np.abs(ow))[0]
    y = out[0].cpu().numpy().astype(np.float64)
    assert float((np.abs(y - hx) / np.maximum(S, 1e-30)).max()) <= 4e-5
    del gr
    torch.cuda.synchronize()


def test_attention_layer_in_graph_order_replays(tfg):
    """Scores, softmax and per-head aggregation with the per-edge arrays in
    the graph order (long rows split into chunks), as one graph."""
    import torch
    n, H, D = 3000, 8, 16
    ei = graphgen.random_graph(64, n, 40_000, hub=5, hub_edges=4000)
    g = tfg.tfg_graph_create(dev(ei), n)
    x_static = dev(graphgen.features(65, n, H * D))
    r = np.random.default_rng(66)
    a_s = dev(r.standard_normal((H, D)).astype(np.float32))
    a_d = dev(r.standard_normal((H, D)).astype(np.float32))

    def layer():
        s = tfg.tfg_gat_graph_scores(g, x_static, a_s, a_d, order="csr")
        a = tfg.tfg_segment_softmax_graph(g, s, order="csr")
        y = tfg.tfg_aggregate(None, x_static, n, "sum", edge_weight=a, heads=H,
                              weight_order="csr", graph=g)
        return [s, a, y]

    gr, out = capture(layer)
    check_replays(tfg, gr, out, layer, x_static,
                  lambda rep: dev(graphgen.features(80 + rep, n, H * D)),
                  lambda: tfg.tfg_gat_aggregate(g, x_static, a_s, a_d, 0.2))
    del gr
    torch.cuda.synchronize()


@pytest.mark.parametrize("plan", ["0", "1"])
def test_aggregation_plans_replay(tfg, monkeypatch, plan):
    """The row plan (chunks and their fix-up) and the source-part plan
    (partial rows and their fix-up) of the sum aggregation, as one graph."""
    import torch
    monkeypatch.setenv("TFG_PART_PLAN", plan)
    n, F = 2500, 128
    ei = graphgen.random_graph(67, n, 60_000, hub=9, hub_edges=9000)
    g = tfg.tfg_graph_create(dev(ei), n, src_parts=4)
    w = dev(np.random.default_rng(68).standard_normal(g.E).astype(np.float32))
    x_static = dev(graphgen.features(69, n, F))

    def agg():
        return [tfg.tfg_aggregate(None, x_static, n, "sum", edge_weight=w, weight_order="csr",
                                  graph=g),
                tfg.tfg_aggregate(None, x_static, n, "max", edge_weight=w, weight_order="csr",
                                  graph=g)[1]]

    gr, out = capture(agg)
    check_replays(tfg, gr, out, agg, x_static, lambda rep: dev(graphgen.features(90 + rep, n, F)),
                  lambda: tfg.tfg_aggregate(None, x_static, n, "mean", graph=g))
    del gr
    torch.cuda.synchronize()
