"""Training through the attention layer with the library's calls: the
gradient of the additive GAT layer (Fig. 5a plus the weighted sum) w.r.t. its
input features, composed from tfg_edge_dot_scores (d alpha),
tfg_segment_softmax_backward (d scores), tfg_aggregate over the forward and
transposed graphs (per-node sums of per-edge values) and
tfg_aggregate_backward (the gradient through the weighted sum), against
central differences of the oracle's layer. Elementwise steps (the LeakyReLU
slope, the per-head broadcast of a_src / a_dst) are plain torch here: they
are not aggregation work."""

import numpy as np
import pytest

import graphgen
from test_parity import dev, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tfg():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no ROCm device")
    import paper_2101_11552_amd as lib
    lib.load()
    return lib


def test_gat_layer_gradient_matches_finite_differences(tfg, orc):
    import torch
    n, e, H, D, slope = 40, 300, 2, 4, 0.2
    ei = graphgen.random_graph(101, n, e, hub=3, hub_edges=150)
    E = ei.shape[1]
    rng = np.random.default_rng(101)
    h = rng.standard_normal((n, H * D)).astype(np.float32)
    a_s = rng.standard_normal((H, D)).astype(np.float32)
    a_d = rng.standard_normal((H, D)).astype(np.float32)
    dout = rng.standard_normal((n, H * D)).astype(np.float32)

    eid = dev(ei)
    g = tfg.tfg_graph_create(eid, n)
    gt = tfg.tfg_graph_create_transposed(eid, n)
    hd = dev(h)
    out, alpha = tfg.tfg_gat_aggregate(g, hd, dev(a_s), dev(a_d), slope, want_alpha=True)
    dod = dev(dout)
    # through the weighted sum: d alpha[e, k] = <dout[t, k], h[s, k]>, dh = sum alpha dout
    dalpha = tfg.tfg_edge_dot_scores(g, dod, hd, H, scale=1.0)
    dh, _ = tfg.tfg_aggregate_backward(g, dod, "sum", graph_t=gt, edge_weight=alpha, heads=H)
    # through the softmax and the LeakyReLU
    ds = tfg.tfg_segment_softmax_backward(alpha, dalpha, eid[1], n, graph=g)
    z = tfg.tfg_gat_edge_scores(eid, hd, dev(a_s), dev(a_d), 1.0)  # slope 1: z itself
    dz = (ds * torch.where(z >= 0, torch.ones_like(z), torch.full_like(z, slope))).contiguous()
    # per-node sums of dz: over the out-edges (a_s) and the in-edges (a_d)
    ones = torch.ones((n, H), device=hd.device)
    das = tfg.tfg_aggregate(None, ones, n, "sum", edge_weight=dz, heads=H, graph=gt)
    dad = tfg.tfg_aggregate(None, ones, n, "sum", edge_weight=dz, heads=H, graph=g)
    proj = (das.reshape(n, H, 1) * dev(a_s).reshape(1, H, D) +
            dad.reshape(n, H, 1) * dev(a_d).reshape(1, H, D)).reshape(n, H * D)
    grad = host(dh + proj).astype(np.float64)
    torch.cuda.synchronize()

    def loss(hh):
        o, _, _ = orc.gat_layer(ei, hh, a_s, a_d, H, slope=np.float32(slope))
        return float((o * dout).sum())
    eps = 1e-3
    for (i, c) in [(0, 0), (3, 5), (7, 7), (n - 1, 2), (11, 3)]:
        hp, hm = h.copy(), h.copy()
        hp[i, c] += eps
        hm[i, c] -= eps
        step = float(np.float32(h[i, c] + eps)) - float(np.float32(h[i, c] - eps))
        fd = (loss(hp) - loss(hm)) / step
        assert fd == pytest.approx(grad[i, c], rel=2e-3, abs=2e-4), (i, c)
    assert E > 0
