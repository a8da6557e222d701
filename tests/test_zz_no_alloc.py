"""The aggregation entry point that allocates nothing (tfg_aggregate_noalloc),
called through the C ABI: its partial rows live in the library's static
device scratch. Two calls in a row, the second on a smaller graph, each
bit-identical to tfg_aggregate (same kernels, same plan) and within the
scaled 1e-5 bar of the oracle; a graph whose partial rows exceed the scratch
is refused before any launch."""

import ctypes

import numpy as np
import pytest

import graphgen
from test_parity import assert_scaled, dev, host, same_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tfg():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no ROCm device")
    import paper_2101_11552_amd as lib
    lib.load()
    return lib


def _noalloc(tfg, g, x, n, reduce, w=None, order="csr"):
    """tfg_aggregate_noalloc through ctypes on torch's current stream."""
    import torch
    lib = tfg.load()
    F = x.shape[1]
    out = torch.full((n, F), 7.0, device=x.device)
    arg = torch.full((n, F), 7, dtype=torch.int32, device=x.device) if reduce == "max" else None
    red = {"sum": 0, "mean": 1, "max": 2}[reduce]
    stream = ctypes.c_void_p(torch.cuda.current_stream(x.device).cuda_stream)
    rc = lib.tfg_aggregate_noalloc(None, 0, g.E, None if w is None else ctypes.c_void_p(w.data_ptr()),
                                   1, 1 if order == "csr" else 0, ctypes.c_void_p(x.data_ptr()),
                                   x.shape[0], F, F, n, red, g.handle,
                                   ctypes.c_void_p(out.data_ptr()),
                                   None if arg is None else ctypes.c_void_p(arg.data_ptr()), stream)
    return rc, out, arg


@pytest.mark.parametrize("reduce,plan", [("sum", "0"), ("max", "0"), ("sum", "1"), ("mean", "1")])
def test_noalloc_matches_tfg_aggregate(tfg, orc, monkeypatch, reduce, plan):
    monkeypatch.setenv("TFG_PART_PLAN", plan)
    import torch
    cases = [(4000, 90_000, 64, 31), (700, 9_000, 32, 32)]  # the second call is smaller
    for n, e, F, seed in cases:
        ei = graphgen.random_graph(seed, n, e, hub=5, hub_edges=3000)  # split rows: partials
        g = tfg.tfg_graph_create(dev(ei), n, add_self_loops=True, src_parts=4)
        norm = tfg.tfg_gcn_norm(dev(ei), n, graph=g)
        x = graphgen.features(seed, n, F)
        xd = dev(x)
        w = norm["edge_weight_csr"]
        rc, out, arg = _noalloc(tfg, g, xd, n, reduce, w)
        assert rc == 0, tfg.load().tfg_last_error()
        torch.cuda.synchronize()
        ref = tfg.tfg_aggregate(None, xd, n, reduce, edge_weight=w, weight_order="csr", graph=g)
        what = f"noalloc {reduce} plan={plan} n={n}"
        oei, ow, _ = orc.gcn_norm(ei, n)
        if reduce == "max":
            assert same_bits(host(out), host(ref[0])) and torch.equal(arg, ref[1]), what
            rv, ra = orc.aggregate(oei, x, n, "max", edge_weight=ow)
            assert same_bits(host(out), rv) and np.array_equal(host(arg), ra), what
        else:
            assert same_bits(host(out), host(ref)), what
            r64, S = orc.aggregate(oei, x, n, reduce, edge_weight=ow)
            assert_scaled(host(out), r64, S, what=what)


def test_noalloc_refuses_oversized_partials(tfg, monkeypatch):
    import torch
    monkeypatch.setenv("TFG_PART_PLAN", "1")
    n, F = 200_000, 128
    ei = graphgen.random_graph(33, n, 2_000_000)
    g = tfg.tfg_graph_create(dev(ei.astype(np.int32)), n, src_parts=8)
    need = tfg.tfg_aggregate_ws_bytes(g.E, n, F, "sum", graph=g)
    assert need > 64 << 20  # TFG_NOALLOC_SCRATCH_BYTES
    x = torch.zeros((n, F), device="cuda:0")
    rc, out, _ = _noalloc(tfg, g, x, n, "sum", order="coo")
    assert rc == tfg.TFG_ERR_WORKSPACE
    assert bool((out == 7.0).all())  # nothing was launched
    with pytest.raises(ValueError):
        tfg.tfg_aggregate_noalloc(None, x, n, g)
