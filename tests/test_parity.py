"""GPU parity: every C-ABI call against the oracle on the same seeded inputs.

Bars: bit-exact for the CSR permutation, degrees, normalised weights and max /
argmax; for sums and means an error scaled by the size of the terms,
|y - ref| / sum|terms| <= 1e-5 (the float32 summation bound; plain relative
error is meaningless where a sum of N(0,1) terms cancels); for softmax a plain
relative error <= 1e-5 (all terms positive).
"""

import numpy as np
import pytest

import graphgen
from graph_order import expected_graph

pytestmark = pytest.mark.gpu

TOL = 1e-5
FLT_MIN = np.finfo(np.float32).tiny


@pytest.fixture(scope="module")
def tfg():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no ROCm device")
    import paper_2101_11552_amd as lib
    lib.load()
    return lib


def dev(a, dtype=None):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to("cuda:0")


def host(t):
    return t.detach().cpu().numpy()


def assert_scaled(y, ref, S, tol=TOL, what=""):
    y = np.asarray(y, np.float64)
    zero = S == 0
    assert np.all(y[zero] == 0), f"{what}: nonzero output where every term is zero"
    err = np.abs(y[~zero] - ref[~zero]) / S[~zero]
    worst = float(err.max()) if err.size else 0.0
    assert worst <= tol, f"{what}: scaled error {worst:.3e} > {tol}"
    return worst


def assert_rel(y, ref, tol=TOL, what=""):
    y = np.asarray(y, np.float64)
    err = np.abs(y - ref) / np.maximum(np.abs(ref), FLT_MIN)
    worst = float(err.max()) if err.size else 0.0
    assert worst <= tol, f"{what}: relative error {worst:.3e} > {tol}"


def same_bits(a, b):
    a, b = np.asarray(a), np.asarray(b)
    return a.shape == b.shape and np.array_equal(a.view(np.uint32), b.view(np.uint32))


# ---------------------------------------------------------------------------
# COO -> CSR
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n,e,loops,idx,parts", [
    (1, 7, False, np.int64, 1),            # N = 1: a single row
    (200, 30_000, False, np.int32, 1),     # one radix pass (8 bits), 4 tiles + ragged tail
    (300, 50_000, False, np.int32, 1),     # two passes (9 bits), 7 tiles + ragged tail
    (5_000, 70_001, True, np.int64, 1),    # two passes, loops appended
    (300_000, 40_000, False, np.int32, 1),  # three passes (19 bits), mostly empty rows
    (1000, 0, True, np.int32, 1),          # no input edges: loops only
    (2000, 90_000, True, np.int32, 8),     # source parts: key (target, part), 3 + 11 bits
    (300, 50_000, False, np.int64, 3),     # parts that do not divide N
    (70_000, 200_000, False, np.int32, 16),  # 21-bit keys: three passes
    (4_096, 40_000, True, np.int32, 1),    # 4096 rows: one-block work lists (largest)
    (4_097, 40_000, True, np.int32, 1),    # one row more: work lists from per-block counts
    (60_000, 500_000, True, np.int32, 1),  # digit tables of 21.5k counts: one-block scan
    (20_000, 1_500_000, False, np.int32, 1),  # digit tables of 58.6k counts: three-kernel scan
])
def test_csr_bit_exact(tfg, orc, n, e, loops, idx, parts):
    ei = graphgen.random_graph(e + n, n, e, hub=n // 2, hub_edges=e // 4)
    g = tfg.tfg_graph_create(dev(ei.astype(idx)), n, add_self_loops=loops, src_parts=parts)
    assert g.info()["src_parts"] == min(parts, n)
    rowptr, col, perm = (host(t) for t in tfg.tfg_graph_csr(g))
    full = ei
    if loops:
        full = np.concatenate([ei, np.stack([np.arange(n), np.arange(n)])], axis=1)
    ref = expected_graph(orc, full, n, parts=min(parts, n))
    r, c, p = ref[:3]
    assert np.array_equal(rowptr, r) and np.array_equal(perm, p) and np.array_equal(col, c)
    # the row plan's lists: rows longer than 128 edges are cut into chunks
    deg = np.diff(r)
    long_rows = deg[deg > 128]
    info = g.info()
    assert info["n_rows_split"] == long_rows.size
    assert info["n_chunks"] == int(((long_rows + 127) // 128).sum())
    if parts > 1:
        assert np.array_equal(host(tfg.tfg_graph_segments(g)), ref[3])


@pytest.mark.parametrize("n,n_src,e,loops,idx,parts,packed", [
    (300_000, 300_000, 40_000, False, np.int32, 1, "0"),  # three passes, three-word payloads
    (70_000, 70_000, 200_000, True, np.int64, 16, "0"),   # 21-bit keys, three-word payloads
    (2000, 2000, 90_000, True, np.int32, 8, "0"),         # two passes, three-word payloads
    (150_000, 300_000, 120_000, False, np.int32, 4, "1"),  # rectangular: source bits in both words
    (300_000, 5_000, 60_000, False, np.int64, 2, "1"),    # rectangular: every source bit in A
])
def test_csr_packed_and_unpacked_payloads(tfg, orc, monkeypatch, n, n_src, e, loops, idx, parts,
                                          packed):
    # the radix passes carry (key, edge id, source) as three words, or, with
    # a power-of-two part count, packed into two; both give the oracle's order
    monkeypatch.setenv("TFG_SORT_PACKED", packed)
    ei = graphgen.random_graph(e + n + 1, n, e, n_src=n_src, hub=n // 3, hub_edges=e // 5)
    g = tfg.tfg_graph_create(dev(ei.astype(idx)), n, N_src=n_src, add_self_loops=loops,
                             src_parts=parts)
    rowptr, col, perm = (host(t) for t in tfg.tfg_graph_csr(g))
    full = ei
    if loops:
        full = np.concatenate([ei, np.stack([np.arange(n), np.arange(n)])], axis=1)
    ref = expected_graph(orc, full, n, parts=g.info()["src_parts"], n_src=n_src)
    assert np.array_equal(rowptr, ref[0]) and np.array_equal(perm, ref[2])
    assert np.array_equal(col, ref[1])
    if g.info()["src_parts"] > 1:
        assert np.array_equal(host(tfg.tfg_graph_segments(g)), ref[3])


@pytest.mark.parametrize("n,n_src,e,loops,parts", [
    (1 << 17, 1 << 17, 300_000, False, 8),            # 17-bit targets: A keeps 15 source bits
    ((1 << 17) + 1, (1 << 17) + 1, 300_000, False, 1),  # one more node: 18-bit ids
    (1 << 20, 1 << 22, 1 << 22, False, 1),            # source bits 10 + 12, 22-bit positions: B full
    (70_000, 1, 500_000, False, 4),                   # a single source (0 source bits), 4 parts
    (1 << 16, 1 << 16, (1 << 20) - (1 << 16), True, 2),  # E' = 2^20 exactly (with the loops)
])
def test_csr_packed_bit_boundaries(tfg, orc, n, n_src, e, loops, parts):
    # the packed passes at the edges of their bit budget: the result is the
    # oracle's order whatever the split of the source bits between A and B
    ei = graphgen.random_graph(e + 7, n, e, n_src=n_src, hub=n // 5, hub_edges=e // 10)
    g = tfg.tfg_graph_create(dev(ei.astype(np.int32)), n, N_src=n_src, add_self_loops=loops,
                             src_parts=parts)
    rowptr, col, perm = (host(t) for t in tfg.tfg_graph_csr(g))
    full = ei
    if loops:
        full = np.concatenate([ei, np.stack([np.arange(n), np.arange(n)])], axis=1)
    ref = expected_graph(orc, full, n, parts=g.info()["src_parts"], n_src=n_src)
    assert np.array_equal(rowptr, ref[0]) and np.array_equal(perm, ref[2])
    assert np.array_equal(col, ref[1])
    if g.info()["src_parts"] > 1:
        assert np.array_equal(host(tfg.tfg_graph_segments(g)), ref[3])


def test_auto_parts(tfg):
    # small source table: one part; large table with long rows: several
    ei = graphgen.random_graph(3, 1000, 20_000)
    assert tfg.tfg_graph_create(dev(ei), 1000).info()["src_parts"] == 1
    n = 70_000
    ei = graphgen.random_graph(4, n, 64 * n)  # 35.8 MB of 512-byte rows, average degree 64
    info = tfg.tfg_graph_create(dev(ei.astype(np.int32)), n).info()
    assert info["src_parts"] == 3 and info["n_part_items"] > 0


def test_csr_rejects_out_of_range(tfg):
    ei = np.array([[0, 1, 2], [1, 2, 9]])
    with pytest.raises(IndexError):
        tfg.tfg_graph_create(dev(ei), 5)
    ei = np.array([[0, -1], [1, 2]])
    with pytest.raises(IndexError):
        tfg.tfg_graph_create(dev(ei.astype(np.int32)), 5)


# ---------------------------------------------------------------------------
# GCN normalisation
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("weighted,idx,parts", [(False, np.int32, 1), (True, np.int64, 1),
                                                (True, np.int32, 6)])
def test_gcn_norm_bit_exact(tfg, orc, weighted, idx, parts):
    n, e = 4000, 60_000
    ei = graphgen.random_graph(21, n, e, hub=3, hub_edges=5000)  # duplicates, loops, a hub
    w = (np.random.default_rng(3).uniform(0.1, 3.0, ei.shape[1]).astype(np.float32)
         if weighted else None)
    g = tfg.tfg_graph_create(dev(ei.astype(idx)), n, add_self_loops=True, src_parts=parts)
    r = tfg.tfg_gcn_norm(dev(ei.astype(idx)), n, edge_weight=None if w is None else dev(w), graph=g)
    oei, ow, odeg = orc.gcn_norm(ei, n, edge_weight=w)
    assert np.array_equal(host(r["edge_index"]), oei)
    assert same_bits(host(r["deg"]), odeg)
    assert same_bits(host(r["edge_weight"]), ow)
    perm = expected_graph(orc, oei, n, parts=parts)[2]
    assert same_bits(host(r["edge_weight_csr"]), ow[perm])
    # functional path without a handle gives the same bits
    r2 = tfg.tfg_gcn_norm(dev(ei.astype(idx)), n, edge_weight=None if w is None else dev(w))
    assert same_bits(host(r2["edge_weight"]), ow)


NORM_SLICE_CASES = [
    # n, e, weighted, idx, parts, loops
    (4000, 60_000, False, np.int32, 1, True),    # one LDS slice
    (4000, 60_000, True, np.int64, 6, True),     # key / parts for the row
    (100_003, 300_000, False, np.int32, 1, True),  # three slices, N % 4 == 3 (tail)
    (100_003, 300_000, True, np.int32, 5, False),  # no loops: E' == E
    (90_001, 50_000, False, np.int64, 1, True),  # int64 ids, more nodes than edges
    (100_003, 400_000, False, np.int32, 7, True),  # graph order by source part, 7 parts
    (4000, 60_000, False, np.int64, 3, False),   # blocks of items straddling two parts
    (81_409, 200_000, False, np.int32, 1, True),  # two full 159 KB slices and one node
]


@pytest.mark.parametrize("n,e,weighted,idx,parts,loops", NORM_SLICE_CASES)
def test_gcn_norm_sliced_and_direct(tfg, orc, monkeypatch, n, e, weighted, idx, parts, loops):
    # the LDS-sliced, the direct-gather and (unit weights, several source
    # parts) the part-range weight kernels, each forced, all equal to the
    # oracle bit for bit (COO and CSR order)
    ei = graphgen.random_graph(23, n, e, hub=11, hub_edges=e // 10)
    w = (np.random.default_rng(5).uniform(0.1, 3.0, ei.shape[1]).astype(np.float32)
         if weighted else None)
    oei, ow, odeg = orc.gcn_norm(ei, n, edge_weight=w, add_self_loops=loops)
    perm = expected_graph(orc, oei, n, parts=parts)[2]
    eid = dev(ei.astype(idx))
    g = tfg.tfg_graph_create(eid, n, add_self_loops=loops, src_parts=parts)
    for mode, by_part in (("1", "0"), ("0", "0"), ("0", "1")):
        monkeypatch.setenv("TFG_NORM_SLICED", mode)
        monkeypatch.setenv("TFG_NORM_PARTS", by_part)
        mode = f"sliced={mode} parts={by_part}"
        r = tfg.tfg_gcn_norm(eid, n, edge_weight=None if w is None else dev(w),
                             add_self_loops=loops, graph=g)
        assert np.array_equal(host(r["edge_index"]), oei), mode
        assert same_bits(host(r["deg"]), odeg), mode
        assert same_bits(host(r["edge_weight"]), ow), mode
        assert same_bits(host(r["edge_weight_csr"]), ow[perm]), mode
        # one order at a time (the sliced path then runs one kernel per order)
        r = tfg.tfg_gcn_norm(eid, n, edge_weight=None if w is None else dev(w),
                             add_self_loops=loops, graph=g, out_edge_index=False,
                             out_edge_weight_csr=False, out_deg=False)
        assert same_bits(host(r["edge_weight"]), ow), mode
        r = tfg.tfg_gcn_norm(eid, n, edge_weight=None if w is None else dev(w),
                             add_self_loops=loops, graph=g, out_edge_index=False,
                             out_edge_weight=False, out_deg=False)
        assert same_bits(host(r["edge_weight_csr"]), ow[perm]), mode


@pytest.mark.parametrize("idx", [np.int32, np.int64])
def test_gcn_norm_sliced_hub_row(tfg, orc, monkeypatch, idx):
    # a target with more than 65535 in-edges (a row longer than any 16-bit
    # count) through the sliced kernels
    n = 3000
    ei = graphgen.random_graph(29, n, 10_000, hub=5, hub_edges=70_000)
    oei, ow, odeg = orc.gcn_norm(ei, n)
    assert odeg.max() > 65535
    perm = orc.csr_by_target(oei, n)[2]
    eid = dev(ei.astype(idx))
    g = tfg.tfg_graph_create(eid, n, add_self_loops=True)
    monkeypatch.setenv("TFG_NORM_SLICED", "1")
    r = tfg.tfg_gcn_norm(eid, n, graph=g)
    assert same_bits(host(r["edge_weight"]), ow)
    assert same_bits(host(r["edge_weight_csr"]), ow[perm])


def test_row_longer_than_float32_integers(tfg, orc, monkeypatch):
    # a target with more than 2^24 in-edges: its unit-weight degree is no
    # longer an exact float32, so the row length is rounded once (to nearest
    # even); weights in both orders, and the hub row of the sum and mean
    # aggregations over the normalised weights, against the oracle
    n, hub, F = 1000, 7, 4
    ei = graphgen.random_graph(31, n, 20_000, hub=hub, hub_edges=2**24 + 3_000_002)
    oei, ow, odeg = orc.gcn_norm(ei, n)
    count = int(np.count_nonzero(oei[1] == hub))
    assert count > 2**24 and float(np.float32(count)) != count
    assert odeg[hub] == np.float32(count)
    perm = orc.csr_by_target(oei, n)[2]
    eid = dev(ei.astype(np.int32))
    g = tfg.tfg_graph_create(eid, n, add_self_loops=True)
    for mode in ("1", "0"):
        monkeypatch.setenv("TFG_NORM_SLICED", mode)
        r = tfg.tfg_gcn_norm(eid, n, graph=g)
        assert same_bits(host(r["deg"]), odeg), mode
        assert same_bits(host(r["edge_weight"]), ow), mode
        assert same_bits(host(r["edge_weight_csr"]), ow[perm]), mode
    x = graphgen.features(32, n, F)
    for red in ("sum", "mean"):
        y = host(tfg.tfg_aggregate(None, dev(x), n, red, edge_weight=r["edge_weight_csr"],
                                   weight_order="csr", graph=g))
        ref, S = orc.aggregate(oei, x, n, red, edge_weight=ow, rows=[hub])
        assert_scaled(y[hub:hub + 1], ref, S, what=f"hub row, {red}")


# ---------------------------------------------------------------------------
# Aggregation
# ---------------------------------------------------------------------------

AGG_CASES = [
    # n_src, n, e, F, ldx, heads
    (600, 600, 20_000, 64, 64, 1),
    (600, 700, 20_000, 128, 128, 1),
    (500, 500, 9_000, 1, 1, 1),
    (500, 500, 9_000, 3, 3, 1),
    (400, 400, 9_000, 130, 133, 1),   # F not a multiple of 4, ldx > F
    (800, 800, 30_000, 128, 136, 8),  # one weight per head
    (300, 900, 6_000, 16, 16, 2),     # rectangular, many empty targets
]


@pytest.mark.parametrize("n_src,n,e,F,ldx,H", AGG_CASES)
@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
def test_aggregate(tfg, orc, n_src, n, e, F, ldx, H, reduce):
    ei = graphgen.random_graph(e + F, n, e, n_src=n_src, hub=1, hub_edges=3 * 1200)  # split row
    E = ei.shape[1]
    big = graphgen.features(F, n_src, ldx)
    x = big[:, :F]
    w = np.random.default_rng(e).standard_normal((E, H) if H > 1 else E).astype(np.float32)
    xd = dev(big)[:, :F]
    g = tfg.tfg_graph_create(dev(ei), n, N_src=n_src)
    assert g.info()["n_rows_split"] >= 1
    res = tfg.tfg_aggregate(dev(ei), xd, n, reduce=reduce, edge_weight=dev(w), heads=H, graph=g)
    if reduce == "max":
        out, arg = (host(t) for t in res)
        ref, refarg = orc.aggregate(ei, x, n, "max", edge_weight=w, heads=H)
        assert same_bits(out, ref) and np.array_equal(arg, refarg)
    else:
        ref, S = orc.aggregate(ei, x, n, reduce, edge_weight=w, heads=H)
        assert_scaled(host(res), ref, S, what=f"{reduce} F={F}")


@pytest.mark.parametrize("F,H", [(128, 1), (64, 1), (32, 4), (5, 1)])
@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
@pytest.mark.parametrize("plan", ["0", "1"])
def test_aggregate_source_parts(tfg, orc, monkeypatch, F, H, reduce, plan):
    """Graphs ordered by (target, source part); the part plan (partials per
    source part, reduced in part order) and the row plan on the same graph."""
    monkeypatch.setenv("TFG_PART_PLAN", plan)
    n, e, parts = 1500, 60_000, 5
    ei = graphgen.random_graph(F + H, n, e, hub=17, hub_edges=9000)
    E = ei.shape[1]
    x = graphgen.features(F, n, F)
    w = np.random.default_rng(F).standard_normal((E, H) if H > 1 else E).astype(np.float32)
    g = tfg.tfg_graph_create(dev(ei), n, src_parts=parts)
    assert g.info()["n_part_items"] > 0
    _, _, perm, _ = expected_graph(orc, ei, n, parts=parts)
    res = tfg.tfg_aggregate(None, dev(x), n, reduce, edge_weight=dev(w[perm]), heads=H,
                            weight_order="csr", graph=g)
    coo = tfg.tfg_aggregate(dev(ei), dev(x), n, reduce, edge_weight=dev(w), heads=H, graph=g)
    if reduce == "max":
        ref, refarg = orc.aggregate(ei, x, n, "max", edge_weight=w, heads=H)
        assert same_bits(host(res[0]), ref) and np.array_equal(host(res[1]), refarg)
        assert same_bits(host(coo[0]), ref) and np.array_equal(host(coo[1]), refarg)
    else:
        ref, S = orc.aggregate(ei, x, n, reduce, edge_weight=w, heads=H)
        assert_scaled(host(res), ref, S, what=f"{reduce} parts plan={plan}")
        assert same_bits(host(res), host(coo))


WIDE_CASES = [
    # F, ldx: the layout the sum / mean kernel with scalar edge ids takes
    (128, 132),  # two edge slots of 32 lanes x 4 columns
    (256, 256),  # the same, two full passes over the columns
    (192, 192),  # one slot of 64 lanes x 2 columns, second pass half full
    (64, 64),    # one slot, one column per lane
    (65, 67),    # one column per lane, a one-column second pass
]


@pytest.mark.parametrize("F,ldx", WIDE_CASES)
@pytest.mark.parametrize("reduce", ["sum", "mean"])
@pytest.mark.parametrize("plan", ["0", "1"])
@pytest.mark.parametrize("wide", ["0", "1"])
def test_aggregate_wide_layouts(tfg, orc, monkeypatch, F, ldx, reduce, plan, wide):
    """Sum and mean over rows of at least 64 columns: the kernel with scalar
    edge ids in each of its column layouts (wide=1), and the general row
    kernel it replaces there (wide=0), on both plans, with weights in COO
    order (gathered through the permutation), in graph order and without."""
    monkeypatch.setenv("TFG_WIDE_ROWS", wide)
    monkeypatch.setenv("TFG_PART_PLAN", plan)
    n, e, parts = 1500, 50_000, 5
    ei = graphgen.random_graph(F + ldx, n, e, hub=23, hub_edges=7000)
    E = ei.shape[1]
    big = graphgen.features(F + 1, n, ldx)
    x = big[:, :F]
    w = np.random.default_rng(F).standard_normal(E).astype(np.float32)
    g = tfg.tfg_graph_create(dev(ei), n, src_parts=parts)
    perm = expected_graph(orc, ei, n, parts=parts)[2]
    xd = dev(big)[:, :F]
    ref, S = orc.aggregate(ei, x, n, reduce, edge_weight=w)
    coo = tfg.tfg_aggregate(dev(ei), xd, n, reduce, edge_weight=dev(w), graph=g)
    csr = tfg.tfg_aggregate(None, xd, n, reduce, edge_weight=dev(w[perm]), weight_order="csr",
                            graph=g)
    what = f"{reduce} F={F} ldx={ldx} plan={plan} wide={wide}"
    assert_scaled(host(coo), ref, S, what=what + " COO weights")
    assert same_bits(host(coo), host(csr))
    ref1, S1 = orc.aggregate(ei, x, n, reduce)
    assert_scaled(host(tfg.tfg_aggregate(None, xd, n, reduce, graph=g)), ref1, S1,
                  what=what + " unweighted")


@pytest.mark.parametrize("plan", ["0", "1"])
def test_aggregate_table_beyond_2gb(tfg, orc, monkeypatch, plan):
    """A feature table whose rows span more than 2 GB (a large leading
    dimension): row offsets no longer fit 32 bits and the gathers take
    64-bit offsets."""
    import torch
    monkeypatch.setenv("TFG_PART_PLAN", plan)
    n_src, n, e, F = 520, 700, 30_000, 128
    ldx = (1 << 20) + 128  # 520 rows x 4 MB = 2.18 GB
    assert n_src * ldx * 4 >= 2 ** 31
    ei = graphgen.random_graph(77, n, e, n_src=n_src, hub=3, hub_edges=3000)
    x = graphgen.features(78, n_src, F)
    w = np.random.default_rng(79).standard_normal(ei.shape[1]).astype(np.float32)
    big = torch.zeros((n_src, ldx), dtype=torch.float32, device="cuda:0")
    big[:, :F] = dev(x)
    g = tfg.tfg_graph_create(dev(ei), n, N_src=n_src, src_parts=4)
    y = tfg.tfg_aggregate(dev(ei), big[:, :F], n, "sum", edge_weight=dev(w), graph=g)
    ref, S = orc.aggregate(ei, x, n, "sum", edge_weight=w)
    assert_scaled(host(y), ref, S, what=f"sum, ldx={ldx}, plan={plan}")
    del big
    torch.cuda.empty_cache()


@pytest.mark.parametrize("reduce", ["sum", "max"])
def test_aggregate_functional_and_csr_weights(tfg, orc, reduce):
    n, e, F = 2000, 40_000, 64
    ei = graphgen.random_graph(9, n, e, hub=11, hub_edges=4000)
    x = graphgen.features(9, n, F)
    w = np.random.default_rng(9).standard_normal(e + 4000).astype(np.float32)
    g = tfg.tfg_graph_create(dev(ei), n)
    _, _, perm = orc.csr_by_target(ei, n)
    a = tfg.tfg_aggregate(dev(ei), dev(x), n, reduce, edge_weight=dev(w))           # no handle
    b = tfg.tfg_aggregate(dev(ei), dev(x), n, reduce, edge_weight=dev(w[perm]),
                          weight_order="csr", graph=g)
    c = tfg.tfg_aggregate(dev(ei), dev(x), n, reduce, edge_weight=dev(w), graph=g)  # COO + handle
    if reduce == "max":
        assert all(same_bits(host(a[0]), host(t[0])) for t in (b, c))
        assert all(np.array_equal(host(a[1]), host(t[1])) for t in (b, c))
    else:
        assert same_bits(host(a), host(b)) and same_bits(host(a), host(c))


def test_aggregate_unweighted_ones_is_degree(tfg):
    n, e = 3000, 100_000
    ei = graphgen.random_graph(4, n, e, hub=0, hub_edges=20_000)
    y = host(tfg.tfg_aggregate(dev(ei), dev(np.ones((n, 4), np.float32)), n, "sum"))
    cnt = np.bincount(ei[1], minlength=n).astype(np.float32)
    assert np.array_equal(y, np.repeat(cnt[:, None], 4, axis=1))  # exact: integers < 2^24
    m = host(tfg.tfg_aggregate(dev(ei), dev(np.ones((n, 4), np.float32)), n, "mean"))
    assert np.array_equal(m[:, 0], (cnt > 0).astype(np.float32))


def test_aggregate_edge_cases(tfg, orc):
    x = graphgen.features(2, 5, 8)
    empty = np.zeros((2, 0), np.int64)
    y = host(tfg.tfg_aggregate(dev(empty), dev(x), 5, "sum"))
    assert np.all(y == 0)
    m, a = tfg.tfg_aggregate(dev(empty), dev(x), 5, "max")
    assert np.all(host(m) == 0) and np.all(host(a) == -1)
    one = np.array([[3], [0]])  # a single edge
    y = host(tfg.tfg_aggregate(dev(one), dev(x), 5, "sum"))
    assert np.array_equal(y[0], x[3]) and np.all(y[1:] == 0)
    # ties and signed zeros: the first edge in input order wins
    ei = np.array([[0, 1, 2, 0], [4, 4, 4, 4]])
    xt = np.array([[-0.0], [0.0], [0.0], [-0.0], [0.0]], np.float32)
    m, a = tfg.tfg_aggregate(dev(ei), dev(xt), 5, "max")
    assert host(a)[4, 0] == 0 and np.signbit(host(m)[4, 0])


def test_aggregate_deterministic(tfg):
    n, e = 5000, 200_000
    ei = graphgen.random_graph(31, n, e, hub=5, hub_edges=30_000)
    x = dev(graphgen.features(31, n, 128))
    w = dev(np.random.default_rng(31).standard_normal(e + 30_000).astype(np.float32))
    g = tfg.tfg_graph_create(dev(ei), n)
    y1 = host(tfg.tfg_aggregate(dev(ei), x, n, "sum", edge_weight=w, graph=g))
    y2 = host(tfg.tfg_aggregate(dev(ei), x, n, "sum", edge_weight=w, graph=g))
    g2 = tfg.tfg_graph_create(dev(ei), n)
    y3 = host(tfg.tfg_aggregate(dev(ei), x, n, "sum", edge_weight=w, graph=g2))
    assert same_bits(y1, y2) and same_bits(y1, y3)


# ---------------------------------------------------------------------------
# Attention: scores and softmax
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("H,D", [(8, 16), (1, 5), (3, 4)])
def test_gat_scores(tfg, orc, H, D):
    n, e = 3000, 50_000
    ei = graphgen.random_graph(H * D, n, e)
    h = graphgen.features(H, n, H * D)
    r = np.random.default_rng(D)
    a_s = r.standard_normal((H, D)).astype(np.float32)
    a_d = r.standard_normal((H, D)).astype(np.float32)
    s = host(tfg.tfg_gat_edge_scores(dev(ei.astype(np.int32)), dev(h), dev(a_s), dev(a_d), 0.2))
    ref, S = orc.gat_scores(ei, h, a_s, a_d, H, slope=np.float32(0.2))
    assert_scaled(s, ref, S, what="gat scores")


@pytest.mark.parametrize("H,parts", [(1, 1), (8, 1), (3, 1), (8, 4)])
def test_segment_softmax(tfg, orc, H, parts):
    n, e = 5000, 80_000
    ei = graphgen.random_graph(H, n, e, hub=2, hub_edges=6000)
    E = ei.shape[1]
    s = (graphgen.features(77, E, H) * 6).astype(np.float32)
    g = tfg.tfg_graph_create(dev(ei), n, src_parts=parts)
    out, out_csr = tfg.tfg_segment_softmax(dev(s), dev(ei[1]), n, graph=g, out_csr=True)
    ref64, _ = orc.segment_softmax(s, ei[1], n)
    assert_rel(host(out), ref64, what="softmax")
    perm = expected_graph(orc, ei, n, parts=parts)[2]
    assert same_bits(host(out_csr), host(out)[perm])
    plain = tfg.tfg_segment_softmax(dev(s), dev(ei[1]), n)  # no handle: a transient graph
    if parts == 1:  # the same graph order and plan: the same bits
        assert same_bits(host(plain), host(out))
    else:  # another edge order inside the rows: the same values up to rounding
        assert_rel(host(plain), ref64, what="softmax, transient graph")
    again = tfg.tfg_segment_softmax(dev(s), dev(ei[1]), n, graph=g)
    assert same_bits(host(again), host(out))
    tot = np.zeros((n, H))
    np.add.at(tot, ei[1], host(out).astype(np.float64))
    has = np.bincount(ei[1], minlength=n) > 0
    assert np.all(np.abs(tot[has] - 1) <= 1e-5)


@pytest.mark.parametrize("H,D,parts,loops,hub_edges", [
    (8, 16, 1, False, 5000), (3, 4, 1, True, 5000), (8, 16, 4, False, 5000),
    (1, 5, 3, True, 5000),
    (80, 2, 1, False, 5000),  # heads in two passes
    (8, 16, 1, True, 1500),   # a hub of 12 chunks: the split row done inside one block
    (6, 8, 2, False, 1900)])  # the same with source parts and six heads
def test_attention_in_graph_order(tfg, orc, H, D, parts, loops, hub_edges):
    """Scores, softmax and its gradient over a graph handle with the per-edge
    arrays in the graph order: the same bits as the calls in the caller's
    order (permuted), and the oracle's values. A hub of more than 16 chunks
    of 128 edges takes the two-launch path of the split rows, a smaller one
    the path inside one block."""
    n, e = 4000, 60_000
    ei = graphgen.random_graph(H * D + parts + hub_edges, n, e, hub=3, hub_edges=hub_edges)
    g = tfg.tfg_graph_create(dev(ei), n, add_self_loops=loops, src_parts=parts)
    oei = orc.gcn_norm(ei, n)[0] if loops else ei  # the handle's edge list (loops appended)
    E = oei.shape[1]
    assert g.E == E
    perm = expected_graph(orc, oei, n, parts=parts)[2]
    h = graphgen.features(H, n, H * D)
    r = np.random.default_rng(D)
    a_s = r.standard_normal((H, D)).astype(np.float32)
    a_d = r.standard_normal((H, D)).astype(np.float32)
    s_coo = host(tfg.tfg_gat_edge_scores(dev(oei.astype(np.int32)), dev(h), dev(a_s), dev(a_d)))
    s_csr = host(tfg.tfg_gat_graph_scores(g, dev(h), dev(a_s), dev(a_d), order="csr"))
    assert same_bits(s_csr, s_coo[perm])
    assert same_bits(host(tfg.tfg_gat_graph_scores(g, dev(h), dev(a_s), dev(a_d), order="coo")),
                     s_coo)
    # softmax: graph order == the COO call's graph-order output, bit for bit
    a_coo, a_csr_ref = tfg.tfg_segment_softmax(dev(s_coo), dev(oei[1]), n, graph=g, out_csr=True)
    a_csr = host(tfg.tfg_segment_softmax_graph(g, dev(s_csr), order="csr"))
    assert same_bits(a_csr, host(a_csr_ref))
    assert same_bits(host(tfg.tfg_segment_softmax_graph(g, dev(s_coo), order="coo")), host(a_coo))
    ref64, a32 = orc.segment_softmax(s_coo, oei[1], n)
    assert_rel(a_csr, ref64[perm], what="softmax in graph order")
    # gradient in both orders
    da = graphgen.features(H + 100, E, H)
    ds_coo = host(tfg.tfg_segment_softmax_backward(a_coo, dev(da), dev(oei[1]), n, graph=g))
    ds_csr = host(tfg.tfg_segment_softmax_graph_backward(g, dev(a_csr), dev(da[perm]),
                                                         order="csr"))
    assert same_bits(ds_csr, ds_coo[perm])
    assert same_bits(host(tfg.tfg_segment_softmax_graph_backward(g, a_coo, dev(da), order="coo")),
                     ds_coo)
    a_h = host(a_coo)
    ref = orc.segment_softmax_backward(a_h, da, oei[1], n)
    dot = np.zeros((n, H))
    np.add.at(dot, oei[1], a_h.astype(np.float64) * np.abs(da))
    S = a_h * (np.abs(da) + dot[oei[1]])
    assert_scaled(ds_csr, ref[perm], S[perm], what="dscores in graph order")
    # a layer kept in the graph order: scores -> softmax -> aggregation, TFG_CSR weights
    y = host(tfg.tfg_aggregate(None, dev(h), n, "sum", edge_weight=dev(a_csr), heads=H,
                               weight_order="csr", graph=g))
    yref, yS = orc.aggregate(oei, h, n, "sum", edge_weight=a32 if H > 1 else a32.reshape(E),
                             heads=H)
    assert_scaled(y, yref, yS, what="aggregation with graph-order alpha")


def test_attention_in_graph_order_degenerate(tfg):
    """A graph without edges gives empty outputs; one node with only its loop
    gives the loop's score and alpha = 1 exactly."""
    import torch
    empty = np.zeros((2, 0), np.int64)
    g0 = tfg.tfg_graph_create(dev(empty), 5)
    h = torch.ones((5, 6), device="cuda:0")
    a = torch.ones((2, 3), device="cuda:0")
    s0 = tfg.tfg_gat_graph_scores(g0, h, a, a)
    assert tuple(s0.shape) == (0, 2)
    assert tuple(tfg.tfg_segment_softmax_graph(g0, s0).shape) == (0, 2)
    assert tuple(tfg.tfg_segment_softmax_graph_backward(g0, s0, s0).shape) == (0, 2)
    seg0 = torch.zeros(0, dtype=torch.int64, device="cuda:0")  # the caller's-order calls too
    assert tuple(tfg.tfg_segment_softmax(s0, seg0, 5).shape) == (0, 2)
    assert tuple(tfg.tfg_segment_softmax_backward(s0, s0, seg0, 5).shape) == (0, 2)
    g1 = tfg.tfg_graph_create(dev(empty), 1, add_self_loops=True)
    h1 = torch.tensor([[1.0, -2.0, 0.5, 3.0]], device="cuda:0")
    a_s = torch.tensor([[1.0, 1.0], [0.0, 2.0]], device="cuda:0")
    a_d = torch.tensor([[0.5, 0.0], [1.0, 1.0]], device="cuda:0")
    s1 = host(tfg.tfg_gat_graph_scores(g1, h1, a_s, a_d))
    # head 0: (1 - 2) + 0.5 = -0.5 -> 0.2 * -0.5; head 1: 2 * 3 + (0.5 + 3) = 9.5
    assert np.array_equal(s1, np.array([[np.float32(0.2) * np.float32(-0.5), 9.5]], np.float32))
    a1 = host(tfg.tfg_segment_softmax_graph(g1, dev(s1)))
    assert np.array_equal(a1, np.ones((1, 2), np.float32))
    d1 = host(tfg.tfg_segment_softmax_graph_backward(g1, dev(a1), dev(np.array([[3.0, -1.0]], np.float32))))
    assert np.array_equal(d1, np.zeros((1, 2), np.float32))


def test_attention_in_graph_order_errors(tfg):
    import torch
    n = 50
    ei = graphgen.random_graph(5, n, 400)
    g = tfg.tfg_graph_create(dev(ei), n)
    gt = tfg.tfg_graph_create_transposed(dev(ei), n)
    h = torch.zeros((n, 8), device="cuda:0")
    a = torch.zeros((2, 4), device="cuda:0")
    with pytest.raises(ValueError):
        tfg.tfg_gat_graph_scores(gt, h, a, a)  # a transposed graph
    with pytest.raises(ValueError):
        tfg.tfg_gat_graph_scores(g, h[:10], a, a)  # h of the wrong shape
    s = torch.zeros((g.E, 2), device="cuda:0")
    with pytest.raises(ValueError):
        tfg.tfg_segment_softmax_graph(g, s[:-1])  # not one row per edge
    with pytest.raises(ValueError):
        tfg.tfg_segment_softmax_graph_backward(gt, s, s)  # a transposed graph
    lib = tfg.load()
    assert lib.tfg_segment_softmax_graph(g.handle, s.data_ptr(), 2, 7, s.data_ptr(), None, 0,
                                         None) == 1  # bad order


def test_segment_softmax_closed_forms(tfg):
    seg = np.array([0, 1, 1, 1, 3])
    s = np.array([5.0, 2.0, 2.0, 2.0, -7.0], np.float32)
    out = host(tfg.tfg_segment_softmax(dev(s), dev(seg), 4))
    assert out[0] == 1.0 and out[4] == 1.0 and np.all(out[1:4] == np.float32(1 / 3))


# ---------------------------------------------------------------------------
# Pooling
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("F,ldx", [(64, 64), (7, 9), (130, 130)])
@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
def test_segment_pool(tfg, orc, F, ldx, reduce):
    sizes = np.random.default_rng(F).integers(0, 40, 700)
    sizes[5] = 3000  # one large graph
    gi = np.repeat(np.arange(700), sizes)
    big = graphgen.features(ldx, gi.shape[0], ldx)
    res = tfg.tfg_segment_pool(dev(big)[:, :F], dev(gi.astype(np.int32)), 703, reduce)
    if reduce == "max":
        ref, refarg = orc.segment_pool(big[:, :F], gi, 703, "max")
        assert same_bits(host(res[0]), ref) and np.array_equal(host(res[1]), refarg)
    else:
        ref, S = orc.segment_pool(big[:, :F], gi, 703, reduce)
        assert_scaled(host(res), ref, S, what=f"pool {reduce}")


def test_segment_pool_errors(tfg):
    x = dev(np.ones((3, 4), np.float32))
    with pytest.raises(ValueError):
        tfg.tfg_segment_pool(x, dev(np.array([0, 2, 1])), 3, "sum")
    with pytest.raises(IndexError):
        tfg.tfg_segment_pool(x, dev(np.array([0, 1, 3])), 3, "sum")
    out = host(tfg.tfg_segment_pool(x, dev(np.array([1, 1, 1])), 4, "mean"))
    assert np.all(out[0] == 0) and np.all(out[1] == 1) and np.all(out[2:] == 0)
    empty = host(tfg.tfg_segment_pool(dev(np.zeros((0, 4), np.float32)),
                                      dev(np.zeros(0, np.int64)), 2, "sum"))
    assert np.all(empty == 0)


# ---------------------------------------------------------------------------
# BatchGraph construction
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("idx", [np.int32, np.int64])
def test_batch_graphs_match_oracle(tfg, orc, idx):
    sizes, graphs = graphgen.batch_of_small_graphs(55, 300, 10, 60, 0.1)
    sizes[7] = 0  # an empty graph
    graphs[7] = np.zeros((2, 0), np.int64)
    counts = np.array([g.shape[1] for g in graphs])
    local = np.concatenate(graphs, axis=1)
    ei, gi, noff, eoff = tfg.tfg_batch_graphs(dev(sizes.astype(idx)), dev(counts.astype(idx)),
                                              dev(local.astype(idx)), int(sizes.sum()))
    ref_ei, ref_gi = orc.batch_graphs(sizes, graphs)
    assert np.array_equal(host(ei), ref_ei) and np.array_equal(host(gi), ref_gi)
    assert np.array_equal(host(noff), orc.batch_offsets(sizes))
    assert np.array_equal(host(eoff), orc.batch_offsets(counts))


@pytest.mark.parametrize("G", [16383, 16384, 40000])
def test_batch_graphs_one_block_and_device_scan(tfg, orc, G):
    # up to 16,383 graphs the offsets come from one block, above from the device-wide scan
    rng = graphgen.rng_for(56, 0)
    sizes = rng.integers(0, 6, G)
    graphs = []
    for n in sizes:
        m = int(rng.integers(0, 2 * n + 1)) if n > 0 else 0
        graphs.append(rng.integers(0, max(n, 1), (2, m)))
    counts = np.array([g.shape[1] for g in graphs])
    local = np.concatenate(graphs, axis=1)
    ei, gi, noff, eoff = tfg.tfg_batch_graphs(dev(sizes.astype(np.int32)),
                                              dev(counts.astype(np.int32)),
                                              dev(local.astype(np.int32)), int(sizes.sum()))
    ref_ei, ref_gi = orc.batch_graphs(sizes, graphs)
    assert np.array_equal(host(ei), ref_ei) and np.array_equal(host(gi), ref_gi)
    assert np.array_equal(host(noff), orc.batch_offsets(sizes))
    assert np.array_equal(host(eoff), orc.batch_offsets(counts))
    bad = sizes.copy()
    bad[G // 2] = -1  # a negative count is reported, whichever path runs
    with pytest.raises(IndexError):
        tfg.tfg_batch_graphs(dev(bad.astype(np.int32)), dev(counts.astype(np.int32)),
                             dev(local.astype(np.int32)), int(sizes.sum()))


def test_batch_graphs_paper_example(tfg):
    import json
    import os
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                       "batch_reindex_paper_example.json")))
    sizes = np.array(gold["sizes"])
    # one edge per graph: its last local node -> its first
    local = np.array([[n - 1 for n in sizes], [0, 0, 0]])
    ei, gi, noff, _ = tfg.tfg_batch_graphs(dev(sizes), dev(np.ones(3, np.int64)), dev(local))
    assert list(host(noff)[1:3]) == gold["offsets_of_graphs_2_and_3"]
    for ex in gold["one_based_examples"]:
        assert host(noff)[ex["graph"] - 1] + ex["node"] == ex["batched_index"]
    assert list(host(gi)) == [0, 0, 0, 0, 1, 1, 2, 2, 2]
    assert host(ei).tolist() == [[3, 5, 8], [0, 4, 6]]


def test_batch_graphs_totals(tfg):
    """The node and edge totals come from the library (summed on the device),
    in 64 bits; a negative count is an index error."""
    sizes = np.array([4, 0, 2, 3])
    counts = np.array([1, 0, 2, 5])
    for idx in (np.int32, np.int64):
        assert tfg.tfg_batch_graphs_totals(dev(sizes.astype(idx)), dev(counts.astype(idx))) == (9, 8)
    big = np.full(3, 2**31 - 1, np.int64)  # totals beyond 32 bits
    assert tfg.tfg_batch_graphs_totals(dev(big), dev(big)) == (3 * (2**31 - 1),) * 2
    assert tfg.tfg_batch_graphs_totals(dev(np.zeros(0, np.int64)), dev(np.zeros(0, np.int64))) == (0, 0)
    with pytest.raises(IndexError):
        tfg.tfg_batch_graphs_totals(dev(np.array([1, -2])), dev(np.array([0, 0])))
    rng = graphgen.rng_for(57, 0)
    many = rng.integers(0, 100, 40_000)
    assert tfg.tfg_batch_graphs_totals(dev(many), dev(many[::-1].copy())) == (int(many.sum()),) * 2


def test_binding_rejects_bad_buffers(tfg):
    """Caller-supplied outputs and workspaces of the wrong device, dtype, shape
    or layout are refused by the binding before any launch, and the output
    stays untouched."""
    import torch
    n, F, G = 200, 8, 5
    ei = dev(graphgen.random_graph(1, n, 600))
    x = dev(graphgen.features(1, n, F))
    g = tfg.tfg_graph_create(ei, n)
    cuda = torch.device("cuda:0")
    bad_out = [torch.empty((n, F)),                                   # host memory
               torch.empty((n, F), dtype=torch.float64, device=cuda),  # dtype
               torch.empty((n - 1, F), device=cuda),                   # too small
               torch.empty((n * F,), device=cuda),                     # flat
               torch.empty((F, n), device=cuda).t()]                   # strided
    for o in bad_out:
        o.fill_(7.0)
        keep = o.clone()
        with pytest.raises((ValueError, TypeError)):
            tfg.tfg_aggregate(ei, x, n, "sum", graph=g, out=o)
        with pytest.raises((ValueError, TypeError)):
            tfg.tfg_propagate(g, x, 2, out=o)
        assert torch.equal(o.cpu(), keep.cpu())
    for a in (torch.empty((n, F), dtype=torch.int64, device=cuda), torch.empty((n, F), dtype=torch.int32)):
        with pytest.raises((ValueError, TypeError)):
            tfg.tfg_aggregate(ei, x, n, "max", graph=g, argmax=a)
    with pytest.raises(ValueError):  # workspace in host memory
        tfg.tfg_aggregate(ei, x, n, "sum", graph=g, ws=torch.empty(1 << 20, dtype=torch.uint8))
    with pytest.raises(ValueError):  # h of another shape
        tfg.tfg_propagate(g, x, 2, alpha=0.1, h=x[:-1])
    gi = dev(np.repeat(np.arange(G), n // G))
    with pytest.raises((ValueError, TypeError)):
        tfg.tfg_segment_pool(x, gi, G, "sum", out=torch.empty((G + 1, F), device=cuda))
    with pytest.raises((ValueError, TypeError)):
        tfg.tfg_segment_pool(x, gi, G, "max", argmax=torch.empty((G, F), device=cuda))
    with pytest.raises(ValueError):  # graph index of another length
        tfg.tfg_segment_pool(x, gi[:-1], G, "sum")
    with pytest.raises((ValueError, TypeError)):
        tfg.tfg_segment_pool_backward(dev(np.ones((G, F), np.float32)), gi, "sum",
                                      out=torch.empty((n, F + 1), device=cuda))
    # a caller workspace of another dtype counts by bytes: 1 MiB of float32 is enough
    y = tfg.tfg_aggregate(ei, x, n, "sum", graph=g, ws=torch.empty(1 << 18, device=cuda))
    assert torch.equal(y, tfg.tfg_aggregate(ei, x, n, "sum", graph=g))


def test_batch_graphs_errors(tfg):
    sizes = np.array([3, 2])
    with pytest.raises(IndexError):  # local id 3 in a graph of 3 nodes
        tfg.tfg_batch_graphs(dev(sizes), dev(np.array([1, 1])), dev(np.array([[3, 0], [0, 1]])))
    with pytest.raises(IndexError):  # edge counts add up to 3, the list has 2 edges
        tfg.tfg_batch_graphs(dev(sizes), dev(np.array([2, 1])), dev(np.array([[0, 0], [1, 1]])))


# ---------------------------------------------------------------------------
# Multi-step propagation (SGC / APPNP)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("K,alpha,parts,plan", [(1, 0.0, 1, "0"), (3, 0.0, 1, "0"),
                                                (4, 0.1, 1, "0"), (5, 0.2, 4, "1"),
                                                (2, 1.0, 4, "1"), (0, 0.0, 1, "0")])
def test_propagate(tfg, orc, monkeypatch, K, alpha, parts, plan):
    monkeypatch.setenv("TFG_PART_PLAN", plan)
    n, e, F = 3000, 80_000, 64
    ei = graphgen.random_graph(7 + K, n, e, hub=9, hub_edges=4000)
    x = graphgen.features(K, n, F)
    g = tfg.tfg_graph_create(dev(ei), n, add_self_loops=True, src_parts=parts)
    norm = tfg.tfg_gcn_norm(dev(ei), n, graph=g)
    oei, ow, _ = orc.gcn_norm(ei, n)
    h = x if alpha > 0 else None
    # stage by stage on the GPU's own intermediate values
    z = dev(x)
    for k in range(K):
        zin = host(z)
        z = tfg.tfg_propagate(g, z, 1, alpha=alpha, h=dev(x) if alpha > 0 else None,
                              edge_weight=norm["edge_weight_csr"])
        ref, S = orc.propagate(oei, zin, 1, alpha=alpha, h=h, edge_weight=ow)
        assert_scaled(host(z), ref, S, what=f"step {k}")
    # the K steps in one call, against the double-precision chain
    zk = tfg.tfg_propagate(g, dev(x), K, alpha=alpha, h=dev(x) if alpha > 0 else None,
                           edge_weight=norm["edge_weight_csr"])
    ref, S = orc.propagate(oei, x, K, alpha=alpha, h=h, edge_weight=ow)
    assert_scaled(host(zk), ref, S + 1e-30, tol=max(K, 1) * 1e-5, what=f"K={K} chain")
    if K == 0:
        assert same_bits(host(zk), x)


# ---------------------------------------------------------------------------
# Fused attention aggregation
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("H,D", [(8, 16), (1, 5), (3, 4), (4, 3), (16, 8)])
def test_gat_aggregate_fused(tfg, orc, H, D):
    n, e = 3000, 40_000
    ei = graphgen.random_graph(H * 10 + D, n, e, hub=3, hub_edges=3000)
    h = graphgen.features(H + D, n, H * D)
    r = np.random.default_rng(D)
    a_s = r.standard_normal((H, D)).astype(np.float32)
    a_d = r.standard_normal((H, D)).astype(np.float32)
    g = tfg.tfg_graph_create(dev(ei), n)
    out, alpha = tfg.tfg_gat_aggregate(g, dev(h), dev(a_s), dev(a_d), 0.2, want_alpha=True)
    ref, ref_alpha, S = orc.gat_layer(ei, h, a_s, a_d, H, slope=np.float32(0.2))
    assert_scaled(host(out), ref, S, what=f"fused GAT H={H} D={D}")
    has = np.bincount(ei[1], minlength=n)[ei[1]] > 0
    assert_rel(host(alpha)[has], ref_alpha[has], what="fused GAT alpha")
    # the unfused chain of the library gives the same layer
    s = tfg.tfg_gat_edge_scores(dev(ei), dev(h), dev(a_s), dev(a_d), 0.2)
    _, a_csr = tfg.tfg_segment_softmax(s, dev(ei[1]), n, graph=g, out_csr=True)
    y = tfg.tfg_aggregate(dev(ei), dev(h), n, "sum", edge_weight=a_csr, heads=H,
                          weight_order="csr", graph=g)
    assert_scaled(host(y), ref, S, what="unfused chain")


# ---------------------------------------------------------------------------
# Transformer-style attention (scaled dot-product scores)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("H,D,order,rect", [(1, 16, "coo", False), (4, 8, "csr", False),
                                            (3, 5, "coo", True), (8, 16, "csr", True)])
def test_edge_dot_scores(tfg, orc, H, D, order, rect):
    n, n_src, e = 2000, (1500 if rect else 2000), 30_000
    ei = graphgen.random_graph(H * 7 + D, n, e, n_src=n_src, hub=4, hub_edges=1000)
    q = graphgen.features(H + 1, n, H * D)
    k = graphgen.features(H + 2, n_src, H * D)
    g = tfg.tfg_graph_create(dev(ei), n, N_src=n_src)
    s = tfg.tfg_edge_dot_scores(g, dev(q), dev(k), H, scale=0.25, order=order)
    ref = orc.dot_scores(ei, q, k, H, 0.25)
    S = orc.dot_scores(ei, np.abs(q), np.abs(k), H, 0.25)
    got = host(s)
    if order == "csr":
        perm = host(tfg.tfg_graph_csr(g)[2])
        back = np.empty_like(got)
        back[perm] = got
        got = back
    assert_scaled(got, ref, S, what=f"dot scores H={H} D={D}")


def dot_alpha_bound(orc, ei, q, k, H, scale, ref_alpha, n):
    """Per-element bound on |alpha - ref| for attention over float32 scaled dot
    products (the oracle's scores are exact in double).

    A float32 dot product of D terms, in any summation order, then scaled,
    is within delta = (D + 2) u scale sum_d |q_d k_d| of the exact score
    (u = 2^-24). Since d log alpha_e / d s_j = [e = j] - alpha_j, score errors
    change alpha_e by at most alpha_e (delta_e + sum_j alpha_j delta_j) over
    the edges j of its segment, to first order. The softmax's own rounding is
    held to the 1e-5 relative bar of every softmax, so the bound is
    alpha_e (1e-5 + delta_e + sum_j alpha_j delta_j), with the FLT_MIN floor."""
    D = q.shape[1] // H
    S = orc.dot_scores(ei, np.abs(q), np.abs(k), H, scale)  # scale * sum_d |q_d k_d|
    delta = (D + 2) * 2.0 ** -24 * S
    seg = np.zeros((n, H))
    np.add.at(seg, ei[1], ref_alpha * delta)
    return np.maximum(ref_alpha, FLT_MIN) * (TOL + delta + seg[ei[1]])


@pytest.mark.parametrize("H,D,rect", [(8, 16, False), (1, 4, False), (4, 8, True), (2, 64, False),
                                      (16, 2, False), (3, 1, True)])
def test_gat_dot_aggregate_fused(tfg, orc, H, D, rect):
    import torch
    n, n_src, e = 3000, (2200 if rect else 3000), 40_000
    ei = graphgen.random_graph(H * 11 + D, n, e, n_src=n_src, hub=3, hub_edges=3000)
    q = graphgen.features(H + 5, n, H * D)
    k = graphgen.features(H + 6, n_src, H * D)
    v = graphgen.features(H + 7, n_src, H * D)
    scale = 1.0 / np.sqrt(D)
    g = tfg.tfg_graph_create(dev(ei), n, N_src=n_src)
    out, alpha = tfg.tfg_gat_dot_aggregate(g, dev(q), dev(k), dev(v), H, scale=scale,
                                           want_alpha=True)
    torch.cuda.synchronize()
    ref, ref_alpha, S = orc.dot_layer(ei, q, k, v, H, np.float32(scale))
    assert_scaled(host(out), ref, S, what=f"fused dot attention H={H} D={D}")
    bound = dot_alpha_bound(orc, ei, q, k, H, np.float32(scale), ref_alpha, n)
    err = np.abs(host(alpha).astype(np.float64) - ref_alpha)
    worst = float((err / bound).max())
    assert worst <= 1.0, f"fused dot attention alpha: {worst:.3f} of the bound"
    empty = np.bincount(ei[1], minlength=n) == 0
    assert np.all(host(out)[empty] == 0)
    # the unfused chain of the library gives the same layer
    s = tfg.tfg_edge_dot_scores(g, dev(q), dev(k), H, scale=scale)
    _, a_csr = tfg.tfg_segment_softmax(s, dev(ei[1]), n, graph=g, out_csr=True)
    y = tfg.tfg_aggregate(dev(ei), dev(v), n, "sum", edge_weight=a_csr, heads=H,
                          weight_order="csr", graph=g)
    assert_scaled(host(y), ref, S, what="unfused dot chain")


def test_gat_dot_rejects_shapes(tfg):
    ei = dev(np.array([[0, 1], [1, 2]]))
    g = tfg.tfg_graph_create(ei, 4)
    x = dev(np.ones((4, 12), np.float32))
    with pytest.raises(ValueError):  # D = 3 is not a power of two
        tfg.tfg_gat_dot_aggregate(g, x, x, x, 4)


_CHUNK_SCRIPT = r"""
import os
import sys
import numpy as np
sys.path.insert(0, sys.argv[1])
sys.path.insert(0, sys.argv[1] + "/tests")
import torch
import graphgen
import oracle
import paper_2101_11552_amd as tfg
from test_parity import assert_scaled, same_bits
from graph_order import expected_graph
n, parts = 5000, 4
ei = graphgen.random_graph(41, n, 150_000, hub=9, hub_edges=20_000)
eid = torch.from_numpy(ei.astype(np.int32)).cuda()
g = tfg.tfg_graph_create(eid, n, add_self_loops=True, src_parts=parts)
assert g.info()["src_parts"] == parts
oei, ow, _ = oracle.gcn_norm(ei, n)
perm = expected_graph(oracle, oei, n, parts=parts)[2]
x = graphgen.features(41, n, 32)
for by_part in ("1", "0"):
    os.environ["TFG_NORM_PARTS"] = by_part
    r = tfg.tfg_gcn_norm(eid, n, graph=g)
    assert same_bits(r["edge_weight_csr"].cpu().numpy(), ow[perm]), by_part
    assert same_bits(r["edge_weight"].cpu().numpy(), ow), by_part
for plan in ("1", "0"):
    os.environ["TFG_PART_PLAN"] = plan
    y = tfg.tfg_aggregate(None, torch.from_numpy(x).cuda(), n, "sum",
                          edge_weight=r["edge_weight_csr"], weight_order="csr", graph=g)
    ref, S = oracle.aggregate(oei, x, n, "sum", edge_weight=ow)
    assert_scaled(y.cpu().numpy(), ref, S, what="chunk knob, plan " + plan)
print("chunk knob ok")
"""


def test_row_chunk_knob_in_a_fresh_process(tfg):
    """TFG_ROW_CHUNK is read once per process, so a longer work item (300
    edges, beyond two rounds of lanes) runs in a child process: normalised
    weights in both orders (part-range kernel on and off) and the sum
    aggregation (both plans) against the oracle."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    env = dict(os.environ, TFG_ROW_CHUNK="300", TFG_NORM_SLICED="0")
    r = subprocess.run([sys.executable, "-c", _CHUNK_SCRIPT, root], env=env,
                       capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    assert "chunk knob ok" in r.stdout


# ---------------------------------------------------------------------------
# Seeded random configurations: graph size and shape, source parts, plan,
# normalisation kernels, index type, feature width, leading dimension, heads
# and reducer drawn together, each case checked against the oracle.
# ---------------------------------------------------------------------------

def _random_case(seed):
    r = np.random.default_rng([9001, seed])
    n = int(r.integers(1, 3000))
    n_src = n if r.random() < 0.7 else int(r.integers(1, 3000))
    e = int(r.integers(0, 40_000))
    H = int(r.choice([1, 1, 2, 4]))
    F = H * int(r.choice([1, 3, 4, 16, 32]))
    return dict(n=n, n_src=n_src, e=e, H=H, F=F, ldx=F + int(r.choice([0, 0, 3])),
                parts=int(r.choice([0, 1, 2, 5, 16])), plan=str(r.choice(["0", "1"])),
                reduce=str(r.choice(["sum", "mean", "max"])),
                idx=np.int64 if r.random() < 0.3 else np.int32,
                hub_edges=int(r.choice([0, 0, 500, 5000])),
                sliced=str(r.choice(["0", "1"])), by_part=str(r.choice(["0", "1"])),
                weighted=bool(r.random() < 0.5))


@pytest.mark.parametrize("seed", range(40))
def test_random_configurations(tfg, orc, monkeypatch, seed):
    c = _random_case(seed)
    monkeypatch.setenv("TFG_PART_PLAN", c["plan"])
    monkeypatch.setenv("TFG_NORM_SLICED", c["sliced"])
    monkeypatch.setenv("TFG_NORM_PARTS", c["by_part"])
    n, n_src, H, F = c["n"], c["n_src"], c["H"], c["F"]
    hub = 0 if c["hub_edges"] else None
    ei = graphgen.random_graph(100 + seed, n, c["e"], n_src=n_src, hub=hub,
                               hub_edges=c["hub_edges"])
    E = ei.shape[1]
    what = f"seed {seed}: {c}"
    eid = dev(ei.astype(c["idx"]))
    g = tfg.tfg_graph_create(eid, n, N_src=n_src, src_parts=c["parts"])
    rowptr, col, perm = tfg.tfg_graph_csr(g)
    parts = g.info()["src_parts"]
    ref_rowptr, ref_col, ref_perm = expected_graph(orc, ei, n, parts=parts, n_src=n_src)[:3]
    assert np.array_equal(host(perm), ref_perm), what
    assert np.array_equal(host(col), ref_col) and np.array_equal(host(rowptr), ref_rowptr), what
    # the aggregation, weighted per edge (or per head) or not
    big = graphgen.features(200 + seed, n_src, c["ldx"])
    x = big[:, :F]
    w = (np.random.default_rng(seed).standard_normal((E, H) if H > 1 else E).astype(np.float32)
         if c["weighted"] else None)
    heads = H if w is not None else 1
    res = tfg.tfg_aggregate(eid, dev(big)[:, :F], n, reduce=c["reduce"],
                            edge_weight=None if w is None else dev(w), heads=heads, graph=g)
    if c["reduce"] == "max":
        out, arg = (host(t) for t in res)
        ref, refarg = orc.aggregate(ei, x, n, "max", edge_weight=w, heads=heads)
        assert same_bits(out, ref) and np.array_equal(arg, refarg), what
    else:
        ref, S = orc.aggregate(ei, x, n, c["reduce"], edge_weight=w, heads=heads)
        assert_scaled(host(res), ref, S, what=what)
    # the normalisation of the square part of the graph (with loops)
    if n_src == n:
        gl = tfg.tfg_graph_create(eid, n, add_self_loops=True, src_parts=c["parts"])
        wn = None if w is None else np.abs(w if H == 1 else w[:, 0]).astype(np.float32) + 0.1
        r = tfg.tfg_gcn_norm(eid, n, edge_weight=None if wn is None else dev(wn), graph=gl)
        oei, ow, odeg = orc.gcn_norm(ei, n, edge_weight=wn)
        assert same_bits(host(r["deg"]), odeg), what
        assert same_bits(host(r["edge_weight"]), ow), what
        lperm = expected_graph(orc, oei, n, parts=gl.info()["src_parts"])[2]
        assert same_bits(host(r["edge_weight_csr"]), ow[lperm]), what


@pytest.mark.parametrize("seed", range(20))
def test_random_attention_and_pooling(tfg, orc, seed):
    """Seeded random attention layers (heads, head width, graph shape, hub
    rows, source parts) through the fused layer and the unfused chain, and
    random pooling batches (graph sizes including empty graphs, width,
    leading dimension, reducer), against the oracle."""
    r = np.random.default_rng([9002, seed])
    n = int(r.integers(2, 3000))
    H = int(r.choice([1, 2, 4, 8]))
    D = int(r.choice([1, 4, 8, 16]))
    hub_edges = int(r.choice([0, 300, 4000]))
    ei = graphgen.random_graph(300 + seed, n, int(r.integers(1, 30_000)),
                               hub=0 if hub_edges else None, hub_edges=hub_edges)
    h = graphgen.features(400 + seed, n, H * D)
    a_s = r.standard_normal((H, D)).astype(np.float32)
    a_d = r.standard_normal((H, D)).astype(np.float32)
    g = tfg.tfg_graph_create(dev(ei), n, src_parts=int(r.choice([0, 1, 3])))
    out = tfg.tfg_gat_aggregate(g, dev(h), dev(a_s), dev(a_d), 0.2)
    ref, ref_alpha, S = orc.gat_layer(ei, h, a_s, a_d, H, slope=np.float32(0.2))
    what = f"seed {seed}: n={n} H={H} D={D} E={ei.shape[1]}"
    assert_scaled(host(out), ref, S, what=what)
    s = tfg.tfg_gat_edge_scores(dev(ei), dev(h), dev(a_s), dev(a_d), 0.2)
    alpha = tfg.tfg_segment_softmax(s, dev(ei[1]), n, graph=g)
    has = np.bincount(ei[1], minlength=n)[ei[1]] > 0
    assert_rel(host(alpha)[has], ref_alpha[has], what=what + " softmax")
    # the same scores and softmax with the per-edge arrays in the graph order
    perm = expected_graph(orc, ei, n, parts=g.info()["src_parts"])[2]
    s_csr = tfg.tfg_gat_graph_scores(g, dev(h), dev(a_s), dev(a_d), 0.2, order="csr")
    assert same_bits(host(s_csr), host(s)[perm]), what + " scores in graph order"
    a_csr = tfg.tfg_segment_softmax_graph(g, s_csr, order="csr")
    assert same_bits(host(a_csr), host(alpha)[perm]), what + " softmax in graph order"
    # the softmax gradient in both orders, and against the oracle
    da = graphgen.features(600 + seed, ei.shape[1], H)
    ds = host(tfg.tfg_segment_softmax_backward(alpha, dev(da), dev(ei[1]), n, graph=g))
    ds_csr = host(tfg.tfg_segment_softmax_graph_backward(g, a_csr, dev(da[perm]), order="csr"))
    assert same_bits(ds_csr, ds[perm]), what + " softmax gradient in graph order"
    a_h = host(alpha)
    dref = orc.segment_softmax_backward(a_h, da, ei[1], n)
    dot = np.zeros((n, H))
    np.add.at(dot, ei[1], a_h.astype(np.float64) * np.abs(da))
    assert_scaled(ds, dref, a_h * (np.abs(da) + dot[ei[1]]), what=what + " softmax gradient")
    # pooling
    G = int(r.integers(1, 800))
    sizes = r.integers(0, 30, G)
    gi = np.repeat(np.arange(G), sizes)
    F = int(r.choice([1, 3, 16, 64, 130]))
    ldx = F + int(r.choice([0, 1, 4]))
    reduce = str(r.choice(["sum", "mean", "max"]))
    if gi.size:
        big = graphgen.features(500 + seed, gi.shape[0], ldx)
        res = tfg.tfg_segment_pool(dev(big)[:, :F], dev(gi.astype(np.int32)), G, reduce)
        if reduce == "max":
            pref, parg = orc.segment_pool(big[:, :F], gi, G, "max")
            assert same_bits(host(res[0]), pref) and np.array_equal(host(res[1]), parg), what
        else:
            pref, pS = orc.segment_pool(big[:, :F], gi, G, reduce)
            assert_scaled(host(res), pref, pS, what=what + f" pool {reduce}")


@pytest.mark.parametrize("seed", range(12))
def test_random_propagation_and_batching(tfg, orc, monkeypatch, seed):
    """Seeded random multi-step propagation (steps, teleport weight, width,
    source parts, plan) one step at a time on the library's own intermediate
    values, and random BatchGraph construction (graph count, sizes, edge
    density, index type) against the oracle."""
    r = np.random.default_rng([9004, seed])
    monkeypatch.setenv("TFG_PART_PLAN", str(r.choice(["0", "1"])))
    n = int(r.integers(2, 2500))
    F = int(r.choice([1, 8, 32, 64]))
    K = int(r.integers(1, 4))
    alpha = float(r.choice([0.0, 0.1, 0.5]))
    ei = graphgen.random_graph(800 + seed, n, int(r.integers(1, 25_000)), hub=0,
                               hub_edges=int(r.choice([0, 3000])))
    x = graphgen.features(900 + seed, n, F)
    g = tfg.tfg_graph_create(dev(ei), n, add_self_loops=True, src_parts=int(r.choice([0, 1, 3])))
    norm = tfg.tfg_gcn_norm(dev(ei), n, graph=g)
    oei, ow, _ = orc.gcn_norm(ei, n)
    z = dev(x)
    for k in range(K):
        zin = host(z)
        z = tfg.tfg_propagate(g, z, 1, alpha=alpha, h=dev(x) if alpha > 0 else None,
                              edge_weight=norm["edge_weight_csr"])
        ref, S = orc.propagate(oei, zin, 1, alpha=alpha, h=x if alpha > 0 else None,
                               edge_weight=ow)
        assert_scaled(host(z), ref, S, what=f"seed {seed} step {k}")
    # BatchGraph construction
    idx = np.int64 if r.random() < 0.3 else np.int32
    G = int(r.integers(1, 2000))
    sizes, graphs = graphgen.batch_of_small_graphs(1000 + seed, G, 0, 40, float(r.uniform(0, 0.3)))
    counts = np.array([gr.shape[1] for gr in graphs])
    local = (np.concatenate(graphs, axis=1) if counts.sum() else np.zeros((2, 0), np.int64))
    bei, bgi, noff, eoff = tfg.tfg_batch_graphs(dev(sizes.astype(idx)), dev(counts.astype(idx)),
                                                dev(local.astype(idx)), int(sizes.sum()))
    ref_ei, ref_gi = orc.batch_graphs(sizes, graphs)
    assert np.array_equal(host(bei), ref_ei) and np.array_equal(host(bgi), ref_gi), seed
    assert np.array_equal(host(noff), orc.batch_offsets(sizes)), seed
    assert np.array_equal(host(eoff), orc.batch_offsets(counts)), seed


def test_every_call_on_a_graph_without_edges(tfg, orc):
    """Each entry point on a graph of 5 nodes and no edges (and, where the call
    takes them, no loops): empty per-edge outputs, zero node outputs, no error."""
    import torch
    cuda = "cuda:0"
    n, F, H, D = 5, 8, 2, 4
    empty = dev(np.zeros((2, 0), np.int64))
    x = dev(graphgen.features(301, n, F))
    g = tfg.tfg_graph_create(empty, n)
    gt = tfg.tfg_graph_create_transposed(empty, n)
    rowptr, col, perm = (host(t) for t in tfg.tfg_graph_csr(g))
    assert np.all(rowptr == 0) and col.size == 0 and perm.size == 0
    tfg.tfg_check(g)
    nz = tfg.tfg_gcn_norm(empty, n, add_self_loops=False, graph=g)
    assert nz["edge_weight"].numel() == 0 and np.all(host(nz["deg"]) == 0)
    nl = tfg.tfg_gcn_norm(empty, n)  # loops only: every weight 1, degree 1
    assert np.all(host(nl["edge_weight"]) == 1) and np.all(host(nl["deg"]) == 1)
    for red in ("sum", "mean"):
        assert np.all(host(tfg.tfg_aggregate(None, x, n, red, graph=g)) == 0)
        assert np.all(host(tfg.tfg_aggregate_noalloc(None, x, n, g, red)) == 0)
    m, a = tfg.tfg_aggregate(None, x, n, "max", graph=g)
    assert np.all(host(m) == 0) and np.all(host(a) == -1)
    dx, dw = tfg.tfg_aggregate_backward(g, x, "sum", graph_t=gt, x=x, want_dw=True)
    assert np.all(host(dx) == 0) and dw.numel() == 0
    assert tfg.tfg_edge_reorder(torch.zeros(0, device=cuda), src=g).numel() == 0
    h = dev(graphgen.features(302, n, H * D))
    a_s = dev(graphgen.features(303, H, D))
    assert tfg.tfg_gat_edge_scores(empty, h, a_s, a_s).shape == (0, H)
    y = tfg.tfg_gat_aggregate(g, h, a_s, a_s)
    assert np.all(host(y) == 0)
    assert tfg.tfg_edge_dot_scores(g, h, h, H).shape == (0, H)
    assert np.all(host(tfg.tfg_gat_dot_aggregate(g, h, h, h, H)) == 0)
    # propagation: no edges leave alpha * h after each step; K = 0 copies x
    assert np.array_equal(host(tfg.tfg_propagate(g, x, 0)), host(x))
    assert np.all(host(tfg.tfg_propagate(g, x, 2)) == 0)
    p = host(tfg.tfg_propagate(g, x, 2, alpha=0.5, h=x))
    assert np.array_equal(p, (np.float32(0.5) * host(x)).astype(np.float32))
    # pooling of no nodes into 3 graphs, and its gradient
    gi = torch.zeros(0, dtype=torch.int64, device=cuda)
    xp = torch.zeros((0, F), device=cuda)
    assert np.all(host(tfg.tfg_segment_pool(xp, gi, 3, "sum")) == 0)
    assert tfg.tfg_segment_pool_backward(torch.ones((3, F), device=cuda), gi).shape == (0, F)
    # a batch of graphs without edges
    nc = torch.tensor([2, 0, 3], dtype=torch.int64, device=cuda)
    ec = torch.zeros(3, dtype=torch.int64, device=cuda)
    bei, bgi, noff, eoff = tfg.tfg_batch_graphs(nc, ec, empty)
    assert bei.shape == (2, 0) and np.array_equal(host(bgi), [0, 0, 2, 2, 2])
    assert np.array_equal(host(noff), [0, 2, 2, 5]) and np.all(host(eoff) == 0)
