"""Pins for the oracle (CPU only).

Each oracle function is checked against something other than itself: dense
brute force written from the mathematical definition, closed forms of small
graphs, library routines (numpy's stable argsort, scipy's softmax), invariants
that hold at any size, and the worked BatchGraph example printed in the paper
(Sec. 2.1.1). The cases are chosen so that a dropped term, a wrong sign or
index, or a transposed operand fails at least one test.
"""

import json
import math
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import graphgen

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def dense_adj(edge_index, n, w=None, n_src=None):
    """A[s, t] = sum of the weights of the edges s -> t (a multigraph adds up)."""
    n_src = n if n_src is None else n_src
    A = np.zeros((n_src, n), np.float64)
    w = np.ones(edge_index.shape[1]) if w is None else np.asarray(w, np.float64)
    np.add.at(A, (edge_index[0], edge_index[1]), w)
    return A


def dense_gcn(edge_index, n, w=None):
    """D^-1/2 (A + I) D^-1/2 in float64, D the weighted in-degree including the loop."""
    A = dense_adj(edge_index, n, w) + np.eye(n)
    deg = A.sum(axis=0)
    dinv = np.where(deg > 0, 1.0 / np.sqrt(np.where(deg > 0, deg, 1.0)), 0.0)
    return dinv[:, None] * A * dinv[None, :], deg


def propagate_dense(Ahat, x):
    """y[t] = sum_s Ahat[s, t] x[s]: messages flow from source rows to target columns."""
    return Ahat.T @ x.astype(np.float64)


# ---------------------------------------------------------------------------
# CSR by target
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed,n,e", [(1, 1, 5), (2, 7, 40), (3, 300, 5000), (4, 5000, 3)])
def test_csr_is_numpy_stable_argsort(orc, seed, n, e):
    ei = graphgen.random_graph(seed, n, e)
    rowptr, col, perm = orc.csr_by_target(ei, n)
    ref_perm = np.argsort(ei[1], kind="stable")
    np.testing.assert_array_equal(perm, ref_perm)
    np.testing.assert_array_equal(col, ei[0][ref_perm])
    np.testing.assert_array_equal(np.diff(rowptr), np.bincount(ei[1], minlength=n))
    assert rowptr[0] == 0 and rowptr[-1] == e


@pytest.mark.parametrize("seed,n,n_src,e,parts", [(5, 40, 40, 3000, 2), (6, 300, 77, 9000, 3),
                                                 (7, 1000, 5000, 20000, 8), (8, 9, 9, 50, 9)])
def test_part_order_from_plain_csr(orc, seed, n, n_src, e, parts):
    """The tests' regrouping of the oracle's plain CSR into the (target, source
    part) order of a handle with several source parts equals numpy's stable
    argsort of that composite key over the edge list."""
    from graph_order import expected_graph, part_rows
    ei = graphgen.random_graph(seed, n, e, n_src=n_src)
    rowptr, col, perm, seg = expected_graph(orc, ei, n, parts=parts, n_src=n_src)
    key = ei[1] * parts + ei[0] // part_rows(n_src, parts)
    ref = np.argsort(key, kind="stable")
    np.testing.assert_array_equal(perm, ref)
    np.testing.assert_array_equal(col, ei[0][ref])
    np.testing.assert_array_equal(np.diff(seg), np.bincount(key, minlength=n * parts))
    np.testing.assert_array_equal(rowptr, seg[::parts])
    # the rows are those of the plain CSR; only the order inside a row changes
    r1, _, p1 = orc.csr_by_target(ei, n, n_src=n_src)
    np.testing.assert_array_equal(rowptr, r1)
    for t in range(0, n, max(1, n // 17)):
        assert sorted(perm[rowptr[t]:rowptr[t + 1]]) == list(p1[r1[t]:r1[t + 1]])


def test_csr_brute_force_tiny(orc):
    ei = graphgen.random_graph(11, 6, 25)
    rowptr, col, perm = orc.csr_by_target(ei, 6)
    k = 0
    for t in range(6):  # O(N * E): scan all edges once per target, in input order
        for e in range(ei.shape[1]):
            if ei[1, e] == t:
                assert perm[k] == e and col[k] == ei[0, e]
                k += 1
        assert rowptr[t + 1] == k


def test_csr_invariants_and_empty(orc):
    rowptr, col, perm = orc.csr_by_target(np.zeros((2, 0), np.int64), 4)
    assert list(rowptr) == [0, 0, 0, 0, 0] and col.size == 0 and perm.size == 0
    ei = graphgen.random_graph(5, 50, 2000, hub=3, hub_edges=500)
    rowptr, col, perm = orc.csr_by_target(ei, 50)
    assert sorted(perm.tolist()) == list(range(ei.shape[1]))
    assert np.all(np.diff(ei[1][perm]) >= 0)
    for t in range(50):
        seg = perm[rowptr[t]:rowptr[t + 1]]
        assert np.all(np.diff(seg) > 0)  # input order kept inside a row


def test_csr_rejects_out_of_range(orc):
    with pytest.raises(orc.OracleError) as ex:
        orc.csr_by_target(np.array([[0, 1], [0, 5]]), 3)
    assert ex.value.code == orc.ERR_INDEX_RANGE


# ---------------------------------------------------------------------------
# GCN normalisation
# ---------------------------------------------------------------------------

def test_gcn_norm_hand_example(orc):
    g = json.load(open(os.path.join(GOLDEN, "gcn_path3_hand.json")))
    ei = np.array(g["edge_index"])
    out_ei, w, deg = orc.gcn_norm(ei, 3)
    np.testing.assert_array_equal(deg, np.array(g["deg"], np.float32))
    np.testing.assert_allclose(w, g["edge_weight_in_order_edges_then_loops"], rtol=4 * 2.0**-24)
    np.testing.assert_array_equal(out_ei, np.array([[0, 1, 1, 2, 0, 1, 2], [1, 0, 2, 1, 0, 1, 2]]))
    x = np.array(g["x"], np.float32)[:, None]
    y, _ = orc.aggregate(out_ei, x, 3, "sum", edge_weight=w)
    np.testing.assert_allclose(y[:, 0], g["y"], rtol=3e-7)


@pytest.mark.parametrize("seed,n,e,weighted", [(1, 5, 12, False), (2, 17, 60, True),
                                               (3, 64, 400, False), (4, 40, 300, True)])
def test_gcn_matches_dense(orc, seed, n, e, weighted):
    ei = graphgen.random_graph(seed, n, e)  # duplicates and self-loops included
    w = (np.random.default_rng(seed).uniform(0.1, 2.0, e).astype(np.float32)
         if weighted else None)
    out_ei, what, deg = orc.gcn_norm(ei, n, edge_weight=w)
    Ahat, ddeg = dense_gcn(ei, n, w)
    np.testing.assert_allclose(deg, ddeg, rtol=1e-7)
    x = graphgen.features(seed, n, 9)
    y, S = orc.aggregate(out_ei, x, n, "sum", edge_weight=what)
    ref = propagate_dense(Ahat, x)
    # weights carry three float32 roundings each: |y - ref| <= 4u * sum |w x|
    assert np.all(np.abs(y - ref) <= 4 * 2.0**-24 * S + 1e-300)


def test_gcn_complete_graph(orc):
    n = 7  # K_n plus loops: every A_hat entry is 1/n, so each output is the column mean
    i, j = np.where(~np.eye(n, dtype=bool))
    ei = np.stack([i, j]).astype(np.int64)
    out_ei, w, deg = orc.gcn_norm(ei, n)
    assert np.all(deg == n)
    np.testing.assert_allclose(w, 1.0 / n, rtol=4 * 2.0**-24)
    x = graphgen.features(1, n, 5)
    y, _ = orc.aggregate(out_ei, x, n, "sum", edge_weight=w)
    np.testing.assert_allclose(y, np.tile(x.astype(np.float64).mean(0), (n, 1)), atol=1e-6)


def test_gcn_star(orc):
    c = 9  # hub 0 with c leaves, both directions
    leaves = np.arange(1, c + 1)
    ei = np.stack([np.concatenate([leaves, np.zeros(c, int)]),
                   np.concatenate([np.zeros(c, int), leaves])]).astype(np.int64)
    out_ei, w, deg = orc.gcn_norm(ei, c + 1)
    assert deg[0] == c + 1 and np.all(deg[1:] == 2)
    np.testing.assert_allclose(w[:2 * c], 1 / math.sqrt(2 * (c + 1)), rtol=4 * 2.0**-24)
    np.testing.assert_allclose(w[2 * c], 1 / (c + 1), rtol=4 * 2.0**-24)  # hub loop
    np.testing.assert_allclose(w[2 * c + 1:], 0.5, rtol=4 * 2.0**-24)  # leaf loops


def test_gcn_isolated_node_is_identity(orc):
    ei = np.array([[0, 1], [1, 0]])  # node 2 isolated
    out_ei, w, deg = orc.gcn_norm(ei, 3)
    assert deg[2] == 1 and w[-1] == 1.0
    x = graphgen.features(3, 3, 4)
    y, _ = orc.aggregate(out_ei, x, 3, "sum", edge_weight=w)
    assert np.array_equal(y[2].astype(np.float32), x[2])  # exactly


def test_gcn_regular_ring(orc):
    n, k = 12, 4  # 4-regular ring: A_hat = (A + I) / (k + 1)
    src, tgt = [], []
    for v in range(n):
        for d in (1, 2):
            src += [v, (v + d) % n]
            tgt += [(v + d) % n, v]
    ei = np.array([src, tgt], np.int64)
    out_ei, w, deg = orc.gcn_norm(ei, n)
    assert np.all(deg == k + 1)
    np.testing.assert_allclose(w, 1 / (k + 1), rtol=4 * 2.0**-24)


def test_gcn_sqrt_degree_is_fixed_point(orc):
    # (A_hat s)_t = dinv_t * sum_{e->t} w_e = sqrt(deg_t) for s = sqrt(deg), at any size
    n = 3000
    ei = graphgen.random_graph(8, n, 60000, hub=5, hub_edges=4000)
    out_ei, w, deg = orc.gcn_norm(ei, n)
    s = np.sqrt(deg.astype(np.float64)).astype(np.float32)[:, None]
    y, S = orc.aggregate(out_ei, s, n, "sum", edge_weight=w)
    assert np.all(np.abs(y[:, 0] - s[:, 0]) <= 1e-6 * S[:, 0])


def test_gcn_without_loops_and_zero_degree(orc):
    ei = np.array([[0, 0], [1, 1]])  # target 0 and 2 have no in-edges, no loops
    out_ei, w, deg = orc.gcn_norm(ei, 3, add_self_loops=False)
    assert list(deg) == [0, 2, 0]
    # src 0 has in-degree 0, so dinv[0] = 0 and its messages vanish
    assert np.all(w == 0.0) and out_ei.shape == (2, 2)


# ---------------------------------------------------------------------------
# Aggregation
# ---------------------------------------------------------------------------

@settings(max_examples=40, deadline=None)
@given(n=st.integers(1, 12), n_src=st.integers(1, 12), e=st.integers(0, 60),
       f=st.integers(1, 6), seed=st.integers(0, 10**6), weighted=st.booleans())
def test_aggregate_sum_mean_dense(orc, n, n_src, e, f, seed, weighted):
    ei = graphgen.random_graph(seed, n, e, n_src=n_src)
    w = np.random.default_rng(seed).standard_normal(e).astype(np.float32) if weighted else None
    x = graphgen.features(seed, n_src, f)
    A = dense_adj(ei, n, w, n_src=n_src)
    ref = A.T @ x.astype(np.float64)
    y, S = orc.aggregate(ei, x, n, "sum", edge_weight=w)
    assert np.all(np.abs(y - ref) <= 1e-12 * (S + 1e-300))
    cnt = np.bincount(ei[1], minlength=n).astype(np.float64)
    ym, _ = orc.aggregate(ei, x, n, "mean", edge_weight=w)
    refm = np.where(cnt[:, None] > 0, ref / np.maximum(cnt, 1)[:, None], 0.0)
    np.testing.assert_allclose(ym, refm, rtol=1e-12, atol=1e-12)


def test_aggregate_per_head_weights(orc):
    n, e, H, D = 9, 50, 3, 4
    ei = graphgen.random_graph(4, n, e)
    w = np.random.default_rng(4).standard_normal((e, H)).astype(np.float32)
    x = graphgen.features(4, n, H * D)
    y, _ = orc.aggregate(ei, x, n, "sum", edge_weight=w, heads=H)
    for h in range(H):
        A = dense_adj(ei, n, w[:, h])
        ref = A.T @ x[:, h * D:(h + 1) * D].astype(np.float64)
        np.testing.assert_allclose(y[:, h * D:(h + 1) * D], ref, rtol=1e-12, atol=1e-12)


def test_aggregate_ones_is_in_degree_and_mean_is_one(orc):
    n = 200
    ei = graphgen.random_graph(9, n, 3000)
    x = np.ones((n, 3), np.float32)
    y, _ = orc.aggregate(ei, x, n, "sum")
    cnt = np.bincount(ei[1], minlength=n)
    assert np.array_equal(y[:, 0], cnt.astype(np.float64))
    ym, _ = orc.aggregate(ei, x, n, "mean")
    assert np.array_equal(ym[:, 1], (cnt > 0).astype(np.float64))


def test_aggregate_ldx_stride(orc):
    n = 20
    ei = graphgen.random_graph(2, n, 100)
    big = graphgen.features(2, n, 11)
    y1, _ = orc.aggregate(ei, big[:, :7], n, "sum")  # ldx = 11 > F = 7
    y2, _ = orc.aggregate(ei, np.ascontiguousarray(big[:, :7]), n, "sum")
    assert np.array_equal(y1, y2)


def brute_max(ei, x, n, w):
    F = x.shape[1]
    out = np.zeros((n, F), np.float32)
    arg = np.full((n, F), -1, np.int64)
    for t in range(n):
        es = [e for e in range(ei.shape[1]) if ei[1, e] == t]
        for c in range(F):
            best = None
            for e in es:  # first maximal edge in input order wins
                m = np.float32(w[e]) * x[ei[0, e], c]
                if best is None or m > best:
                    best, arg[t, c] = m, e
            if best is not None:
                out[t, c] = best
    return out, arg


def test_aggregate_max_brute_force_with_ties(orc):
    n = 10
    ei = graphgen.random_graph(6, n, 80)
    w = np.random.default_rng(6).choice(np.float32([0.5, 1.0, -1.0, 2.0]), 80).astype(np.float32)
    x = np.random.default_rng(7).integers(-2, 3, (n, 5)).astype(np.float32)  # many ties
    x[0, 0] = -0.0
    out, arg = orc.aggregate(ei, x, n, "max", edge_weight=w)
    ref, refarg = brute_max(ei, x, n, w)
    assert np.array_equal(out.view(np.int32), ref.view(np.int32))
    assert np.array_equal(arg, refarg)


def test_aggregate_max_signed_zero_is_a_tie(orc):
    ei = np.array([[0, 1], [2, 2]])
    x = np.array([[0.0], [-0.0], [5.0]], np.float32)
    x[0, 0] = -0.0
    x[1, 0] = 0.0
    out, arg = orc.aggregate(ei, x, 3, "max")
    assert arg[2, 0] == 0 and np.signbit(out[2, 0])  # -0 first, +0 does not replace it
    assert arg[0, 0] == -1 and out[0, 0] == 0.0  # empty target


def test_aggregate_max_properties(orc):
    n = 300
    ei = graphgen.random_graph(12, n, 5000)
    w = np.random.default_rng(12).standard_normal(5000).astype(np.float32)
    x = graphgen.features(12, n, 8)
    out, arg = orc.aggregate(ei, x, n, "max", edge_weight=w)
    cnt = np.bincount(ei[1], minlength=n)
    for t in range(n):
        for c in range(8):
            if cnt[t] == 0:
                assert arg[t, c] == -1 and out[t, c] == 0
                continue
            e = arg[t, c]
            assert ei[1, e] == t
            assert out[t, c] == np.float32(w[e]) * x[ei[0, e], c]
            members = np.float32(w[ei[1] == t]) * x[ei[0][ei[1] == t], c]
            assert np.all(members <= out[t, c])


def test_aggregate_sampled_rows_equal_full(orc):
    n = 500
    ei = graphgen.random_graph(13, n, 8000)
    x = graphgen.features(13, n, 6)
    y, S = orc.aggregate(ei, x, n, "sum")
    rows = np.array([3, 499, 0, 250])
    ys, Ss = orc.aggregate(ei, x, n, "sum", rows=rows)
    assert np.array_equal(ys, y[rows]) and np.array_equal(Ss, S[rows])
    m, a = orc.aggregate(ei, x, n, "max")
    ms, as_ = orc.aggregate(ei, x, n, "max", rows=rows)
    assert np.array_equal(ms, m[rows]) and np.array_equal(as_, a[rows])


# ---------------------------------------------------------------------------
# Segment softmax
# ---------------------------------------------------------------------------

def test_softmax_matches_scipy(orc):
    from scipy.special import softmax
    n, e, H = 30, 400, 3
    seg = graphgen.random_graph(3, n, e)[1]
    s = (graphgen.features(3, e, H) * 4).astype(np.float32)
    a64, a32 = orc.segment_softmax(s, seg, n)
    for t in range(n):
        idx = np.nonzero(seg == t)[0]
        if idx.size:
            ref = softmax(s[idx].astype(np.float64), axis=0)
            np.testing.assert_allclose(a64[idx], ref, rtol=1e-13)
    assert np.array_equal(a32, a64.astype(np.float32))


def test_softmax_closed_forms(orc):
    seg = np.array([0, 1, 1, 1, 2, 2, 3])
    s = np.array([5.0, 2.0, 2.0, 2.0, -100.0, 100.0, -3e38], np.float32)
    a64, a32 = orc.segment_softmax(s, seg, 5)
    assert a32[0] == 1.0 and a32[6] == 1.0  # size-1 segments
    assert np.all(a32[1:4] == np.float32(1.0 / 3.0))  # constant scores
    assert a32[5] == 1.0 and a64[4] == pytest.approx(math.exp(-200.0), rel=1e-12)


def test_softmax_wide_spread_stays_finite(orc):
    # exp(1000) overflows double: only a shift by the segment maximum keeps every term finite
    seg = np.array([0, 0, 0])
    s = np.array([-500.0, 500.0, 499.0], np.float32)
    a64, a32 = orc.segment_softmax(s, seg, 1)
    assert np.all(np.isfinite(a64))
    np.testing.assert_allclose(a64, [0.0, 1 / (1 + math.exp(-1)), math.exp(-1) / (1 + math.exp(-1))],
                               rtol=1e-14, atol=1e-300)


def test_softmax_sums_to_one_and_shift_invariant(orc):
    n, e, H = 1000, 30000, 4
    seg = graphgen.random_graph(21, n, e, hub=7, hub_edges=3000)[1]
    s = graphgen.features(21, seg.shape[0], H) * 5
    a64, _ = orc.segment_softmax(s, seg, n)
    tot = np.zeros((n, H))
    np.add.at(tot, seg, a64)
    has = np.bincount(seg, minlength=n) > 0
    np.testing.assert_allclose(tot[has], 1.0, rtol=1e-12)
    shift = np.random.default_rng(1).integers(-8, 8, n).astype(np.float32)  # exact in fp32
    b64, _ = orc.segment_softmax(s + shift[seg][:, None], seg, n)
    np.testing.assert_allclose(b64, a64, rtol=1e-5)


# ---------------------------------------------------------------------------
# Pooling
# ---------------------------------------------------------------------------

def test_pool_single_graph_is_column_reduction(orc):
    x = graphgen.features(5, 37, 6)
    gi = np.zeros(37, np.int64)
    s, _ = orc.segment_pool(x, gi, 1, "sum")
    np.testing.assert_allclose(s[0], x.astype(np.float64).sum(0), rtol=1e-12)
    m, _ = orc.segment_pool(x, gi, 1, "mean")
    np.testing.assert_allclose(m[0], x.astype(np.float64).mean(0), rtol=1e-12, atol=1e-15)
    mx, arg = orc.segment_pool(x, gi, 1, "max")
    assert np.array_equal(mx[0], x.max(0)) and np.array_equal(arg[0], x.argmax(0))


def test_pool_equals_aggregation_over_membership_edges(orc):
    sizes = np.array([3, 0, 5, 1, 4])  # an empty graph included
    gi = np.repeat(np.arange(5), sizes)
    nb = gi.shape[0]
    x = graphgen.features(6, nb, 7)
    ei = np.stack([np.arange(nb), gi])  # node n -> graph gi[n]
    for red in ("sum", "mean"):
        p, ps = orc.segment_pool(x, gi, 5, red)
        a, as_ = orc.aggregate(ei, x, 5, red)
        assert np.array_equal(p, a) and np.array_equal(ps, as_)
    p, pa = orc.segment_pool(x, gi, 5, "max")
    a, aa = orc.aggregate(ei, x, 5, "max")
    assert np.array_equal(p, a) and np.array_equal(pa, aa)  # edge id == node id here
    assert np.all(pa[1] == -1) and np.all(p[1] == 0)


def test_pool_total_and_mean(orc):
    sizes = np.random.default_rng(2).integers(1, 30, 50)
    gi = np.repeat(np.arange(50), sizes)
    x = graphgen.features(7, gi.shape[0], 5)
    s, S = orc.segment_pool(x, gi, 50, "sum")
    np.testing.assert_allclose(s.sum(0), x.astype(np.float64).sum(0), rtol=1e-10, atol=1e-10)
    m, _ = orc.segment_pool(x, gi, 50, "mean")
    np.testing.assert_allclose(m, s / sizes[:, None], rtol=1e-14)


def test_pool_errors(orc):
    x = np.zeros((3, 2), np.float32)
    with pytest.raises(orc.OracleError) as ex:
        orc.segment_pool(x, np.array([0, 2, 1]), 3)
    assert ex.value.code == orc.ERR_UNSORTED
    with pytest.raises(orc.OracleError) as ex:
        orc.segment_pool(x, np.array([0, 1, 3]), 3)
    assert ex.value.code == orc.ERR_INDEX_RANGE


# ---------------------------------------------------------------------------
# GAT scores
# ---------------------------------------------------------------------------

def test_gat_scores_dense(orc):
    n, e, H, D = 15, 90, 4, 3
    ei = graphgen.random_graph(8, n, e)
    h = graphgen.features(8, n, H * D)
    r = np.random.default_rng(9)
    a_s = r.standard_normal((H, D)).astype(np.float32)
    a_d = r.standard_normal((H, D)).astype(np.float32)
    s, S = orc.gat_scores(ei, h, a_s, a_d, H, slope=0.2)
    h3 = h.astype(np.float64).reshape(n, H, D)
    z = np.einsum("nhd,hd->nh", h3, a_s)[ei[0]] + np.einsum("nhd,hd->nh", h3, a_d)[ei[1]]
    ref = np.where(z >= 0, z, np.float64(np.float32(0.2)) * z)
    np.testing.assert_allclose(s, ref, rtol=1e-12, atol=1e-12)
    assert np.all(S >= np.abs(s) - 1e-12)


# ---------------------------------------------------------------------------
# BatchGraph (Sec. 2.1.1)
# ---------------------------------------------------------------------------

def test_batch_reindex_paper_example(orc):
    g = json.load(open(os.path.join(GOLDEN, "batch_reindex_paper_example.json")))
    off = orc.batch_offsets(np.array(g["sizes"]))
    assert list(off[1:3]) == g["offsets_of_graphs_2_and_3"]
    for ex in g["one_based_examples"]:
        zero_based = ex["node"] - 1 + off[ex["graph"] - 1]
        assert zero_based + 1 == ex["batched_index"]


def test_batch_equals_per_graph(orc):
    """Applying the GNN to each graph separately equals applying it to the
    BatchGraph (Sec. 2.1.1): 3 GCN propagations then sum / mean / max pooling."""
    sizes, graphs = graphgen.batch_of_small_graphs(77, 40, 10, 60, 0.1)
    ei, gi = orc.batch_graphs(sizes, graphs)
    ei2, gi2 = graphgen.stack_batch(sizes, graphs)  # the input generator's own batching
    assert np.array_equal(ei, ei2) and np.array_equal(gi, gi2)
    nb = int(sizes.sum())
    x = graphgen.features(77, nb, 6)
    out_ei, w, _ = orc.gcn_norm(ei, nb)
    h = x
    for _ in range(3):
        h, _ = orc.aggregate(out_ei, h, nb, "sum", edge_weight=w)
        h = h.astype(np.float32)
    pooled = {r: orc.segment_pool(h, gi, len(sizes), r)[0] for r in ("sum", "mean", "max")}
    off = orc.batch_offsets(sizes)
    for i, (n, g) in enumerate(zip(sizes.tolist(), graphs)):
        oe, ow, _ = orc.gcn_norm(g, n)
        hl = x[off[i]:off[i + 1]]
        for _ in range(3):
            hl, _ = orc.aggregate(oe, hl, n, "sum", edge_weight=ow)
            hl = hl.astype(np.float32)
        assert np.array_equal(hl, h[off[i]:off[i + 1]])
        loc = np.zeros(n, np.int64)
        for r in ("sum", "mean", "max"):
            assert np.array_equal(orc.segment_pool(hl, loc, 1, r)[0][0], pooled[r][i])


# ---------------------------------------------------------------------------
# Propagation (SGC / APPNP)
# ---------------------------------------------------------------------------

def test_propagate_dense_closed_form(orc):
    n, K, alpha = 30, 5, 0.15
    ei = graphgen.random_graph(41, n, 200)
    out_ei, w, _ = orc.gcn_norm(ei, n)
    x = graphgen.features(41, n, 4)
    h = graphgen.features(42, n, 4)
    M = (1 - alpha) * dense_adj(out_ei, n, w).T  # messages: y[t] = sum_s A[s, t] z[s]
    ref = np.linalg.matrix_power(M, K) @ x.astype(np.float64)
    ref += alpha * sum(np.linalg.matrix_power(M, j) for j in range(K)) @ h.astype(np.float64)
    z, S = orc.propagate(out_ei, x, K, alpha=alpha, h=h, edge_weight=w)
    np.testing.assert_allclose(z, ref, rtol=1e-12, atol=1e-12)
    assert np.all(S >= np.abs(z) - 1e-12)


def test_propagate_special_cases(orc):
    n = 50
    ei = graphgen.random_graph(43, n, 400)
    out_ei, w, deg = orc.gcn_norm(ei, n)
    x = graphgen.features(43, n, 3)
    h = graphgen.features(44, n, 3)
    z0, _ = orc.propagate(out_ei, x, 0, edge_weight=w)
    assert np.array_equal(z0, x.astype(np.float64))  # K = 0
    z1, _ = orc.propagate(out_ei, x, 4, alpha=1.0, h=h, edge_weight=w)
    assert np.array_equal(z1, h.astype(np.float64))  # alpha = 1: only the teleport term
    y, _ = orc.propagate(out_ei, x, 1, edge_weight=w)
    agg, _ = orc.aggregate(out_ei, x, n, "sum", edge_weight=w)
    np.testing.assert_allclose(y, agg, rtol=1e-14, atol=1e-15)
    # sqrt(deg) is a fixed point of A_hat, hence of every APPNP step with h = sqrt(deg)
    s = np.sqrt(deg.astype(np.float64)).astype(np.float32)[:, None]
    zs, _ = orc.propagate(out_ei, s, 7, alpha=0.3, h=s, edge_weight=w)
    np.testing.assert_allclose(zs, s.astype(np.float64), rtol=2e-6)


def test_propagate_appnp_limit(orc):
    # many steps converge to alpha (I - (1 - alpha) A^T)^-1 h
    n, alpha = 25, 0.2
    ei = graphgen.random_graph(45, n, 150)
    out_ei, w, _ = orc.gcn_norm(ei, n)
    h = graphgen.features(45, n, 2)
    z, _ = orc.propagate(out_ei, h, 300, alpha=alpha, h=h, edge_weight=w)
    M = (1 - alpha) * dense_adj(out_ei, n, w).T
    ref = alpha * np.linalg.solve(np.eye(n) - M, h.astype(np.float64))
    np.testing.assert_allclose(z, ref, rtol=1e-9, atol=1e-12)


# ---------------------------------------------------------------------------
# GAT layer (scores -> softmax -> weighted aggregation)
# ---------------------------------------------------------------------------

def test_gat_layer_zero_attention_is_mean(orc):
    # a_src = a_dst = 0: every score is 0, attention is uniform, output = mean of in-neighbours
    n, e, H, D = 40, 300, 4, 3
    ei = graphgen.random_graph(51, n, e)
    h = graphgen.features(51, n, H * D)
    z = np.zeros((H, D), np.float32)
    out, alpha, _ = orc.gat_layer(ei, h, z, z, H)
    mean, _ = orc.aggregate(ei, h, n, "mean")
    np.testing.assert_allclose(out, mean, rtol=1e-13, atol=1e-15)
    cnt = np.bincount(ei[1], minlength=n)
    np.testing.assert_allclose(alpha[:, 0], 1.0 / cnt[ei[1]], rtol=1e-15)


def test_gat_layer_single_edge_and_dense(orc):
    n, H, D = 12, 2, 3
    ei = graphgen.random_graph(52, n, 40)
    h = graphgen.features(52, n, H * D)
    r = np.random.default_rng(52)
    a_s = r.standard_normal((H, D)).astype(np.float32)
    a_d = r.standard_normal((H, D)).astype(np.float32)
    out, alpha, S = orc.gat_layer(ei, h, a_s, a_d, H, slope=0.2)
    # dense: per target and head, softmax over the in-edge scores, then the weighted sum
    h3 = h.astype(np.float64).reshape(n, H, D)
    z = (np.einsum("nhd,hd->nh", h3, a_s)[ei[0]] + np.einsum("nhd,hd->nh", h3, a_d)[ei[1]])
    s = np.where(z >= 0, z, np.float64(np.float32(0.2)) * z).astype(np.float32).astype(np.float64)
    ref = np.zeros((n, H, D))
    for t in range(n):
        idx = np.nonzero(ei[1] == t)[0]
        if idx.size == 0:
            continue
        a = np.exp(s[idx] - s[idx].max(0))
        a /= a.sum(0)
        ref[t] = np.einsum("eh,ehd->hd", a, h3[ei[0][idx]])
        if idx.size == 1:
            assert np.array_equal(out[t], h3[ei[0][idx[0]]].reshape(-1))  # alpha = 1 exactly
    np.testing.assert_allclose(out, ref.reshape(n, H * D), rtol=1e-12, atol=1e-12)
    assert np.all(S >= np.abs(out) - 1e-12)


# ---------------------------------------------------------------------------
# Backward: finite differences of the forward oracle
# ---------------------------------------------------------------------------

def _loss(orc, ei, x, n, dy, reduce, w, heads):
    if reduce == "max":
        out, _ = orc.aggregate(ei, x, n, "max", edge_weight=w, heads=heads)
        return float((out.astype(np.float64) * dy).sum())
    out, _ = orc.aggregate(ei, x, n, reduce, edge_weight=w, heads=heads)
    return float((out * dy).sum())


@pytest.mark.parametrize("reduce,heads", [("sum", 1), ("mean", 1), ("sum", 2), ("max", 1)])
def test_aggregate_backward_finite_differences(orc, reduce, heads):
    n, n_src, e, F = 9, 11, 60, 4
    ei = graphgen.random_graph(61, n, e, n_src=n_src)
    rng = np.random.default_rng(61)
    x = rng.standard_normal((n_src, F)).astype(np.float32)
    w = rng.uniform(0.5, 2.0, (e, heads) if heads > 1 else e).astype(np.float32)
    dy = rng.standard_normal((n, F))
    arg = orc.aggregate(ei, x, n, "max", edge_weight=w, heads=heads)[1] if reduce == "max" else None
    dx, dw = orc.aggregate_backward(ei, x, n, dy, reduce, edge_weight=w, heads=heads, arg=arg)
    # the loss is linear (piecewise linear for max) in x and in w; the sums are taken in double,
    # the max of float32 products, whose rounding (2^-24 relative) over a step of 2^-10 leaves
    # an error near 2^-14 in the quotient
    eps = 2.0 ** -10
    rel = 2e-4 if reduce == "max" else 1e-6
    for (i, c) in [(0, 0), (3, 2), (n_src - 1, 3), (5, 1)]:
        xp, xm = x.copy(), x.copy()
        xp[i, c] += eps
        xm[i, c] -= eps
        fd = (_loss(orc, ei, xp, n, dy, reduce, w, heads) -
              _loss(orc, ei, xm, n, dy, reduce, w, heads)) / (2 * eps)
        assert fd == pytest.approx(dx[i, c], rel=rel, abs=1e-9)
    for j in [0, 7, e - 1]:
        for k in range(heads):
            wp, wm = w.copy(), w.copy()
            if heads > 1:
                wp[j, k] += eps
                wm[j, k] -= eps
            else:
                wp[j] += eps
                wm[j] -= eps
            fd = (_loss(orc, ei, x, n, dy, reduce, wp, heads) -
                  _loss(orc, ei, x, n, dy, reduce, wm, heads)) / (2 * eps)
            assert fd == pytest.approx(dw[j, k], rel=rel, abs=1e-9 if reduce != "max" else 1e-4)


def test_aggregate_backward_is_transpose(orc):
    # dx of a sum aggregation is the aggregation over the reversed edges
    n, e, F = 40, 500, 5
    ei = graphgen.random_graph(62, n, e)
    w = np.random.default_rng(62).standard_normal(e).astype(np.float32)
    x = graphgen.features(62, n, F)
    dy = graphgen.features(63, n, F)
    dx, _ = orc.aggregate_backward(ei, x, n, dy, "sum", edge_weight=w)
    rev, _ = orc.aggregate(ei[::-1], dy, n, "sum", edge_weight=w)
    np.testing.assert_allclose(dx, rev, rtol=1e-12, atol=1e-12)


def test_softmax_backward_finite_differences(orc):
    n, e, H = 6, 40, 2
    seg = graphgen.random_graph(64, n, e)[1]
    rng = np.random.default_rng(64)
    s = rng.standard_normal((e, H)).astype(np.float32)
    da = rng.standard_normal((e, H)).astype(np.float32)
    a64, a32 = orc.segment_softmax(s, seg, n)
    ds = orc.segment_softmax_backward(a64.astype(np.float32), da, seg, n)
    eps = 1e-3
    for (i, h) in [(0, 0), (5, 1), (e - 1, 0), (17, 1)]:
        sp, sm = s.astype(np.float64), s.astype(np.float64)
        sp = sp.copy(); sm = sm.copy()
        sp[i, h] += eps
        sm[i, h] -= eps
        lp = (orc.segment_softmax(sp.astype(np.float32), seg, n)[0] * da).sum()
        lm = (orc.segment_softmax(sm.astype(np.float32), seg, n)[0] * da).sum()
        # float32 perturbed scores: compare with the rounding-aware step
        step = float(np.float32(s[i, h] + eps)) - float(np.float32(s[i, h] - eps))
        assert (lp - lm) / step == pytest.approx(ds[i, h], rel=2e-4, abs=1e-6)


# ---------------------------------------------------------------------------
# Transformer-style attention (scaled dot-product scores)
# ---------------------------------------------------------------------------

def test_dot_scores_brute_force(orc):
    n, e, H, D = 7, 30, 3, 4
    ei = graphgen.random_graph(71, n, e)
    rng = np.random.default_rng(71)
    q = rng.standard_normal((n, H * D)).astype(np.float32)
    k = rng.standard_normal((n, H * D)).astype(np.float32)
    s = orc.dot_scores(ei, q, k, H, 0.5)
    q3 = q.astype(np.float64).reshape(n, H, D)
    k3 = k.astype(np.float64).reshape(n, H, D)
    for j in range(e):
        for h in range(H):
            ref = 0.5 * sum(q3[ei[1, j], h, d] * k3[ei[0, j], h, d] for d in range(D))
            assert s[j, h] == pytest.approx(ref, rel=1e-14, abs=1e-14)


def test_dot_layer_zero_query_is_mean(orc):
    # q = 0: every score is 0, the attention is uniform, the output is the mean of v
    n, e, H, D = 30, 200, 2, 4
    ei = graphgen.random_graph(72, n, e)
    k = graphgen.features(72, n, H * D)
    v = graphgen.features(73, n, H * D)
    out, alpha, _ = orc.dot_layer(ei, np.zeros_like(k), k, v, H, 0.25)
    mean, _ = orc.aggregate(ei, v, n, "mean")
    np.testing.assert_allclose(out, mean, rtol=1e-13, atol=1e-15)
    cnt = np.bincount(ei[1], minlength=n)
    np.testing.assert_allclose(alpha[:, 1], 1.0 / cnt[ei[1]], rtol=1e-15)


def test_dot_layer_dense(orc):
    # a dense check: per target and head, softmax of the float32 scores, then the weighted sum
    n, H, D = 9, 2, 3
    ei = graphgen.random_graph(74, n, 35)
    rng = np.random.default_rng(74)
    q, k, v = (rng.standard_normal((n, H * D)).astype(np.float32) for _ in range(3))
    scale = 1 / np.sqrt(D)
    out, alpha, _ = orc.dot_layer(ei, q, k, v, H, scale)
    s = np.einsum("ehd,ehd->eh", q.astype(np.float64).reshape(n, H, D)[ei[1]],
                  k.astype(np.float64).reshape(n, H, D)[ei[0]]) * scale
    s = s.astype(np.float32).astype(np.float64)
    ref = np.zeros((n, H, D))
    for t in range(n):
        m = ei[1] == t
        if not m.any():
            continue
        a = np.exp(s[m] - s[m].max(0))
        a /= a.sum(0)
        ref[t] = np.einsum("eh,ehd->hd", a, v.astype(np.float64).reshape(n, H, D)[ei[0][m]])
    np.testing.assert_allclose(out, ref.reshape(n, H * D), rtol=1e-12, atol=1e-13)
    tot = np.zeros((n, H))
    np.add.at(tot, ei[1], alpha)
    has = np.bincount(ei[1], minlength=n) > 0
    np.testing.assert_allclose(tot[has], 1.0, rtol=1e-13)


def test_dot_layer_single_edge_copies_value(orc):
    # a target with one in-edge gets exactly the value row of its source
    ei = np.array([[3, 1, 2], [0, 2, 2]])
    rng = np.random.default_rng(75)
    q, k, v = (rng.standard_normal((4, 8)).astype(np.float32) for _ in range(3))
    out, alpha, _ = orc.dot_layer(ei, q, k, v, 2, 0.5)
    np.testing.assert_array_equal(out[0], v[3].astype(np.float64))
    assert np.all(out[[1, 3]] == 0) and np.all(alpha[0] == 1.0)


@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
def test_pool_backward_finite_differences(orc, reduce):
    sizes = np.array([3, 1, 4, 2])
    gi = np.repeat(np.arange(4), sizes)
    Nb, F, G = gi.shape[0], 3, 4
    rng = np.random.default_rng(81)
    x = rng.standard_normal((Nb, F)).astype(np.float32)
    dy = rng.standard_normal((G, F))
    arg = orc.segment_pool(x, gi, G, "max")[1] if reduce == "max" else None
    dx = orc.segment_pool_backward(dy, gi, G, reduce, arg=arg)

    def loss(xx):
        out = orc.segment_pool(xx, gi, G, reduce)[0]
        return float((np.asarray(out, np.float64) * dy).sum())
    eps = 2.0 ** -10  # the pooled values are exact sums / copies at these magnitudes
    for n in range(Nb):
        for c in range(F):
            xp, xm = x.copy(), x.copy()
            xp[n, c] += eps
            xm[n, c] -= eps
            fd = (loss(xp) - loss(xm)) / (2 * eps)
            assert fd == pytest.approx(dx[n, c], rel=1e-6, abs=1e-9)


def test_pool_backward_mean_sums_to_dy(orc):
    # every graph's mean gradient adds back up to its dy row
    sizes = np.array([5, 2, 7])
    gi = np.repeat(np.arange(3), sizes)
    dy = np.random.default_rng(82).standard_normal((3, 4)).astype(np.float32)
    dx = orc.segment_pool_backward(dy, gi, 3, "mean")
    tot = np.zeros((3, 4))
    np.add.at(tot, gi, dx)
    np.testing.assert_allclose(tot, dy.astype(np.float64), rtol=1e-14)
