"""GPU parity at the largest size the ABI accepts: E' = 2^31 - 2^20 - 1 edges
(the input edges plus one self-loop per node) over N = 65,536 nodes, so that
32-bit positions run up to the limit in the CSR conversion, the
normalisation (COO and graph order) and the sum aggregation. It needs about
160 GB of device memory and is skipped on a device with less free.

The checks scale to that size: the CSR permutation through properties that
fix a stable sort uniquely, checked in slices on the device; sampled
normalised weights bit for bit against the oracle (run on a small graph with
the same degrees at the sampled endpoints); sampled rows of an unweighted
aggregation against the oracle; and the identity A_hat sqrt(deg) = sqrt(deg)
on every row of the weighted aggregation.
"""

import numpy as np
import pytest

from test_parity import assert_scaled, host, same_bits

pytestmark = pytest.mark.gpu

LIMIT = 2**31 - 2**20  # counts must stay below this
N = 65_536
SLICE = 1 << 27


@pytest.fixture(scope="module")
def tfg():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no ROCm device")
    import paper_2101_11552_amd as lib
    lib.load()
    return lib


def slices(n):
    for a in range(0, n, SLICE):
        yield a, min(n, a + SLICE)


def test_maximum_edge_count(tfg, orc):
    import torch
    free, _ = torch.cuda.mem_get_info()
    if free < 200 * 2**30:
        pytest.skip("needs about 160 GB of free device memory")
    Ep = LIMIT - 1
    E = Ep - N
    gen = torch.Generator(device="cuda").manual_seed(2_101_115)
    eid = torch.randint(0, N, (2, E), dtype=torch.int32, device="cuda", generator=gen)
    loops = torch.arange(N, dtype=torch.int32, device="cuda")

    def src_of(lo, hi):  # sources of positions [lo, hi) of the edge list with loops
        return torch.cat([eid[0, lo:min(hi, E)], loops[max(lo, E) - E:max(hi, E) - E]])

    def tgt_of(lo, hi):
        return torch.cat([eid[1, lo:min(hi, E)], loops[max(lo, E) - E:max(hi, E) - E]])

    g = tfg.tfg_graph_create(eid, N, add_self_loops=True)
    info = g.info()
    assert info["E"] == Ep and info["n_rows_split"] == N  # every row is long
    P = info["src_parts"]
    R = -(-N // P)

    # CSR by (target, source part): row lengths, a permutation, keys in order,
    # input order among equal keys, sources along -> the stable sort, unique
    rowptr, col, perm = tfg.tfg_graph_csr(g)
    cnt = torch.zeros(N, dtype=torch.long, device="cuda")
    segcnt = torch.zeros(N * P, dtype=torch.long, device="cuda")
    for a, b in slices(Ep):
        t, s = tgt_of(a, b).long(), src_of(a, b).long()
        cnt += torch.bincount(t, minlength=N)
        segcnt += torch.bincount(t * P + s // R, minlength=N * P)
    assert rowptr[0].item() == 0 and torch.equal(rowptr[1:].long() - rowptr[:-1].long(), cnt)
    if P > 1:
        seg = tfg.tfg_graph_segments(g).long()
        assert torch.equal(seg[1:] - seg[:-1], segcnt)
    assert int(perm.min()) == 0 and int(perm.max()) == Ep - 1
    seen = torch.zeros(Ep, dtype=torch.bool, device="cuda")
    prev_key = prev_e = None
    for a, b in slices(Ep):
        pl = perm[a:b].long()
        seen[pl] = True
        is_loop = pl >= E
        pe = torch.where(is_loop, 0, pl)
        t = torch.where(is_loop, pl - E, eid[1][pe].long())
        s = torch.where(is_loop, pl - E, eid[0][pe].long())
        key = t * P + s // R
        assert torch.equal(col[a:b].long(), s)
        if prev_key is not None:
            key = torch.cat([prev_key, key])
            pl = torch.cat([prev_e, pl])
        assert bool((key[1:] >= key[:-1]).all())
        same = key[1:] == key[:-1]
        assert bool((pl[1:][same] > pl[:-1][same]).all())
        prev_key, prev_e = key[-1:], pl[-1:]
    assert bool(seen.all())  # Ep positions cover Ep distinct ids: a permutation
    del seen, pl, pe, t, s, key, same, segcnt

    # normalisation: the edge list with loops, degrees, both weight orders
    norm = tfg.tfg_gcn_norm(eid, N, graph=g)
    for a, b in slices(Ep):
        assert torch.equal(norm["edge_index"][0, a:b], src_of(a, b))
        assert torch.equal(norm["edge_index"][1, a:b], tgt_of(a, b))
    assert torch.equal(norm["deg"].double(), cnt.double())  # cnt counts the loops
    w_coo, w_csr = norm["edge_weight"], norm["edge_weight_csr"]
    for a, b in slices(Ep):
        assert torch.equal(w_csr[a:b].view(torch.int32),
                           w_coo[perm[a:b].long()].view(torch.int32))

    # sampled weights against the oracle: a small graph whose nodes have the
    # sampled endpoints' degrees (extra edges from one spare node) gives the
    # oracle the same dinv at both ends of every sampled edge
    rng = np.random.default_rng(5)
    pos = np.concatenate([rng.choice(E, 192, replace=False), E + rng.choice(N, 16, replace=False),
                          [0, E - 1, E, Ep - 1]])
    pos_t = torch.from_numpy(pos).to("cuda")
    ps = torch.where(pos_t < E, eid[0][torch.clamp(pos_t, max=E - 1)].long(), pos_t - E)
    pt = torch.where(pos_t < E, eid[1][torch.clamp(pos_t, max=E - 1)].long(), pos_t - E)
    es, et = host(ps), host(pt)
    in_deg = host(cnt)
    nodes = np.unique(np.concatenate([es, et]))
    local = {int(v): i for i, v in enumerate(nodes)}
    spare = len(nodes)
    ls = np.array([local[int(v)] for v in es])
    lt = np.array([local[int(v)] for v in et])
    sampled_in = np.bincount(lt, minlength=spare)
    # the oracle appends one loop per node, so node v needs in_deg[v] - 1 edges
    fill = np.array([in_deg[v] - 1 for v in nodes]) - sampled_in
    assert (fill >= 0).all()
    extra_t = np.repeat(np.arange(spare), fill)
    small = np.stack([np.concatenate([ls, np.full(extra_t.size, spare)]),
                      np.concatenate([lt, extra_t])]).astype(np.int64)
    _, ow_small, odeg_small = orc.gcn_norm(small, spare + 1)
    assert np.array_equal(odeg_small[:spare], in_deg[nodes].astype(np.float32))
    assert same_bits(host(w_coo[pos_t]), ow_small[:pos.size])

    # unweighted sum aggregation, sampled rows against the oracle
    x = torch.randn(N, 4, generator=gen, device="cuda")
    y = tfg.tfg_aggregate(None, x, N, "sum", graph=g)  # unit weights on all E' edges
    rows = np.unique(np.concatenate([rng.choice(N, 12, replace=False), [0, N - 1]]))
    rows_t = torch.from_numpy(rows.astype(np.int32)).to("cuda")
    picks = [torch.nonzero(torch.isin(eid[1, a:b], rows_t)).flatten() + a
             for a, b in slices(E)]
    ids = torch.cat(picks)
    sub = np.stack([host(eid[0][ids]), host(eid[1][ids])]).astype(np.int64)
    sub = np.concatenate([sub, np.stack([rows, rows])], axis=1)  # their self-loops
    ref, S = orc.aggregate(sub, host(x), N, "sum", rows=rows)
    assert_scaled(host(y)[rows], ref, S, what="largest graph, sampled rows")

    # weighted aggregation in graph order: A_hat sqrt(deg) = sqrt(deg), every row
    sq = torch.sqrt(norm["deg"]).reshape(N, 1).repeat(1, 4).contiguous()
    ys = tfg.tfg_aggregate(None, sq, N, "sum", edge_weight=w_csr, weight_order="csr", graph=g)
    assert float(((ys - sq).abs() / sq).max()) <= 1e-5
    del g, norm, eid, perm, col, w_coo, w_csr
    torch.cuda.empty_cache()
