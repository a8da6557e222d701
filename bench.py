"""Benchmark of the GCN sum-aggregation hot path on one MI355X.

Workload: the large power-law graph (Chung-Lu, gamma = 2): N = 232,965 nodes,
E = 114.6M directed edges plus N self-loops, x ~ N(0, 1) of shape [N, 128],
float32, all seeded and synthetic. One step is the whole path on that graph:
COO -> CSR by target (validation, histogram, stable radix sort, work list),
GCN normalisation D^-1/2 (A + I) D^-1/2 (COO and CSR order outputs), and the
sum aggregation out = A_hat x. Inputs are resident in HBM before timing.

Prints one JSON line: throughput in aggregated edges per second (E' / step
time), the roofline of the aggregation call (algorithmic bytes / its average
duration from HIP events on the launch stream), and the oracle's throughput
on a bounded sample of the same workload on the host.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E
METRIC = "aggregated edges/sec (GE/s) and achieved HBM GB/s for fp32 GCN sum-aggregation"
AGG_SRC = [os.path.join(ROOT, "paper_2101_11552_amd", "csrc", f) for f in ("spmm.h", "aggregate.hip")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_aggregate_powerlaw.txt")


def algorithmic_bytes(E_total: int, N: int, F: int) -> int:
    """Per launch: per edge one column index, one weight and one gathered
    feature row; per target one output row and one row pointer."""
    return E_total * (8 + 4 * F) + N * 4 * F + 4 * (N + 1)


def compulsory_bytes(E_total: int, N: int, N_src: int, F: int, n_items: int) -> int:
    """Bytes one aggregation launch must move to or from memory at least: the
    column index and weight of every edge, x once, the output, the row or
    segment pointers and the work items (16 bytes each). Gathered rows that
    the caches serve again are not counted, nor the part plan's partial rows
    (reported apart)."""
    return E_total * 8 + N_src * 4 * F + N * 4 * F + 4 * (N + 1) + 16 * n_items


def part_plan_items(segptr: np.ndarray, N: int, P: int, chunk: int) -> np.ndarray:
    """(kbeg, kend) of the part plan's work items in dispatch order: part by
    part, row by row, each (row, part) segment cut into chunks of `chunk`."""
    seg = segptr.astype(np.int64)
    start = seg[:-1].reshape(N, P).T.reshape(-1)  # part-major
    end = seg[1:].reshape(N, P).T.reshape(-1)
    length = end - start
    nch = (length + chunk - 1) // chunk
    first = np.repeat(start, nch)
    idx = np.arange(first.size) - np.repeat(np.cumsum(nch) - nch, nch)
    kb = first + idx * chunk
    ke = np.minimum(kb + chunk, np.repeat(end, nch))
    return np.stack([kb, ke], axis=1).astype(np.int32)


def probe_lib():
    import ctypes
    path = os.path.join(ROOT, "paper_2101_11552_amd", "libtfg_probe.so")
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(path)
    p, i64 = ctypes.c_void_p, ctypes.c_int64
    lib.tfg_probe_gather_window.argtypes = [p, i64, i64, i64, i64, p, p]
    lib.tfg_probe_gather_items.argtypes = [p, p, p, i64, p, p]
    lib.tfg_probe_stream.argtypes = [p, ctypes.c_int, p, ctypes.c_int, i64, p]
    return lib


# read / write mixes of the streaming kernels, in 4-byte words per element
STREAM_MIXES = (("read 2", 2, 0, "first counting pass (both id rows)"),
                ("read 1 + write 1", 1, 1, "a plain copy"),
                ("read 2 + write 1", 2, 1, "graph-order weights (ids, key -> weight)"),
                ("read 2 + write 2", 2, 2, "radix scatter passes over two-word payloads"),
                ("read 2 + write 3", 2, 3, "last radix pass; COO-order weights with the edge list"),
                ("read 8 + write 1", 8, 1, "fix-up of the partial rows (8 parts)"))


def stream_ceiling(torch, n_edges: int, n_rows_words: int, device, reps: int = 5):
    """Rates (GB/s of bytes read + written) of plain streams with the read /
    write mixes of the CSR build, the normalisation and the fix-up, over as
    many elements as those kernels move on the workload (E' per plane; the
    fix-up mix over the output's N * F words). Best of `reps` launches."""
    import ctypes
    lib = probe_lib()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    out = {}
    for name, r, w, what in STREAM_MIXES:
        n = n_rows_words if r == 8 else n_edges
        n = -(-n // 4) * 4
        src = torch.ones(r * n, dtype=torch.float32, device=device)
        dst = torch.empty(max(w, 1) * n, dtype=torch.float32, device=device)
        ts = []
        for _ in range(reps + 1):
            a0 = torch.cuda.Event(enable_timing=True)
            a1 = torch.cuda.Event(enable_timing=True)
            a0.record()
            rc = lib.tfg_probe_stream(ctypes.c_void_p(src.data_ptr()), r,
                                      ctypes.c_void_p(dst.data_ptr()), w, n, stream)
            a1.record()
            assert rc == 0, rc
            torch.cuda.synchronize()
            ts.append(a0.elapsed_time(a1))
        ms = min(ts[1:])
        out[name] = {"ms": round(ms, 4), "GBps": round((r + w) * n * 4 / (ms * 1e-3) / 1e9, 1),
                     "words": n, "like": what}
        del src, dst
    torch.cuda.empty_cache()
    return out


def gather_ceiling(torch, x, items=None, col=None, reps: int = 5):
    """Rates (GB/s of 512-byte rows) of bare row gathers from x, the
    aggregation's table: E' rows drawn uniformly from a window that moves
    every E'/P gathers, for windows from the whole table down to 256 rows;
    with (items, col), also the part plan's own row stream. Each figure is
    the best of `reps` timed launches (HIP events on the launch stream)."""
    import ctypes
    lib = probe_lib()
    N, F = x.shape
    assert F == 128
    n = int(items.shape[0]) if items is not None else 0
    n_gathers = int(col.shape[0]) if col is not None else 114_832_965
    sink = torch.empty(max((n_gathers + 127) // 128, n, 1), dtype=torch.float32, device=x.device)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    out = {}

    def best(fn):
        ts = []
        for _ in range(reps + 1):
            a0 = torch.cuda.Event(enable_timing=True)
            a1 = torch.cuda.Event(enable_timing=True)
            a0.record()
            rc = fn()
            a1.record()
            assert rc == 0, rc
            torch.cuda.synchronize()
            ts.append(a0.elapsed_time(a1))
        return min(ts[1:])

    for name, wr in (("table", N), ("table/8", -(-N // 8)), ("table/16", -(-N // 16)),
                     ("table/32", -(-N // 32)), ("table/64", -(-N // 64)),
                     ("table/128", -(-N // 128)), ("1024 rows", 1024), ("256 rows", 256)):
        windows = -(-N // wr)
        per = -(-n_gathers // windows)
        per = -(-per // 128) * 128
        ms = best(lambda: lib.tfg_probe_gather_window(ctypes.c_void_p(x.data_ptr()), N, wr,
                                                      n_gathers, per,
                                                      ctypes.c_void_p(sink.data_ptr()), stream))
        out[name] = {"ms": round(ms, 4), "GBps": round(n_gathers * 4 * F / (ms * 1e-3) / 1e9, 1),
                     "window_rows": wr}
    if items is not None:
        it = torch.from_numpy(items).to(x.device)
        ms = best(lambda: lib.tfg_probe_gather_items(ctypes.c_void_p(x.data_ptr()),
                                                     ctypes.c_void_p(col.data_ptr()),
                                                     ctypes.c_void_p(it.data_ptr()), n,
                                                     ctypes.c_void_p(sink.data_ptr()), stream))
        out["part plan stream"] = {"ms": round(ms, 4),
                                   "GBps": round(n_gathers * 4 * F / (ms * 1e-3) / 1e9, 1),
                                   "items": n}
    return out


def row_chunk() -> int:
    """Edges per work item of the row plan (the library's default unless
    TFG_ROW_CHUNK overrides it)."""
    v = os.environ.get("TFG_ROW_CHUNK")
    return int(v) if v and int(v) >= 64 else 128


def source_sha(paths) -> str:
    h = hashlib.sha256()
    for p in paths:
        h.update(open(p, "rb").read())
    return h.hexdigest()[:16]


def stored_traffic():
    """Bytes per launch that the L2s request from the fabric (Infinity Cache
    and HBM together), from the committed rocprofv3 counter summary, if it was
    taken on the current aggregation source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    vals = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line:
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("kernel_source_sha256_16") != source_sha(AGG_SRC):
        return None
    if vals.get("row_chunk") != str(row_chunk()):
        return None
    try:
        return int(float(vals["hbm_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def load_workload(cache: str | None):
    import graphgen
    if cache and os.path.exists(cache):
        z = np.load(cache)
        return z["edge_index"], z["x"]
    c = graphgen.power_law(dtype=np.int32)
    if cache:
        np.savez(cache, edge_index=c["edge_index"], x=c["x"])
    return c["edge_index"], c["x"]


def cpu_baseline(ei: np.ndarray, x: np.ndarray, n: int, n_edges: int):
    """The oracle (single-threaded C, double accumulation) on the first
    ``n_edges`` edges of the same edge list over all N nodes: GCN
    normalisation then sum aggregation, timed end to end."""
    import oracle
    sub = np.ascontiguousarray(ei[:, :n_edges].astype(np.int64))
    t0 = time.perf_counter()
    oei, ow, _ = oracle.gcn_norm(sub, n)
    oracle.aggregate(oei, x, n, "sum", edge_weight=ow)
    dt = time.perf_counter() - t0
    e_total = n_edges + n
    return {"value": round(e_total / dt / 1e9, 6), "unit": "GE/s", "cores": 1, "kind": "oracle",
            "sample": f"first {n_edges} of the {ei.shape[1]} edges (+{n} self-loops), all "
                      f"{n} nodes, F={x.shape[1]}: gcn_norm + sum aggregation, {dt:.1f} s",
            "cpu_model": cpu_model(), "nproc": os.cpu_count()}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline_threads(ei: np.ndarray, x: np.ndarray, n: int, n_edges: int):
    """The same sample with the aggregation over all host threads (rows split
    by target range, bit-identical to one thread); the normalisation, about
    1% of the work, stays on one thread."""
    import oracle
    threads = oracle.host_threads()
    sub = np.ascontiguousarray(ei[:, :n_edges].astype(np.int64))
    t0 = time.perf_counter()
    oei, ow, _ = oracle.gcn_norm(sub, n)
    oracle.aggregate_by_row_ranges(oei, x, n, "sum", edge_weight=ow, threads=threads)
    dt = time.perf_counter() - t0
    e_total = n_edges + n
    return {"value": round(e_total / dt / 1e9, 6), "unit": "GE/s", "cores": threads,
            "kind": "oracle",
            "sample": f"the single-thread sample, aggregation rows split over {threads} "
                      f"threads, {dt:.1f} s",
            "cpu_model": cpu_model(), "nproc": os.cpu_count()}


def _replayed(torch, fn, reps: int) -> float:
    """Average ms per replay of fn() captured as one HIP graph (two warm-up
    runs on a side stream, then the capture), replays timed back to back by
    events on the current stream."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    gr = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gr):
        fn()
    ms = _timed(torch, gr.replay, reps)
    del gr
    return ms


def _timed(torch, fn, reps: int, warm: int = 2) -> float:
    """Average ms of fn() over reps back-to-back calls, by events on the
    current stream (the stream the library launches on)."""
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    a0 = torch.cuda.Event(enable_timing=True)
    a1 = torch.cuda.Event(enable_timing=True)
    a0.record()
    for _ in range(reps):
        fn()
    a1.record()
    torch.cuda.synchronize()
    return a0.elapsed_time(a1) / reps


def _oracle(fn, units: int, unit: str, sample: str):
    """The oracle on the host (one thread), timed on a bounded sample: the rate
    in `unit` (units per second, scaled like the GPU figure)."""
    t0 = time.perf_counter()
    fn()
    dt = time.perf_counter() - t0
    scale = 1e9 if unit == "GE/s" else 1.0
    return {"value": round(units / dt / scale, 6), "unit": unit, "cores": 1, "kind": "oracle",
            "sample": f"{sample}, {dt:.2f} s"}


def _oracle_threads(fn, units: int, unit: str, sample: str):
    """As _oracle, for a callable that splits the oracle's work over
    oracle.host_threads() threads by target range (each range's results are
    bit-identical to one thread's)."""
    import oracle
    threads = oracle.host_threads()
    t0 = time.perf_counter()
    fn(threads)
    dt = time.perf_counter() - t0
    scale = 1e9 if unit == "GE/s" else 1.0
    return {"value": round(units / dt / scale, 6), "unit": unit, "cores": threads,
            "kind": "oracle", "sample": f"{sample}, split over {threads} threads by target "
                                        f"range, {dt:.2f} s"}


def _by_target_range(fn, edge_index, n, threads):
    """Runs fn(sub_edge_index) for the edges of each target range [n*i/T,
    n*(i+1)/T) in parallel threads (input order kept inside a range)."""
    from concurrent.futures import ThreadPoolExecutor
    tgt = edge_index[1]
    bounds = [n * i // threads for i in range(threads + 1)]

    def part(i):
        m = (tgt >= bounds[i]) & (tgt < bounds[i + 1])
        return fn(np.ascontiguousarray(edge_index[:, m]))

    with ThreadPoolExecutor(threads) as pool:
        return list(pool.map(part, range(threads)))


def _row(name: str, workload: str, ms: float, edges: int | None, nbytes: int | None,
         compulsory: int | None = None, gathered: int | None = None,
         ceiling: tuple | None = None, **extra):
    """One suite line. nbytes: the algorithmic bytes of the row (one gathered
    row per edge where the kernel gathers). For gathering kernels whose rows
    the caches serve, `compulsory` (bytes that must cross HBM) is set against
    8 TB/s and `gathered` (the row bytes) against the measured gather ceiling
    (name, GB/s)."""
    line = {"row": name, "workload": workload, "ms": round(ms, 4)}
    if edges is not None:
        line["GE_per_s"] = round(edges / (ms * 1e-3) / 1e9, 3)
    if nbytes is not None:
        t = ms * 1e-3
        hbm = compulsory if compulsory is not None else nbytes
        gbs = hbm / t / 1e9
        roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                "frac": round(gbs / PEAK_HBM_GBPS, 4), "algorithmic_bytes_per_launch": int(nbytes),
                "algorithmic_GBps": round(nbytes / t / 1e9, 1)}
        if compulsory is not None:
            roof["compulsory_bytes_per_launch"] = int(compulsory)
        if gathered is not None and ceiling is not None:
            rate = gathered / t / 1e9
            roof["gather"] = {"bytes_per_launch": int(gathered), "achieved": round(rate, 1),
                              "ceiling": ceiling[1], "ceiling_from": ceiling[0],
                              "frac": round(rate / ceiling[1], 4), "unit": "GB/s"}
        line["roofline"] = roof
    line.update(extra)
    print(json.dumps(line), flush=True)


def run_suite(args):
    """One JSON line per measured row of the path besides the headline step:
    the backward aggregation, multi-step propagation, attention (fused and
    unfused), segment softmax, BatchGraph construction and pooling, and the
    GCN step on the two small graphs. Each figure is the average of
    back-to-back calls on resident inputs."""
    import torch
    import graphgen
    import paper_2101_11552_amd as tfg

    tfg.load()
    dev = torch.device("cuda:0")
    reps = max(args.steps, 5)

    # --- the large power-law graph: backward aggregation and propagation
    ei_np, x_np = load_workload(args.cache)
    N, F = x_np.shape
    E = ei_np.shape[1]
    Ep = E + N
    ei = torch.from_numpy(ei_np).to(dev)
    x = torch.from_numpy(x_np).to(dev)
    g = tfg.tfg_graph_create(ei, N, add_self_loops=True)
    gt = tfg.tfg_graph_create_transposed(ei, N, add_self_loops=True)
    norm = tfg.tfg_gcn_norm(ei, N, graph=g)
    dy = torch.randn((N, F), generator=torch.Generator(device=dev).manual_seed(7), device=dev)
    wl = f"Chung-Lu power-law graph N={N}, E'={Ep} (with self-loops), F={F}"
    ws = torch.empty(max(tfg.load().tfg_aggregate_backward_ws_bytes(
        g.handle, gt.handle, F, 1, 0, 0, 1), 256), dtype=torch.uint8, device=dev)
    # the normalised weights in the transposed graph's order, cached once per graph
    w_t = tfg.tfg_edge_reorder(norm["edge_weight_csr"], src=g, dst=gt)
    # the gather ceiling on this table (the rows gathered by dx, dw and APPNP)
    ceil = gather_ceiling(torch, x, reps=5)
    ceiling = max(((k, v["GBps"]) for k, v in ceil.items()), key=lambda kv: kv[1])
    info_f, info_t = g.info(), gt.info()

    def items(inf):
        return inf["n_part_items"] if inf["src_parts"] > 1 else inf["n_chunks"] + N

    ms = _timed(torch, lambda: tfg.tfg_aggregate_backward(
        g, dy, "sum", graph_t=gt, edge_weight=w_t, weight_order="csr_t", want_dx=True, ws=ws),
        reps)
    ms_coo = _timed(torch, lambda: tfg.tfg_aggregate_backward(
        g, dy, "sum", graph_t=gt, edge_weight=norm["edge_weight"], weight_order="coo",
        want_dx=True, ws=ws), reps)
    import oracle
    cpu = {}
    if not args.no_cpu_baseline:
        m = 4_000_000
        sub = np.ascontiguousarray(ei_np[:, :m].astype(np.int64))
        w_sub = np.random.default_rng(7).uniform(0.1, 1.0, m).astype(np.float32)
        dy_h = dy.cpu().numpy()
        cpu["bw"] = _oracle(lambda: oracle.aggregate_backward(sub, x_np, N, dy_h, "sum",
                                                              edge_weight=w_sub),
                            m, "GE/s", f"first {m} edges, all {N} nodes, F={F}: dx and dw together")
        cpu["appnp"] = _oracle(lambda: oracle.propagate(sub, x_np, 3, alpha=0.1, h=x_np,
                                                        edge_weight=w_sub),
                               3 * m, "GE/s", f"first {m} edges, all {N} nodes, F={F}, K=3")
        del sub, dy_h
    # per edge: target id, the weight and a dy row; per source: a dx row
    _row("backward dx (transposed sum aggregation)", wl, ms, Ep,
         Ep * (8 + 4 * F) + N * 4 * F + 4 * (N + 1),
         compulsory=compulsory_bytes(Ep, N, N, F, items(info_t)), gathered=Ep * 4 * F,
         ceiling=ceiling, kernel="spmm_wide over the transposed graph",
         src_parts=gt.info()["src_parts"], weights="transposed graph order",
         ms_with_edge_order_weights=round(ms_coo, 4), cpu_baseline=cpu.get("bw"))
    ms = _timed(torch, lambda: tfg.tfg_aggregate_backward(
        g, dy, "sum", x=x, want_dx=False, want_dw=True, dw_order="csr", ws=ws), reps)
    # per edge: source id, an x row, the dw value; per target: a dy row
    _row("backward dw (per-edge dot products)", wl, ms, Ep,
         Ep * (8 + 4 * F) + N * 4 * F + 4 * (N + 1),
         compulsory=Ep * 8 + 2 * N * 4 * F + 4 * (N + 1) + 16 * items(info_f),
         gathered=Ep * 4 * F, ceiling=ceiling, kernel="edge_grad_rows",
         cpu_baseline=cpu.get("bw"))
    K = 3
    ms = _timed(torch, lambda: tfg.tfg_propagate(g, x, K, alpha=0.1, h=x,
                                                edge_weight=norm["edge_weight_csr"]), reps)
    _row(f"APPNP propagation, K={K}, alpha=0.1", wl, ms, K * Ep,
         K * (Ep * (8 + 4 * F) + N * 8 * F + 4 * (N + 1)),
         compulsory=K * (compulsory_bytes(Ep, N, N, F, items(info_f)) + N * 4 * F),
         gathered=K * Ep * 4 * F, ceiling=ceiling, ms_per_step=round(ms / K, 4),
         cpu_baseline=cpu.get("appnp"))
    del g, gt, norm, dy, ws, ei, x
    torch.cuda.empty_cache()

    # --- attention on the preferential-attachment graph
    c = graphgen.attention_graph()
    n3, H, D = c["N"], c["H"], c["D"]
    Fh = H * D
    ei3 = torch.from_numpy(c["edge_index"].astype(np.int32)).to(dev)
    E3 = ei3.shape[1]
    h = torch.from_numpy(c["h"]).to(dev)
    a_s, a_d = torch.from_numpy(c["a_src"]).to(dev), torch.from_numpy(c["a_dst"]).to(dev)
    g3 = tfg.tfg_graph_create(ei3, n3)
    wl3 = f"Barabasi-Albert graph (m=7) N={n3}, E={E3}, H={H} heads x {D} dims"
    ms_f = _timed(torch, lambda: tfg.tfg_gat_aggregate(g3, h, a_s, a_d, c["slope"]), reps)

    def chain():
        s = tfg.tfg_gat_edge_scores(ei3, h, a_s, a_d, c["slope"])
        _, a_csr = tfg.tfg_segment_softmax(s, ei3[1], n3, graph=g3, out_csr=True)
        return tfg.tfg_aggregate(ei3, h, n3, "sum", edge_weight=a_csr, heads=H,
                                 weight_order="csr", graph=g3)
    ms_c = _timed(torch, chain, reps)
    # the same chain with scores, alpha and weights kept in the graph order
    sg_out = torch.empty((E3, H), dtype=torch.float32, device=dev)
    ag_out = torch.empty_like(sg_out)
    sg_ws = torch.empty(max(tfg.load().tfg_gat_graph_scores_ws_bytes(g3.handle, H), 256),
                        dtype=torch.uint8, device=dev)
    ag_ws = torch.empty(max(tfg.load().tfg_segment_softmax_graph_ws_bytes(g3.handle, H), 256),
                        dtype=torch.uint8, device=dev)

    def chain_graph_order():
        s = tfg.tfg_gat_graph_scores(g3, h, a_s, a_d, c["slope"], order="csr", out=sg_out, ws=sg_ws)
        a = tfg.tfg_segment_softmax_graph(g3, s, order="csr", out=ag_out, ws=ag_ws)
        return tfg.tfg_aggregate(None, h, n3, "sum", edge_weight=a, heads=H, weight_order="csr",
                                 graph=g3)
    ms_cg = _timed(torch, chain_graph_order, reps)
    ms_cg_replay = _replayed(torch, chain_graph_order, reps)
    ei3_np = c["edge_index"]
    if not args.no_cpu_baseline:
        cpu["gat"] = _oracle(lambda: oracle.gat_layer(ei3_np, c["h"], c["a_src"], c["a_dst"], H,
                                                      slope=np.float32(c["slope"])),
                             E3, "GE/s", "the whole attention graph")
        cpu["gat_t"] = _oracle_threads(
            lambda T: _by_target_range(lambda sub: oracle.gat_layer(
                sub, c["h"], c["a_src"], c["a_dst"], H, slope=np.float32(c["slope"])),
                ei3_np, n3, T), E3, "GE/s", "the whole attention graph")
    _row("fused attention aggregation", wl3, ms_f, E3,
         E3 * (4 + 4 * H + 4 * Fh) + n3 * (4 * Fh + 8 * H) + n3 * (4 * H + 4 * Fh + 4),
         kernel="node_projections_vec + gat_short + gat_items + gat_merge",
         unfused_chain_ms=round(ms_c, 4), speedup_vs_unfused=round(ms_c / ms_f, 3),
         unfused_chain_graph_order_ms=round(ms_cg, 4),
         unfused_chain_graph_order_hip_graph_ms=round(ms_cg_replay, 4),
         cpu_baseline=cpu.get("gat"), cpu_baseline_threads=cpu.get("gat_t"))
    # the Transformer-style variant: q, key, v of the same shape as h
    gen = torch.Generator(device=dev).manual_seed(3)
    qd, kd, vd = (torch.randn((n3, Fh), generator=gen, device=dev) for _ in range(3))
    ms_f = _timed(torch, lambda: tfg.tfg_gat_dot_aggregate(g3, qd, kd, vd, H), reps)

    def dot_chain():
        s = tfg.tfg_edge_dot_scores(g3, qd, kd, H)
        _, a_csr = tfg.tfg_segment_softmax(s, ei3[1], n3, graph=g3, out_csr=True)
        return tfg.tfg_aggregate(ei3, vd, n3, "sum", edge_weight=a_csr, heads=H,
                                 weight_order="csr", graph=g3)
    ms_c = _timed(torch, dot_chain, reps)

    def dot_chain_graph_order():
        s = tfg.tfg_edge_dot_scores(g3, qd, kd, H, order="csr", out=sg_out)
        a = tfg.tfg_segment_softmax_graph(g3, s, order="csr", out=ag_out, ws=ag_ws)
        return tfg.tfg_aggregate(None, vd, n3, "sum", edge_weight=a, heads=H, weight_order="csr",
                                 graph=g3)
    ms_cg = _timed(torch, dot_chain_graph_order, reps)
    if not args.no_cpu_baseline:
        qh, kh, vh = (t.cpu().numpy() for t in (qd, kd, vd))
        cpu["dot"] = _oracle(lambda: oracle.dot_layer(ei3_np, qh, kh, vh, H, 1.0 / np.sqrt(c["D"])),
                             E3, "GE/s", "the whole attention graph")
        del qh, kh, vh
    # per edge: source id, the key and value rows; per node: q row, output row
    _row("fused Transformer-style attention (scaled dot product)", wl3, ms_f, E3,
         E3 * (4 + 8 * Fh) + n3 * (8 * Fh + 4), kernel="gat_short + gat_items (dot) + gat_merge",
         unfused_chain_ms=round(ms_c, 4), speedup_vs_unfused=round(ms_c / ms_f, 3),
         unfused_chain_graph_order_ms=round(ms_cg, 4),
         cpu_baseline=cpu.get("dot"))
    del qd, kd, vd
    s = tfg.tfg_gat_edge_scores(ei3, h, a_s, a_d, c["slope"])
    ms = _timed(torch, lambda: tfg.tfg_segment_softmax(s, ei3[1], n3, graph=g3), reps)
    # per edge: edge id, the scores (read twice by the kernel, counted once), alpha
    if not args.no_cpu_baseline:
        s_h = s.cpu().numpy()
        cpu["sm"] = _oracle(lambda: oracle.segment_softmax(s_h, ei3_np[1], n3), E3, "GE/s",
                            "the whole attention graph")
    _row("segment softmax", wl3, ms, E3, E3 * (4 + 8 * H) + 4 * (n3 + 1),
         kernel="softmax_items + softmax_split",
         cpu_baseline=cpu.get("sm"))
    # scores and alpha in the graph order: no permutation, one run per row
    s_g = tfg.tfg_gat_graph_scores(g3, h, a_s, a_d, c["slope"], order="csr")
    ms = _timed(torch, lambda: tfg.tfg_segment_softmax_graph(g3, s_g, order="csr", out=ag_out,
                                                             ws=ag_ws), reps)
    _row("segment softmax, scores and alpha in graph order", wl3, ms, E3,
         E3 * 8 * H + 4 * (n3 + 1), kernel="softmax_items + softmax_split (no permutation)",
         cpu_baseline=cpu.get("sm"))
    alpha = tfg.tfg_segment_softmax(s, ei3[1], n3, graph=g3)
    dal = torch.randn_like(alpha)
    if not args.no_cpu_baseline:
        a_h, d_h = alpha.cpu().numpy(), dal.cpu().numpy()
        cpu["smb"] = _oracle(lambda: oracle.segment_softmax_backward(a_h, d_h, ei3_np[1], n3), E3,
                             "GE/s", "the whole attention graph")
    ms = _timed(torch, lambda: tfg.tfg_segment_softmax_backward(alpha, dal, ei3[1], n3, graph=g3),
                reps)
    _row("segment softmax backward", wl3, ms, E3, E3 * (4 + 12 * H) + 4 * (n3 + 1),
         kernel="softmax_grad_items + softmax_grad_split",
         cpu_baseline=cpu.get("smb"))
    a_g = tfg.tfg_segment_softmax_graph(g3, s_g, order="csr")
    dal_g = torch.randn_like(a_g)
    ms = _timed(torch, lambda: tfg.tfg_segment_softmax_graph_backward(g3, a_g, dal_g, order="csr"),
                reps)
    _row("segment softmax backward, in graph order", wl3, ms, E3, E3 * 12 * H + 4 * (n3 + 1),
         kernel="softmax_grad_items + softmax_grad_split (no permutation)",
         cpu_baseline=cpu.get("smb"))
    del g3, ei3, h, s, alpha, dal, s_g, a_g, dal_g, sg_out, ag_out
    torch.cuda.empty_cache()

    # --- mini-batch of small graphs: BatchGraph, 3 GCN layers, pooling
    c = graphgen.graph_batch()
    sizes, graphs = c["sizes"], c["graphs"]
    G, Fb = c["G"], c["F"]
    nc = torch.from_numpy(sizes.astype(np.int32)).to(dev)
    ec = torch.from_numpy(np.array([gr.shape[1] for gr in graphs], np.int32)).to(dev)
    local = torch.from_numpy(np.concatenate(graphs, axis=1).astype(np.int32)).to(dev)
    Nb = int(sizes.sum())
    Eb = local.shape[1]
    xb = torch.from_numpy(c["x"]).to(dev)
    wl5 = f"{G} graphs, {Nb} nodes, {Eb} edges (+ self-loops), F={Fb}"
    bout = tfg.tfg_batch_graphs(nc, ec, local, Nb, validate=False)
    bws = torch.empty(max(tfg.load().tfg_batch_graphs_ws_bytes(G), 256), dtype=torch.uint8,
                      device=dev)
    ms = _timed(torch, lambda: tfg.tfg_batch_graphs(nc, ec, local, Nb, validate=False, out=bout,
                                                    ws=bws), reps)
    if not args.no_cpu_baseline:
        cpu["batch"] = _oracle(lambda: oracle.batch_graphs(sizes, graphs), Eb, "GE/s",
                               "the whole batch")

        def oracle_step():
            oei, ow, _ = oracle.gcn_norm(c["edge_index"], Nb)
            hb = c["x"]
            for _ in range(c["layers"]):
                hb = oracle.aggregate(oei, hb, Nb, "sum", edge_weight=ow)[0].astype(np.float32)
            return [oracle.segment_pool(hb, c["graph_index"], G, r) for r in ("sum", "mean", "max")]
        cpu["mb"] = _oracle(oracle_step, 3 * (Eb + Nb), "GE/s",
                            "the whole batch (normalisation, 3 layers, 3 pools)")

        def oracle_step_threads(T):
            oei, ow, _ = oracle.gcn_norm(c["edge_index"], Nb)
            hb = c["x"]
            for _ in range(c["layers"]):
                hb = oracle.aggregate_by_row_ranges(oei, hb, Nb, "sum", edge_weight=ow,
                                                    threads=T)[0].astype(np.float32)
            return [oracle.segment_pool(hb, c["graph_index"], G, r) for r in ("sum", "mean", "max")]
        cpu["mb_t"] = _oracle_threads(oracle_step_threads, 3 * (Eb + Nb), "GE/s",
                                      "the whole batch (normalisation and pools on one thread, "
                                      "the 3 layers)")
        cpu["pool"] = _oracle(lambda: oracle.segment_pool(c["x"], c["graph_index"], G, "sum"),
                              Nb, "nodes/s", "the whole batch")
    _row("BatchGraph construction", wl5, ms, Eb,
         Eb * 16 + G * 8 + Nb * 4, kernel="batch_offsets_small + batch_fill",
         cpu_baseline=cpu.get("batch"))

    def batch_step():
        bei, bgi, _, _ = tfg.tfg_batch_graphs(nc, ec, local, Nb, validate=False)
        gb = tfg.tfg_graph_create(bei, Nb, add_self_loops=True)
        nb = tfg.tfg_gcn_norm(bei, Nb, graph=gb, out_edge_index=False, out_edge_weight=False,
                              out_deg=False)
        hb = xb
        for _ in range(c["layers"]):
            hb = tfg.tfg_aggregate(None, hb, Nb, "sum", edge_weight=nb["edge_weight_csr"],
                                   weight_order="csr", graph=gb)
        return [tfg.tfg_segment_pool(hb, bgi, G, r, validate=False) for r in ("sum", "mean", "max")]
    ms = _timed(torch, batch_step, reps)
    _row("mini-batch step: BatchGraph + CSR + gcn_norm + 3 GCN layers + 3 pools", wl5, ms,
         3 * (Eb + Nb), None, cpu_baseline=cpu.get("mb"), cpu_baseline_threads=cpu.get("mb_t"))
    gi = torch.from_numpy(c["graph_index"].astype(np.int32)).to(dev)
    # the forward on a cached BatchGraph (normalisation, 3 layers, 3 pools):
    # eager calls, then the same calls replayed as one HIP graph
    bei_c, bgi_c, _, _ = tfg.tfg_batch_graphs(nc, ec, local, Nb, validate=False)
    gb_c = tfg.tfg_graph_create(bei_c, Nb, add_self_loops=True)

    def cached_forward():
        nb = tfg.tfg_gcn_norm(bei_c, Nb, graph=gb_c, out_edge_index=False,
                              out_edge_weight=False, out_deg=False)
        hb = xb
        for _ in range(c["layers"]):
            hb = tfg.tfg_aggregate(None, hb, Nb, "sum", edge_weight=nb["edge_weight_csr"],
                                   weight_order="csr", graph=gb_c)
        return [tfg.tfg_segment_pool(hb, bgi_c, G, r, validate=False)
                for r in ("sum", "mean", "max")]
    ms_e = _timed(torch, cached_forward, reps)
    ms_r = _replayed(torch, cached_forward, reps)
    _row("mini-batch forward on a cached BatchGraph (gcn_norm + 3 GCN layers + 3 pools), "
         "HIP graph replay", wl5, ms_r, 3 * (Eb + Nb), None, eager_ms=round(ms_e, 4),
         speedup_vs_eager=round(ms_e / ms_r, 3))
    del gb_c, bei_c, bgi_c
    pout = torch.empty((G, Fb), dtype=torch.float32, device=dev)
    pws = torch.empty(max(tfg.load().tfg_segment_pool_ws_bytes(Nb, G), 256), dtype=torch.uint8,
                      device=dev)
    ms = _timed(torch, lambda: tfg.tfg_segment_pool(xb, gi, G, "sum", validate=False, out=pout,
                                                    ws=pws), reps)
    _row("segment pool (sum)", wl5, ms, None, Nb * 4 * Fb + Nb * 4 + G * 4 * Fb,
         kernel="segment_bounds + pool_rows", nodes_per_s=round(Nb / (ms * 1e-3), 1),
         cpu_baseline=cpu.get("pool"))

    # --- the GCN step on the two small uniform graphs
    for cfg in (graphgen.uniform_small(), graphgen.uniform_medium()):
        n, Fc = cfg["N"], cfg["F"]
        eic = torch.from_numpy(cfg["edge_index"].astype(np.int32)).to(dev)
        xc = torch.from_numpy(cfg["x"]).to(dev)
        Ec = eic.shape[1] + n

        def gcn_step():
            gc = tfg.tfg_graph_create(eic, n, add_self_loops=True)
            nm = tfg.tfg_gcn_norm(eic, n, graph=gc)
            return tfg.tfg_aggregate(None, xc, n, "sum", edge_weight=nm["edge_weight_csr"],
                                     weight_order="csr", graph=gc)
        ms = _timed(torch, gcn_step, reps)
        cb = cbt = None
        if not args.no_cpu_baseline:
            def oracle_gcn():
                oei, ow, _ = oracle.gcn_norm(cfg["edge_index"], n)
                return oracle.aggregate(oei, cfg["x"], n, "sum", edge_weight=ow)

            def oracle_gcn_threads(T):
                oei, ow, _ = oracle.gcn_norm(cfg["edge_index"], n)
                return oracle.aggregate_by_row_ranges(oei, cfg["x"], n, "sum", edge_weight=ow,
                                                      threads=T)
            cb = _oracle(oracle_gcn, Ec, "GE/s", "the whole graph")
            cbt = _oracle_threads(oracle_gcn_threads, Ec, "GE/s",
                                  "the whole graph (normalisation on one thread)")
        _row("GCN step: CSR + gcn_norm + sum aggregation", f"uniform graph N={n}, "
             f"E'={Ec}, F={Fc}", ms, Ec, None, cpu_baseline=cb, cpu_baseline_threads=cbt)
        # a GCN layer on the cached graph: eager, then replayed as one HIP graph
        gcc = tfg.tfg_graph_create(eic, n, add_self_loops=True)

        def gcn_layer():
            nm = tfg.tfg_gcn_norm(eic, n, graph=gcc, out_edge_index=False, out_edge_weight=False,
                                  out_deg=False)
            return tfg.tfg_aggregate(None, xc, n, "sum", edge_weight=nm["edge_weight_csr"],
                                     weight_order="csr", graph=gcc)
        ms_e = _timed(torch, gcn_layer, reps)
        ms_r = _replayed(torch, gcn_layer, reps)
        _row("GCN layer on the cached graph (graph-order gcn_norm + sum aggregation), "
             "HIP graph replay", f"uniform graph N={n}, E'={Ec}, F={Fc}", ms_r, Ec, None,
             eager_ms=round(ms_e, 4), speedup_vs_eager=round(ms_e / ms_r, 3))
        del gcc


def run_ceiling(args):
    """The gather probes on the power-law workload's table and graph, with
    more repetitions than the headline run takes: one JSON line."""
    import torch
    import paper_2101_11552_amd as tfg
    tfg.load()
    dev = torch.device("cuda:0")
    ei_np, x_np = load_workload(args.cache)
    N, F = x_np.shape
    ei = torch.from_numpy(ei_np).to(dev)
    x = torch.from_numpy(x_np).to(dev)
    g = tfg.tfg_graph_create(ei, N, add_self_loops=True, src_parts=args.src_parts)
    info = g.info()
    P = info["src_parts"]
    items = col = None
    if P > 1:
        items = part_plan_items(tfg.tfg_graph_segments(g).cpu().numpy(), N, P, row_chunk())
        col = tfg.tfg_graph_csr(g)[1]
    res = gather_ceiling(torch, x, items, col, reps=max(args.steps, 5))
    print(json.dumps({"row": "gather ceiling", "workload": f"power-law table [{N}, {F}] float32, "
                      f"{info['E']} gathers of 512-byte rows", "src_parts": P, "probes": res}),
          flush=True)
    del g, items, col
    torch.cuda.empty_cache()
    st = stream_ceiling(torch, int(info["E"]), N * F, dev, reps=max(args.steps, 5))
    print(json.dumps({"row": "stream ceiling", "workload": f"plain streams over E' = {info['E']} "
                      f"elements per plane (the fix-up mix over N * F = {N * F} words)",
                      "probes": st}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-edges", type=int, default=20_000_000)
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run a plain 1 GiB device copy (counter calibration)")
    ap.add_argument("--cache", default=None, help="npz file to reuse the generated graph")
    ap.add_argument("--src-parts", type=int, default=0,
                    help="source parts of the graph (0: the library's choice)")
    ap.add_argument("--suite", action="store_true",
                    help="instead of the headline line, one line per other measured row")
    ap.add_argument("--ceiling", action="store_true",
                    help="instead of the headline line, the gather-ceiling probes (one line)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: runs on one GPU only; --gpus {args.gpus} is not supported",
              file=sys.stderr)
        sys.exit(2)
    if args.suite:
        run_suite(args)
        return
    if args.ceiling:
        run_ceiling(args)
        return

    import torch
    import paper_2101_11552_amd as tfg

    tfg.load()
    dev = torch.device("cuda:0")
    t_gen = time.perf_counter()
    ei_np, x_np = load_workload(args.cache)
    t_gen = time.perf_counter() - t_gen
    N, F = x_np.shape
    E = ei_np.shape[1]
    E_total = E + N
    print(f"# workload generated in {t_gen:.1f} s: N={N} E={E} F={F}", file=sys.stderr, flush=True)

    ei = torch.from_numpy(ei_np).to(dev)
    x = torch.from_numpy(x_np).to(dev)
    nb, ns = tfg.tfg_graph_bytes(E, N, True, src_parts=args.src_parts)
    buf = torch.empty(nb, dtype=torch.uint8, device=dev)
    scratch = torch.empty(ns, dtype=torch.uint8, device=dev)
    out = torch.empty((N, F), dtype=torch.float32, device=dev)
    torch.cuda.synchronize()

    if args.calib_copy:
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev)  # 1 GiB
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    ev = {k: [] for k in ("create", "norm", "agg")}
    agg_ws = None

    def step(record: bool):
        nonlocal agg_ws
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e2 = torch.cuda.Event(enable_timing=True)
        e3 = torch.cuda.Event(enable_timing=True)
        e0.record()
        g = tfg.tfg_graph_create(ei, N, add_self_loops=True, src_parts=args.src_parts, buf=buf,
                                 scratch=scratch)
        e1.record()
        norm = tfg.tfg_gcn_norm(ei, N, graph=g)
        e2.record()
        if agg_ws is None:
            agg_ws = torch.empty(max(tfg.tfg_aggregate_ws_bytes(E_total, N, F, "sum", g), 256),
                                 dtype=torch.uint8, device=dev)
        tfg.tfg_aggregate(None, x, N, "sum", edge_weight=norm["edge_weight_csr"],
                          weight_order="csr", graph=g, out=out, ws=agg_ws)
        e3.record()
        if record:
            ev["create"].append((e0, e1))
            ev["norm"].append((e1, e2))
            ev["agg"].append((e2, e3))
        return g, norm

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        g, norm = step(True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    avg = {k: sum(a.elapsed_time(b) for a, b in v) / len(v) for k, v in ev.items()}

    # the aggregation alone, back to back (the paper caches the normalised graph)
    info = g.info()
    a0 = torch.cuda.Event(enable_timing=True)
    a1 = torch.cuda.Event(enable_timing=True)
    reps = max(args.steps, 20)
    a0.record()
    for _ in range(reps):
        tfg.tfg_aggregate(None, x, N, "sum", edge_weight=norm["edge_weight_csr"],
                          weight_order="csr", graph=g, out=out, ws=agg_ws)
    a1.record()
    torch.cuda.synchronize()
    agg_ms = a0.elapsed_time(a1) / reps
    # the same launches one by one (events around each): median and minimum
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    marks[0].record()
    for i in range(reps):
        tfg.tfg_aggregate(None, x, N, "sum", edge_weight=norm["edge_weight_csr"],
                          weight_order="csr", graph=g, out=out, ws=agg_ws)
        marks[i + 1].record()
    torch.cuda.synchronize()
    each = sorted(marks[i].elapsed_time(marks[i + 1]) for i in range(reps))

    B = algorithmic_bytes(E_total, N, F)
    value = E_total / (ms_step * 1e-3) / 1e9
    traffic = stored_traffic()
    P = info["src_parts"]
    n_items = info["n_part_items"] if P > 1 else info["n_chunks"] + N
    n_partials = info["n_part_items"] if P > 1 else info["n_chunks"]
    C = compulsory_bytes(E_total, N, N, F, n_items)
    partial_bytes = 2 * n_partials * 4 * F  # written once, read once by the fix-up
    achieved = C / (agg_ms * 1e-3) / 1e9
    gathered = E_total * 4 * F
    gather_rate = gathered / (agg_ms * 1e-3) / 1e9
    # the gather ceiling, measured in this run: bare gathers of the same number
    # of rows from the same table (random windows, and the part plan's stream)
    items = col = None
    if P > 1:
        seg = tfg.tfg_graph_segments(g).cpu().numpy()
        items = part_plan_items(seg, N, P, row_chunk())
        col = tfg.tfg_graph_csr(g)[1]
    ceil = gather_ceiling(torch, x, items, col)
    del col
    ceiling_name, ceiling = max(((k, v["GBps"]) for k, v in ceil.items()), key=lambda kv: kv[1])

    cpu = cpu_mt = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(ei_np, x_np, N, min(args.cpu_edges, E))
        cpu_mt = cpu_baseline_threads(ei_np, x_np, N, min(args.cpu_edges, E))

    line = {
        "metric": METRIC,
        "value": round(value, 4),
        "unit": "GE/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "GCN sum-aggregation on a Chung-Lu power-law graph (gamma=2): "
                        "N=232965, E=114.6M directed edges + N self-loops, F=128, "
                        "step = COO->CSR + gcn_norm + sum aggregation",
            "N": N, "E": E, "E_total": E_total, "F": F, "seed": 1004,
            "row_chunk": row_chunk(),
        },
        "stages_ms": {"csr_build": round(avg["create"], 4), "gcn_norm": round(avg["norm"], 4),
                      "aggregate": round(avg["agg"], 4)},
        "aggregate_cached_graph": {"ms": round(agg_ms, 4),
                                   "ms_median": round(each[len(each) // 2], 4),
                                   "ms_min": round(each[0], 4), "launches": reps,
                                   "GE_per_s": round(E_total / (agg_ms * 1e-3) / 1e9, 3),
                                   "src_parts": info["src_parts"],
                                   "n_part_items": info["n_part_items"],
                                   "n_chunks": info["n_chunks"],
                                   "n_rows_split": info["n_rows_split"]},
        # achieved / frac: the bytes the aggregation must move to or from HBM (col,
        # weights, x once, out, pointers, work items) per call against 8 TB/s. The
        # gathered rows (one 512-byte row per edge) are served by the L2s and the
        # Infinity Cache: their rate is set against the measured gather ceiling.
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS,
                     "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
                     "traffic": traffic,
                     "traffic_source": ("stored: profiles/traffic_aggregate_powerlaw.txt, rocprofv3 "
                                        "FETCH_SIZE + WRITE_SIZE per launch, taken on the "
                                        "current kernel source" if traffic else None),
                     "traffic_GBps": (round(traffic / (agg_ms * 1e-3) / 1e9, 1)
                                      if traffic else None),
                     "kernel": "tfg_aggregate (spmm_wide + fixup_rows)",
                     "compulsory_bytes_per_launch": C,
                     "partial_row_bytes_per_launch": partial_bytes,
                     "frac_with_partials": round((C + partial_bytes) / (agg_ms * 1e-3) / 1e9
                                                 / PEAK_HBM_GBPS, 4),
                     "gather": {"bytes_per_launch": gathered, "achieved": round(gather_rate, 1),
                                "ceiling": ceiling, "ceiling_from": ceiling_name,
                                "frac": round(gather_rate / ceiling, 4), "unit": "GB/s",
                                "probes": ceil},
                     "algorithmic_bytes_per_launch": B,
                     "algorithmic_GBps": round(B / (agg_ms * 1e-3) / 1e9, 1)},
        "cpu_baseline": cpu,
        "cpu_baseline_threads": cpu_mt,
    }
    if cpu_mt and cpu_mt.get("value"):  # the step's rate over the threaded oracle's
        line["speedup_vs_cpu_baseline_threads"] = round(value / cpu_mt["value"], 1)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
