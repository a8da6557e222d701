"""Command-line contract of bench.py that needs no GPU: more than one GPU is
refused with a message and a non-zero status."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_several_gpus():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr and "--gpus 2" in r.stderr
    assert r.stdout == ""


@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
def test_threaded_oracle_is_bit_identical(reduce):
    """The oracle split over threads by target range (the benchmark's threaded
    CPU baseline and the full-size GPU checks) reduces every row over its
    edges in input order, so it equals the single-thread oracle bit for bit
    (ragged split: 97 rows over 5 threads)."""
    import numpy as np
    sys.path.insert(0, ROOT)
    import oracle
    rng = np.random.default_rng(7)
    n, E, F = 97, 2_000, 16
    ei = rng.integers(0, n, size=(2, E), dtype=np.int64)
    x = rng.standard_normal((n, F)).astype(np.float32)
    oei, ow, _ = oracle.gcn_norm(ei, n)
    one = oracle.aggregate(oei, x, n, reduce, edge_weight=ow)
    for threads in (1, 5, 8):
        many = oracle.aggregate_by_row_ranges(oei, x, n, reduce, edge_weight=ow, threads=threads)
        assert all(m.dtype == o.dtype and np.array_equal(m, o) for m, o in zip(many, one))
