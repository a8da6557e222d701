"""Command-line contract of bench.py that needs no GPU: more than one GPU is
refused with a message and a non-zero status."""

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_several_gpus():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr and "--gpus 2" in r.stderr
    assert r.stdout == ""


def test_threaded_oracle_baseline_is_bit_identical():
    """The threaded CPU baseline splits target rows over threads; every row is
    still summed over its edges in input order, so the result equals the
    single-thread oracle bit for bit (ragged split: 97 rows over 5 threads)."""
    import numpy as np
    sys.path.insert(0, ROOT)
    import bench
    import oracle
    rng = np.random.default_rng(7)
    n, E, F = 97, 2_000, 16
    ei = rng.integers(0, n, size=(2, E), dtype=np.int64)
    x = rng.standard_normal((n, F)).astype(np.float32)
    oei, ow, _ = oracle.gcn_norm(ei, n)
    one, _ = oracle.aggregate(oei, x, n, "sum", edge_weight=ow)
    for threads in (1, 5, 8):
        many = bench.oracle_sum_by_row_ranges(oei, ow, x, n, threads)
        assert many.dtype == np.float64 and many.shape == (n, F)
        assert np.array_equal(many, one)
