"""Expected edge order of a graph handle, derived in the tests from the
oracle's plain CSR by target.

A handle built with P source parts orders each row's edges by source part
(part = source // ceil(N_src / P)), keeping input order among the edges of
one (row, part) segment. That order is a stable regrouping of the plain
stable CSR by target (the paper's reduce key, Sec. 2.1.2): inside each row,
positions move by part and keep their relative order. The oracle only knows
the plain CSR; the regrouping is written here.
"""

import numpy as np


def part_rows(n_src: int, parts: int) -> int:
    return max(-(-n_src // parts), 1)


def regroup_by_part(rowptr, col, perm, parts, n_src):
    """(col, perm, seg) of the (target, source part) order from the plain CSR
    (rowptr, col, perm); seg [N * parts + 1] is the start of every segment."""
    n = rowptr.shape[0] - 1
    col = np.asarray(col, np.int64)
    perm = np.asarray(perm, np.int64)
    if parts == 1:
        return col, perm, np.asarray(rowptr, np.int64)
    row = np.repeat(np.arange(n, dtype=np.int64), np.diff(rowptr))
    key = row * parts + col // part_rows(n_src, parts)
    order = np.argsort(key, kind="stable")  # rows are already in order: moves within rows only
    seg = np.zeros(n * parts + 1, np.int64)
    np.cumsum(np.bincount(key, minlength=n * parts), out=seg[1:])
    return col[order], perm[order], seg


def expected_graph(orc, edge_index, n, parts=1, n_src=None):
    """(rowptr, col, perm, seg) that a handle with `parts` source parts must
    hold for this edge list (self-loops, if any, already appended)."""
    n_src = n if n_src is None else n_src
    rowptr, col, perm = orc.csr_by_target(edge_index, n, n_src=n_src)
    col, perm, seg = regroup_by_part(rowptr, col, perm, parts, n_src)
    return rowptr, col, perm, seg
