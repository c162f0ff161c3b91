"""The interleave decision of Dual-interleaved Attention (§3.2): when the
topology-induced pattern alone may be used, and when a fully connected layer
must be interleaved.

Oracle - test infrastructure only (see the package docstring).

The paper lists three conditions for the sparse pattern and checks them with
quick heuristics, Dirac's theorem for the Hamiltonian path.  Readings (the
graph is taken as undirected, i.e. the CSR as symmetric; node i reaches what it
can attend to through its out-edges):

* C1, every node attends to itself: exact, the rows missing their self-loop
  are counted.
* C2, a Hamiltonian path through all nodes: Dirac's condition on the minimum
  degree without self-loops, 2 min_deg >= n with n >= 3, confirms it; a single
  node holds trivially and two nodes hold iff they are adjacent.  Otherwise the
  heuristic cannot confirm it and C2 counts as not holding.
* C3, every node reaches every node within L layers (diameter <= L): a
  breadth-first search from node 0, cut at depth L + 1, gives its eccentricity
  e.  A node at depth L + 1, or a node not reached, fails C3; 2 e <= L confirms
  it (the diameter is at most twice any eccentricity).  Otherwise a second
  search from the smallest-id node at depth e (the double sweep) gives a
  lower bound e2 on the diameter: a node at depth L + 1 fails C3, else C3 is
  undetermined.
* The sparse pattern is used alone iff C1, C2 and C3 all hold; in every other
  case a dense layer is interleaved.
"""

from __future__ import annotations

import numpy as np


def self_loop_rows(rowptr, col) -> np.ndarray:
    """Boolean per row: does row i contain column i."""
    rowptr = np.asarray(rowptr, np.int64)
    col = np.asarray(col, np.int64)
    n = len(rowptr) - 1
    rows = np.repeat(np.arange(n, dtype=np.int64), np.diff(rowptr))
    has = np.zeros(n, dtype=bool)
    has[rows[rows == col]] = True
    return has


def bfs_levels(rowptr, col, root: int, cap: int) -> np.ndarray:
    """Breadth-first depth of every node from ``root`` along out-edges, -1 where deeper than ``cap`` or unreached."""
    rowptr = np.asarray(rowptr, np.int64)
    col = np.asarray(col, np.int64)
    n = len(rowptr) - 1
    lev = np.full(n, -1, dtype=np.int64)
    lev[root] = 0
    frontier = np.array([root], dtype=np.int64)
    d = 0
    while len(frontier) and d < cap:
        # every edge position of the frontier rows: rowptr[v] + 0 .. deg(v) - 1 for each v
        lens = rowptr[frontier + 1] - rowptr[frontier]
        starts = np.repeat(rowptr[frontier] - (np.cumsum(lens) - lens), lens)
        nbr = np.unique(col[starts + np.arange(int(lens.sum()))])
        new = nbr[lev[nbr] < 0]
        d += 1
        lev[new] = d
        frontier = new
    return lev


def interleave_report(rowptr, col, L: int) -> dict:
    """The three conditions and the decision (fields as in the library's report)."""
    rowptr = np.asarray(rowptr, np.int64)
    col = np.asarray(col, np.int64)
    n = len(rowptr) - 1
    has = self_loop_rows(rowptr, col)
    missing = int(n - has.sum())
    deg = np.diff(rowptr) - has
    min_deg = int(deg.min()) if n else 0
    c1 = 1 if missing == 0 else 0
    if n <= 1:
        c2 = 1
    elif n == 2:
        c2 = 1 if min_deg >= 1 else 0
    else:
        c2 = 1 if n >= 3 and 2 * min_deg >= n else 0
    lev = bfs_levels(rowptr, col, 0, L + 1) if n else np.zeros(0, np.int64)
    reached = int((lev >= 0).sum())
    ecc = int(lev.max()) if n else 0
    ecc_far = -1
    if n == 0:
        c3 = 1
    elif ecc > L or reached < n:
        c3 = 0
    elif 2 * ecc <= L:
        c3 = 1
    else:
        far = int(np.flatnonzero(lev == ecc)[0])
        lev2 = bfs_levels(rowptr, col, far, L + 1)
        ecc_far = int(lev2.max())
        c3 = 0 if ecc_far > L or (lev2 < 0).any() else -1
    return {"n": n, "missing_self_loops": missing, "min_degree": min_deg, "reached": reached, "ecc_root": ecc,
            "ecc_far": ecc_far, "c1": c1, "c2": c2, "c3": c3,
            "use_sparse": 1 if (c1 == 1 and c2 == 1 and c3 == 1) else 0}
