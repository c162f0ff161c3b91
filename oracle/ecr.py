"""The paper's lossy Elastic Computation Reformation and its Auto Tuner (§3.4).

Oracle - test infrastructure only (see the package docstring).

Cluster sparsity (§3.4).  The clustered N x N layout is cut into a k x k grid of
clusters; the scattered edges of a sparse cluster are moved into a few compact
d_b x d_b sub-blocks, as many as the cluster's edges fill, which changes the
attended graph.  The paper leaves the placement of the sub-blocks open (its
figure shows them scattered inside the cluster, obtained by compacting edges to
nearby positions); this oracle fixes the rule below.

* c = ceil(N / k); cluster (I, J) holds the edges (i, j) with i div c = I and
  j div c = J; cnt(I, J) counts them (self-loops included) and
  area(I, J) = rows(I) * rows(J), rows(I) = min(c, N - I c).
* The cluster is transferred iff cnt >= 1 and cnt / area < beta_thre, tested
  exactly as cnt * den < num * area with beta_thre = num / den (the paper's
  "smaller than" the threshold; the indolent rule is beta_thre = beta_G =
  nnz / N^2).
* In a transferred cluster the self-loops stay (condition C1 of §3.2: every node
  attends to itself); its other edges, moved = cnt - self-loops of them, are
  replaced by m = ceil(moved / d_b^2) full sub-blocks.  The cluster is cut into
  d_b x d_b blocks from its corner (block (a, b) covers local rows
  [a d_b, (a + 1) d_b) and columns [b d_b, (b + 1) d_b), clipped to the cluster);
  the m blocks holding the most moved edges are chosen, ties to the smaller
  (a, b) in row-major order, and every (i, j) inside them becomes an edge.  A
  block holds at most d_b^2 edges, so at least m blocks are non-empty and only
  non-empty blocks are chosen.
* Every edge of a cluster that is not transferred is kept.  E' is the union of
  kept edges, self-loops and sub-block cells, as a sorted duplicate-free CSR.

Auto Tuner (§3.4, transfer threshold).  Running loss F_t = 0.9 F_{t-1} + 0.1
L_t with F_0 = L_0; loss descent rate LDR_t = (F_t - F_{t-1}) / et_t from the
second epoch on; the threshold walks the ladder
{0, beta_G, 1.5 beta_G, 5 beta_G, 7 beta_G, 10 beta_G, 1} starting at beta_G.
Readings: a decision is taken at epoch t once LDR_{t - delta} exists and delta
epochs have passed since the previous change (or since the start); LDR_t >=
LDR_{t - delta} moves one step up the ladder, LDR_t < LDR_{t - delta} one step
down, clamped at both ends.  Thresholds are kept as exact fractions.
"""

from __future__ import annotations

from fractions import Fraction

import numpy as np


def cluster_edge(n: int, k: int) -> int:
    """c = ceil(N / k), the edge length of a cluster."""
    return max(1, -(-int(n) // int(k)))


def ecr_compact(rowptr, col, k: int, d_b: int, num: int, den: int, progress=None):
    """E' of the lossy reformation: (rowptr', col', info) with info the per-cluster counts and choices.
    ``progress`` (optional) is called with a short text after each stage."""
    say = progress or (lambda *_: None)
    rowptr = np.asarray(rowptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    n = len(rowptr) - 1
    if k < 1 or d_b < 1 or den < 1 or num < 0:
        raise ValueError("k, d_b, den must be positive and num non-negative")
    c = cluster_edge(n, k)
    rows = np.repeat(np.arange(n, dtype=np.int64), np.diff(rowptr))
    I, J = rows // c, col // c
    cid = I * k + J
    cnt = np.bincount(cid, minlength=k * k).astype(np.int64)
    size = np.array([max(0, min(c, n - a * c)) for a in range(k)], dtype=np.int64)
    area = np.outer(size, size).reshape(-1)
    # exact comparison cnt / area < num / den in Python integers
    transfer = np.array([cnt[x] >= 1 and int(cnt[x]) * int(den) < int(num) * int(area[x]) for x in range(k * k)],
                        dtype=bool)

    say("clusters counted")
    self_loop = rows == col
    moved = transfer[cid] & ~self_loop
    keep = ~moved
    out_r = [rows[keep]]
    out_c = [col[keep]]
    # moved edges per transferred cluster and its sub-block count m
    mcnt = np.bincount(cid[moved], minlength=k * k)
    m_of = {int(x): -(-int(mcnt[x]) // (d_b * d_b)) for x in np.flatnonzero(transfer)}
    # edges per block (cluster, block row a, block column b) of the moved edges
    nb = -(-c // d_b)
    mc = cid[moved]
    a = (rows[moved] - I[moved] * c) // d_b
    b = (col[moved] - J[moved] * c) // d_b
    bkey, counts = np.unique((mc * nb + a) * nb + b, return_counts=True)
    say(f"{len(bkey)} blocks counted")
    bc, ba, bb = bkey // (nb * nb), (bkey // nb) % nb, bkey % nb
    # inside each cluster: most edges first, ties to the smaller (a, b); the first m are chosen
    order = np.lexsort((bb, ba, -counts, bc))
    bc, ba, bb = bc[order], ba[order], bb[order]
    first = np.searchsorted(bc, bc, side="left")
    rank = np.arange(len(bc)) - first
    m_arr = np.zeros(k * k, dtype=np.int64)
    for x, m in m_of.items():
        m_arr[x] = m
    pick = rank < m_arr[bc]
    say(f"{int(pick.sum())} sub-blocks chosen")
    chosen = {x: [] for x in m_of}
    for x, aa, bbb in zip(bc[pick].tolist(), ba[pick].tolist(), bb[pick].tolist()):
        chosen[x].append((aa, bbb))
        Ix, Jx = divmod(x, k)
        r0, c0 = Ix * c + aa * d_b, Jx * c + bbb * d_b
        rr = np.arange(r0, min(r0 + d_b, Ix * c + size[Ix]), dtype=np.int64)
        cc = np.arange(c0, min(c0 + d_b, Jx * c + size[Jx]), dtype=np.int64)
        out_r.append(np.repeat(rr, len(cc)))
        out_c.append(np.tile(cc, len(rr)))
    say("cells emitted")
    R = np.concatenate(out_r)
    C = np.concatenate(out_c)
    key = np.unique(R * max(n, 1) + C)
    R, C = key // max(n, 1), key % max(n, 1)
    rp = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(np.bincount(R, minlength=n), out=rp[1:])
    info = {"c": c, "cnt": cnt, "area": area, "transfer": transfer, "m": m_of, "chosen": chosen}
    return rp, C.astype(np.int32), info


def max_nnz(nnz: int, k: int, d_b: int) -> int:
    """An upper bound on |E'|: the kept edges plus, per cluster, its moved edges rounded up to whole sub-blocks."""
    return int(nnz) + int(k) * int(k) * (int(d_b) * int(d_b) - 1)


def ladder(nnz: int, n: int):
    """The Auto Tuner's thresholds {0, bG, 1.5 bG, 5 bG, 7 bG, 10 bG, 1} as fractions, each capped at 1."""
    bG = Fraction(int(nnz), max(1, int(n) * int(n)))
    steps = [Fraction(0), bG, Fraction(3, 2) * bG, 5 * bG, 7 * bG, 10 * bG, Fraction(1)]
    return [min(s, Fraction(1)) for s in steps]


class AutoTuner:
    """The transfer-threshold controller (readings in the module docstring)."""

    def __init__(self, nnz: int, n: int, delta: int = 10):
        if delta < 1:
            raise ValueError("delta must be >= 1")
        self.values = ladder(nnz, n)
        self.level = 1  # beta_G
        self.delta = delta
        self.F = None
        self.ldr = []  # LDR_1, LDR_2, ... (index t - 1)
        self.t = -1
        self.last_change = 0

    @property
    def threshold(self) -> Fraction:
        return self.values[self.level]

    def step(self, loss: float, epoch_seconds: float) -> int:
        """Feed epoch t's loss and time; returns the ladder level to use for the next epoch."""
        self.t += 1
        t = self.t
        if self.F is None:
            self.F = float(loss)
            return self.level
        F_prev = self.F
        self.F = 0.9 * F_prev + 0.1 * float(loss)
        self.ldr.append((self.F - F_prev) / float(epoch_seconds))
        if t - self.delta >= 1 and t - self.last_change >= self.delta:
            now, then = self.ldr[t - 1], self.ldr[t - self.delta - 1]
            new = min(self.level + 1, len(self.values) - 1) if now >= then else max(self.level - 1, 0)
            if new != self.level:
                self.level = new
                self.last_change = t
        return self.level
