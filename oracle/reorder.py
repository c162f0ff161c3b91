"""Cluster reordering of the node set, in integer arithmetic.

Oracle - test infrastructure only (see the package docstring).

§3.3 (utilisation of graph cluster) reorders the nodes so that each cluster's
nodes get neighbouring ids, using METIS.  METIS is a third-party multilevel
partitioner whose output cannot be reproduced bit for bit, so the library reads
the step as "any deterministic community-finding node order" and fixes one:
label propagation with hashed tie-breaks and hashed partial activation,
followed by a sort by (label, -degree, id).  The definition:

* k_t = seed + (t + 1) * 0x9E3779B97F4A7C15  (mod 2^64), for sweep t = 0, 1, ...
* mix64 is the SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014):
  z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27; z *= 0x94D049BB133111EB;
  z ^= z >> 31 (all mod 2^64).
* label priority  h_t(l) = mix64(l XOR k_t)
* node activity   a_t(v) = the top three bits of mix64(v XOR k_t XOR
  0xD6E8FEB86659FD93) are not all zero (about 7 nodes in 8 are active)
* lab_0[v] = v.
* Sweep t computes lab_{t+1} from lab_t alone.  For node v let C_v be the
  multiset of lab_t[u] over neighbours u of v with u != v, and M_v the labels
  of largest multiplicity in C_v.  The candidate c_v is lab_t[v] if C_v is empty
  or lab_t[v] is in M_v, otherwise the l in M_v with the smallest (h_t(l), l).
  If c_v == lab_t[v] for every node, propagation stops (no later sweep could
  change anything).  Otherwise lab_{t+1}[v] = c_v for active nodes and
  lab_t[v] for the others.
* After at most ``iters`` sweeps the new order sorts the nodes by
  (lab[v], -deg(v), v), deg counting neighbours other than v itself.
  perm[new] = old and iperm[old] = new.

The partial activation keeps synchronous propagation from oscillating on
bipartite pieces (a star, a single edge), where every node would otherwise swap
labels with its neighbours on every sweep.  Twenty sweeps is the default: on the
block-model workloads it recovers an order whose dense-tile edge share matches
the planted block order's.
"""

from __future__ import annotations

import numpy as np

GOLDEN = np.uint64(0x9E3779B97F4A7C15)
ACTIVITY_SALT = np.uint64(0xD6E8FEB86659FD93)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def mix64(x) -> np.ndarray:
    """SplitMix64 output function on uint64 values (wrapping arithmetic)."""
    z = np.asarray(x, dtype=np.uint64).copy()
    with np.errstate(over="ignore"):
        z ^= z >> np.uint64(30)
        z *= _M1
        z ^= z >> np.uint64(27)
        z *= _M2
        z ^= z >> np.uint64(31)
    return z


def sweep_key(seed: int, t: int) -> np.uint64:
    return np.uint64((int(seed) + (t + 1) * int(GOLDEN)) % (1 << 64))


def _offdiag_edges(rowptr, col):
    n = len(rowptr) - 1
    r = np.repeat(np.arange(n, dtype=np.int64), np.diff(rowptr))
    c = np.asarray(col, dtype=np.int64)
    keep = r != c
    return n, r[keep], c[keep]


def lp_sweep(n, r, c, lab, t, seed):
    """One synchronous sweep; returns (candidate labels c_v, new labels)."""
    k = sweep_key(seed, t)
    L = lab[c]
    order = np.lexsort((L, r))
    rs, Ls = r[order], L[order]
    cand = lab.copy()
    if len(rs):
        brk = np.ones(len(rs), dtype=bool)
        brk[1:] = (rs[1:] != rs[:-1]) | (Ls[1:] != Ls[:-1])
        starts = np.flatnonzero(brk)
        run_row = rs[starts]
        run_lab = Ls[starts]
        run_cnt = np.diff(np.append(starts, len(rs)))
        best = np.zeros(n, dtype=np.int64)
        np.maximum.at(best, run_row, run_cnt)
        top = run_cnt == best[run_row]
        own_top = np.zeros(n, dtype=bool)
        own_top[run_row[top & (run_lab == lab[run_row])]] = True
        t_row = run_row[top]
        t_lab = run_lab[top]
        t_pri = mix64(t_lab.astype(np.uint64) ^ k)
        pick = np.lexsort((t_lab, t_pri, t_row))
        t_row, t_lab = t_row[pick], t_lab[pick]
        first = np.ones(len(t_row), dtype=bool)
        first[1:] = t_row[1:] != t_row[:-1]
        win_row, win_lab = t_row[first], t_lab[first]
        move = ~own_top[win_row]
        cand[win_row[move]] = win_lab[move]
    active = (mix64(np.arange(n, dtype=np.uint64) ^ k ^ ACTIVITY_SALT) >> np.uint64(61)) != 0
    new = np.where(active, cand, lab)
    return cand, new


def lp_labels(rowptr, col, iters: int = 20, seed: int = 0):
    """Final labels and the number of sweeps that changed something."""
    n, r, c = _offdiag_edges(np.asarray(rowptr, np.int64), col)
    lab = np.arange(n, dtype=np.int64)
    done = 0
    for t in range(iters):
        cand, new = lp_sweep(n, r, c, lab, t, seed)
        if np.array_equal(cand, lab):
            break
        lab = new
        done = t + 1
    return lab, done


def cluster_order(rowptr, col, labels):
    """perm (new -> old) sorting nodes by (label, -deg, id); iperm its inverse."""
    rowptr = np.asarray(rowptr, np.int64)
    n = len(rowptr) - 1
    r = np.repeat(np.arange(n, dtype=np.int64), np.diff(rowptr))
    deg = np.bincount(r[r != np.asarray(col, np.int64)], minlength=n).astype(np.int64)
    perm = np.lexsort((np.arange(n), -deg, np.asarray(labels, np.int64))).astype(np.int64)
    iperm = np.empty(n, dtype=np.int64)
    iperm[perm] = np.arange(n)
    return perm, iperm


def reorder(rowptr, col, iters: int = 20, seed: int = 0):
    """perm, iperm, labels of the cluster reordering."""
    labels, _ = lp_labels(rowptr, col, iters, seed)
    perm, iperm = cluster_order(rowptr, col, labels)
    return perm, iperm, labels
