"""Seeded synthetic graphs shaped like the paper's workloads.

The paper trains on large, sparse, clustered graphs (evaluation datasets of
§4: node counts from thousands to millions, densities of 1e-5 to 1e-4, strong
community structure).  None of those datasets is used here; these generators
produce graphs of the same regime:

* a stochastic block model with an exact share of cross-block edges, equal or
  log-normally distributed block sizes, and a random node order;
* a Chung-Lu power-law graph with capped expected degrees, also shuffled.

Every graph comes out as a symmetric CSR: rows sorted, columns strictly
increasing inside each row, duplicates removed, and (by default) a self-loop on
every node, which is the paper's condition C1 of §3.2 (every node attends to
itself).  ``rowptr`` is int64[N+1] and ``col`` int32[nnz].
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass
class Graph:
    n: int
    rowptr: np.ndarray  # int64[n+1]
    col: np.ndarray  # int32[nnz]
    block: np.ndarray | None = None  # planted block of each node (after shuffling), or None
    info: dict = field(default_factory=dict)

    @property
    def nnz(self) -> int:
        return int(self.rowptr[-1])

    def degrees(self) -> np.ndarray:
        return np.diff(self.rowptr)


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def csr_from_pairs(n: int, u: np.ndarray, v: np.ndarray, symmetric: bool = True,
                   self_loops: bool = True) -> tuple[np.ndarray, np.ndarray]:
    """Build a sorted, duplicate-free CSR from (u, v) pairs.

    With ``symmetric`` both directions are inserted; with ``self_loops`` the
    pair (i, i) is inserted for every node.
    """
    u = np.asarray(u, dtype=np.int64)
    v = np.asarray(v, dtype=np.int64)
    parts_r = [u]
    parts_c = [v]
    if symmetric:
        parts_r.append(v)
        parts_c.append(u)
    if self_loops:
        diag = np.arange(n, dtype=np.int64)
        parts_r.append(diag)
        parts_c.append(diag)
    r = np.concatenate(parts_r)
    c = np.concatenate(parts_c)
    keys = np.unique(r * np.int64(n) + c)
    rows = keys // n
    cols = (keys - rows * n).astype(np.int32)
    counts = np.bincount(rows, minlength=n)
    rowptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(counts, out=rowptr[1:])
    return rowptr, cols


def lognormal_block_sizes(n: int, n_blocks: int, sigma: float, seed: int, min_size: int = 2) -> np.ndarray:
    """Block sizes drawn log-normal, scaled to sum to ``n`` by largest-remainder rounding."""
    rng = _rng(seed)
    raw = rng.lognormal(mean=0.0, sigma=sigma, size=n_blocks)
    spare = n - min_size * n_blocks
    if spare < 0:
        raise ValueError("n too small for the requested number of blocks")
    share = raw / raw.sum() * spare
    base = np.floor(share).astype(np.int64)
    rem = spare - int(base.sum())
    order = np.argsort(-(share - base), kind="stable")
    base[order[:rem]] += 1
    return base + min_size


def sbm_graph(block_sizes, avg_degree: float, cross_frac: float, seed: int,
              shuffle: bool = True, self_loops: bool = True) -> Graph:
    """Stochastic block model with an exact number of drawn pairs.

    ``round(N * avg_degree / 2)`` undirected pairs are drawn; a ``cross_frac``
    share of them joins two different blocks (uniform over such pairs), the
    rest join two distinct nodes of one block, the block being picked with
    probability proportional to its number of node pairs (so the in-block edge
    probability is the same for every block).  Duplicates are dropped, so the
    realised degree is slightly below ``avg_degree``.
    """
    rng = _rng(seed)
    sizes = np.asarray(block_sizes, dtype=np.int64)
    n = int(sizes.sum())
    nb = len(sizes)
    starts = np.zeros(nb, dtype=np.int64)
    np.cumsum(sizes[:-1], out=starts[1:])
    n_pairs = int(round(n * avg_degree / 2.0))
    n_cross = int(round(cross_frac * n_pairs)) if nb > 1 else 0
    n_in = n_pairs - n_cross

    pair_w = sizes * (sizes - 1) / 2.0
    b = rng.choice(nb, size=n_in, p=pair_w / pair_w.sum())
    u = rng.integers(0, sizes[b])
    v = rng.integers(0, sizes[b] - 1)
    v = v + (v >= u)
    u = u + starts[b]
    v = v + starts[b]

    block_of = np.repeat(np.arange(nb, dtype=np.int64), sizes)
    cu = np.empty(0, dtype=np.int64)
    cv = np.empty(0, dtype=np.int64)
    while len(cu) < n_cross:
        need = n_cross - len(cu)
        a = rng.integers(0, n, size=need + need // 8 + 16)
        c = rng.integers(0, n, size=len(a))
        ok = block_of[a] != block_of[c]
        cu = np.concatenate([cu, a[ok]])[:n_cross]
        cv = np.concatenate([cv, c[ok]])[:n_cross]

    u = np.concatenate([u, cu])
    v = np.concatenate([v, cv])
    block = block_of
    if shuffle:
        new_id = rng.permutation(n).astype(np.int64)
        u = new_id[u]
        v = new_id[v]
        block = np.empty(n, dtype=np.int64)
        block[new_id] = block_of
    rowptr, col = csr_from_pairs(n, u, v, symmetric=True, self_loops=self_loops)
    info = {"kind": "sbm", "n_blocks": nb, "pairs_drawn": n_pairs, "cross_pairs_drawn": n_cross,
            "avg_degree_nominal": avg_degree, "cross_frac": cross_frac, "seed": seed}
    return Graph(n=n, rowptr=rowptr, col=col, block=block, info=info)


def chung_lu_weights(n: int, gamma: float, avg_degree: float, max_degree: float) -> np.ndarray:
    """Expected degrees w_i = c * i^(-1/(gamma-1)), capped, with c set so mean(w) = avg_degree."""
    base = np.arange(1, n + 1, dtype=np.float64) ** (-1.0 / (gamma - 1.0))
    lo, hi = 0.0, float(max_degree) / base[-1] + 1.0
    for _ in range(200):
        c = 0.5 * (lo + hi)
        m = np.minimum(c * base, max_degree).mean()
        if m < avg_degree:
            lo = c
        else:
            hi = c
    return np.minimum(0.5 * (lo + hi) * base, max_degree)


def chung_lu_graph(n: int, gamma: float, avg_degree: float, max_degree: float, seed: int,
                   shuffle: bool = True, self_loops: bool = True) -> Graph:
    """Chung-Lu graph: ``round(N*avg_degree/2)`` pairs, both endpoints drawn with
    probability proportional to the expected degrees; loops and duplicates dropped."""
    rng = _rng(seed)
    w = chung_lu_weights(n, gamma, avg_degree, max_degree)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    m = int(round(n * avg_degree / 2.0))
    u = np.searchsorted(cdf, rng.random(m), side="right").astype(np.int64)
    v = np.searchsorted(cdf, rng.random(m), side="right").astype(np.int64)
    np.minimum(u, n - 1, out=u)
    np.minimum(v, n - 1, out=v)
    keep = u != v
    u, v = u[keep], v[keep]
    if shuffle:
        new_id = rng.permutation(n).astype(np.int64)
        u = new_id[u]
        v = new_id[v]
    rowptr, col = csr_from_pairs(n, u, v, symmetric=True, self_loops=self_loops)
    info = {"kind": "chung_lu", "gamma": gamma, "avg_degree_nominal": avg_degree,
            "max_degree_cap": max_degree, "pairs_drawn": m, "seed": seed,
            "n_at_cap": int((w >= max_degree).sum())}
    return Graph(n=n, rowptr=rowptr, col=col, block=None, info=info)


def batched_graphs(sizes, avg_degree: float, seed: int, global_token: bool = False,
                   self_loops: bool = True) -> Graph:
    """Many small graphs as one block-diagonal graph (graph-level batching).

    Graph g gets ``sizes[g]`` consecutive node ids.  Each is a random spanning
    tree (every node links to a uniformly chosen earlier node, so the graph is
    connected) plus extra uniformly random in-graph pairs up to
    ``round(size * avg_degree / 2)`` pairs in total (molecule-like rings when
    avg_degree is near 2).  With ``global_token`` one more node (the last id)
    is linked to every node in both directions, a degree-N row and column.
    Nodes keep the batch order: each graph is contiguous.
    """
    rng = _rng(seed)
    sizes = np.asarray(sizes, dtype=np.int64)
    starts = np.concatenate([[0], np.cumsum(sizes)[:-1]])
    n_real = int(sizes.sum())
    us, vs = [], []
    # spanning trees: node k > 0 of a graph links to a uniform earlier node of the same graph
    local = np.arange(n_real, dtype=np.int64) - np.repeat(starts, sizes)
    first = local > 0
    parent_local = (rng.random(n_real) * np.maximum(local, 1)).astype(np.int64)
    node = np.arange(n_real, dtype=np.int64)
    us.append(node[first])
    vs.append((node - local + parent_local)[first])
    # extra in-graph pairs
    extra = np.maximum(0, np.round(sizes * avg_degree / 2.0).astype(np.int64) - (sizes - 1))
    g_of = np.repeat(np.arange(len(sizes)), extra)
    a = starts[g_of] + (rng.random(len(g_of)) * sizes[g_of]).astype(np.int64)
    b = starts[g_of] + (rng.random(len(g_of)) * sizes[g_of]).astype(np.int64)
    keep = a != b
    us.append(a[keep])
    vs.append(b[keep])
    n = n_real + (1 if global_token else 0)
    if global_token:
        us.append(np.full(n_real, n_real, dtype=np.int64))
        vs.append(np.arange(n_real, dtype=np.int64))
    rowptr, col = csr_from_pairs(n, np.concatenate(us), np.concatenate(vs), symmetric=True, self_loops=self_loops)
    block = np.repeat(np.arange(len(sizes)), sizes)
    if global_token:
        block = np.concatenate([block, [-1]])
    info = {"kind": "batched", "graphs": len(sizes), "mean_size": float(sizes.mean()),
            "avg_degree_nominal": avg_degree, "global_token": global_token, "seed": seed}
    return Graph(n=n, rowptr=rowptr, col=col, block=block, info=info)
