"""Softmax attention over graph neighbourhoods and over all pairs, in fp64.

Oracle - test infrastructure only (see the package docstring).

Definitions followed:

* Full attention, §2.1 Eq. (1): O = softmax(Q K^T / sqrt(d_K)) V, applied per
  head with d_K the per-head key width.
* Local topology-induced pattern, §3.2: node i attends only to the nodes j of
  its neighbourhood N(i); the coefficients are the softmax over j in N(i) of the
  scaled dot products, and the new feature is the coefficient-weighted sum of
  the neighbours' value rows.  N(i) is row i of the CSR exactly as given (the
  caller adds the self-loop of condition C1, §3.2).

Per head h and row i with neighbourhood N(i):

    s_ij  = scale * <Q[i,h], K[j,h]>              j in N(i)
    LSE_i = log sum_j exp(s_ij)                    (-inf for an empty row)
    P_ij  = exp(s_ij - LSE_i)
    O[i,h] = sum_j P_ij V[j,h]                     (0 for an empty row)

Backward, for an upstream gradient dO:

    D_i   = <dO[i,h], O[i,h]>
    dP_ij = <dO[i,h], V[j,h]>
    dS_ij = P_ij (dP_ij - D_i)
    dQ_i  = scale * sum_{j in N(i)} dS_ij K[j,h]
    dK_j  = scale * sum_{i : j in N(i)} dS_ij Q[i,h]
    dV_j  = sum_{i : j in N(i)} P_ij dO[i,h]

With a per-edge bias b (the graph encoding of §2.1 Eq. (3), added to the
scaled product; it shares the attention's sparse layout, §3.3), given as
[nnz, H] in CSR order:

    s_ij  = scale * <Q[i,h], K[j,h]> + b_ij[h]
    dB_ij = dS_ij

All arrays are [N, H, d] (node, head, feature); LSE and D are [N, H].
Inputs are upcast to fp64; bfloat16 workloads pass the already-rounded values.
"""

from __future__ import annotations

import numpy as np

_EDGE_BUDGET = 1 << 22  # edge x head x feature elements per chunk


def _f64(x):
    return np.asarray(x, dtype=np.float64)


class _Widen:
    """Rows of a feature array as fp64 on selection.  The inputs hold fp32 (or bf16-rounded) values, which
    fp64 holds exactly, so widening the selected rows equals widening the whole array first; large arrays are
    never copied whole."""

    def __init__(self, x):
        self.x = x.x if isinstance(x, _Widen) else np.asarray(x)
        self.shape = self.x.shape

    def __getitem__(self, key):
        return np.asarray(self.x[key], dtype=np.float64)


def _row_chunks(rowptr: np.ndarray, rows: np.ndarray, per_edge: int):
    """Split the row list into consecutive chunks holding about _EDGE_BUDGET elements."""
    deg = rowptr[rows + 1] - rowptr[rows]
    budget = max(1, _EDGE_BUDGET // max(1, per_edge))
    cum = np.cumsum(deg)
    start = 0
    while start < len(rows):
        base = cum[start - 1] if start else 0
        # rows while the chunk stays within the budget; a row above the budget on its own is a chunk alone
        stop = int(np.searchsorted(cum, base + budget, side="right"))
        stop = min(max(stop, start + 1), len(rows))
        yield rows[start:stop]
        start = stop


def _edges_of(rowptr, col, rows, with_pos=False):
    """Edge list (local row index, neighbour id) for the given rows, in CSR order (and the CSR positions)."""
    deg = (rowptr[rows + 1] - rowptr[rows]).astype(np.int64)
    local = np.repeat(np.arange(len(rows)), deg)
    first = np.zeros(len(rows), dtype=np.int64)
    if len(rows):
        np.cumsum(deg[:-1], out=first[1:])
    idx = np.arange(int(deg.sum()), dtype=np.int64) - np.repeat(first, deg) + np.repeat(rowptr[rows], deg)
    if with_pos:
        return local, col[idx].astype(np.int64), deg, idx
    return local, col[idx].astype(np.int64), deg


def _segments(local, n_rows):
    """Rows with at least one edge and the offset of each one's first edge; ``local`` is non-decreasing (the
    edges of a row are contiguous in CSR order)."""
    counts = np.bincount(local, minlength=n_rows)
    nz = np.nonzero(counts)[0]
    first = np.concatenate([[0], np.cumsum(counts)[:-1]])
    return nz, first[nz]


def _segment_softmax_stats(s, local, n_rows):
    """Per local row and head: max and log-sum-exp of the scores s[e, h] of its edges."""
    H = s.shape[1]
    m = np.full((n_rows, H), -np.inf)
    total = np.zeros((n_rows, H))
    if len(s):
        nz, first = _segments(local, n_rows)
        m[nz] = np.maximum.reduceat(s, first, axis=0)
        p = np.exp(s - m[local])
        total[nz] = np.add.reduceat(p, first, axis=0)
    with np.errstate(divide="ignore"):
        lse = m + np.log(total)
    return lse


def sparse_attn_fwd(rowptr, col, Q, K, V, scale, rows=None, bias=None):
    """O[rows], LSE[rows] of neighbourhood softmax attention (all rows when ``rows`` is None); ``bias`` is the
    optional per-edge term [nnz, H] in CSR order."""
    Q, K, V = _Widen(Q), _Widen(K), _Widen(V)
    B = None if bias is None else np.asarray(bias, dtype=np.float64)
    N, H, d = Q.shape
    rowptr = np.asarray(rowptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    rows = np.arange(N) if rows is None else np.asarray(rows, dtype=np.int64)
    O = np.zeros((len(rows), H, d))
    LSE = np.full((len(rows), H), -np.inf)
    pos = 0
    for chunk in _row_chunks(rowptr, rows, H * d):
        local, nbr, _, epos = _edges_of(rowptr, col, chunk, with_pos=True)
        n = len(chunk)
        if n == 1 and len(nbr) > 4096:
            # one long row (a hub, a global token): the same definition per head, as contractions over its
            # partners without edge-major temporaries
            r = chunk[0]
            Kn, Vn = K[nbr], V[nbr]
            for h in range(H):
                s = scale * (Kn[:, h, :] @ Q[r, h, :])
                if B is not None:
                    s = s + B[epos, h]
                m = s.max()
                p = np.exp(s - m)
                tot = p.sum()
                O[pos, h] = (p @ Vn[:, h, :]) / tot
                LSE[pos, h] = m + np.log(tot)
        elif len(nbr):
            i = chunk[local]
            s = scale * np.einsum("ehc,ehc->eh", Q[i], K[nbr])
            if B is not None:
                s = s + B[epos]
            lse = _segment_softmax_stats(s, local, n)
            p = np.exp(s - lse[local])
            o = np.zeros((n, H, d))
            nz, first = _segments(local, n)
            o[nz] = np.add.reduceat(p[:, :, None] * V[nbr], first, axis=0)
            O[pos:pos + n] = o
            LSE[pos:pos + n] = lse
        pos += n
    return O, LSE


def _csc(rowptr, col, N, with_pos=False):
    """In-neighbour lists: for each column j, the rows i with j in N(i), ascending (and each entry's CSR
    position)."""
    rowptr = np.asarray(rowptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    rows = np.repeat(np.arange(N), np.diff(rowptr))
    order = np.argsort(col, kind="stable")
    colptr = np.zeros(N + 1, dtype=np.int64)
    np.cumsum(np.bincount(col, minlength=N), out=colptr[1:])
    if with_pos:
        return colptr, rows[order], order
    return colptr, rows[order]


def sparse_attn_bwd(rowptr, col, Q, K, V, dO, scale, bias=None):
    """dQ, dK, dV of neighbourhood softmax attention for the whole graph (and dB [nnz, H] with a bias)."""
    Q, K, V, dO = _f64(Q), _f64(K), _f64(V), _f64(dO)
    N, H, d = Q.shape
    rowptr = np.asarray(rowptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    B = None if bias is None else np.asarray(bias, dtype=np.float64)
    O, LSE = sparse_attn_fwd(rowptr, col, Q, K, V, scale, bias=B)
    D = np.einsum("nhc,nhc->nh", dO, O)
    dQ = np.zeros_like(Q)
    dK = np.zeros_like(K)
    dV = np.zeros_like(V)
    dB = None if B is None else np.zeros_like(B)
    for chunk in _row_chunks(rowptr, np.arange(N), H * d):
        local, j, _, epos = _edges_of(rowptr, col, chunk, with_pos=True)
        if not len(j):
            continue
        i = chunk[local]
        s = scale * np.einsum("ehc,ehc->eh", Q[i], K[j])
        if B is not None:
            s = s + B[epos]
        p = np.exp(s - LSE[i])
        dp = np.einsum("ehc,ehc->eh", dO[i], V[j])
        ds = p * (dp - D[i])
        if dB is not None:
            dB[epos] = ds
        np.add.at(dQ, i, scale * ds[:, :, None] * K[j])
        np.add.at(dK, j, scale * ds[:, :, None] * Q[i])
        np.add.at(dV, j, p[:, :, None] * dO[i])
    if dB is not None:
        return dQ, dK, dV, dB
    return dQ, dK, dV


def sparse_attn_bwd_sampled(rowptr, col, Q, K, V, dO, scale, rows, cols, bias=None):
    """dQ[rows], dK[cols], dV[cols] computed from only the rows they depend on.

    dQ_i needs row i alone; dK_j and dV_j need every row i that has j as a
    neighbour (with that row's LSE_i and D_i, each row-local).  With a bias, a
    fourth result (positions, dB) holds dB of the sampled rows' edges with their
    CSR positions.
    """
    Q, K, V, dO = _Widen(Q), _Widen(K), _Widen(V), _Widen(dO)
    B = None if bias is None else np.asarray(bias, dtype=np.float64)
    N, H, d = Q.shape
    rowptr = np.asarray(rowptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    rows = np.asarray(rows, dtype=np.int64)
    cols = np.asarray(cols, dtype=np.int64)

    colptr, inrow, inpos = _csc(rowptr, col, N, with_pos=True)
    # LSE_i and D_i of the sampled rows and of every source row a sampled column needs, each computed once
    need = np.unique(np.concatenate([rows] + [inrow[colptr[jj]:colptr[jj + 1]] for jj in cols]))
    slot = np.full(N, -1, dtype=np.int64)
    slot[need] = np.arange(len(need))
    O_n, L_n = sparse_attn_fwd(rowptr, col, Q, K, V, scale, rows=need, bias=B)
    D_n = np.einsum("nhc,nhc->nh", dO[need], O_n)
    L_r, D_r = L_n[slot[rows]], D_n[slot[rows]]
    dQ = np.zeros((len(rows), H, d))
    local, j, _, epos = _edges_of(rowptr, col, rows, with_pos=True)
    dB_r = np.zeros((len(j), H))
    if len(j):
        i = rows[local]
        s = scale * np.einsum("ehc,ehc->eh", Q[i], K[j])
        if B is not None:
            s = s + B[epos]
        p = np.exp(s - L_r[local])
        dp = np.einsum("ehc,ehc->eh", dO[i], V[j])
        ds = p * (dp - D_r[local])
        dB_r = ds
        nz, first = _segments(local, len(rows))
        dQ[nz] = np.add.reduceat(scale * ds[:, :, None] * K[j], first, axis=0)

    dK = np.zeros((len(cols), H, d))
    dV = np.zeros((len(cols), H, d))
    for k, jj in enumerate(cols):
        srcs = inrow[colptr[jj]:colptr[jj + 1]]
        if not len(srcs):
            continue
        L_s, D_s = L_n[slot[srcs]], D_n[slot[srcs]]
        s = scale * np.einsum("ehc,hc->eh", Q[srcs], K[jj])
        if B is not None:
            s = s + B[inpos[colptr[jj]:colptr[jj + 1]]]
        p = np.exp(s - L_s)
        dp = np.einsum("ehc,hc->eh", dO[srcs], V[jj])
        ds = p * (dp - D_s)
        dK[k] = scale * np.einsum("eh,ehc->hc", ds, Q[srcs])
        dV[k] = np.einsum("eh,ehc->hc", p, dO[srcs])
    if B is not None:
        return dQ, dK, dV, (epos, dB_r)
    return dQ, dK, dV


# ---------------------------------------------------------------------------
# Full softmax attention, §2.1 Eq. (1), per head.
# ---------------------------------------------------------------------------

def dense_attn_fwd(Q, K, V, scale, rows=None):
    """O[rows], LSE[rows] of softmax(scale Q K^T) V over all N keys, per head."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    N, H, d = Q.shape
    rows = np.arange(N) if rows is None else np.asarray(rows, dtype=np.int64)
    O = np.zeros((len(rows), H, d))
    LSE = np.zeros((len(rows), H))
    step = max(1, (1 << 22) // max(1, N))
    for a in range(0, len(rows), step):
        r = rows[a:a + step]
        for h in range(H):
            s = scale * (Q[r, h, :] @ K[:, h, :].T)  # [R, N]
            m = s.max(axis=1, keepdims=True)
            e = np.exp(s - m)
            tot = e.sum(axis=1, keepdims=True)
            O[a:a + len(r), h, :] = (e / tot) @ V[:, h, :]
            LSE[a:a + len(r), h] = (m + np.log(tot))[:, 0]
    return O, LSE


def dense_attn_bwd(Q, K, V, dO, scale):
    """dQ, dK, dV of full softmax attention (materialises N x N per head: small N only)."""
    Q, K, V, dO = _f64(Q), _f64(K), _f64(V), _f64(dO)
    N, H, d = Q.shape
    dQ = np.zeros_like(Q)
    dK = np.zeros_like(K)
    dV = np.zeros_like(V)
    for h in range(H):
        s = scale * (Q[:, h, :] @ K[:, h, :].T)
        s -= s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        o = p @ V[:, h, :]
        Dv = (dO[:, h, :] * o).sum(axis=1, keepdims=True)
        dp = dO[:, h, :] @ V[:, h, :].T
        ds = p * (dp - Dv)
        dQ[:, h, :] = scale * ds @ K[:, h, :]
        dK[:, h, :] = scale * ds.T @ Q[:, h, :]
        dV[:, h, :] = p.T @ dO[:, h, :]
    return dQ, dK, dV


def dense_attn_dq_rows(Q, K, V, dO, scale, rows):
    """dQ[rows] of full softmax attention; each row needs only its own scores against all keys."""
    Q, K, V, dO = _f64(Q), _f64(K), _f64(V), _f64(dO)
    N, H, d = Q.shape
    rows = np.asarray(rows, dtype=np.int64)
    dQ = np.zeros((len(rows), H, d))
    step = max(1, (1 << 22) // max(1, N))
    for a in range(0, len(rows), step):
        r = rows[a:a + step]
        for h in range(H):
            s = scale * (Q[r, h, :] @ K[:, h, :].T)
            s -= s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            o = p @ V[:, h, :]
            Dv = (dO[r, h, :] * o).sum(axis=1, keepdims=True)
            dp = dO[r, h, :] @ V[:, h, :].T
            ds = p * (dp - Dv)
            dQ[a:a + len(r), h, :] = scale * ds @ K[:, h, :]
    return dQ


def dense_attn_row_stats(Q, K, V, dO, scale):
    """LSE_i and D_i = <dO_i, O_i> of every row of full softmax attention ([N, H] each), O in fp64."""
    dO = _f64(dO)
    O, LSE = dense_attn_fwd(Q, K, V, scale)
    return LSE, np.einsum("nhc,nhc->nh", dO, O)


def dense_attn_dkdv_cols(Q, K, V, dO, scale, cols, stats=None):
    """dK[cols], dV[cols] of full softmax attention: column j gathers dS_ij Q_i and P_ij dO_i over all N rows,
    with P_ij = exp(s_ij - LSE_i) and dS_ij = P_ij (dP_ij - D_i), so it needs every row's LSE and D
    (``stats`` = dense_attn_row_stats(...), computed here when not given)."""
    Q, K, V, dO = _f64(Q), _f64(K), _f64(V), _f64(dO)
    N, H, d = Q.shape
    cols = np.asarray(cols, dtype=np.int64)
    LSE, Dv = stats if stats is not None else dense_attn_row_stats(Q, K, V, dO, scale)
    dK = np.zeros((len(cols), H, d))
    dV = np.zeros((len(cols), H, d))
    step = max(1, (1 << 22) // max(1, N))
    for a in range(0, len(cols), step):
        c = cols[a:a + step]
        for h in range(H):
            p = np.exp(scale * (Q[:, h, :] @ K[c, h, :].T) - LSE[:, h:h + 1])  # [N, C]
            ds = p * (dO[:, h, :] @ V[c, h, :].T - Dv[:, h:h + 1])
            dK[a:a + len(c), h, :] = scale * ds.T @ Q[:, h, :]
            dV[a:a + len(c), h, :] = p.T @ dO[:, h, :]
    return dK, dV
