"""Relabelled CSR and the dense/sparse tile plan, in integer arithmetic.

Oracle - test infrastructure only (see the package docstring).

Relabelling (§3.3: after gathering the full sequence the layout is reorganised
by cluster; token order is free for graph tasks, §3.3 "specialized graph
parallelism"): row r of the new CSR is {iperm[c] : c in row perm[r] of the old
CSR}, ascending.

Tiles (§3.4, cluster sparsity and transfer strategy).  The paper cuts the
clustered S x S layout into a grid of square blocks and treats each block by
how full it is, the fullness being the share of non-zero entries.  The library
reads that as an exact execution plan on T x T tiles:

* R = ceil(N / T) tile rows and columns; tile (I, J) holds the edges (i, j) with
  i div T = I and j div T = J; cnt(I, J) is their number and
  area(I, J) = min(T, N - I T) * min(T, N - J T) its clipped size.
* A tile is dense iff cnt >= 1 and cnt * 10^6 >= tau_ppm * area (exact integer
  comparison; equality counts as dense).  tau_ppm = 0 makes every non-empty
  tile dense; tau_ppm > 10^6 makes none dense.
* The dense tiles, sorted by (I, J): tile_rowptr[R+1], tile_col, tile_nnz and a
  T x T bit mask per tile (uint32 words, row-major; bit b of word w of local row
  r marks column J T + 32 w + b).
* The sparse remainder: every edge outside the dense tiles, in CSR order
  (sp_rowptr[N+1], sp_col), and its transpose (sp_colptr[N+1], sp_row, rows
  ascending inside each column).
* The dense tiles grouped by column tile, sorted by (J, I): tileT_ptr[R+1] and
  tileT_idx (index into the (I, J)-sorted list).

The split never changes which pairs are attended: every edge is in exactly one
of the two parts.
"""

from __future__ import annotations

import numpy as np


def permute_csr(rowptr, col, perm, iperm):
    """CSR of P A P^T: row r holds iperm of the neighbours of node perm[r], sorted."""
    rowptr = np.asarray(rowptr, np.int64)
    col = np.asarray(col, np.int64)
    perm = np.asarray(perm, np.int64)
    iperm = np.asarray(iperm, np.int64)
    n = len(rowptr) - 1
    deg = np.diff(rowptr)
    new_deg = deg[perm]
    rp = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(new_deg, out=rp[1:])
    new_row_of_edge = iperm[np.repeat(np.arange(n, dtype=np.int64), deg)]
    new_col = iperm[col]
    order = np.lexsort((new_col, new_row_of_edge))
    return rp, new_col[order].astype(np.int32)


def tau_to_ppm(tau: float) -> int:
    """Density threshold as parts per million, rounded to nearest."""
    return int(round(float(tau) * 1e6))


def build_tiles(rowptr, col, T: int, tau_ppm: int):
    """The tile plan as a dict of numpy arrays (see the module docstring)."""
    rowptr = np.asarray(rowptr, np.int64)
    col = np.asarray(col, np.int64)
    n = len(rowptr) - 1
    R = (n + T - 1) // T
    rows = np.repeat(np.arange(n, dtype=np.int64), np.diff(rowptr))
    I = rows // T
    J = col // T
    key = I * R + J
    ukey, cnt = np.unique(key, return_counts=True)
    uI, uJ = ukey // R, ukey % R
    area = np.minimum(T, n - uI * T) * np.minimum(T, n - uJ * T)
    dense = (cnt.astype(np.int64) * 1_000_000 >= np.int64(tau_ppm) * area) & (cnt >= 1)

    d_key = ukey[dense]  # ascending = sorted by (I, J)
    d_I, d_J = uI[dense], uJ[dense]
    tile_rowptr = np.zeros(R + 1, dtype=np.int64)
    np.cumsum(np.bincount(d_I, minlength=R), out=tile_rowptr[1:])
    n_dense = len(d_key)
    words = T // 32
    mask = np.zeros((n_dense, T, words), dtype=np.uint32)

    pos = np.searchsorted(d_key, key)
    in_dense = np.zeros(len(key), dtype=bool)
    ok = pos < n_dense
    in_dense[ok] = d_key[pos[ok]] == key[ok]
    e_tile = pos[in_dense]
    e_r = rows[in_dense] - I[in_dense] * T
    e_c = col[in_dense] - J[in_dense] * T
    np.bitwise_or.at(mask, (e_tile, e_r, e_c // 32), (np.uint32(1) << (e_c % 32).astype(np.uint32)))
    tile_nnz = np.bincount(e_tile, minlength=n_dense).astype(np.int32)

    sp_rows = rows[~in_dense]
    sp_col = col[~in_dense]
    sp_rowptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(np.bincount(sp_rows, minlength=n), out=sp_rowptr[1:])
    corder = np.argsort(sp_col, kind="stable")
    sp_colptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(np.bincount(sp_col, minlength=n), out=sp_colptr[1:])
    sp_row = sp_rows[corder]

    torder = np.lexsort((d_I, d_J))
    tileT_ptr = np.zeros(R + 1, dtype=np.int64)
    np.cumsum(np.bincount(d_J, minlength=R), out=tileT_ptr[1:])

    return {
        "T": T,
        "n_row_tiles": R,
        "tile_rowptr": tile_rowptr,
        "tile_col": d_J.astype(np.int32),
        "tile_nnz": tile_nnz,
        "tile_mask": mask.reshape(-1),
        "sp_rowptr": sp_rowptr,
        "sp_col": sp_col.astype(np.int32),
        "sp_colptr": sp_colptr,
        "sp_row": sp_row.astype(np.int32),
        "tileT_ptr": tileT_ptr,
        "tileT_idx": torder.astype(np.int32),
    }


def tile_counts(rowptr, col, T: int, tau_ppm: int):
    """(number of dense tiles, number of remainder edges) of the plan."""
    p = build_tiles(rowptr, col, T, tau_ppm)
    return len(p["tile_col"]), len(p["sp_col"])
