"""Partition set-up of Algorithm 1, in plain NumPy (integers only).

Definitions followed (Algorithm 1's set-up block and Section 3.1):

* inner set   V_i = nodes owned by partition i;
* boundary    B_i = nodes not in V_i that are neighbours of a node in V_i;
* send sets   S_{i,j} = B_j ∩ V_i  (rows partition i sends to partition j);
* receive     S_{j,i} = B_i ∩ V_j  (the owner-j block of B_i);
* the local propagation matrix P_i keeps the inner rows of the row-normalised
  D̃⁻¹(A + I) and the columns of V_i ∪ B_i (Appendix A.1 splits P into
  P_in + P_bd; here both halves are columns of one matrix);
* for the GraphSAGE layer (Section 2: the update takes CONCAT(z_v, h_v) with
  z_v aggregated over N(v)) the matrix is the mean over N(v) alone,
  D⁻¹A, with no self loop (``self_loop=False``); a row without neighbours
  is zero.

Canonical numbering (the papers leaves numbering open; this one makes the
C++ builder's output comparable bit for bit):

* inner local id   = rank of the global id among the nodes with owner i;
* boundary local id = n_inner + rank by (owner, global id);
* CSR columns ascending by local id, duplicates removed, one self loop per
  inner row (none with ``self_loop=False``);
* the transpose CSR has rows 0 .. n_inner+n_bd-1, columns ascending;
* the concatenated send list holds S_{i,j} for ascending j, each ascending by
  global id (equal to ascending local id);
* the inverse send map lists, per inner row u, the positions k of the send
  list with send[k] == u, ascending.

Symmetric normalisation (the D̃^{-1/2} Ã D̃^{-1/2} of the paper's appendix,
``norm="sym"`` in ``propagation_matrix``): entry (v, u) of P_i is
1 / sqrt(d̃_v d̃_u) with d̃ = degree + 1 of the whole graph, so the degrees of
the boundary nodes (``deg``) come from their full neighbourhoods, not only
from the edges to partition i.

Pinned by: a pure-Python brute force from the dense adjacency (tests).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass
class Partition:
    part: int
    nparts: int
    inner_gid: np.ndarray      # int64 [n]
    bd_gid: np.ndarray         # int64 [b]
    bd_owner: np.ndarray       # int32 [b]
    recv_ptr: np.ndarray       # int64 [nparts+1]  boundary rows owned by j: [recv_ptr[j], recv_ptr[j+1])
    rowptr: np.ndarray         # int64 [n+1]   CSR of P_i (pattern; values are 1/row length)
    col: np.ndarray            # int32 [nnz]
    rowptr_t: np.ndarray       # int64 [n+b+1] CSR of P_iᵀ (pattern)
    col_t: np.ndarray          # int32 [nnz]
    send_ptr: np.ndarray       # int64 [nparts+1]
    send_idx: np.ndarray       # int32 [s]  inner local ids, S_{i,0} .. S_{i,nparts-1}
    inv_ptr: np.ndarray        # int64 [n+1]
    inv_k: np.ndarray          # int32 [s]
    deg: np.ndarray            # int64 [n+b]  whole-graph degree + 1 of every local node

    @property
    def n_inner(self) -> int:
        return len(self.inner_gid)

    @property
    def n_bd(self) -> int:
        return len(self.bd_gid)

    @property
    def nnz(self) -> int:
        return len(self.col)

    @property
    def row_len(self) -> np.ndarray:
        return np.diff(self.rowptr)


def _row_pairs(rowptr: np.ndarray, col: np.ndarray, rows: np.ndarray):
    """(row, neighbour) pairs of the given global rows, self loops and duplicates removed."""
    starts = rowptr[rows]
    lens = rowptr[rows + 1] - starts
    total = int(lens.sum())
    r = np.repeat(rows.astype(np.int64), lens)
    if total:
        offs = np.repeat(starts - np.concatenate([[0], np.cumsum(lens)[:-1]]), lens)
        c = col[np.arange(total, dtype=np.int64) + offs].astype(np.int64)
    else:
        c = np.zeros(0, dtype=np.int64)
    keep = r != c
    return r[keep], c[keep]


def _csr(nrows: int, r: np.ndarray, c: np.ndarray):
    """CSR with columns ascending inside each row; (r, c) pairs must be unique."""
    order = np.lexsort((c, r))
    r, c = r[order], c[order]
    rowptr = np.zeros(nrows + 1, dtype=np.int64)
    np.cumsum(np.bincount(r, minlength=nrows), out=rowptr[1:])
    return rowptr, c.astype(np.int32)


def build_partition(n: int, rowptr: np.ndarray, col: np.ndarray, owner: np.ndarray,
                    part: int, nparts: int, self_loop: bool = True) -> Partition:
    rowptr = np.asarray(rowptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    owner = np.asarray(owner, dtype=np.int64)

    # V_i: nodes owned by partition i, local id = rank of global id
    inner_gid = np.flatnonzero(owner == part).astype(np.int64)
    n_in = len(inner_gid)
    local_of = np.full(n, -1, dtype=np.int64)
    local_of[inner_gid] = np.arange(n_in)

    # N(v) for v in V_i (deduplicated, self loops dropped)
    r, c = _row_pairs(rowptr, col, inner_gid)
    key = np.unique(r * n + c)
    r, c = key // n, key % n

    # B_i: non-inner neighbours of inner nodes, ordered by (owner, global id)
    nb = np.unique(c[owner[c] != part])
    order = np.lexsort((nb, owner[nb]))
    bd_gid = nb[order]
    bd_owner = owner[bd_gid].astype(np.int32)
    local_of[bd_gid] = n_in + np.arange(len(bd_gid))
    recv_ptr = np.zeros(nparts + 1, dtype=np.int64)
    np.cumsum(np.bincount(bd_owner, minlength=nparts), out=recv_ptr[1:])

    # P_i pattern: N(v) ∪ {v} for inner v (N(v) alone without self loops), in local ids
    diag = np.arange(n_in) if self_loop else np.zeros(0, dtype=np.int64)
    lr = np.concatenate([local_of[r], diag])
    lc = np.concatenate([local_of[c], diag])
    p_rowptr, p_col = _csr(n_in, lr, lc)
    # P_iᵀ pattern
    t_rowptr, t_col = _csr(n_in + len(bd_gid), lc, lr)

    # S_{i,j} = B_j ∩ V_i: inner u with a neighbour w owned by j (w's row lists u)
    send_parts = []
    for j in range(nparts):
        if j == part:
            send_parts.append(np.zeros(0, dtype=np.int64))
            continue
        vj = np.flatnonzero(owner == j)
        rj, cj = _row_pairs(rowptr, col, vj)
        bj = np.unique(cj[owner[cj] == part])          # B_j ∩ V_i, ascending global id
        send_parts.append(local_of[bj])
    send_ptr = np.zeros(nparts + 1, dtype=np.int64)
    np.cumsum([len(s) for s in send_parts], out=send_ptr[1:])
    send_idx = np.concatenate(send_parts).astype(np.int32) if send_ptr[-1] else np.zeros(0, np.int32)

    # inverse send map: for each inner u, positions k with send_idx[k] == u, ascending k
    k = np.arange(len(send_idx), dtype=np.int64)
    o = np.lexsort((k, send_idx))
    inv_k = k[o].astype(np.int32)
    inv_ptr = np.zeros(n_in + 1, dtype=np.int64)
    np.cumsum(np.bincount(send_idx, minlength=n_in), out=inv_ptr[1:])

    # whole-graph degree + 1 of the inner and boundary nodes (distinct neighbours, no self loop)
    loc_gid = np.concatenate([inner_gid, bd_gid])
    rr, cc = _row_pairs(rowptr, col, loc_gid)
    rr = np.unique(rr * n + cc) // n
    deg = np.bincount(np.searchsorted(np.sort(loc_gid), rr), minlength=len(loc_gid))
    deg = deg[np.argsort(np.argsort(loc_gid))].astype(np.int64) + 1

    return Partition(part, nparts, inner_gid, bd_gid, bd_owner, recv_ptr,
                     p_rowptr, p_col, t_rowptr, t_col, send_ptr, send_idx, inv_ptr, inv_k, deg)


def propagation_matrix(p: Partition, norm: str = "mean"):
    """P_i as a SciPy CSR matrix.  ``mean``: entries 1/d_v with d_v the row length (degree + 1,
    or the degree without self loops).  ``sym``: entries 1/sqrt(d̃_v d̃_u), d̃ = whole-graph
    degree + 1 (self loops required)."""
    import scipy.sparse as sp
    d = np.diff(p.rowptr)
    if norm == "sym":
        assert np.array_equal(d, p.deg[: p.n_inner]), "symmetric normalisation needs the self loops"
        rows = np.repeat(np.arange(p.n_inner), d)
        vals = 1.0 / np.sqrt(p.deg[rows].astype(np.float64) * p.deg[p.col].astype(np.float64))
    else:
        assert norm == "mean", norm
        inv = np.zeros(len(d))
        inv[d > 0] = 1.0 / d[d > 0]
        vals = np.repeat(inv, d)
    return sp.csr_matrix((vals, p.col.astype(np.int64), p.rowptr),
                         shape=(p.n_inner, p.n_inner + p.n_bd))
