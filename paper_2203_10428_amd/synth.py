"""Seeded synthetic inputs shaped like the paper's partition workloads.

This module only draws random numbers and assembles graphs in compressed
sparse row (CSR) form; it holds none of the method's arithmetic (no
aggregation, no normalisation, no layer maths).  Both the fp64 oracle
(through the tests) and the HIP path consume exactly the arrays produced
here, so a given (workload, seed) pair always yields the same bytes.

Graph model of one partition (Section 3.1 of the paper describes a partition
as inner nodes plus boundary nodes replicated from other partitions):

* nodes ``0 .. n_inner-1`` are owned by partition 0 (the one that is built);
* nodes ``n_inner .. n_inner+pool-1`` form a pool owned by the peer
  partitions ``1 .. nparts-1``; the pool nodes that end up adjacent to an
  inner node become the boundary set;
* every edge has at least one inner endpoint (edges between two pool nodes
  never influence partition 0 and are not generated), except for the Tiny
  workload which is a complete global graph split into two halves.

The returned global graph is symmetric, has no self loops and no duplicate
edges; node ids inside the inner range and inside the pool are randomly
permuted so that degree is not correlated with id (as in real datasets).

Random streams: one ``numpy.random.PCG64`` child stream per array, spawned
from ``SeedSequence(seed)`` in a fixed order, so adding an array never
changes the existing ones.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np


@dataclass
class GlobalGraph:
    """A symmetric global graph in CSR form plus the node -> partition map."""

    n: int                      # global node count
    rowptr: np.ndarray          # int64 [n+1]
    col: np.ndarray             # int32 [nnz]
    owner: np.ndarray           # int32 [n]
    nparts: int
    self_part: int = 0
    stats: dict = field(default_factory=dict)


# ---------------------------------------------------------------------------
# helpers
# ---------------------------------------------------------------------------

def _streams(seed: int, count: int):
    ss = np.random.SeedSequence(seed)
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(count)]


def _csr_from_pairs(n: int, u: np.ndarray, v: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """Symmetrise an undirected edge list, drop self loops and duplicates."""
    u = u.astype(np.int64, copy=False)
    v = v.astype(np.int64, copy=False)
    keep = u != v
    u, v = u[keep], v[keep]
    src = np.concatenate([u, v])
    dst = np.concatenate([v, u])
    key = np.unique(src * n + dst)
    src = key // n
    dst = (key - src * n).astype(np.int32)
    counts = np.bincount(src, minlength=n)
    rowptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(counts, out=rowptr[1:])
    return rowptr, dst


def _power_law_weights(n: int, mean: float, wmax: float, tau: float) -> np.ndarray:
    """Expected-degree sequence w_i = wmax (i/i0 + 1)^(-1/(tau-1)) with mean ``mean``."""
    beta = 1.0 / (tau - 1.0)
    i = np.arange(n, dtype=np.float64)
    lo, hi = 1e-9, 1e9
    for _ in range(200):
        i0 = (lo * hi) ** 0.5
        w = wmax * (i / i0 + 1.0) ** (-beta)
        if w.mean() > mean:
            hi = i0
        else:
            lo = i0
    return wmax * (i / ((lo * hi) ** 0.5) + 1.0) ** (-beta)


def _draw(rng, w: np.ndarray, m: int) -> np.ndarray:
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    r = rng.random(m)
    return np.minimum(np.searchsorted(cdf, r, side="right"), len(w) - 1)


def _owners_local(n_inner: int, pool: int, nparts: int) -> np.ndarray:
    owner = np.zeros(n_inner + pool, dtype=np.int32)
    # pool ids are split into nparts-1 contiguous blocks, one per peer
    owner[n_inner:] = 1 + (np.arange(pool, dtype=np.int64) * (nparts - 1) // max(pool, 1)).astype(np.int32)
    return owner


def _relabel(n_inner: int, pool: int, u, v, rng):
    """Random permutation of ids inside the inner range and inside the pool."""
    perm_in = rng.permutation(n_inner)
    perm_pool = rng.permutation(pool) + n_inner
    perm = np.concatenate([perm_in, perm_pool]).astype(np.int64)
    return perm[u], perm[v]


def _stats(g: GlobalGraph) -> dict:
    inner = np.flatnonzero(g.owner == g.self_part)
    deg = g.rowptr[inner + 1] - g.rowptr[inner]
    # boundary = distinct non-inner neighbours of inner rows
    mask = np.zeros(g.n, dtype=bool)
    starts, ends = g.rowptr[inner], g.rowptr[inner + 1]
    idx = _ranges(starts, ends)
    cols = g.col[idx]
    nonin = cols[g.owner[cols] != g.self_part]
    mask[nonin] = True
    return {
        "n_inner": int(len(inner)),
        "n_boundary": int(mask.sum()),
        "nnz_with_self_loops": int(deg.sum() + len(inner)),
        "mean_row_len": float((deg + 1).mean()) if len(inner) else 0.0,
        "max_row_len": int((deg + 1).max()) if len(inner) else 0,
    }


def _ranges(starts: np.ndarray, ends: np.ndarray) -> np.ndarray:
    lens = (ends - starts).astype(np.int64)
    total = int(lens.sum())
    if total == 0:
        return np.zeros(0, dtype=np.int64)
    offs = np.repeat(starts - np.concatenate([[0], np.cumsum(lens)[:-1]]), lens)
    return np.arange(total, dtype=np.int64) + offs


# ---------------------------------------------------------------------------
# graph generators
# ---------------------------------------------------------------------------

def tiny_uniform(n: int = 2000, pairs: int = 10000, nparts: int = 2, seed: int = 0) -> GlobalGraph:
    """Uniform random global graph split into ``nparts`` id ranges."""
    (rg,) = _streams(seed, 1)
    u = rg.integers(0, n, size=pairs)
    v = rg.integers(0, n - 1, size=pairs)
    v = v + (v >= u)                       # u != v by construction
    rowptr, col = _csr_from_pairs(n, u, v)
    owner = (np.arange(n, dtype=np.int64) * nparts // n).astype(np.int32)
    g = GlobalGraph(n, rowptr, col, owner, nparts, 0)
    g.stats = _stats(g)
    return g


def chung_lu_partition(n_inner: int, pool: int, nparts: int, mean_row: float, max_deg: float,
                       tau: float, frac_inner: float, seed: int, oversample: float = 1.0) -> GlobalGraph:
    """Power-law (Chung-Lu) partition: inner + pool, every edge touches an inner node.

    ``mean_row`` is the target mean row length of the partition's propagation
    matrix (degree + 1); ``frac_inner`` is the share of inner-node edge
    endpoints that land on other inner nodes.
    """
    rg_w, rg_e, rg_p = _streams(seed, 3)
    w_in = _power_law_weights(n_inner, mean_row - 1.0, max_deg, tau)
    w_pool = _power_law_weights(pool, (mean_row - 1.0) * n_inner * (1 - frac_inner) / pool,
                                max_deg * 0.5, tau)
    total = n_inner * (mean_row - 1.0) * oversample
    m_ii = int(round(total * frac_inner / 2.0))
    m_ib = int(round(total * (1.0 - frac_inner)))
    u = np.concatenate([_draw(rg_e, w_in, m_ii), _draw(rg_e, w_in, m_ib)])
    v = np.concatenate([_draw(rg_e, w_in, m_ii), n_inner + _draw(rg_e, w_pool, m_ib)])
    u, v = _relabel(n_inner, pool, u, v, rg_p)
    n = n_inner + pool
    rowptr, col = _csr_from_pairs(n, u, v)
    g = GlobalGraph(n, rowptr, col, _owners_local(n_inner, pool, nparts), nparts, 0)
    g.stats = _stats(g)
    return g


def er_hubs_partition(n_inner: int, pool: int, nparts: int, mean_row: float, hub_deg: int,
                      hub_share: float, frac_inner: float, seed: int) -> GlobalGraph:
    """Erdos-Renyi partition plus hub nodes that carry ``hub_share`` of the endpoints."""
    rg_e, rg_h, rg_p = _streams(seed, 3)
    total = n_inner * (mean_row - 1.0)
    hub_endpoints = hub_share * total
    n_hub = max(1, int(round(hub_endpoints / hub_deg)))
    er_total = total - n_hub * hub_deg
    m_ii = int(round(er_total * frac_inner / 2.0))
    m_ib = int(round(er_total * (1.0 - frac_inner)))
    u = [rg_e.integers(0, n_inner, m_ii), rg_e.integers(0, n_inner, m_ib)]
    v = [rg_e.integers(0, n_inner, m_ii), n_inner + rg_e.integers(0, pool, m_ib)]
    hubs = rg_h.choice(n_inner, size=n_hub, replace=False)
    hu = np.repeat(hubs, hub_deg)
    to_inner = rg_h.random(len(hu)) < frac_inner
    hv = np.where(to_inner, rg_h.integers(0, n_inner, len(hu)), n_inner + rg_h.integers(0, pool, len(hu)))
    u.append(hu)
    v.append(hv)
    u = np.concatenate(u)
    v = np.concatenate(v)
    u, v = _relabel(n_inner, pool, u, v, rg_p)
    n = n_inner + pool
    rowptr, col = _csr_from_pairs(n, u, v)
    g = GlobalGraph(n, rowptr, col, _owners_local(n_inner, pool, nparts), nparts, 0)
    g.stats = _stats(g)
    g.stats["n_hubs"] = int(n_hub)
    return g


def _rmat_ids(rng, m: int, scale: int, a: float, b: float, c: float):
    """Recursive-matrix (R-MAT) edge coordinates, one quadrant draw per bit."""
    u = np.zeros(m, dtype=np.int64)
    v = np.zeros(m, dtype=np.int64)
    ab, abc = a + b, a + b + c
    for _ in range(scale):
        r = rng.random(m, dtype=np.float32)
        ubit = r >= ab                      # quadrants c, d
        vbit = ((r >= a) & (r < ab)) | (r >= abc)   # quadrants b, d
        u = (u << 1) | ubit
        v = (v << 1) | vbit
    return u, v


def rmat_partition(n_inner: int, pool_scale: int, nparts: int, mean_row: float,
                   frac_inner: float, seed: int, abcd=(0.57, 0.19, 0.19, 0.05),
                   oversample: float = 1.0) -> GlobalGraph:
    """R-MAT partition: inner-inner and inner-pool edges from R-MAT coordinates."""
    rg_e, rg_p = _streams(seed, 2)
    a, b, c, _ = abcd
    scale_in = int(np.ceil(np.log2(n_inner)))
    pool = 1 << pool_scale
    total = n_inner * (mean_row - 1.0) * oversample
    m_ii = int(round(total * frac_inner / 2.0))
    m_ib = int(round(total * (1.0 - frac_inner)))
    u1, v1 = _rmat_ids(rg_e, m_ii, scale_in, a, b, c)
    u2, v2 = _rmat_ids(rg_e, m_ib, max(scale_in, pool_scale), a, b, c)
    u2 = u2 >> max(0, pool_scale - scale_in)
    v2 = v2 >> max(0, scale_in - pool_scale)
    keep1 = (u1 < n_inner) & (v1 < n_inner)
    keep2 = u2 < n_inner
    u = np.concatenate([u1[keep1], u2[keep2]])
    v = np.concatenate([v1[keep1], n_inner + v2[keep2]])
    u, v = _relabel(n_inner, pool, u, v, rg_p)
    n = n_inner + pool
    rowptr, col = _csr_from_pairs(n, u, v)
    g = GlobalGraph(n, rowptr, col, _owners_local(n_inner, pool, nparts), nparts, 0)
    g.stats = _stats(g)
    return g


# ---------------------------------------------------------------------------
# dense inputs
# ---------------------------------------------------------------------------

def features(rng, rows: int, cols: int) -> np.ndarray:
    return rng.standard_normal((rows, cols), dtype=np.float32)


def glorot_uniform(rng, f_in: int, f_out: int) -> np.ndarray:
    a = np.sqrt(6.0 / (f_in + f_out))
    return rng.uniform(-a, a, size=(f_in, f_out)).astype(np.float32)


def labels_single(rng, rows: int, classes: int) -> np.ndarray:
    return rng.integers(0, classes, size=rows).astype(np.int32)


def labels_multi(rng, rows: int, classes: int, p: float = 0.05) -> np.ndarray:
    return (rng.random((rows, classes)) < p).astype(np.float32)


def dense_streams(seed: int, count: int):
    """Child streams for dense arrays, disjoint from the graph streams."""
    return _streams(seed + 0x5EED, count)
