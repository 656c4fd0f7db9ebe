"""Pins of the oracle's symmetric normalisation, P = D̃^{-1/2} (A + I) D̃^{-1/2}
(the normalisation of the paper's appendix), against what fixes it
independently of the oracle's code:

* every partition's P_i equals the rows of the dense symmetric-normalised
  adjacency of the whole graph, built here from the edge list;
* the matrix assembled from all partitions' rows is symmetric and has
  sqrt(d̃) as an eigenvector of eigenvalue 1 (closed form), which fails if a
  boundary node's degree is counted from the partition's edges only;
* vanilla training with it equals dense full-graph GCN with that matrix, in
  both associations of the layer product, and one partition makes PipeGCN
  equal to vanilla;
* central finite differences of the partition-local loss match its gradients.
"""
import numpy as np
import pytest

from oracle import layers
from oracle.partition import build_partition, propagation_matrix
from oracle.pipegcn import Options, run
from test_oracle_pins import SMALL_GRAPHS, assemble, tiny_problem
from test_oracle_transform_pins import local_loss_and_grads


def dense_sym(n, rowptr, col):
    A = np.zeros((n, n))
    for v in range(n):
        for k in range(rowptr[v], rowptr[v + 1]):
            if col[k] != v:
                A[v, col[k]] = 1.0
    A = np.maximum(A, A.T) + np.eye(n)
    d = A.sum(1)
    return A / np.sqrt(np.outer(d, d)), d


@pytest.mark.parametrize("gi", range(len(SMALL_GRAPHS)))
def test_sym_matrix_is_dense_symmetric_adjacency(gi):
    n, rowptr, col, owner = SMALL_GRAPHS[gi]
    nparts = int(owner.max()) + 1
    P_full, d = dense_sym(n, rowptr, col)
    for i in range(nparts):
        p = build_partition(n, rowptr, col, owner, i, nparts)
        gids = np.concatenate([p.inner_gid, p.bd_gid])
        assert np.array_equal(p.deg, d[gids].astype(np.int64))
        P = propagation_matrix(p, "sym").toarray()
        assert np.allclose(P, P_full[np.ix_(p.inner_gid, gids)], rtol=0, atol=1e-15)
        # rows of P_full outside V_i ∪ B_i are zero for inner rows
        rest = np.setdiff1d(np.arange(n), gids)
        assert not P_full[np.ix_(p.inner_gid, rest)].any()


@pytest.mark.parametrize("gi", range(len(SMALL_GRAPHS)))
def test_assembled_sym_matrix_closed_form(gi):
    n, rowptr, col, owner = SMALL_GRAPHS[gi]
    nparts = int(owner.max()) + 1
    M = np.zeros((n, n))
    deg = np.zeros(n)
    for i in range(nparts):
        p = build_partition(n, rowptr, col, owner, i, nparts)
        gids = np.concatenate([p.inner_gid, p.bd_gid])
        M[np.ix_(p.inner_gid, gids)] = propagation_matrix(p, "sym").toarray()
        deg[p.inner_gid] = p.deg[: p.n_inner]
    assert np.allclose(M, M.T, atol=1e-15)
    s = np.sqrt(deg)
    assert np.allclose(M @ s, s, rtol=1e-13)


def dense_full_graph_sym(n, rowptr, col, X, labels, W, T, eta, scale):
    P, _ = dense_sym(n, rowptr, col)
    W = [w.astype(float).copy() for w in W]
    out = []
    for _ in range(T):
        H = X.astype(float)
        As, Zs, Hs = [], [], []
        for l, w in enumerate(W):
            A = P @ H
            Z = A @ w
            H = np.maximum(Z, 0) if l < len(W) - 1 else Z
            As.append(A); Zs.append(Z); Hs.append(H)
        val, J = layers.softmax_ce(H, labels, scale)
        G = [None] * len(W)
        for l in range(len(W) - 1, -1, -1):
            M = J * (Zs[l] > 0) if l < len(W) - 1 else J
            G[l] = As[l].T @ M
            J = P.T @ (M @ W[l].T)
        out.append(dict(loss=val, H=Hs, G=G))
        W = [w - eta * g for w, g in zip(W, G)]
    return out, W


@pytest.mark.parametrize("order", ["agg", "transform"])
@pytest.mark.parametrize("gi", [0, 2, 3])
def test_sym_vanilla_equals_dense_full_graph(gi, order):
    n, rowptr, col, owner = SMALL_GRAPHS[gi]
    nparts = int(owner.max()) + 1
    widths = [6, 5, 4, 3]
    X, W, y = tiny_problem((n, rowptr, col, owner), widths)
    opts = Options(mode="vanilla", eta=0.3, loss_scale=1.0 / n, norm="sym", order=order)
    sim, recs = run(n, rowptr, col, owner, nparts, X, y, W, 3, opts)
    ref, W_ref = dense_full_graph_sym(n, rowptr, col, X, y, W, 3, 0.3, 1.0 / n)
    for t in range(3):
        assert np.isclose(sum(r["loss"] for r in recs[t]), ref[t]["loss"], rtol=1e-12)
        for l in range(1, 4):
            assert np.allclose(assemble(sim, recs[t], "H", l), ref[t]["H"][l - 1], atol=1e-12)
            assert np.allclose(recs[t][0]["G_sum"][l - 1], ref[t]["G"][l - 1], atol=1e-12)
    for w, wr in zip(sim.W, W_ref):
        assert np.allclose(w, wr, atol=1e-12)


def test_sym_single_partition_pipe_equals_vanilla():
    n, rowptr, col, _ = SMALL_GRAPHS[2]
    owner = np.zeros(n, np.int32)
    X, W, y = tiny_problem((n, rowptr, col, owner), [4, 6, 3])
    a = run(n, rowptr, col, owner, 1, X, y, W, 4,
            Options(mode="pipe", smooth_f=True, smooth_g=True, eta=0.2, norm="sym"))[1]
    b = run(n, rowptr, col, owner, 1, X, y, W, 4, Options(mode="vanilla", eta=0.2, norm="sym"))[1]
    for ra, rb in zip(a, b):
        assert np.isclose(ra[0]["loss"], rb[0]["loss"], rtol=1e-13)


@pytest.mark.parametrize("order", ["agg", "transform"])
def test_sym_gradients_match_finite_differences(order):
    n, rowptr, col, owner = SMALL_GRAPHS[0]
    p = build_partition(n, rowptr, col, owner, 0, 3)
    P = propagation_matrix(p, "sym")
    rng = np.random.default_rng(31)
    widths = [5, 3, 4, 2]
    X_in = rng.standard_normal((p.n_inner, widths[0]))
    Hbd = [rng.standard_normal((p.n_bd, widths[l])) for l in range(3)]
    W = [rng.standard_normal((widths[l], widths[l + 1])) * 0.7 for l in range(3)]
    y = rng.integers(0, widths[-1], p.n_inner)
    _, G, Jbd = local_loss_and_grads(p, P, X_in, Hbd, W, y, 0.29, order)
    eps = 1e-6

    def f(W_, Hbd_):
        return local_loss_and_grads(p, P, X_in, Hbd_, W_, y, 0.29, order)[0]

    for l in range(3):
        for (a, b) in [(0, 0), (widths[l] - 1, widths[l + 1] - 1)]:
            Wp = [w.copy() for w in W]; Wm = [w.copy() for w in W]
            Wp[l][a, b] += eps; Wm[l][a, b] -= eps
            fd = (f(Wp, Hbd) - f(Wm, Hbd)) / (2 * eps)
            assert abs(fd - G[l][a, b]) <= 1e-7 * max(1.0, abs(fd))
        for (r, c) in [(0, 0), (p.n_bd - 1, widths[l] - 1)]:
            Hp = [h.copy() for h in Hbd]; Hm = [h.copy() for h in Hbd]
            Hp[l][r, c] += eps; Hm[l][r, c] -= eps
            fd = (f(W, Hp) - f(W, Hm)) / (2 * eps)
            assert abs(fd - Jbd[l][r, c]) <= 1e-7 * max(1.0, abs(fd))
