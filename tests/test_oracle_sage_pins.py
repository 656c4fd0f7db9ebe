"""Pins of the oracle's GraphSAGE layer, dropout and Adam (the paper's experiment model).

Nothing here retypes an oracle formula to compare it with itself:

* Philox4x32-10 reproduces the published known-answer vectors of its
  authors (counter, key -> output);
* the dropout mask drops the requested fraction of elements (binomial
  bounds), scales the kept ones by 1/(1-p), and is a pure function of
  (seed, partition, layer, iteration, element);
* the no-self-loop local matrix is the dense row-normalised adjacency D⁻¹A
  of the whole graph, restricted to the partition's rows and columns;
* the layer gradients (with dropout masks held fixed) are central finite
  differences of the partition-local loss, both for a stack composed here
  and for the oracle's per-partition step itself (gradient of the received
  boundary rows included);
* vanilla partition-parallel GraphSAGE reproduces dense full-graph
  GraphSAGE (Section 2's CONCAT update) and one partition makes both modes
  equal;
* Adam equals torch.optim.Adam on the same gradient sequence.
"""
import numpy as np
import pytest

from oracle import layers
from oracle.partition import build_partition, propagation_matrix
from oracle.philox import drop_threshold, dropout_mask, dropout_mask_rows, philox4x32_10
from oracle.pipegcn import Options, partition_step, run
from paper_2203_10428_amd import synth
from test_oracle_pins import SMALL_GRAPHS, assemble, tiny_problem


# published known-answer vectors of Philox4x32-10: (counter, key) -> output
KAT = [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2, (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


@pytest.mark.parametrize("ctr,key,out", KAT)
def test_philox_known_answers(ctr, key, out):
    got = philox4x32_10(np.array([ctr], dtype=np.uint64), key)[0]
    assert tuple(int(x) for x in got) == out


@pytest.mark.parametrize("p", [0.1, 0.3, 0.5])
def test_dropout_mask_statistics(p):
    rows, cols = 700, 150
    m = dropout_mask(rows, cols, p, seed=7, part=1, layer=2, iteration=5)
    assert set(np.unique(m)) <= {0.0, 1.0 / (1.0 - p)}
    N = rows * cols
    dropped = (m == 0).sum()
    assert abs(dropped - p * N) < 5 * np.sqrt(N * p * (1 - p)), (dropped, p * N)
    # a pure function of its arguments; rows can be drawn on their own
    assert np.array_equal(m, dropout_mask(rows, cols, p, 7, 1, 2, 5))
    ids = np.array([0, 3, 699, 350])
    assert np.array_equal(dropout_mask_rows(ids, cols, p, 7, 1, 2, 5), m[ids])
    for other in [dict(seed=8, part=1, layer=2, iteration=5), dict(seed=7, part=0, layer=2, iteration=5),
                  dict(seed=7, part=1, layer=3, iteration=5), dict(seed=7, part=1, layer=2, iteration=6)]:
        m2 = dropout_mask(rows, cols, p, **other)
        assert 0.3 * N * 2 * p * (1 - p) < (m2 != m).sum(), other     # about 2p(1-p) N differ


def test_dropout_threshold_and_identity():
    assert drop_threshold(0.5) == 1 << 31
    assert drop_threshold(0.0) == 0
    assert np.array_equal(dropout_mask(5, 3, 0.0, 1, 0, 1, 1), np.ones((5, 3)))


def dense_mean_no_self(n, rowptr, col):
    """D⁻¹A of the whole graph (no self loops; rows without neighbours are zero), dense."""
    A = np.zeros((n, n))
    for v in range(n):
        for k in range(rowptr[v], rowptr[v + 1]):
            A[v, col[k]] = 1.0
    np.fill_diagonal(A, 0.0)
    d = A.sum(axis=1, keepdims=True)
    return np.divide(A, d, out=np.zeros_like(A), where=d > 0)


@pytest.mark.parametrize("gi", range(len(SMALL_GRAPHS)))
def test_sage_matrix_is_dense_mean_adjacency(gi):
    n, rowptr, col, owner = SMALL_GRAPHS[gi]
    nparts = int(owner.max()) + 1
    D = dense_mean_no_self(n, rowptr, col)
    for i in range(nparts):
        p = build_partition(n, rowptr, col, owner, i, nparts, self_loop=False)
        q = build_partition(n, rowptr, col, owner, i, nparts)
        for a in ("inner_gid", "bd_gid", "send_idx", "send_ptr", "recv_ptr", "inv_ptr", "inv_k"):
            assert np.array_equal(getattr(p, a), getattr(q, a)), a          # same sets, other matrix
        P = propagation_matrix(p).toarray()
        gids = np.concatenate([p.inner_gid, p.bd_gid])
        assert np.allclose(P, D[np.ix_(p.inner_gid, gids)], atol=1e-15)
        assert np.allclose(D[p.inner_gid].sum(axis=1), P.sum(axis=1))     # no neighbour outside


def sage_local_loss(p, P, X_in, Hbd, masks, W, y, scale):
    """Partition-local loss of a GraphSAGE stack with dropout masks held fixed, and its gradients."""
    L = len(W)
    H = X_in
    cache = []
    for l in range(L):
        X = np.vstack([H, Hbd[l]]) * masks[l]
        z, Z, Hn = layers.sage_forward(P, X, p.n_inner, W[l], l < L - 1)
        cache.append((z, X[: p.n_inner], Z))
        H = Hn
    val, J = layers.softmax_ce(H, y, scale)
    G, Jbd = [None] * L, [None] * L
    for l in range(L - 1, -1, -1):
        z, Xi, Z = cache[l]
        G[l], Jf = layers.sage_backward(P, z, Xi, Z, J, W[l], l < L - 1, True)
        Jf = Jf * masks[l]
        Jbd[l] = Jf[p.n_inner:]
        J = Jf[: p.n_inner]
    return val, G, Jbd


@pytest.mark.parametrize("gi,p_drop", [(0, 0.0), (0, 0.4), (3, 0.25)])
def test_sage_gradients_match_finite_differences(gi, p_drop):
    n, rowptr, col, owner = SMALL_GRAPHS[gi]
    nparts = int(owner.max()) + 1
    p = build_partition(n, rowptr, col, owner, 0, nparts, self_loop=False)
    P = propagation_matrix(p)
    rng = np.random.default_rng(5)
    widths = [5, 6, 4, 3]
    X_in = rng.standard_normal((p.n_inner, widths[0]))
    Hbd = [rng.standard_normal((p.n_bd, widths[l])) for l in range(3)]
    W = [rng.standard_normal((2 * widths[l], widths[l + 1])) * 0.6 for l in range(3)]
    masks = [dropout_mask(p.n_inner + p.n_bd, widths[l], p_drop, 3, 0, l + 1, 2) for l in range(3)]
    y = rng.integers(0, widths[-1], p.n_inner)
    _, G, Jbd = sage_local_loss(p, P, X_in, Hbd, masks, W, y, 0.41)
    eps = 1e-6

    def f(W_, Hbd_):
        return sage_local_loss(p, P, X_in, Hbd_, masks, W_, y, 0.41)[0]

    for l in range(3):
        for (a, b) in [(0, 0), (2 * widths[l] - 1, widths[l + 1] - 1), (widths[l], 1), (1, 2)]:
            Wp = [w.copy() for w in W]; Wm = [w.copy() for w in W]
            Wp[l][a, b] += eps; Wm[l][a, b] -= eps
            fd = (f(Wp, Hbd) - f(Wm, Hbd)) / (2 * eps)
            assert abs(fd - G[l][a, b]) <= 1e-7 * max(1.0, abs(fd)), (l, a, b, fd, G[l][a, b])
        for (r, c) in [(0, 0), (p.n_bd - 1, widths[l] - 1), (p.n_bd // 2, 1)]:
            Hp = [h.copy() for h in Hbd]; Hm = [h.copy() for h in Hbd]
            Hp[l][r, c] += eps; Hm[l][r, c] -= eps
            fd = (f(W, Hp) - f(W, Hm)) / (2 * eps)
            assert abs(fd - Jbd[l][r, c]) <= 1e-7 * max(1.0, abs(fd)), (l, r, c, fd, Jbd[l][r, c])


def dense_full_graph_sage(n, rowptr, col, X, labels, W, T, eta, scale):
    """Full-graph GraphSAGE (CONCAT update, mean over N(v)) with a dense matrix and SGD."""
    P = dense_mean_no_self(n, rowptr, col)
    W = [w.astype(float).copy() for w in W]
    out = []
    for _ in range(T):
        H = X.astype(float)
        Xs, Zs, Hs = [], [], []
        for l, w in enumerate(W):
            Xc = np.hstack([P @ H, H])
            Z = Xc @ w
            Xs.append((Xc, H.shape[1])); Zs.append(Z)
            H = np.maximum(Z, 0) if l < len(W) - 1 else Z
            Hs.append(H)
        val, J = layers.softmax_ce(H, labels, scale)
        G = [None] * len(W)
        for l in range(len(W) - 1, -1, -1):
            M = J * (Zs[l] > 0) if l < len(W) - 1 else J
            Xc, f = Xs[l]
            G[l] = Xc.T @ M
            dX = M @ W[l].T
            J = P.T @ dX[:, :f] + dX[:, f:]
        out.append(dict(loss=val, H=Hs, G=G))
        W = [w - eta * g for w, g in zip(W, G)]
    return out, W


def sage_problem(graph, widths, seed=0):
    X, W, y = tiny_problem(graph, widths, seed=seed)
    rng = np.random.default_rng(seed + 100)
    W = [rng.uniform(-0.5, 0.5, (2 * widths[l], widths[l + 1])) for l in range(len(widths) - 1)]
    return X, W, y


@pytest.mark.parametrize("gi", [0, 3, "tiny"])
def test_sage_vanilla_equals_dense_full_graph(gi):
    if gi == "tiny":
        g = synth.tiny_uniform()
        graph = (g.n, g.rowptr, g.col, g.owner)
    else:
        graph = SMALL_GRAPHS[gi]
    n, rowptr, col, owner = graph
    nparts = int(owner.max()) + 1
    widths = [6, 5, 4, 3]
    X, W, y = sage_problem(graph, widths)
    opts = Options(mode="vanilla", model="sage", eta=0.3, loss_scale=1.0 / n)
    sim, recs = run(n, rowptr, col, owner, nparts, X, y, W, 3, opts)
    ref, W_ref = dense_full_graph_sage(n, rowptr, col, X, y, W, 3, 0.3, 1.0 / n)
    for t in range(3):
        assert np.isclose(sum(r["loss"] for r in recs[t]), ref[t]["loss"], rtol=1e-12)
        for l in range(1, 4):
            assert np.allclose(assemble(sim, recs[t], "H", l), ref[t]["H"][l - 1], atol=1e-12)
            assert np.allclose(recs[t][0]["G_sum"][l - 1], ref[t]["G"][l - 1], atol=1e-12)
    for w, wr in zip(sim.W, W_ref):
        assert np.allclose(w, wr, atol=1e-12)


def test_sage_single_partition_pipe_equals_vanilla():
    n, rowptr, col, _ = SMALL_GRAPHS[2]
    owner = np.zeros(n, np.int32)
    widths = [4, 6, 3]
    X, W, y = sage_problem((n, rowptr, col, owner), widths)
    kw = dict(model="sage", dropout=0.3, seed=4, optimizer="adam", eta=0.01)
    a = run(n, rowptr, col, owner, 1, X, y, W, 4, Options(mode="pipe", smooth_f=True, smooth_g=True, **kw))[1]
    b = run(n, rowptr, col, owner, 1, X, y, W, 4, Options(mode="vanilla", **kw))[1]
    for ra, rb in zip(a, b):
        assert np.isclose(ra[0]["loss"], rb[0]["loss"], rtol=1e-13)
        for wa, wb in zip(ra[0]["W_out"], rb[0]["W_out"]):
            assert np.allclose(wa, wb, atol=1e-14)


def test_adam_matches_torch():
    import torch
    rng = np.random.default_rng(9)
    W0 = rng.standard_normal((7, 5))
    grads = [rng.standard_normal((7, 5)) * s for s in (1.0, 0.1, 3.0, 0.01, 1.0)]
    w = torch.tensor(W0.copy(), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([w], lr=0.003, betas=(0.9, 0.999), eps=1e-8)
    W, m, v = W0.copy(), np.zeros_like(W0), np.zeros_like(W0)
    for t, g in enumerate(grads, start=1):
        w.grad = torch.tensor(g)
        opt.step()
        W, m, v = layers.adam(W, g, m, v, t, 0.003)
        assert np.allclose(W, w.detach().numpy(), rtol=0, atol=1e-15)


@pytest.mark.parametrize("model,p_drop", [("sage", 0.3), ("gcn", 0.2), ("sage", 0.0)])
def test_partition_step_matches_simulation_with_dropout(model, p_drop):
    g = synth.tiny_uniform()
    n, rowptr, col, owner = g.n, g.rowptr, g.col, g.owner
    widths = [5, 4, 3]
    X, W, y = sage_problem((n, rowptr, col, owner), widths) if model == "sage" else \
        tiny_problem((n, rowptr, col, owner), widths)
    opts = Options(model=model, dropout=p_drop, seed=11, smooth_f=True, smooth_g=True, gamma=0.9, eta=0.01,
                   optimizer="adam", loss_scale=1.0 / n)
    sim, recs = run(n, rowptr, col, owner, 2, X, y, W, 4, opts)
    p, P = sim.parts[0], sim.P[0]
    for t in range(1, 5):
        r = recs[t - 1][0]
        si = r["state_in"]
        ema_f = {k: v.copy() for k, v in si.ema_f.items()}
        ema_g = {k: v.copy() for k, v in si.ema_g.items()}
        out = partition_step(p, P, X[p.inner_gid], y[p.inner_gid], r["W_in"], si.feat_buf, si.grad_buf,
                             ema_f, ema_g, t, opts)
        assert np.isclose(out["loss"], r["loss"], rtol=1e-14)
        for l in (1, 2):
            assert np.array_equal(out["H"][l], r["H"][l])
            assert np.array_equal(out["G"][l], r["G"][l])
            assert np.array_equal(out["mask"][l], r["mask"][l])
        assert np.array_equal(out["J_full"][2], r["J_full"][2])


@pytest.mark.parametrize("model", ["sage", "gcn"])
def test_partition_step_gradients_match_finite_differences(model):
    """The per-partition step (dropout on, masks fixed by t): G = dloss/dW and the boundary rows of
    J_full = dloss/d(received boundary features)."""
    g = synth.tiny_uniform()
    n, rowptr, col, owner = g.n, g.rowptr, g.col, g.owner
    p = build_partition(n, rowptr, col, owner, 0, 2, self_loop=model == "gcn")
    P = propagation_matrix(p)
    rng = np.random.default_rng(21)
    widths = [4, 5, 3]
    k = 2 if model == "sage" else 1
    W = [rng.uniform(-0.6, 0.6, (k * widths[l], widths[l + 1])) for l in range(2)]
    X = rng.standard_normal((p.n_inner, widths[0]))
    y = rng.integers(0, widths[-1], p.n_inner)
    rf = {l: rng.standard_normal((p.n_bd, widths[l - 1])) for l in (1, 2)}
    rg = {2: np.zeros((len(p.send_idx), widths[1]))}
    opts = Options(model=model, dropout=0.35, seed=2, loss_scale=0.5)

    def step(W_, rf_):
        return partition_step(p, P, X, y, W_, rf_, rg, {}, {}, 3, opts)

    rec = step(W, rf)
    eps = 1e-6
    for l in (1, 2):
        for (a, b) in [(0, 0), (k * widths[l - 1] - 1, widths[l] - 1), (1, 1)]:
            Wp = [w.copy() for w in W]; Wm = [w.copy() for w in W]
            Wp[l - 1][a, b] += eps; Wm[l - 1][a, b] -= eps
            fd = (step(Wp, rf)["loss"] - step(Wm, rf)["loss"]) / (2 * eps)
            assert abs(fd - rec["G"][l][a, b]) <= 1e-7 * max(1.0, abs(fd)), (l, a, b)
    for (r, c) in [(0, 0), (p.n_bd - 1, widths[1] - 1), (p.n_bd // 3, 2), (7, 1)]:
        fp = {q: v.copy() for q, v in rf.items()}; fm = {q: v.copy() for q, v in rf.items()}
        fp[2][r, c] += eps; fm[2][r, c] -= eps
        fd = (step(W, fp)["loss"] - step(W, fm)["loss"]) / (2 * eps)
        assert abs(fd - rec["J_full"][2][p.n_inner + r, c]) <= 1e-7 * max(1.0, abs(fd)), (r, c)
