"""Pins of the oracle's transform-first association of the GCN layer.

The layer's product P H W may be evaluated as P (H W); the backward then
aggregates M before the transform: T = Pᵀ M, G = H_fullᵀ T, J_full = T Wᵀ.
Pinned against what fixes it independently of the oracle's own code:

* central finite differences of the partition-local loss in that association
  (G and the boundary-row gradients);
* vanilla training in that association (and in "auto") reproduces dense
  full-graph GCN, and the pipelined simulation equals the aggregate-first one
  to rounding;
* the bf16 reading (operands H, W and T rounded to bf16, exact products):
  single elements recomputed term by term with torch's float32 -> bfloat16
  conversion, the standard error bound of a product of rounded operands
  against the fp64 result, and exactness when nothing needs rounding.

The GraphSAGE layer in the same association (z W_top = P (X_full W_top)) is
pinned by finite differences of its partition loss (with and without dropout
masks), vanilla training equal to dense full-graph GraphSAGE, and bf16
exactness when nothing needs rounding.
"""
import numpy as np
import pytest
import torch

from oracle import layers
from oracle.partition import build_partition, propagation_matrix
from oracle.pipegcn import Options, layer_order, partition_step, run
from paper_2203_10428_amd import synth
from test_oracle_pins import SMALL_GRAPHS, assemble, dense_full_graph, random_graph, tiny_problem


def local_loss_and_grads(p, P, X_in, Hbd, W, y, scale, order):
    L = len(W)
    H = X_in
    cache = []
    for l in range(L):
        relu = l < L - 1
        Hf = np.vstack([H, Hbd[l]])
        A, Z, Hn = layers.layer_forward(P, Hf, W[l], relu, order=order)
        cache.append((A, Z, relu, Hf))
        H = Hn
    val, J = layers.softmax_ce(H, y, scale)
    G, Jbd = [None] * L, [None] * L
    for l in range(L - 1, -1, -1):
        A, Z, relu, Hf = cache[l]
        G[l], Jf = layers.layer_backward(P, A, Z, J, W[l], relu, True, order=order, H_full=Hf)
        Jbd[l] = Jf[p.n_inner:]
        J = Jf[: p.n_inner]
    return val, G, Jbd


@pytest.mark.parametrize("gi", [0, 1])
def test_transform_gradients_match_finite_differences(gi):
    n, rowptr, col, owner = SMALL_GRAPHS[gi]
    nparts = int(owner.max()) + 1
    p = build_partition(n, rowptr, col, owner, 0, nparts)
    P = propagation_matrix(p)
    rng = np.random.default_rng(21)
    widths = [7, 3, 5, 2]                          # narrowing and widening layers
    X_in = rng.standard_normal((p.n_inner, widths[0]))
    Hbd = [rng.standard_normal((p.n_bd, widths[l])) for l in range(3)]
    W = [rng.standard_normal((widths[l], widths[l + 1])) * 0.7 for l in range(3)]
    y = rng.integers(0, widths[-1], p.n_inner)
    _, G, Jbd = local_loss_and_grads(p, P, X_in, Hbd, W, y, 0.41, "transform")
    eps = 1e-6

    def f(W_, Hbd_):
        return local_loss_and_grads(p, P, X_in, Hbd_, W_, y, 0.41, "transform")[0]

    for l in range(3):
        for (a, b) in [(0, 0), (widths[l] - 1, widths[l + 1] - 1), (2, 1)]:
            Wp = [w.copy() for w in W]; Wm = [w.copy() for w in W]
            Wp[l][a, b] += eps; Wm[l][a, b] -= eps
            fd = (f(Wp, Hbd) - f(Wm, Hbd)) / (2 * eps)
            assert abs(fd - G[l][a, b]) <= 1e-7 * max(1.0, abs(fd)), (l, a, b, fd, G[l][a, b])
        for (r, c) in [(0, 0), (p.n_bd - 1, widths[l] - 1), (p.n_bd // 2, 1)]:
            Hp = [h.copy() for h in Hbd]; Hm = [h.copy() for h in Hbd]
            Hp[l][r, c] += eps; Hm[l][r, c] -= eps
            fd = (f(W, Hp) - f(W, Hm)) / (2 * eps)
            assert abs(fd - Jbd[l][r, c]) <= 1e-7 * max(1.0, abs(fd)), (l, r, c, fd, Jbd[l][r, c])


@pytest.mark.parametrize("order", ["transform", "auto"])
@pytest.mark.parametrize("gi", [0, 3])
def test_transform_vanilla_equals_dense_full_graph(order, gi):
    n, rowptr, col, owner = SMALL_GRAPHS[gi]
    nparts = int(owner.max()) + 1
    widths = [6, 3, 5, 2]
    X, W, y = tiny_problem((n, rowptr, col, owner), widths)
    opts = Options(mode="vanilla", eta=0.3, loss_scale=1.0 / n, order=order)
    sim, recs = run(n, rowptr, col, owner, nparts, X, y, W, 3, opts)
    ref, W_ref = dense_full_graph(n, rowptr, col, X, y, W, 3, 0.3, "softmax_ce", 1.0 / n)
    for t in range(3):
        assert np.isclose(sum(r["loss"] for r in recs[t]), ref[t]["loss"], rtol=1e-12)
        for l in range(1, 4):
            assert np.allclose(assemble(sim, recs[t], "H", l), ref[t]["H"][l - 1], atol=1e-12)
            assert np.allclose(recs[t][0]["G_sum"][l - 1], ref[t]["G"][l - 1], atol=1e-12)
    for w, wr in zip(sim.W, W_ref):
        assert np.allclose(w, wr, atol=1e-12)


def test_layer_order_rule():
    o = Options(order="auto")
    assert layer_order(o, np.zeros((602, 256))) == "transform"
    assert layer_order(o, np.zeros((256, 256))) == "agg"
    assert layer_order(o, np.zeros((300, 512))) == "agg"
    assert layer_order(Options(order="transform"), np.zeros((3, 9))) == "transform"


@pytest.mark.parametrize("sf,sg", [(False, False), (True, True)])
def test_pipelined_transform_equals_aggregate_first(sf, sg):
    """Same iteration semantics in both associations: the pipelined runs agree to rounding."""
    g = synth.tiny_uniform()
    n, rowptr, col, owner = g.n, g.rowptr, g.col, g.owner
    X, W, y = tiny_problem((n, rowptr, col, owner), [6, 3, 4, 2])
    base = dict(smooth_f=sf, smooth_g=sg, gamma=0.8, eta=0.3, loss_scale=1.0 / n)
    a = run(n, rowptr, col, owner, 2, X, y, W, 4, Options(**base))[1]
    b = run(n, rowptr, col, owner, 2, X, y, W, 4, Options(order="transform", **base))[1]
    for ra, rb in zip(a, b):
        for i in range(2):
            assert np.isclose(ra[i]["loss"], rb[i]["loss"], rtol=1e-12)
            for l in (1, 2, 3):
                assert np.allclose(ra[i]["H"][l], rb[i]["H"][l], rtol=1e-11, atol=1e-13)
                assert np.allclose(ra[i]["G"][l], rb[i]["G"][l], rtol=1e-11, atol=1e-13)
            for l in (2, 3):
                assert np.allclose(ra[i]["J_full"][l], rb[i]["J_full"][l], rtol=1e-11, atol=1e-13)


def test_transform_partition_step_matches_simulation():
    g = synth.tiny_uniform()
    n, rowptr, col, owner = g.n, g.rowptr, g.col, g.owner
    X, W, y = tiny_problem((n, rowptr, col, owner), [5, 2, 3])
    opts = Options(smooth_f=True, smooth_g=True, gamma=0.9, eta=0.3, loss_scale=1.0 / n, order="transform",
                   gemm="bf16")
    sim, recs = run(n, rowptr, col, owner, 2, X, y, W, 3, opts)
    p, P = sim.parts[0], sim.P[0]
    for t in range(1, 4):
        r = recs[t - 1][0]
        si = r["state_in"]
        ema_f = {k: v.copy() for k, v in si.ema_f.items()}
        ema_g = {k: v.copy() for k, v in si.ema_g.items()}
        out = partition_step(p, P, X[p.inner_gid], y[p.inner_gid], r["W_in"], si.feat_buf, si.grad_buf,
                             ema_f, ema_g, t, opts)
        for l in (1, 2):
            assert np.array_equal(out["H"][l], r["H"][l])
            assert np.array_equal(out["G"][l], r["G"][l])
        assert np.array_equal(out["J_full"][2], r["J_full"][2])


# ---------------------------------------------------------------------------
# bf16 reading
# ---------------------------------------------------------------------------

def torch_bf16(x: float) -> float:
    return float(torch.tensor(x, dtype=torch.float32).to(torch.bfloat16).to(torch.float64))


def bf16_case(seed=5):
    n, rowptr, col, owner = random_graph(30, 90, 2, seed)
    p = build_partition(n, rowptr, col, owner, 0, 2)
    P = propagation_matrix(p)
    rng = np.random.default_rng(seed)
    Hf = rng.standard_normal((p.n_inner + p.n_bd, 9))
    W = rng.standard_normal((9, 4)) * 0.5
    J = rng.standard_normal((p.n_inner, 4))
    return p, P, Hf, W, J


def test_bf16_transform_elements_term_by_term():
    """A few outputs recomputed with Python loops and torch's bf16 conversion."""
    p, P, Hf, W, J = bf16_case()
    Pd = P.toarray()
    A, Z, H = layers.layer_forward(P, Hf, W, True, gemm="bf16", order="transform")
    G, Jf = layers.layer_backward(P, A, Z, J, W, True, True, gemm="bf16", order="transform", H_full=Hf)
    nt = Pd.shape[1]
    for (v, j) in [(0, 0), (p.n_inner - 1, 3), (p.n_inner // 2, 1)]:
        y = [sum(torch_bf16(Hf[u, k]) * torch_bf16(W[k, j]) for k in range(9)) for u in range(nt)]
        z = sum(Pd[v, u] * y[u] for u in range(nt))
        assert abs(z - Z[v, j]) <= 1e-12 * max(1.0, abs(z))
    M = [[J[v, j] if Z[v, j] > 0 else 0.0 for j in range(4)] for v in range(p.n_inner)]
    T = [[torch_bf16(sum(Pd[v, u] * M[v][j] for v in range(p.n_inner))) for j in range(4)] for u in range(nt)]
    for (a, b) in [(0, 0), (8, 3), (4, 2)]:
        g = sum(torch_bf16(Hf[u, a]) * T[u][b] for u in range(nt))
        assert abs(g - G[a, b]) <= 1e-12 * max(1.0, abs(g))
    for (u, c) in [(0, 0), (nt - 1, 8), (p.n_inner, 5)]:
        jf = sum(T[u][k] * torch_bf16(W[c, k]) for k in range(4))
        assert abs(jf - Jf[u, c]) <= 1e-12 * max(1.0, abs(jf))


def test_bf16_transform_within_rounding_bound():
    """|x_bf16 - x| <= (2u + u^2) * (sum of |terms|), u = 2^-8, for every product."""
    p, P, Hf, W, J = bf16_case(7)
    u = 2.0 ** -8
    k = 2 * u + u * u
    A, Z, _ = layers.layer_forward(P, Hf, W, True, order="transform")
    _, Zq, _ = layers.layer_forward(P, Hf, W, True, gemm="bf16", order="transform")
    assert np.all(np.abs(Zq - Z) <= k * (abs(P) @ (np.abs(Hf) @ np.abs(W))) + 1e-15)
    # backward from the same mask: the fp64 Z decides it for both
    G, Jf = layers.layer_backward(P, A, Z, J, W, True, True, order="transform", H_full=Hf)
    Gq, Jq = layers.layer_backward(P, A, Z, J, W, True, True, gemm="bf16", order="transform", H_full=Hf)
    T = np.abs(P.T @ (J * (Z > 0)))
    # T is rounded too: its error enters each product once more (bound with 3u)
    kb = 3 * u + 3 * u * u
    assert np.all(np.abs(Gq - G) <= kb * (np.abs(Hf).T @ T) + 1e-15)
    assert np.all(np.abs(Jq - Jf) <= kb * (T @ np.abs(W).T) + 1e-15)
    assert np.abs(Gq - G).max() > 0                 # the reading does round


def test_bf16_transform_exact_without_rounding():
    """Isolated inner nodes (P = I) and bf16-representable inputs: the bf16 reading is exact."""
    n = 12
    rowptr = np.zeros(n + 1, np.int64)
    col = np.zeros(0, np.int32)
    owner = np.zeros(n, np.int32)
    p = build_partition(n, rowptr, col, owner, 0, 1)
    P = propagation_matrix(p)
    rng = np.random.default_rng(2)
    q = lambda a: layers.round_bf16(a)
    Hf, W, J = q(rng.standard_normal((n, 5))), q(rng.standard_normal((5, 3))), q(rng.standard_normal((n, 3)))
    for relu in (False, True):
        A, Z, H = layers.layer_forward(P, Hf, W, relu, order="transform")
        _, Zq, Hq = layers.layer_forward(P, Hf, W, relu, gemm="bf16", order="transform")
        assert np.array_equal(Z, Zq)
        G, Jf = layers.layer_backward(P, A, Z, J, W, relu, True, order="transform", H_full=Hf)
        Gq, Jq = layers.layer_backward(P, A, Z, J, W, relu, True, gemm="bf16", order="transform", H_full=Hf)
        assert np.array_equal(G, Gq) and np.array_equal(Jf, Jq)


# ---------------------------------------------------------------------------
# GraphSAGE layer in the transform-first association
# ---------------------------------------------------------------------------

def sage_local_loss_tf(p, P, X_in, Hbd, masks, W, y, scale):
    L = len(W)
    H = X_in
    cache = []
    for l in range(L):
        X = np.vstack([H, Hbd[l]]) * masks[l]
        z, Z, Hn = layers.sage_forward(P, X, p.n_inner, W[l], l < L - 1, order="transform")
        cache.append((z, X, Z))
        H = Hn
    val, J = layers.softmax_ce(H, y, scale)
    G, Jbd = [None] * L, [None] * L
    for l in range(L - 1, -1, -1):
        z, X, Z = cache[l]
        G[l], Jf = layers.sage_backward(P, z, X[: p.n_inner], Z, J, W[l], l < L - 1, True, order="transform",
                                        X_full=X)
        Jf = Jf * masks[l]
        Jbd[l] = Jf[p.n_inner:]
        J = Jf[: p.n_inner]
    return val, G, Jbd


@pytest.mark.parametrize("p_drop", [0.0, 0.35])
def test_sage_transform_gradients_match_finite_differences(p_drop):
    from oracle.philox import dropout_mask
    n, rowptr, col, owner = SMALL_GRAPHS[0]
    p = build_partition(n, rowptr, col, owner, 0, 3, self_loop=False)
    P = propagation_matrix(p)
    rng = np.random.default_rng(41)
    widths = [7, 3, 5, 2]
    X_in = rng.standard_normal((p.n_inner, widths[0]))
    Hbd = [rng.standard_normal((p.n_bd, widths[l])) for l in range(3)]
    W = [rng.standard_normal((2 * widths[l], widths[l + 1])) * 0.6 for l in range(3)]
    masks = [dropout_mask(p.n_inner + p.n_bd, widths[l], p_drop, 3, 0, l + 1, 2) for l in range(3)]
    y = rng.integers(0, widths[-1], p.n_inner)
    _, G, Jbd = sage_local_loss_tf(p, P, X_in, Hbd, masks, W, y, 0.37)
    eps = 1e-6

    def f(W_, Hbd_):
        return sage_local_loss_tf(p, P, X_in, Hbd_, masks, W_, y, 0.37)[0]

    for l in range(3):
        for (a, b) in [(0, 0), (2 * widths[l] - 1, widths[l + 1] - 1), (widths[l], 1), (1, 0)]:
            Wp = [w.copy() for w in W]; Wm = [w.copy() for w in W]
            Wp[l][a, b] += eps; Wm[l][a, b] -= eps
            fd = (f(Wp, Hbd) - f(Wm, Hbd)) / (2 * eps)
            assert abs(fd - G[l][a, b]) <= 1e-7 * max(1.0, abs(fd)), (l, a, b, fd, G[l][a, b])
        for (r, c) in [(0, 0), (p.n_bd - 1, widths[l] - 1), (p.n_bd // 2, 1)]:
            Hp = [h.copy() for h in Hbd]; Hm = [h.copy() for h in Hbd]
            Hp[l][r, c] += eps; Hm[l][r, c] -= eps
            fd = (f(W, Hp) - f(W, Hm)) / (2 * eps)
            assert abs(fd - Jbd[l][r, c]) <= 1e-7 * max(1.0, abs(fd)), (l, r, c, fd, Jbd[l][r, c])


@pytest.mark.parametrize("order", ["transform", "auto"])
def test_sage_transform_vanilla_equals_dense_full_graph(order):
    from test_oracle_sage_pins import dense_full_graph_sage, sage_problem
    n, rowptr, col, owner = SMALL_GRAPHS[3]
    nparts = int(owner.max()) + 1
    widths = [6, 3, 5, 2]
    X, W, y = sage_problem((n, rowptr, col, owner), widths)
    opts = Options(mode="vanilla", model="sage", eta=0.3, loss_scale=1.0 / n, order=order)
    sim, recs = run(n, rowptr, col, owner, nparts, X, y, W, 3, opts)
    ref, W_ref = dense_full_graph_sage(n, rowptr, col, X, y, W, 3, 0.3, 1.0 / n)
    for t in range(3):
        assert np.isclose(sum(r["loss"] for r in recs[t]), ref[t]["loss"], rtol=1e-12)
        for l in range(1, 4):
            assert np.allclose(assemble(sim, recs[t], "H", l), ref[t]["H"][l - 1], atol=1e-12)
            assert np.allclose(recs[t][0]["G_sum"][l - 1], ref[t]["G"][l - 1], atol=1e-12)
    for w, wr in zip(sim.W, W_ref):
        assert np.allclose(w, wr, atol=1e-12)


def test_sage_layer_order_rule():
    o = Options(order="auto")
    assert layer_order(o, np.zeros((2 * 602, 256)), sage=True) == "transform"
    assert layer_order(o, np.zeros((2 * 256, 256)), sage=True) == "agg"
    assert layer_order(o, np.zeros((2 * 100, 128)), sage=True) == "agg"


def test_sage_bf16_transform_exact_without_rounding():
    """Isolated nodes (z = 0) and bf16-representable inputs: the bf16 reading equals fp64."""
    n = 10
    rowptr = np.zeros(n + 1, np.int64)
    col = np.zeros(0, np.int32)
    owner = np.zeros(n, np.int32)
    p = build_partition(n, rowptr, col, owner, 0, 1, self_loop=False)
    P = propagation_matrix(p)
    rng = np.random.default_rng(3)
    q = layers.round_bf16
    X, W, J = q(rng.standard_normal((n, 4))), q(rng.standard_normal((8, 3))), q(rng.standard_normal((n, 3)))
    z, Z, _ = layers.sage_forward(P, X, n, W, True, order="transform")
    _, Zq, _ = layers.sage_forward(P, X, n, W, True, gemm="bf16", order="transform")
    assert np.array_equal(Z, Zq)
    G, Jf = layers.sage_backward(P, z, X, Z, J, W, True, True, order="transform", X_full=X)
    Gq, Jq = layers.sage_backward(P, z, X, Z, J, W, True, True, gemm="bf16", order="transform", X_full=X)
    assert np.array_equal(G, Gq) and np.array_equal(Jf, Jq)
