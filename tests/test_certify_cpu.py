"""CPU checks of the parity tests' decision certification (tests/certify.py):
the element-wise rounding bound really bounds fp32 and bf16-operand
evaluations of a layer, in both associations, and a ReLU decision that
differs beyond it is refused."""
import numpy as np
import pytest

from certify import certify_relu, input_rounding, z_bound
from gpu_helpers import random_partition_graph
from oracle import layers
from oracle.partition import build_partition, propagation_matrix


def setup(seed, f=48, f_out=24, sage=False):
    n_g, rowptr, col, owner = random_partition_graph(400, 200, 3, 30, seed, hub_deg=300)
    ref = build_partition(n_g, rowptr, col, owner, 0, 3, self_loop=not sage)
    P = propagation_matrix(ref)
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((ref.n_inner + ref.n_bd, f))
    W = rng.uniform(-0.3, 0.3, ((2 if sage else 1) * f, f_out)).astype(np.float32).astype(np.float64)
    return ref, P, X, W


def split3(x):
    """fp32 x as hi + mid + lo: hi = x with its low 16 bits cleared, mid = x - hi rounded to
    bf16 (nearest even), lo = the rest (the split of the fp32 update GEMMs)."""
    def rne(v):
        vb = v.view(np.uint32).astype(np.uint64)
        return (((vb + 0x7FFF + ((vb >> 16) & 1)) & 0xFFFF0000).astype(np.uint32)).view(np.float32)

    x = np.asarray(x, dtype=np.float32)
    hi = (x.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32)
    r = (x - hi).astype(np.float32)
    mid = rne(r)
    return hi, mid, rne((r - mid).astype(np.float32))


def is_bf16(v):
    return np.all((np.asarray(v, dtype=np.float32).view(np.uint32) & np.uint32(0xFFFF)) == 0)


def test_split_is_exact_and_small():
    rng = np.random.default_rng(4)
    x = (rng.standard_normal(400_000) * np.exp2(rng.integers(-100, 100, 400_000))).astype(np.float32)
    x[:4] = [0.0, -0.0, np.finfo(np.float32).max, -np.finfo(np.float32).tiny]
    hi, mid, lo = split3(x)
    assert is_bf16(hi) and is_bf16(mid) and is_bf16(lo)
    # exact for |x| >= 2^-111: the three parts add up to x in fp64 (and so in any order);
    # below, the last part is a bf16 subnormal, within half its spacing (2^-134)
    ax = np.abs(x.astype(np.float64))
    err = np.abs(hi.astype(np.float64) + mid.astype(np.float64) + lo.astype(np.float64) - ax * np.sign(x))
    assert (ax < 2.0 ** -111).sum() > 0
    assert np.all(err[ax >= 2.0 ** -111] == 0) and np.all(err <= 2.0 ** -134)
    assert np.all(np.abs(mid) < 2.0 ** -7 * ax + (ax == 0)) and np.all(np.abs(lo) <= 2.0 ** -15 * ax)


def test_dropped_part_products_are_below_the_bound():
    rng = np.random.default_rng(6)
    a = (rng.standard_normal(200_000) * np.exp2(rng.integers(-20, 20, 200_000))).astype(np.float32)
    b = (rng.standard_normal(200_000) * np.exp2(rng.integers(-20, 20, 200_000))).astype(np.float32)
    (a1, a2, a3), (b1, b2, b3) = [[p.astype(np.float64) for p in split3(v)] for v in (a, b)]
    kept = a1 * b1 + a1 * b2 + a2 * b1 + a1 * b3 + a2 * b2 + a3 * b1
    exact = a.astype(np.float64) * b.astype(np.float64)
    assert np.all(np.abs(exact - kept) <= 2.0 ** -21 * (1 + 2.0 ** -7) * np.abs(exact))
    # the part products are exact in fp32 (8 x 8 significant bits)
    for p, q in ((a1, b1), (a1, b2), (a2, b1), (a1, b3), (a2, b2), (a3, b1)):
        assert np.array_equal((p * q).astype(np.float32).astype(np.float64), p * q)


def fp32_by_parts(A32, W32):
    """A32 @ W32 as the fp32 GEMM by parts computes it: six part products, summed in fp32."""
    (a1, a2, a3), (w1, w2, w3) = split3(A32), split3(W32)
    out = np.zeros((A32.shape[0], W32.shape[1]), dtype=np.float32)
    for p, q in ((a3, w1), (a2, w2), (a1, w3), (a2, w1), (a1, w2), (a1, w1)):
        out = (out + (p @ q).astype(np.float32)).astype(np.float32)
    return out


def fp32_layer(P, X, W, order, bf16, parts=False):
    """The layer evaluated as the GPU does: fp32 inputs, fp32 sums, bf16 operands on the bf16 path."""
    P32 = P.astype(np.float32)
    X32 = X.astype(np.float32)
    W32 = W.astype(np.float32)
    q = (lambda a: layers.round_bf16(a).astype(np.float32)) if bf16 else (lambda a: a)
    mm = fp32_by_parts if parts else (lambda a, w: a @ w)
    if order == "transform":
        return (P32 @ mm(q(X32), q(W32))).astype(np.float64)
    A32 = (P32 @ X32).astype(np.float32)
    return mm(q(A32), q(W32)).astype(np.float64)


@pytest.mark.parametrize("order", ["agg", "transform"])
@pytest.mark.parametrize("dt", ["f32", "f32-parts", "bf16"])
@pytest.mark.parametrize("seed", [0, 1])
def test_bound_holds_for_fp32_and_bf16_evaluations(order, dt, seed):
    ref, P, X, W = setup(seed)
    Z = P @ X @ W
    parts = dt == "f32-parts"
    dt = "f32" if parts else dt
    Zg = fp32_layer(P, X, W, order, dt == "bf16", parts)
    B = z_bound(P, X, input_rounding(X), W, dt)
    assert np.all(np.abs(Zg - Z) <= B)
    # the bound is not vacuous: a decision is certified only for |Z| well below the layer's scale
    assert B.max() < (1e-1 if dt == "bf16" else 1e-3) * np.abs(Z).max()
    if dt == "bf16":
        _, Zr, _ = layers.layer_forward(P, X, W, False, "bf16", order=order)
        assert np.all(np.abs(Zg - Zr) <= z_bound(P, X, input_rounding(X), W, dt, reading="bf16"))


def test_bound_carries_input_error():
    ref, P, X, W = setup(2)
    rng = np.random.default_rng(5)
    E = np.abs(X) * 1e-3
    Xp = X + E * rng.uniform(-1, 1, X.shape)
    Z, Zp = P @ X @ W, fp32_layer(P, Xp, W, "agg", False)
    assert np.all(np.abs(Zp - Z) <= z_bound(P, X, E, W, "f32"))


def test_sage_bound():
    ref, P, X, W = setup(3, sage=True)
    n = ref.n_inner
    _, Z, _ = layers.sage_forward(P, X, n, W, False)
    P32, X32, W32 = P.astype(np.float32), X.astype(np.float32), W.astype(np.float32)
    Zg = (np.hstack([P32 @ X32, X32[:n]]) @ W32).astype(np.float64)
    assert np.all(np.abs(Zg - Z) <= z_bound(P, X, input_rounding(X), W, "f32", sage=True))


def test_certify_accepts_flips_within_the_bound_and_refuses_others():
    Z = np.array([[1e-9, -2e-9, 0.5], [-0.3, 0.2, 3e-10]])
    bound = np.full(Z.shape, 1e-8)
    gpu = np.array([[0.0, 1e-9, 0.5], [0.0, 0.2, 0.0]])         # three decisions differ, all within the bound
    mask, flips = certify_relu(Z, gpu, bound)
    assert flips == 3
    assert np.array_equal(mask, gpu > 0)
    gpu_bad = gpu.copy()
    gpu_bad[1, 0] = 0.1                                          # Z = -0.3 decided positive: not a rounding effect
    with pytest.raises(AssertionError, match="beyond the rounding bound"):
        certify_relu(Z, gpu_bad, bound)
