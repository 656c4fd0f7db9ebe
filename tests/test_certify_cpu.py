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


def fp32_layer(P, X, W, order, bf16):
    """The layer evaluated as the GPU does: fp32 inputs, fp32 sums, bf16 operands on the bf16 path."""
    P32 = P.astype(np.float32)
    X32 = X.astype(np.float32)
    W32 = W.astype(np.float32)
    q = (lambda a: layers.round_bf16(a).astype(np.float32)) if bf16 else (lambda a: a)
    if order == "transform":
        return (P32 @ (q(X32) @ q(W32))).astype(np.float64)
    A32 = (P32 @ X32).astype(np.float32)
    return (q(A32) @ q(W32)).astype(np.float64)


@pytest.mark.parametrize("order", ["agg", "transform"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("seed", [0, 1])
def test_bound_holds_for_fp32_and_bf16_evaluations(order, dt, seed):
    ref, P, X, W = setup(seed)
    Z = P @ X @ W
    Zg = fp32_layer(P, X, W, order, dt == "bf16")
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
