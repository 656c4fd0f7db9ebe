"""One GCN layer, its gradients, the losses, moving average and SGD, in float64.

Layer (Appendix A.1, the layer function and its two gradients, with P the
local propagation matrix of Algorithm 1 and the mean aggregator of the
PipeGCN forward equation in Section 3.2):

    A = P H_full            (aggregation; H_full = [H_inner; H_boundary])
    Z = A W                 (update)
    H = relu(Z)             (every layer except the last, which returns Z)

    M      = J ∘ 1[Z > 0]   (J itself at the last layer)
    G      = Aᵀ M           (weight gradient, from the saved A)
    J_full = Pᵀ (M Wᵀ)      (gradient of every input row, inner and boundary)

The paper fixes no precision.  ``gemm="bf16"`` is the reading used for the
bf16 update-GEMM path: the aggregation stays exact, and the operands of the
three products (A, W, M) are rounded to bfloat16 before an exact product, so
that the ReLU mask is decided from the same rounded operands as on the GPU.

The paper writes the aggregation as the product P H W; aggregating first and
transforming first in the backward are the same matrix products in another
association (the reading is listed with the others in the design notes).

``order="transform"`` evaluates the same layer in the other association,
worth it when the layer narrows (f_out < f_in: fewer columns to aggregate):

    Z      = P (H_full W)
    T      = Pᵀ M               (n + b rows)
    G      = H_fullᵀ T
    J_full = T Wᵀ

With ``gemm="bf16"`` the rounded operands are then H_full, W and T (the
products' inputs in this association).

GraphSAGE layer (Section 2: the update takes CONCAT(z_v, h_v); the paper's
experiments train GraphSAGE), with P the mean over N(v) without a self loop
and X the layer input after dropout (dropout is applied to the received rows
too, after communication, with one mask for the forward and the backward):

    z     = P X_full                      (n x f)
    Z     = [z, X_inner] W                (W is 2f x f_out: rows 0..f-1 act on z)
    H     = relu(Z)

    M      = J ∘ 1[Z > 0]
    G      = [z, X_inner]ᵀ M
    [dz, ds] = M Wᵀ
    J_full = Pᵀ dz, plus ds on the inner rows   (gradient of the dropped input;
                                                  the caller applies the mask)

Transform-first (``order="transform"``): z W_top = P (X_full W_top), so
Z = P (X_full W_top) + X_inner W_bot, and in the backward T = Pᵀ M gives the
top half of G as X_fullᵀ T and the top part of J_full as T W_topᵀ.

Adam (Kingma and Ba, ICLR 2015, Algorithm 1), the experiments' optimiser.

Pinned by: dense brute force of P (tests), central finite differences of the
partition-local loss (tests), reduction to full-graph GCN / GraphSAGE (tests),
torch.optim.Adam (tests).
"""
from __future__ import annotations

import numpy as np


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to bfloat16, nearest-even, through float32 (the GPU rounds its fp32 values).

    bfloat16 keeps the sign, the 8 exponent bits and the top 7 mantissa bits of
    a float32; rounding adds half of the dropped part's unit, with ties to the
    even kept value.  NaN stays NaN.
    """
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = (((u + 0x7FFF + lsb) >> 16) << 16).astype(np.uint32)
    out = r.view(np.float32).astype(np.float64)
    nan = np.isnan(f)
    if nan.any():
        out[nan] = np.nan
    return out


def _operand(x, gemm: str):
    return round_bf16(x) if gemm == "bf16" else x


def layer_forward(P, H_full: np.ndarray, W: np.ndarray, relu: bool, gemm: str = "f64", order: str = "agg"):
    """``gemm="bf16"`` rounds both GEMM operands to bf16 first (products and sums stay fp64).
    Returns (A, Z, H) with A = P H_full in both orders."""
    A = P @ H_full
    if order == "transform":
        Z = P @ (_operand(H_full, gemm) @ _operand(W, gemm))
    else:
        Z = _operand(A, gemm) @ _operand(W, gemm)
    H = np.maximum(Z, 0.0) if relu else Z
    return A, Z, H


def relu_mask(Z: np.ndarray, mask=None) -> np.ndarray:
    """The ReLU derivative 1[Z > 0] (reading: 0 at Z = 0), or a given decision.

    The decision is an integer taken from a floating-point value; where the
    value lies within rounding of zero, either side is a correct result, and a
    caller comparing two computations passes the decision it has certified
    (as it passes the received messages) instead of re-deciding here."""
    return (Z > 0.0) if mask is None else np.asarray(mask, dtype=bool)


def layer_backward(P, A: np.ndarray, Z: np.ndarray, J: np.ndarray, W: np.ndarray,
                   relu: bool, input_grad: bool, gemm: str = "f64", order: str = "agg", H_full=None, mask=None):
    """``order="transform"`` needs the layer input H_full (inner and boundary rows) instead of A.
    ``mask`` (bool, Z's shape) replaces the decision Z > 0 when given."""
    M = J * relu_mask(Z, mask) if relu else J
    if order == "transform":
        Tq = _operand(P.T @ M, gemm)
        G = _operand(H_full, gemm).T @ Tq
        J_full = (Tq @ _operand(W, gemm).T) if input_grad else None
        return G, J_full
    Mq = _operand(M, gemm)
    G = _operand(A, gemm).T @ Mq
    J_full = (P.T @ (Mq @ _operand(W, gemm).T)) if input_grad else None
    return G, J_full


def softmax_ce(Z: np.ndarray, y: np.ndarray, scale: float):
    """Sum over rows of -log softmax(Z)[y], times ``scale``; and its gradient in Z."""
    zmax = Z.max(axis=1, keepdims=True)
    e = np.exp(Z - zmax)
    s = e.sum(axis=1, keepdims=True)
    logp = Z - zmax - np.log(s)
    rows = np.arange(Z.shape[0])
    loss = -logp[rows, y].sum() * scale
    J = e / s
    J[rows, y] -= 1.0
    return loss, J * scale


def sigmoid_bce(Z: np.ndarray, Y: np.ndarray, scale: float):
    """Sum of binary cross-entropy with logits over all entries, times ``scale``."""
    loss = (np.maximum(Z, 0.0) - Z * Y + np.log1p(np.exp(-np.abs(Z)))).sum() * scale
    sig = 1.0 / (1.0 + np.exp(-Z))
    return loss, (sig - Y) * scale


def ema(state: np.ndarray, incoming: np.ndarray, gamma: float) -> np.ndarray:
    """Moving average of Section 3.4: ŝ_t = γ ŝ_{t-1} + (1-γ) s_t."""
    return gamma * state + (1.0 - gamma) * incoming


def sgd(W: np.ndarray, G: np.ndarray, eta: float) -> np.ndarray:
    """Algorithm 1's update W_t = W_{t-1} - η G."""
    return W - eta * G


def sage_forward(P, X_full: np.ndarray, n_inner: int, W: np.ndarray, relu: bool, gemm: str = "f64",
                 order: str = "agg"):
    """Returns (z, Z, H); X_full = [X_inner; X_boundary] is the (dropped) layer input.
    ``order="transform"``: Z = P (X_full W_top) + X_inner W_bot (z is still returned)."""
    z = P @ X_full
    f = X_full.shape[1]
    if order == "transform":
        Z = P @ (_operand(X_full, gemm) @ _operand(W[:f], gemm)) + \
            _operand(X_full[:n_inner], gemm) @ _operand(W[f:], gemm)
    else:
        Xc = np.hstack([z, X_full[:n_inner]])
        Z = _operand(Xc, gemm) @ _operand(W, gemm)
    H = np.maximum(Z, 0.0) if relu else Z
    return z, Z, H


def sage_backward(P, z: np.ndarray, X_inner: np.ndarray, Z: np.ndarray, J: np.ndarray, W: np.ndarray,
                  relu: bool, input_grad: bool, gemm: str = "f64", order: str = "agg", X_full=None, mask=None):
    """Returns (G, J_full): J_full is the gradient of the dropped input rows (inner, then boundary).
    ``order="transform"`` (needs X_full): T = Pᵀ M, G = [X_fullᵀ T ; X_innerᵀ M],
    J_full = T W_topᵀ plus M W_botᵀ on the inner rows.  ``mask`` as in ``layer_backward``."""
    M = J * relu_mask(Z, mask) if relu else J
    Mq = _operand(M, gemm)
    f = X_inner.shape[1]
    n = X_inner.shape[0]
    if order == "transform":
        Tq = _operand(P.T @ M, gemm)
        G = np.vstack([_operand(X_full, gemm).T @ Tq, _operand(X_inner, gemm).T @ Mq])
        if not input_grad:
            return G, None
        J_full = Tq @ _operand(W[:f], gemm).T
        J_full[:n] += Mq @ _operand(W[f:], gemm).T
        return G, J_full
    Xc = np.hstack([z, X_inner])
    G = _operand(Xc, gemm).T @ Mq
    if not input_grad:
        return G, None
    dX = Mq @ _operand(W, gemm).T
    J_full = P.T @ dX[:, :f]
    J_full[:n] += dX[:, f:]
    return G, J_full


def adam(W: np.ndarray, G: np.ndarray, m: np.ndarray, v: np.ndarray, t: int, lr: float,
         beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8):
    """One Adam step (t >= 1): moments m, v updated; returns (W, m, v)."""
    m = beta1 * m + (1.0 - beta1) * G
    v = beta2 * v + (1.0 - beta2) * G * G
    m_hat = m / (1.0 - beta1 ** t)
    v_hat = v / (1.0 - beta2 ** t)
    return W - lr * m_hat / (np.sqrt(v_hat) + eps), m, v
