"""Certification of the floating-point decisions the parity tests meet.

The ReLU mask 1[Z > 0] is an integer decision taken from a floating-point
value.  The GPU takes it from its own Z; the oracle from its fp64 Z.  Where
the two disagree, the GPU's decision is a correct one only if the oracle's Z
lies within the error the GPU's arithmetic can make on that element.  These
helpers bound that error element by element, check every disagreement
against the bound (failing the test otherwise), and hand the oracle's
backward a mask that is its own decision everywhere except at the certified
positions, where it takes the GPU's.  The flip count is reported.

Error model (standard forward error analysis of sums of products, Higham,
"Accuracy and Stability of Numerical Algorithms", 2nd ed., Sec. 3.1):
|fl(sum_k x_k y_k) - sum_k x_k y_k| <= gamma_n sum_k |x_k y_k|, with
gamma_n = n u / (1 - n u) for n terms in any order.  One GCN output is
Z_vc = sum_u P_vu sum_k X_uk W_kc.  The GPU sums the d_v rows of P (each as
one term, or as three exact bf16 parts in the dense block the matrix cores
take, plus up to four roundings for the 1/d or d^-1/2 scales and their
products) and K products, in fp32; on the bf16 path both product operands are
first rounded once to bf16 (nearest even).  The fp32 path takes each product
as six exact products of bf16 parts (x = hi + mid + lo exactly, |mid| <
2^-7 |x|, |lo| <= 2^-15 |x|; the three dropped part products are below
2^-21 (1 + 2^-7) |x y| <= p = 2^-20 |x y|), so it sums 6K terms whose
magnitudes add up to at most |x y| per product.  So

    |Z_gpu - Z| <= c_v (P|X|)|W| + (1 + c_v) (P E_X)|W|,
    c_v = (1 + b)^2 (1 + 2^-24) (1 + p) (1 + gamma_{6K}) (1 + gamma_{3 d_v + 4}) - 1,

with b = 2^-8 on the bf16 path and 0 on the fp32 path (p = 0 and 6K -> K
on the bf16 path; the plain fp32 matrix-core kernel is within the same bound),
2^-24 for the weights handed over in fp32, and E_X a bound on the
error of the layer's input as the GPU holds it (rounding of the given inputs,
the previous layer's own bound, the moving average's roundings).  u is taken
as 2^-23, one unit in the last place of fp32, which bounds any faithful
rounding: the hardware documents no rounding mode for the matrix cores'
internal sums.  A GraphSAGE output adds the self term X_inner W_bot
(K = 2f terms).

Also here: the element-wise error metric |g - o| / (|o| + 1e-6 max|o|), which
the parity tests report beside the per-tensor max|g - o| / max|o|.
"""
from __future__ import annotations

import numpy as np

U32 = 2.0 ** -23
UBF16 = 2.0 ** -8


def gamma(n, u=U32):
    n = np.asarray(n, dtype=np.float64)
    return n * u / (1.0 - n * u)


def product_factor(dt: str, K: int, row_terms: np.ndarray) -> np.ndarray:
    """c_v per output row (column vector) for K products and row_terms aggregated rows."""
    bf16 = dt == "bf16"
    b = UBF16 if bf16 else 0.0
    w = 2.0 ** -24                     # the weights are handed to the GPU rounded to fp32
    # fp32: six part products per product, the dropped ones below p |x y|
    p, terms = (0.0, K) if bf16 else (2.0 ** -20, 6 * K)
    # each aggregated row may enter as three exact bf16 parts (the dense block on the matrix cores)
    return ((1.0 + b) ** 2 * (1.0 + w) * (1.0 + p) * (1.0 + gamma(terms))
            * (1.0 + gamma(3 * np.asarray(row_terms) + 4)) - 1.0)[:, None]


def row_lengths(P) -> np.ndarray:
    P = P.tocsr()
    return np.diff(P.indptr)


_TORCH_CSR = {}


def spmm(P, X: np.ndarray) -> np.ndarray:
    """|P| @ X in fp64 with torch's multithreaded CPU sparse product (the bounds need several such
    products per layer; the oracle's own products stay SciPy's)."""
    import warnings

    import torch

    key = id(P)
    if key not in _TORCH_CSR or _TORCH_CSR[key][0] is not P:
        Pc = P.tocsr()
        _TORCH_CSR.clear()
        with warnings.catch_warnings():              # the CSR layout is marked beta
            warnings.simplefilter("ignore")
            t = torch.sparse_csr_tensor(torch.from_numpy(Pc.indptr.astype(np.int64)),
                                        torch.from_numpy(Pc.indices.astype(np.int64)),
                                        torch.from_numpy(np.abs(Pc.data).astype(np.float64)), size=Pc.shape)
        _TORCH_CSR[key] = (P, t)
    return (_TORCH_CSR[key][1] @ torch.from_numpy(np.ascontiguousarray(X, dtype=np.float64))).numpy()


def z_bound(P, X: np.ndarray, E_X: np.ndarray, W: np.ndarray, dt: str, sage: bool = False,
            reading: str = "f64") -> np.ndarray:
    """Bound on |Z_gpu - Z_ref| for one layer.

    X: the oracle's layer input [n + b, f] (after dropout); E_X: bound on the
    GPU's input error, same shape; W: the weights ([f, f_out], GraphSAGE
    [2 f, f_out]).  ``reading="bf16"``: Z_ref is the oracle's reading with
    bf16-rounded operands, itself within (2b + b^2) (P|X|)|W| of the exact Z,
    which is added.  Returns [n, f_out]."""
    X, E_X = np.abs(np.asarray(X, dtype=np.float64)), np.asarray(E_X, dtype=np.float64)
    W = np.abs(np.asarray(W, dtype=np.float64))
    f = X.shape[1]
    n = P.shape[0]
    Wt = W[:f]
    f_out = W.shape[1]
    # (|P| |X|) |W| in whichever association aggregates fewer columns (equal, all terms >= 0)
    if f_out < f:
        both = spmm(P, np.hstack([X @ Wt, E_X @ Wt]))
    else:
        both = spmm(P, np.hstack([X, E_X]))
        both = np.hstack([both[:, :f] @ Wt, both[:, f:] @ Wt])
    T, TE = both[:, :f_out], both[:, f_out:]
    K = f
    if sage:
        T = T + X[:n] @ W[f:]
        TE = TE + E_X[:n] @ W[f:]
        K = 2 * f
    c = product_factor(dt, K, row_lengths(P))
    out = c * T + (1.0 + c) * TE
    if reading == "bf16":
        out += (2.0 * UBF16 + UBF16 ** 2) * T
    return out


def input_rounding(X: np.ndarray) -> np.ndarray:
    """Error of an fp64 value handed to the GPU as fp32 (nearest)."""
    return np.abs(np.asarray(X, dtype=np.float64)) * 2.0 ** -24


def ema_error(state_in: np.ndarray, incoming: np.ndarray, gamma_: float) -> np.ndarray:
    """Bound on the GPU's fp32 moving average gamma*s + (1-gamma)*B of fp32-rounded s and B:
    both inputs rounded once, the two coefficients, two products and the sum (5 roundings)."""
    return 5.0 * U32 * (abs(gamma_) * np.abs(state_in) + abs(1.0 - gamma_) * np.abs(incoming))


def dropout_error(X_dropped: np.ndarray, E_in: np.ndarray, mask: np.ndarray) -> np.ndarray:
    """Inverted dropout x * (1/(1-p)) in fp32: the scale rounded once and the product once,
    plus the input error carried through the mask (whose values are 0 or 1/(1-p))."""
    return np.abs(mask) * E_in + 2.0 * U32 * np.abs(X_dropped)


def certify_relu(Z_ref: np.ndarray, H_gpu: np.ndarray, bound: np.ndarray, what: str = ""):
    """Returns (mask, flips): the oracle's decision Z_ref > 0, except where the GPU decided
    otherwise (H_gpu > 0) and |Z_ref| <= bound (certified).  Fails on an uncertified flip."""
    own = Z_ref > 0.0
    gpu = H_gpu > 0.0
    diff = own != gpu
    flips = int(diff.sum())
    if flips:
        bad = diff & (np.abs(Z_ref) > bound)
        if bad.any():
            r, c = np.nonzero(bad)
            worst = np.max(np.abs(Z_ref[bad]) / np.maximum(bound[bad], 1e-300))
            raise AssertionError(f"{what}: {int(bad.sum())} of {flips} ReLU decisions differ beyond the rounding "
                                 f"bound (first at row {r[0]} col {c[0]}: Z = {Z_ref[r[0], c[0]]:.3e}, bound "
                                 f"{bound[r[0], c[0]]:.3e}; worst |Z|/bound = {worst:.3g})")
    return np.where(diff, gpu, own), flips


def sign_array(mask: np.ndarray) -> np.ndarray:
    """A stand-in Z whose only use by the oracle's backward is the decision Z > 0."""
    return np.where(mask, 1.0, -1.0)


def elem_err(gpu, ref) -> float:
    """max over elements of |g - o| / (|o| + 1e-6 max|o|)."""
    ref = np.asarray(ref, dtype=np.float64)
    gpu = np.asarray(gpu, dtype=np.float64)
    if ref.size == 0:
        return 0.0
    den = np.abs(ref) + 1e-6 * max(np.abs(ref).max(), 1e-300)
    return float((np.abs(gpu - ref) / den).max())


def readings(dt: str):
    """The oracle readings a GPU result of this GEMM precision is compared with: the plain fp64
    oracle always; on the bf16 path also the reading with bf16-rounded operands."""
    return ("f64", "bf16") if dt == "bf16" else ("f64",)


def certified_step(p, P, X_in, y, W, state_in, t, opts, H_gpu: dict, dt: str, rec=None):
    """One partition step of the oracle (``partition_step``, reading ``opts.gemm``) whose ReLU
    decisions are certified against the GPU's.

    ``state_in`` holds what the GPU was given before the iteration (received
    features and gradients, smoothing states, each handed over in fp32);
    ``H_gpu[l]`` is the GPU's layer-l output.  Each layer's error bound is
    carried into the next layer's input (ReLU is 1-Lipschitz).  Returns the
    oracle record (re-run with the certified decisions when any differ), the
    smoothing states it left, and the flip count per layer.  ``rec``: the
    plain step's record when already computed (its smoothing states are then
    recomputed only on a re-run)."""
    from oracle.pipegcn import partition_step

    sage = opts.model == "sage"
    L = len(W)
    copy = lambda d: {k: v.copy() for k, v in d.items()}
    ema_f, ema_g = copy(state_in.ema_f), copy(state_in.ema_g)
    if rec is None:
        rec = partition_step(p, P, X_in, y, W, state_in.feat_buf, state_in.grad_buf, ema_f, ema_g, t, opts)
    else:
        rec, (ema_f, ema_g) = rec
    n = p.n_inner
    E_prev = input_rounding(X_in)
    masks, flips = {}, {}
    for l in range(1, L + 1):
        fb = state_in.feat_buf[l]
        if t == 1:
            E_bd = np.zeros_like(fb)
        elif opts.smooth_f:
            E_bd = ema_error(state_in.ema_f[l], fb, opts.gamma)
        else:
            E_bd = input_rounding(fb)
        E_X = np.vstack([E_prev, E_bd])
        drop = rec["mask"][l]
        if opts.dropout > 0.0:
            E_X = dropout_error(rec["X_full"][l], E_X, drop)
        E = z_bound(P, rec["X_full"][l], E_X, W[l - 1], dt, sage, opts.gemm)
        if l < L or opts.relu_last:
            masks[l], flips[l] = certify_relu(rec["Z"][l], H_gpu[l], E, f"layer {l}")
        E_prev = E
    if any(flips.values()):
        ema_f, ema_g = copy(state_in.ema_f), copy(state_in.ema_g)
        rec = partition_step(p, P, X_in, y, W, state_in.feat_buf, state_in.grad_buf, ema_f, ema_g, t, opts,
                             relu_masks=masks)
    return rec, ema_f, ema_g, flips


def certified_reference(sim, r0, r1, opts, H_gpu: dict, dt: str):
    """Partition 0's expected outputs for an injected iteration of a simulation record pair
    (r0 for partition 0, r1 for its peer): ``certified_step`` from r0's injected inputs under
    ``opts`` (its ``gemm`` reading), then the update with the peer's gradient as the second
    AllReduce operand.  Returns a dict with the keys the step comparisons read."""
    from oracle import layers

    p, P = sim.parts[0], sim.P[0]
    X_in = sim.X[p.inner_gid]
    y = sim.labels[p.inner_gid]
    W = r0["W_in"]
    rec, ema_f, ema_g, flips = certified_step(p, P, X_in, y, W, r0["state_in"], r0["t"], opts, H_gpu, dt)
    L = len(W)
    G_sum = [rec["G"][l + 1] + r1["G"][l + 1] for l in range(L)]
    if opts.optimizer == "adam":
        m, v = r0["adam_in"]
        W_out = [layers.adam(W[l], G_sum[l], m[l], v[l], r0["t"], opts.eta, opts.beta1, opts.beta2, opts.eps)[0]
                 for l in range(L)]
    else:
        W_out = [layers.sgd(W[l], G_sum[l], opts.eta) for l in range(L)]
    return dict(rec, ema_f=ema_f, ema_g=ema_g, flips=flips, G_sum=G_sum, W_out=W_out)


def adam_within_gradient_error(W_gpu, W_in, G_sum, delta, m_in, v_in, t, opts, tol_abs, samples=257):
    """Adam's update is not Lipschitz in the gradient where the moments are near zero (its first
    steps move every weight by about lr * sign(g)).  So instead of comparing with the update of
    the oracle's G alone, check that every GPU weight lies (within tol_abs) in the range of
    updates over gradients g' in [G_sum - delta, G_sum + delta], delta being the certified bound
    of the GPU's gradient error.  Returns the number of weights that needed more than the
    point comparison."""
    from oracle import layers

    s = np.linspace(-1.0, 1.0, samples)
    lo = np.full(W_in.shape, np.inf)
    hi = np.full(W_in.shape, -np.inf)
    for k in s:
        w = layers.adam(W_in, G_sum + k * delta, m_in, v_in, t, opts.eta, opts.beta1, opts.beta2, opts.eps)[0]
        lo, hi = np.minimum(lo, w), np.maximum(hi, w)
    point = layers.adam(W_in, G_sum, m_in, v_in, t, opts.eta, opts.beta1, opts.beta2, opts.eps)[0]
    inside = (W_gpu >= lo - tol_abs) & (W_gpu <= hi + tol_abs)
    assert inside.all(), (f"{int((~inside).sum())} weights outside Adam's range over the certified gradient "
                          f"interval; worst excess {np.max(np.maximum(lo - tol_abs - W_gpu, W_gpu - hi - tol_abs)):.3e}")
    return int((np.abs(W_gpu - point) > tol_abs).sum())
