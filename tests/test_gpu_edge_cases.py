"""Degenerate partitions through the C ABI, for every layer form the library
offers (aggregate-first and transform-first GCN, mean and symmetric
normalisation, GraphSAGE in both associations), against the oracle:

* one partition: no boundary rows and no send list (n_bd = 0), so the split
  weight-gradient GEMM has no second matrix and the transposed aggregation no
  outgoing rows;
* an empty partition (owns no node): every call succeeds, dW = 0;
* a partition whose inner nodes have no edges (P = I with self loops, zero
  rows of the GraphSAGE mean);
* the widest layers the entry points accept (PGCN_MAX_WIDTH columns in or
  out: 32 aggregation launches per row), and one column more, which every
  layer entry point rejects before launching anything;
* a partition whose aggregation plans differ by row width (2 column chunks
  for wide rows, 1 for rows of at most 64 floats), with one narrow and one
  wide width per layer (also 64 against 65, either side of the threshold), so
  that each order runs each plan in each direction.

At the widest layers some of the 19 million pre-activations lie within
rounding of zero, so the GPU's ReLU decisions may differ from the oracle's:
each such difference is certified against the element's rounding bound
(tests/certify.py) before the oracle's backward takes it.  bf16 results are
held to the plain fp64 oracle and to its bf16-operand reading alike.
"""
import numpy as np
import pytest
import torch

from certify import certify_relu, elem_err, input_rounding, readings, z_bound
from gpu_helpers import TOL, dev, host, random_partition_graph, rel_err
from oracle import layers
from oracle.partition import build_partition, propagation_matrix
from paper_2203_10428_amd import binding as B
from paper_2203_10428_amd.step import ld_of

pytestmark = pytest.mark.gpu

FORMS = [("gcn", "mean", "agg"), ("gcn", "mean", "transform"), ("gcn", "sym", "agg"), ("gcn", "sym", "transform"),
         ("sage", "mean", "agg"), ("sage", "mean", "transform")]
ORDER = {"agg": B.PGCN_ORDER_AGG, "transform": B.PGCN_ORDER_TRANSFORM}


def graph(kind):
    if kind == "small":
        n, rowptr, col, owner = random_partition_graph(300, 150, 3, 8, 7)
        return n, rowptr, col, owner, 3
    if kind == "one_partition":
        n, rowptr, col, _ = random_partition_graph(900, 300, 2, 10, 4)
        return n, rowptr, col, np.zeros(n, np.int32), 1
    if kind == "two_plans":       # 12,000 columns, ~100 non-zeros per row: wide plans 2 chunks, narrow 1
        n, rowptr, col, owner = random_partition_graph(9000, 3000, 2, 120, 13)
        return n, rowptr, col, owner, 2
    if kind == "empty":
        n, rowptr, col, owner = random_partition_graph(600, 300, 3, 8, 5)
        owner = np.where(owner == 0, 1, owner).astype(np.int32)      # partition 0 owns nothing
        return n, rowptr, col, owner, 3
    n = 700                                                          # no edges at all
    return n, np.zeros(n + 1, np.int64), np.zeros(0, np.int32), (np.arange(n) % 2).astype(np.int32), 2


def run_layer(kind, model, norm, order, dt, f_in=37, f_out=21):
    n_g, rowptr, col, owner, nparts = graph(kind)
    sage = model == "sage"
    ref = build_partition(n_g, rowptr, col, owner, 0, nparts, self_loop=not sage)
    P = propagation_matrix(ref, norm)
    part = B.pgcn_partition_setup(n_g, rowptr, col, owner, nparts, 0, self_loop=not sage, symmetric=norm == "sym")
    n, b = ref.n_inner, ref.n_bd
    rng = np.random.default_rng(n + b + f_in)
    X = rng.standard_normal((n + b, f_in))
    k = 2 if sage else 1
    W = rng.uniform(-0.3, 0.3, (k * f_in, f_out)).astype(np.float32)
    J = rng.standard_normal((n, f_out)) * 1e-2
    dtype = B.PGCN_BF16 if dt == "bf16" else B.PGCN_F32
    nb = max(B.pgcn_layer_workspace_size(part, f_in, f_out, dtype, ORDER[order]), 256)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    dX, dXbd = dev(X[:n]), dev(X[n:])
    dX16 = dev(X[:n], dtype=torch.bfloat16) if dt == "bf16" else None
    agg = order == "agg"
    A = dev(np.zeros((n, f_in))) if agg else None
    A16 = torch.zeros((n, ld_of(f_in)), dtype=torch.bfloat16, device="cuda") if agg and dt == "bf16" else None
    H = dev(np.zeros((n, f_out)))
    common = dict(f_in=f_in, f_out=f_out, gemm_dtype=dtype, relu=True, ld_in=ld_of(f_in), ld_out=ld_of(f_out),
                  W=torch.from_numpy(W).cuda(), workspace=ws, workspace_bytes=nb, order=ORDER[order])
    if sage:
        B.pgcn_sage_layer_fwd(part, X_in=dX, X_in_bf16=dX16, X_bd=dXbd if b else None, A=A, A_bf16=A16, H_out=H,
                              **common)
    else:
        B.pgcn_layer_fwd(part, H_in=dX, H_bd=dXbd if b else None, A=A, A_bf16=A16, H_out=H, **common)
    dG = torch.full((k * f_in, f_out), 3.0, device="cuda")
    J_in, J_bd = dev(np.zeros((n, f_in))), (dev(np.zeros((b, f_in))) if b else None)
    if sage:
        B.pgcn_sage_layer_bwd(part, J_out=dev(J), H_out=H, A=A, A_bf16=A16, X_in=dX, X_in_bf16=dX16,
                              X_bd=dXbd if b else None, dW=dG, J_in=J_in, J_bd_out=J_bd, **common)
    else:
        B.pgcn_layer_bwd(part, J_out=dev(J), H_out=H, A=A, A_bf16=A16, dW=dG, J_in=J_in, J_bd_out=J_bd,
                         H_in=dX, H_bd=dXbd if b else None, **common)
    torch.cuda.synchronize()
    H_gpu = host(H, f_out)
    Wd = W.astype(np.float64)
    refs = {}
    for gm in readings(dt):
        # the ReLU mask is a decision taken by floating point: where the GPU's differs from the
        # oracle's, the oracle's Z must lie within the rounding bound; only there the GPU's is taken
        if sage:
            z_ref, Z, H_ref = layers.sage_forward(P, X, n, Wd, True, gm, order=order)
        else:
            A_ref, Z, H_ref = layers.layer_forward(P, X, Wd, True, gm, order=order)
        mask, flips = certify_relu(Z, H_gpu, z_bound(P, X, input_rounding(X), Wd, dt, sage, gm),
                                   f"{kind} {model} {norm} {order} {dt} vs {gm}")
        if sage:
            G_ref, Jf_ref = layers.sage_backward(P, z_ref, X[:n], Z, J, Wd, True, True, gm, order=order, X_full=X,
                                                 mask=mask)
        else:
            G_ref, Jf_ref = layers.layer_backward(P, A_ref, Z, J, Wd, True, True, gm, order=order, H_full=X,
                                                  mask=mask)
        refs[gm] = dict(H_ref=H_ref, G_ref=G_ref, Jf_ref=Jf_ref, flips=flips)
    return dict(info=B.pgcn_partition_info(part), n=n, b=b, H=H_gpu, G=dG.cpu().numpy(),
                J_in=host(J_in, f_in), J_bd=host(J_bd, f_in) if b else np.zeros((0, f_in)), refs=refs)


def check(r, dt, what):
    """Every reading of the oracle at the path's tolerance; both error metrics reported."""
    tol = TOL[dt]
    n = r["n"]
    for gm, ref in r["refs"].items():
        pairs = {"H": (r["H"], ref["H_ref"], tol["act"]), "G": (r["G"], ref["G_ref"], tol["grad"]),
                 "J_in": (r["J_in"], ref["Jf_ref"][:n], tol["grad"]),
                 "J_bd": (r["J_bd"], ref["Jf_ref"][n:], tol["grad"])}
        errs = {k: (rel_err(g, o), elem_err(g, o), t) for k, (g, o, t) in pairs.items()}
        print(f"{what} vs {gm}: flips {ref['flips']}, " +
              ", ".join(f"{k} {e:.2e} (elem {el:.2e})" for k, (e, el, _) in errs.items()))
        bad = {k: v for k, v in errs.items() if not v[0] < v[2]}
        assert not bad, (what, gm, bad)


@pytest.mark.parametrize("model,norm,order", FORMS)
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("kind", ["one_partition", "no_edges"])
def test_degenerate_partitions(kind, model, norm, order, dt):
    r = run_layer(kind, model, norm, order, dt)
    if kind == "one_partition":
        assert r["b"] == 0
    check(r, dt, f"{kind} {model} {norm} {order}")


@pytest.mark.parametrize("model,norm,order", FORMS)
def test_empty_partition(model, norm, order):
    r = run_layer("empty", model, norm, order, "f32")
    assert r["n"] == 0 and r["b"] == 0
    assert np.all(r["G"] == 0)


@pytest.mark.parametrize("model,norm,order", [("gcn", "mean", "agg"), ("gcn", "mean", "transform"),
                                              ("sage", "mean", "agg"), ("sage", "mean", "transform")])
@pytest.mark.parametrize("f_in,f_out", [(B.PGCN_MAX_WIDTH, 8), (8, B.PGCN_MAX_WIDTH)])
def test_maximum_width(model, norm, order, f_in, f_out):
    r = run_layer("small", model, norm, order, "f32", f_in=f_in, f_out=f_out)
    check(r, "f32", f"max width {model} {order} {f_in}x{f_out}")


@pytest.mark.parametrize("entry", ["fwd", "bwd", "sage_fwd", "sage_bwd"])
@pytest.mark.parametrize("wide", ["in", "out"])
def test_width_above_maximum_is_rejected(entry, wide):
    n_g, rowptr, col, owner, nparts = graph("small")
    sage = entry.startswith("sage")
    part = B.pgcn_partition_setup(n_g, rowptr, col, owner, nparts, 0, self_loop=not sage)
    info = B.pgcn_partition_info(part)
    n, b = info["n_inner"], info["n_bd"]
    f_in, f_out = (B.PGCN_MAX_WIDTH + 1, 8) if wide == "in" else (8, B.PGCN_MAX_WIDTH + 1)
    li, lo = ld_of(f_in), ld_of(f_out)
    k = 2 if sage else 1
    # buffers of the full sizes the call would use, so nothing could go out of bounds
    z = lambda r, c: torch.zeros((max(r, 1), c), device="cuda")
    nb = max(B.pgcn_workspace_size(part, f_in, f_out, B.PGCN_F32), 256)
    common = dict(f_in=f_in, f_out=f_out, gemm_dtype=B.PGCN_F32, relu=True, ld_in=li, ld_out=lo,
                  W=z(k * f_in, f_out), workspace=torch.zeros(nb, dtype=torch.uint8, device="cuda"), workspace_bytes=nb)
    with pytest.raises(B.PgcnError) as e:
        if entry == "fwd":
            B.pgcn_layer_fwd(part, H_in=z(n, li), H_bd=z(b, li), A=z(n, li), A_bf16=None, H_out=z(n, lo), **common)
        elif entry == "bwd":
            B.pgcn_layer_bwd(part, J_out=z(n, lo), H_out=z(n, lo), A=z(n, li), A_bf16=None, dW=z(f_in, f_out),
                             J_in=z(n, li), J_bd_out=z(b, li), **common)
        elif entry == "sage_fwd":
            B.pgcn_sage_layer_fwd(part, X_in=z(n, li), X_in_bf16=None, X_bd=z(b, li), A=z(n, li), A_bf16=None,
                                  H_out=z(n, lo), **common)
        else:
            B.pgcn_sage_layer_bwd(part, J_out=z(n, lo), H_out=z(n, lo), A=z(n, li), A_bf16=None, X_in=z(n, li),
                                  X_in_bf16=None, X_bd=z(b, li), dW=z(2 * f_in, f_out), J_in=z(n, li),
                                  J_bd_out=z(b, li), **common)
    assert e.value.code == B.PGCN_EINVAL
    assert "PGCN_MAX_WIDTH" in str(e.value)


@pytest.mark.parametrize("model,norm,order", FORMS)
@pytest.mark.parametrize("f_in,f_out", [(41, 72), (72, 41), (64, 65), (65, 64)])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_narrow_and_wide_plans(model, norm, order, f_in, f_out, dt):
    r = run_layer("two_plans", model, norm, order, dt, f_in=f_in, f_out=f_out)
    info = r["info"]
    assert (info["spmm_chunks"], info["spmm_chunks_narrow"]) == (2, 1)
    assert (info["spmmt_chunks"], info["spmmt_chunks_narrow"]) == (2, 1)
    check(r, dt, f"two plans {model} {norm} {order} {f_in}x{f_out}")
