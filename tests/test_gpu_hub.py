"""The dense block on the matrix cores (PGCN_HUB_ROWS / PGCN_HUB_COLS force its
size on small graphs; the Reddit-like partition selects one by itself):
layer forward and backward of every form through the C ABI against the
oracle, element by element, with the block's rows and columns padded
(sizes not multiples of the 512-row and 32-column tiles), three column
chunks or one, a narrow plan (rows of at most 64 floats) with chunks of its
own sharing the block, split rows in the rest of the plan, widths of one, several and a partial
64-float4 pass, and both GEMM precisions (bf16 against both oracle
readings).  ReLU decisions that differ from the oracle's are certified
(tests/certify.py)."""
import os

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

ORDER = {"agg": B.PGCN_ORDER_AGG, "transform": B.PGCN_ORDER_TRANSFORM}
ENV = {"PGCN_HUB_ROWS": "600", "PGCN_HUB_COLS": "1000", "PGCN_AGG_CHUNKS": "3", "PGCN_SEGMENT": "64"}
# one column chunk: the block sums are the rows' only other contribution
ENV_ONE = {"PGCN_HUB_ROWS": "600", "PGCN_HUB_COLS": "1000", "PGCN_AGG_CHUNKS": "1"}
# a narrow plan (rows of at most 64 floats, 2 chunks) beside the 3-chunk wide one, both with the block
ENV_NARROW = {"PGCN_HUB_ROWS": "600", "PGCN_HUB_COLS": "1000", "PGCN_AGG_CHUNKS": "3", "PGCN_AGG_CHUNKS_NARROW": "2",
              "PGCN_SEGMENT": "64"}
_PARTS = {}


def part(model, norm, env=None):
    env = env or ENV
    key = (model, norm, tuple(sorted(env.items())))
    if key not in _PARTS:
        n_g, rowptr, col, owner = random_partition_graph(3000, 2000, 3, 40, 21, hub_deg=2500)
        sage = model == "sage"
        ref = build_partition(n_g, rowptr, col, owner, 0, 3, self_loop=not sage)
        old = {k: os.environ.get(k) for k in env}
        os.environ.update(env)
        try:
            h = B.pgcn_partition_setup(n_g, rowptr, col, owner, 3, 0, self_loop=not sage, symmetric=norm == "sym")
        finally:
            for k, v in old.items():
                if v is None:
                    os.environ.pop(k, None)
                else:
                    os.environ[k] = v
        info = B.pgcn_partition_info(h)
        assert (info["spmm_hub_rows"], info["spmm_hub_cols"]) == (600, 1000)
        assert (info["spmmt_hub_rows"], info["spmmt_hub_cols"]) == (600, 1000)
        assert info["spmm_hub_nnz"] > 0 and info["spmmt_hub_nnz"] > 0
        assert info["spmm_chunks"] == int(env["PGCN_AGG_CHUNKS"])
        narrow = int(env.get("PGCN_AGG_CHUNKS_NARROW", env["PGCN_AGG_CHUNKS"]))
        assert (info["spmm_chunks_narrow"], info["spmmt_chunks_narrow"]) == (narrow, narrow)
        _PARTS[key] = (ref, propagation_matrix(ref, norm), h)
    return _PARTS[key]


FORMS = [("gcn", "mean", "agg"), ("gcn", "mean", "transform"), ("gcn", "sym", "agg"), ("gcn", "sym", "transform"),
         ("sage", "mean", "agg"), ("sage", "mean", "transform")]


@pytest.mark.parametrize("model,norm,order", FORMS)
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("f_in,f_out", [(256, 256), (41, 47), (300, 72), (602, 256), (64, 300)])
def test_layer_with_dense_block(model, norm, order, dt, f_in, f_out):
    check_layer(model, norm, order, dt, f_in, f_out, ENV)


@pytest.mark.parametrize("model,norm,order", [("gcn", "mean", "agg"), ("gcn", "sym", "transform"),
                                              ("sage", "mean", "agg")])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("f_in,f_out", [(256, 256), (41, 47)])
def test_layer_with_dense_block_one_chunk(model, norm, order, dt, f_in, f_out):
    check_layer(model, norm, order, dt, f_in, f_out, ENV_ONE)


@pytest.mark.parametrize("model,norm,order", FORMS)
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("f_in,f_out", [(41, 47), (64, 300), (300, 64), (7, 5)])
def test_layer_with_dense_block_narrow_plan(model, norm, order, dt, f_in, f_out):
    check_layer(model, norm, order, dt, f_in, f_out, ENV_NARROW)


def check_layer(model, norm, order, dt, f_in, f_out, env):
    ref, P, part_h = part(model, norm, env)
    sage = model == "sage"
    n, b = ref.n_inner, ref.n_bd
    rng = np.random.default_rng(f_in * 131 + f_out)
    X = rng.standard_normal((n + b, f_in))
    k = 2 if sage else 1
    W = rng.uniform(-0.3, 0.3, (k * f_in, f_out)).astype(np.float32)
    J = rng.standard_normal((n, f_out)) * 1e-2
    dtype = B.PGCN_BF16 if dt == "bf16" else B.PGCN_F32
    nb = max(B.pgcn_layer_workspace_size(part_h, f_in, f_out, dtype, ORDER[order]), 256)
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
        B.pgcn_sage_layer_fwd(part_h, X_in=dX, X_in_bf16=dX16, X_bd=dXbd, A=A, A_bf16=A16, H_out=H, **common)
    else:
        B.pgcn_layer_fwd(part_h, H_in=dX, H_bd=dXbd, A=A, A_bf16=A16, H_out=H, **common)
    dG = torch.full((k * f_in, f_out), 3.0, device="cuda")
    J_in, J_bd = dev(np.zeros((n, f_in))), dev(np.zeros((b, f_in)))
    if sage:
        B.pgcn_sage_layer_bwd(part_h, J_out=dev(J), H_out=H, A=A, A_bf16=A16, X_in=dX, X_in_bf16=dX16, X_bd=dXbd,
                              dW=dG, J_in=J_in, J_bd_out=J_bd, **common)
    else:
        B.pgcn_layer_bwd(part_h, J_out=dev(J), H_out=H, A=A, A_bf16=A16, dW=dG, J_in=J_in, J_bd_out=J_bd,
                         H_in=dX, H_bd=dXbd, **common)
    torch.cuda.synchronize()
    H_gpu = host(H, f_out)
    got = {"H": H_gpu, "G": dG.cpu().numpy(), "J_in": host(J_in, f_in), "J_bd": host(J_bd, f_in)}
    if agg and dt == "f32":
        got["A"] = host(A, f_in)
    Wd = W.astype(np.float64)
    tol = TOL[dt]
    for gm in readings(dt):
        if sage:
            z_ref, Z, H_ref = layers.sage_forward(P, X, n, Wd, True, gm, order=order)
            A_ref = z_ref
        else:
            A_ref, Z, H_ref = layers.layer_forward(P, X, Wd, True, gm, order=order)
        mask, flips = certify_relu(Z, H_gpu, z_bound(P, X, input_rounding(X), Wd, dt, sage, gm),
                                   f"{model} {norm} {order} {dt} vs {gm}")
        if sage:
            G_ref, Jf_ref = layers.sage_backward(P, z_ref, X[:n], Z, J, Wd, True, True, gm, order=order, X_full=X,
                                                 mask=mask)
        else:
            G_ref, Jf_ref = layers.layer_backward(P, A_ref, Z, J, Wd, True, True, gm, order=order, H_full=X,
                                                  mask=mask)
        ref_v = {"H": (H_ref, tol["act"]), "G": (G_ref, tol["grad"]), "J_in": (Jf_ref[:n], tol["grad"]),
                 "J_bd": (Jf_ref[n:], tol["grad"])}
        if "A" in got:
            ref_v["A"] = (A_ref, 1e-5)          # the aggregation itself stays fp32
        errs = {k: (rel_err(got[k], r), elem_err(got[k], r), t) for k, (r, t) in ref_v.items()}
        print(f"{model} {norm} {order} {dt} {f_in}x{f_out} vs {gm}: flips {flips}; " +
              ", ".join(f"{k} {e:.1e}/{el:.1e}" for k, (e, el, _) in errs.items()))
        bad = {k: v for k, v in errs.items() if not v[0] < v[2]}
        assert not bad, bad


def test_dense_block_is_deterministic():
    ref, P, part_h = part("gcn", "mean")
    n, b = ref.n_inner, ref.n_bd
    f = 256
    rng = np.random.default_rng(3)
    X = rng.standard_normal((n + b, f))
    W = torch.from_numpy(rng.uniform(-0.3, 0.3, (f, f)).astype(np.float32)).cuda()
    nb = B.pgcn_layer_workspace_size(part_h, f, f, B.PGCN_F32, B.PGCN_ORDER_AGG)
    outs = []
    for _ in range(2):
        ws = torch.full((nb,), 7, dtype=torch.uint8, device="cuda")
        A, H = dev(np.zeros((n, f))), dev(np.zeros((n, f)))
        B.pgcn_layer_fwd(part_h, f_in=f, f_out=f, gemm_dtype=B.PGCN_F32, relu=True, ld_in=f, ld_out=f, H_in=dev(X[:n]),
                         H_bd=dev(X[n:]), W=W, A=A, A_bf16=None, H_out=H, workspace=ws, workspace_bytes=nb)
        torch.cuda.synchronize()
        outs.append((A.clone(), H.clone()))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
