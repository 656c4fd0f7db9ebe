"""GPU parity of the GraphSAGE layer, dropout and Adam entry points against the
fp64 oracle (the paper's experiment model: Section 2's CONCAT update, dropout
after the boundary receive, Adam), on seeded random partitions built without
self loops (several tiles, ragged widths, split rows, empty boundary input)."""
import os

import numpy as np
import pytest
import torch

from certify import readings
from gpu_helpers import TOL, dev, host, random_partition_graph, rel_err
from oracle import layers
from oracle.partition import build_partition, propagation_matrix
from oracle.philox import dropout_mask_rows
from paper_2203_10428_amd import binding as B
from paper_2203_10428_amd.step import ld_of

pytestmark = pytest.mark.gpu


class SageGraph:
    def __init__(self, n_inner=3000, n_pool=1500, nparts=4, mean_deg=12, seed=0, hub_deg=0, env=None):
        self.n, self.rowptr, self.col, self.owner = random_partition_graph(n_inner, n_pool, nparts, mean_deg, seed,
                                                                           hub_deg)
        self.ref = build_partition(self.n, self.rowptr, self.col, self.owner, 0, nparts, self_loop=False)
        self.P = propagation_matrix(self.ref)
        old = {k: os.environ.get(k) for k in (env or {})}
        os.environ.update(env or {})
        try:
            self.part = B.pgcn_partition_setup(self.n, self.rowptr, self.col, self.owner, nparts, 0, self_loop=False)
        finally:
            for k, v in old.items():
                if v is None:
                    os.environ.pop(k, None)
                else:
                    os.environ[k] = v
        self.info = B.pgcn_partition_info(self.part)


@pytest.fixture(scope="module")
def graphs():
    # mean_deg 3 leaves inner rows without neighbours (zero rows of the mean)
    return {"plain": SageGraph(), "sparse": SageGraph(n_inner=2000, n_pool=800, seed=3, mean_deg=1.5),
            "chunked": SageGraph(n_inner=2000, n_pool=1200, seed=2, mean_deg=60, hub_deg=2000,
                                 env={"PGCN_AGG_CHUNKS": "3", "PGCN_SEGMENT": "16"}),
            # 5,000 inner rows: 40 row tiles of the node-major GEMMs, the last one ragged
            "tall": SageGraph(n_inner=5000, n_pool=1500, seed=4, mean_deg=8)}


def ws_for(g, f_in, f_out, dt):
    nbytes = max(B.pgcn_workspace_size(g.part, f_in, f_out, dt), 256)
    return torch.empty(nbytes, dtype=torch.uint8, device="cuda"), nbytes


def test_sage_partition_matches_oracle(graphs):
    for g in graphs.values():
        ex = B.pgcn_partition_export(g.part)
        for k in ("inner_gid", "bd_gid", "rowptr", "col", "rowptr_t", "col_t", "send_idx", "inv_ptr", "inv_k"):
            assert np.array_equal(ex[k], getattr(g.ref, k).astype(ex[k].dtype)), k
    assert (np.diff(graphs["sparse"].ref.rowptr) == 0).any()          # rows without neighbours exist


@pytest.mark.parametrize("cols", [1, 3, 4, 41, 602])
@pytest.mark.parametrize("p", [0.0, 0.1, 0.5])
@pytest.mark.parametrize("row0", [0, 12345])
def test_dropout_mask_is_the_oracles(cols, p, row0):
    rows = 1537
    rng = np.random.default_rng(cols)
    x = rng.standard_normal((rows, cols)).astype(np.float32)
    dx = dev(x)
    out = torch.full_like(dx, 7.0)
    o16 = torch.zeros(dx.shape, dtype=torch.bfloat16, device="cuda")
    ld = ld_of(cols)
    B.pgcn_dropout(out, dx, rows, cols, ld, row0, p, 99, 2, 3, 17, o16, ld)
    keep = dropout_mask_rows(np.arange(row0, row0 + rows), cols, p, 99, 2, 3, 17) != 0
    scale = np.float32(1.0 / (1.0 - p))
    expect = np.where(keep, x * scale, np.float32(0.0)).astype(np.float32)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert np.array_equal(got[:, :cols] != 0, expect != 0)
    assert np.array_equal(got[:, :cols], expect)
    assert np.all(got[:, cols:(cols + 3) // 4 * 4] == 0)                 # padding written as zeros
    assert torch.equal(o16[:, :cols], out[:, :cols].to(torch.bfloat16))   # bf16 copy, nearest even
    # in place (the backward applies the forward's mask to a gradient)
    B.pgcn_dropout(dx, dx, rows, cols, ld, row0, p, 99, 2, 3, 17)
    torch.cuda.synchronize()
    assert np.array_equal(dx.cpu().numpy()[:, :cols], expect)


@pytest.mark.parametrize("t", [1, 2, 7])
@pytest.mark.parametrize("peer", [False, True])
def test_adam_update(t, peer):
    rng = np.random.default_rng(t)
    count = 70001
    W, G, Gp = (rng.standard_normal(count) for _ in range(3))
    m = rng.standard_normal(count) * 0.1
    v = rng.random(count) * 0.01
    d = {k: torch.from_numpy(a.astype(np.float32)).cuda() for k, a in dict(W=W, G=G, Gp=Gp, m=m, v=v).items()}
    B.pgcn_adam_update(d["W"], d["G"], d["Gp"] if peer else None, d["m"], d["v"], count, 0.003, 0.9, 0.999, 1e-8, t)
    W32, m32, v32 = (a.astype(np.float32).astype(np.float64) for a in (W, m, v))
    g32 = (G.astype(np.float32) + Gp.astype(np.float32)).astype(np.float64) if peer else \
        G.astype(np.float32).astype(np.float64)
    W_ref, m_ref, v_ref = layers.adam(W32, g32, m32, v32, t, 0.003)
    torch.cuda.synchronize()
    assert rel_err(d["m"].cpu().numpy(), m_ref) < 1e-6
    assert rel_err(d["v"].cpu().numpy(), v_ref) < 1e-6
    # |W| <= ~4.5: within two fp32 ulps; the steps themselves are 1e-3 .. 3e-2
    W_gpu = d["W"].cpu().numpy().astype(np.float64)
    assert np.abs(W_gpu - W_ref).max() < 1e-6
    step_gpu, step_ref = np.abs(W_gpu - W32).mean(), np.abs(W_ref - W32).mean()
    assert abs(step_gpu - step_ref) < 1e-3 * step_ref           # the update is applied


@pytest.mark.parametrize("gname", ["plain", "sparse", "chunked", "tall"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("f_in,f_out", [(3, 5), (41, 47), (100, 128), (300, 512), (602, 256)])
@pytest.mark.parametrize("with_bd", [True, False])
def test_sage_layer_forward(graphs, gname, dt, f_in, f_out, with_bd):
    g = graphs[gname]
    rng = np.random.default_rng(f_in * 1000 + f_out)
    n, b = g.ref.n_inner, g.ref.n_bd
    X_in = rng.standard_normal((n, f_in))
    X_bd = rng.standard_normal((b, f_in)) if with_bd else np.zeros((b, f_in))
    W = rng.uniform(-0.2, 0.2, (2 * f_in, f_out)).astype(np.float32)
    relu = f_out != 5
    bf16 = dt == "bf16"
    z_ref, _, _ = layers.sage_forward(g.P, np.vstack([X_in, X_bd]), n, W.astype(np.float64), relu)
    dtype = B.PGCN_BF16 if bf16 else B.PGCN_F32
    dX = dev(X_in)
    dX16 = dev(X_in, dtype=torch.bfloat16) if bf16 else None
    dXbd = dev(X_bd) if with_bd else None
    A = None if bf16 else dev(np.zeros((n, f_in)))
    A16 = torch.zeros((n, ld_of(f_in)), dtype=torch.bfloat16, device="cuda") if bf16 else None
    H = dev(np.zeros((n, f_out)))
    ws, nb = ws_for(g, f_in, f_out, dtype)
    B.pgcn_sage_layer_fwd(g.part, f_in=f_in, f_out=f_out, gemm_dtype=dtype, relu=relu, ld_in=ld_of(f_in),
                          ld_out=ld_of(f_out), X_in=dX, X_in_bf16=dX16, X_bd=dXbd, W=torch.from_numpy(W).cuda(),
                          A=A, A_bf16=A16, H_out=H, workspace=ws, workspace_bytes=nb)
    if A is not None:
        assert rel_err(host(A, f_in), z_ref) < 1e-5
    else:
        assert rel_err(host(A16, f_in), z_ref) < 1e-2
    for gm in readings(dt):             # bf16: the fp64 oracle and its bf16-operand reading
        _, _, H_ref = layers.sage_forward(g.P, np.vstack([X_in, X_bd]), n, W.astype(np.float64), relu, gm)
        assert rel_err(host(H, f_out), H_ref) < TOL[dt]["act"], gm


@pytest.mark.parametrize("gname", ["plain", "sparse", "chunked", "tall"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("f_in,f_out", [(5, 3), (47, 41), (128, 100), (256, 256), (602, 256)])
@pytest.mark.parametrize("input_grad", [True, False])
def test_sage_layer_backward(graphs, gname, dt, f_in, f_out, input_grad):
    g = graphs[gname]
    rng = np.random.default_rng(f_in * 7 + f_out)
    n, b = g.ref.n_inner, g.ref.n_bd
    z = rng.standard_normal((n, f_in))
    X_in = rng.standard_normal((n, f_in))
    Z = rng.standard_normal((n, f_out))
    J = rng.standard_normal((n, f_out)) * 1e-2
    W = rng.uniform(-0.2, 0.2, (2 * f_in, f_out)).astype(np.float32)
    relu = f_out != 3
    bf16 = dt == "bf16"
    dtype = B.PGCN_BF16 if bf16 else B.PGCN_F32
    if bf16:   # the bf16 path reads z and X_in as bf16: give the oracle the same rounded operands
        z = torch.from_numpy(z).to(torch.bfloat16).double().numpy()
        X_in = torch.from_numpy(X_in).to(torch.bfloat16).double().numpy()
    H_out = np.maximum(Z, 0) if relu else Z
    dz = None if bf16 else dev(z)
    dz16 = dev(z, dtype=torch.bfloat16) if bf16 else None
    dX = None if bf16 else dev(X_in)
    dX16 = dev(X_in, dtype=torch.bfloat16) if bf16 else None
    dG = torch.zeros((2 * f_in, f_out), device="cuda")
    J_in = dev(np.zeros((n, f_in))) if input_grad else None
    J_bd = dev(np.zeros((b, f_in))) if input_grad else None
    ws, nb = ws_for(g, f_in, f_out, dtype)
    B.pgcn_sage_layer_bwd(g.part, f_in=f_in, f_out=f_out, gemm_dtype=dtype, relu=relu, ld_in=ld_of(f_in),
                          ld_out=ld_of(f_out), J_out=dev(J), H_out=dev(H_out), A=dz, A_bf16=dz16, X_in=dX,
                          X_in_bf16=dX16, W=torch.from_numpy(W).cuda(), dW=dG, J_in=J_in, J_bd_out=J_bd,
                          workspace=ws, workspace_bytes=nb)
    tol = TOL[dt]["grad"]
    torch.cuda.synchronize()
    for gm in readings(dt):             # bf16: the fp64 oracle and its bf16-operand reading
        G_ref, Jf_ref = layers.sage_backward(g.P, z, X_in, Z, J, W.astype(np.float64), relu, input_grad, gm)
        assert rel_err(dG.cpu().numpy(), G_ref) < tol, gm
        if input_grad:
            assert rel_err(host(J_in, f_in), Jf_ref[:n]) < tol, gm
            assert rel_err(host(J_bd, f_in), Jf_ref[n:]) < tol, gm


@pytest.mark.parametrize("gname", ["plain", "sparse", "chunked", "tall"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("f_in,f_out", [(5, 3), (47, 41), (602, 256), (128, 100), (100, 128)])
@pytest.mark.parametrize("with_bd", [True, False])
def test_sage_layer_transform(graphs, gname, dt, f_in, f_out, with_bd):
    """Forward and backward in the transform-first association against the oracle's reading of it."""
    g = graphs[gname]
    rng = np.random.default_rng(f_in * 31 + f_out)
    n, b = g.ref.n_inner, g.ref.n_bd
    X_in = rng.standard_normal((n, f_in))
    X_bd = rng.standard_normal((b, f_in)) if with_bd else np.zeros((b, f_in))
    X_full = np.vstack([X_in, X_bd])
    W = rng.uniform(-0.2, 0.2, (2 * f_in, f_out)).astype(np.float32)
    relu = f_out != 3
    bf16 = dt == "bf16"
    dtype = B.PGCN_BF16 if bf16 else B.PGCN_F32
    dX, dXbd = dev(X_in), (dev(X_bd) if with_bd else None)
    dX16 = dev(X_in, dtype=torch.bfloat16) if bf16 else None
    H = dev(np.zeros((n, f_out)))
    nb = B.pgcn_layer_workspace_size(g.part, f_in, f_out, dtype, B.PGCN_ORDER_TRANSFORM)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    common = dict(f_in=f_in, f_out=f_out, gemm_dtype=dtype, relu=relu, ld_in=ld_of(f_in), ld_out=ld_of(f_out),
                  W=torch.from_numpy(W).cuda(), A=None, A_bf16=None, workspace=ws, workspace_bytes=nb,
                  order=B.PGCN_ORDER_TRANSFORM)
    B.pgcn_sage_layer_fwd(g.part, X_in=dX, X_in_bf16=dX16, X_bd=dXbd, H_out=H, **common)
    for gm in readings(dt):             # bf16: the fp64 oracle and its bf16-operand reading
        _, _, H_ref = layers.sage_forward(g.P, X_full, n, W.astype(np.float64), relu, gm, order="transform")
        assert rel_err(host(H, f_out), H_ref) < TOL[dt]["act"], gm
    # backward from a fixed Z (mask) and J
    Z = rng.standard_normal((n, f_out))
    J = rng.standard_normal((n, f_out)) * 1e-2
    dG = torch.zeros((2 * f_in, f_out), device="cuda")
    J_in, J_bd = dev(np.zeros((n, f_in))), dev(np.zeros((b, f_in)))
    B.pgcn_sage_layer_bwd(g.part, J_out=dev(J), H_out=dev(np.maximum(Z, 0) if relu else Z), X_in=dX, X_in_bf16=dX16,
                          X_bd=dXbd, dW=dG, J_in=J_in, J_bd_out=J_bd, **common)
    tol = TOL[dt]["grad"]
    torch.cuda.synchronize()
    for gm in readings(dt):
        G_ref, Jf_ref = layers.sage_backward(g.P, None, X_in, Z, J, W.astype(np.float64), relu, True, gm,
                                             order="transform", X_full=X_full)
        assert rel_err(dG.cpu().numpy(), G_ref) < tol, gm
        assert rel_err(host(J_in, f_in), Jf_ref[:n]) < tol, gm
        assert rel_err(host(J_bd, f_in), Jf_ref[n:]) < tol, gm


def test_layer_entry_points_check_the_partition_kind(graphs):
    g = graphs["plain"]
    n = g.ref.n_inner
    X = dev(np.zeros((n, 8)))
    ws, nb = ws_for(g, 8, 8, B.PGCN_F32)
    with pytest.raises(B.PgcnError, match="self loops"):
        B.pgcn_layer_fwd(g.part, f_in=8, f_out=8, gemm_dtype=B.PGCN_F32, relu=True, ld_in=8, ld_out=8, H_in=X,
                         H_bd=None, W=torch.zeros((8, 8), device="cuda"), A=X, A_bf16=None, H_out=X, workspace=ws,
                         workspace_bytes=nb)
    gcn = B.pgcn_partition_setup(g.n, g.rowptr, g.col, g.owner, 4, 0)
    with pytest.raises(B.PgcnError, match="NO_SELF_LOOP"):
        B.pgcn_sage_layer_fwd(gcn, f_in=8, f_out=8, gemm_dtype=B.PGCN_F32, relu=True, ld_in=8, ld_out=8, X_in=X,
                              X_in_bf16=None, X_bd=None, W=torch.zeros((16, 8), device="cuda"), A=X, A_bf16=None,
                              H_out=X, workspace=ws, workspace_bytes=nb)
    with pytest.raises(B.PgcnError, match="p must be"):
        B.pgcn_dropout(X, X, n, 8, 8, 0, 1.0, 1, 0, 1, 1)
