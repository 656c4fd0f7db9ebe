"""GPU parity of the transform-first GCN layer (P (H W); T = Pᵀ M, G = H_fullᵀ T,
J_full = T Wᵀ) against the oracle's reading of the same association, through
the C ABI: layer by layer on random partitions (plain, a split hub row,
column-chunked and segmented plans; with and without boundary rows; fp32 and
bf16), and Partition 0's whole step on the Tiny workload (injected state and
the autonomous pipeline) with every layer, or only the narrowing ones,
transform-first."""
import numpy as np
import pytest
import torch

from gpu_helpers import TOL, dev, host, rel_err
from oracle import layers
from oracle.pipegcn import Options, run
from paper_2203_10428_amd import binding as B
from paper_2203_10428_amd import configs
from paper_2203_10428_amd.step import PartitionTrainer, StepOptions, ld_of
from test_gpu_kernels import Graph
from dataclasses import replace

from certify import certified_reference, readings
from test_gpu_pipegcn import compare_step, exact_decisions, inject, put, sim_reference

pytestmark = pytest.mark.gpu

TF = B.PGCN_ORDER_TRANSFORM


@pytest.fixture(scope="module")
def graphs():
    return {"plain": Graph(), "hub": Graph(n_inner=2500, n_pool=900, seed=1, hub_deg=3000),
            "chunked": Graph(n_inner=2000, n_pool=1200, seed=2, mean_deg=60, hub_deg=2000,
                             env={"PGCN_AGG_CHUNKS": "3", "PGCN_SEGMENT": "16"}),
            # 5,000 inner and several thousand boundary rows: many row tiles in both GEMM halves
            "tall": Graph(n_inner=5000, n_pool=6000, nparts=2, seed=3, mean_deg=10)}


def ws_tf(g, f_in, f_out, dt):
    nbytes = B.pgcn_layer_workspace_size(g.part, f_in, f_out, dt, TF)
    assert nbytes > 0
    return torch.empty(nbytes, dtype=torch.uint8, device="cuda"), nbytes


@pytest.mark.parametrize("gname", ["plain", "hub", "chunked", "tall"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("f_in,f_out", [(3, 1), (47, 41), (128, 47), (602, 256), (256, 41), (512, 100), (1100, 16),
                                        (100, 128)])
@pytest.mark.parametrize("with_bd", [True, False])
def test_transform_forward(graphs, gname, dt, f_in, f_out, with_bd):
    g = graphs[gname]
    rng = np.random.default_rng(f_in * 1000 + f_out + 17)
    n, b = g.ref.n_inner, g.ref.n_bd
    H_in = rng.standard_normal((n, f_in))
    H_bd = rng.standard_normal((b, f_in)) if with_bd else np.zeros((b, f_in))
    W = rng.uniform(-0.2, 0.2, (f_in, f_out)).astype(np.float32)
    relu = f_out not in (1, 41)
    dtype = B.PGCN_BF16 if dt == "bf16" else B.PGCN_F32
    H = dev(np.full((n, f_out), 7.0))
    ws, nb = ws_tf(g, f_in, f_out, dtype)
    B.pgcn_layer_fwd(g.part, f_in=f_in, f_out=f_out, gemm_dtype=dtype, relu=relu, ld_in=ld_of(f_in),
                     ld_out=ld_of(f_out), H_in=dev(H_in), H_bd=dev(H_bd) if with_bd else None,
                     W=torch.from_numpy(W).cuda(), A=None, A_bf16=None, H_out=H, workspace=ws, workspace_bytes=nb,
                     order=TF)
    for gm in readings(dt):             # bf16: the fp64 oracle and its bf16-operand reading
        _, _, H_ref = layers.layer_forward(g.P, np.vstack([H_in, H_bd]), W.astype(np.float64), relu, gm,
                                           order="transform")
        assert rel_err(host(H, f_out), H_ref) < TOL[dt]["act"], gm
    pad = host(H, ld_of(f_out))[:, f_out:(f_out + 3) // 4 * 4]       # padding columns written as zeros
    assert np.all(pad == 0)


@pytest.mark.parametrize("gname", ["plain", "hub", "chunked", "tall"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("f_in,f_out", [(3, 1), (47, 41), (602, 256), (256, 41), (512, 100), (1100, 16), (100, 128)])
@pytest.mark.parametrize("input_grad", [True, False])
@pytest.mark.parametrize("with_bd", [True, False])
def test_transform_backward(graphs, gname, dt, f_in, f_out, input_grad, with_bd):
    g = graphs[gname]
    rng = np.random.default_rng(f_in * 7 + f_out + 3)
    n, b = g.ref.n_inner, g.ref.n_bd
    H_in = rng.standard_normal((n, f_in))
    H_bd = rng.standard_normal((b, f_in)) if with_bd else np.zeros((b, f_in))
    Z = rng.standard_normal((n, f_out))
    J = rng.standard_normal((n, f_out)) * 1e-2
    W = rng.uniform(-0.2, 0.2, (f_in, f_out)).astype(np.float32)
    relu = f_out not in (1, 41)
    H_out = np.maximum(Z, 0) if relu else Z                          # mask source: H > 0 <=> Z > 0
    dtype = B.PGCN_BF16 if dt == "bf16" else B.PGCN_F32
    dG = torch.full((f_in, f_out), 5.0, device="cuda")
    J_in = dev(np.zeros((n, f_in))) if input_grad else None
    J_bd = dev(np.zeros((b, f_in))) if input_grad else None
    ws, nb = ws_tf(g, f_in, f_out, dtype)
    B.pgcn_layer_bwd(g.part, f_in=f_in, f_out=f_out, gemm_dtype=dtype, relu=relu, ld_in=ld_of(f_in),
                     ld_out=ld_of(f_out), J_out=dev(J), H_out=dev(H_out), A=None, A_bf16=None,
                     W=torch.from_numpy(W).cuda(), dW=dG, J_in=J_in, J_bd_out=J_bd, workspace=ws, workspace_bytes=nb,
                     order=TF, H_in=dev(H_in), H_bd=dev(H_bd) if with_bd else None)
    tol = TOL[dt]["grad"]
    torch.cuda.synchronize()
    for gm in readings(dt):             # bf16: the fp64 oracle and its bf16-operand reading
        G_ref, Jf_ref = layers.layer_backward(g.P, None, Z, J, W.astype(np.float64), relu, input_grad, gm,
                                              order="transform", H_full=np.vstack([H_in, H_bd]))
        assert rel_err(dG.cpu().numpy(), G_ref) < tol, gm
        if input_grad:
            assert rel_err(host(J_in, f_in), Jf_ref[:n]) < tol, gm
            assert rel_err(host(J_bd, f_in), Jf_ref[n:]) < tol, gm


@pytest.mark.parametrize("gname", ["hub", "chunked"])
def test_transform_backward_is_deterministic(graphs, gname):
    g = graphs[gname]
    rng = np.random.default_rng(4)
    n, b = g.ref.n_inner, g.ref.n_bd
    f_in, f_out = 300, 100
    args = dict(f_in=f_in, f_out=f_out, gemm_dtype=B.PGCN_F32, relu=True, ld_in=ld_of(f_in), ld_out=ld_of(f_out),
                J_out=dev(rng.standard_normal((n, f_out))), H_out=dev(rng.standard_normal((n, f_out))),
                A=None, A_bf16=None, W=torch.from_numpy(rng.standard_normal((f_in, f_out)).astype(np.float32)).cuda(),
                order=TF, H_in=dev(rng.standard_normal((n, f_in))), H_bd=dev(rng.standard_normal((b, f_in))))
    outs = []
    for _ in range(2):
        dG = torch.zeros((f_in, f_out), device="cuda")
        J_in, J_bd = dev(np.zeros((n, f_in))), dev(np.zeros((b, f_in)))
        ws, nb = ws_tf(g, f_in, f_out, B.PGCN_F32)
        B.pgcn_layer_bwd(g.part, dW=dG, J_in=J_in, J_bd_out=J_bd, workspace=ws, workspace_bytes=nb, **args)
        torch.cuda.synchronize()
        outs.append((dG.cpu(), J_in.cpu(), J_bd.cpu()))
    for a, b_ in zip(*outs):
        assert torch.equal(a, b_)


def test_transform_argument_errors(graphs):
    g = graphs["plain"]
    n = g.ref.n_inner
    f_in, f_out = 64, 16
    ws, nb = ws_tf(g, f_in, f_out, B.PGCN_F32)
    common = dict(f_in=f_in, f_out=f_out, gemm_dtype=B.PGCN_F32, relu=True, ld_in=ld_of(f_in), ld_out=ld_of(f_out),
                  H_in=dev(np.zeros((n, f_in))), H_bd=None, W=torch.zeros((f_in, f_out), device="cuda"), A=None,
                  A_bf16=None, H_out=dev(np.zeros((n, f_out))))
    with pytest.raises(B.PgcnError, match="bad order"):
        B.pgcn_layer_fwd(g.part, workspace=ws, workspace_bytes=nb, order=7, **common)
    with pytest.raises(B.PgcnError, match="workspace"):
        B.pgcn_layer_fwd(g.part, workspace=ws, workspace_bytes=1024, order=TF, **common)
    assert B.pgcn_layer_workspace_size(g.part, f_in, f_out, B.PGCN_F32, 5) == 0
    assert B.pgcn_layer_workspace_size(g.part, f_in, f_out, B.PGCN_F32, B.PGCN_ORDER_AGG) == \
        B.pgcn_workspace_size(g.part, f_in, f_out, B.PGCN_F32)
    with pytest.raises(B.PgcnError, match="H_in"):
        B.pgcn_layer_bwd(g.part, f_in=f_in, f_out=f_out, gemm_dtype=B.PGCN_F32, relu=True, ld_in=ld_of(f_in),
                         ld_out=ld_of(f_out), J_out=dev(np.zeros((n, f_out))), H_out=dev(np.zeros((n, f_out))),
                         A=None, A_bf16=None, W=torch.zeros((f_in, f_out), device="cuda"),
                         dW=torch.zeros((f_in, f_out), device="cuda"), J_in=None, J_bd_out=None, workspace=ws,
                         workspace_bytes=nb, order=TF, H_in=None)


def tiny_setup(T, sf, sg, gemm, order):
    w = configs.TINY
    g = configs.make_graph(w)
    d = configs.make_dense(w, g.n)
    opts = Options(mode="pipe", smooth_f=sf, smooth_g=sg, gamma=w.gamma, eta=w.eta, loss=w.loss,
                   loss_scale=w.loss_scale, gemm=gemm, order=order)
    sim, recs = run(g.n, g.rowptr, g.col, g.owner, g.nparts, d.X, d.labels, d.W, T, opts)
    return w, g, d, sim, recs


@pytest.mark.parametrize("sf,sg", [(False, False), (True, True)])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_tiny_injected_transform(sf, sg, dt):
    T = 3
    w, g, d, sim, recs = tiny_setup(T, sf, sg, "f64", "transform")
    L = w.layers
    tr = PartitionTrainer(g, d.X, d.labels, d.W, w.widths, w.loss, w.loss_scale, dt,
                          StepOptions(smooth_f=sf, smooth_g=sg, gamma=w.gamma, eta=w.eta, copy_mode="none",
                                      order="transform"))
    assert all(tr.order[l] == TF and tr.A[l] is None for l in range(1, L + 1))
    for t in range(1, T + 1):
        r0, r1 = recs[t - 1][0], recs[t - 1][1]
        inject(tr, r0, r1, L)
        torch.cuda.synchronize()
        tr.step()
        tr.synchronize()
        H_gpu = {l: host(tr.H[l], w.widths[l]) for l in range(1, L + 1)}
        for gm in readings(dt):
            ref = certified_reference(sim, r0, r1, replace(sim.opts, gemm=gm), H_gpu, dt)
            compare_step(tr, ref, dt, L, w.widths, f"transform {dt} t={t} vs {gm}")


@pytest.mark.parametrize("order", ["transform", "auto"])
def test_tiny_autonomous_transform(order):
    T = 4
    w, g, d, sim, recs = tiny_setup(T, True, True, "f64", order)
    L = w.layers
    tr = PartitionTrainer(g, d.X, d.labels, d.W, w.widths, w.loss, w.loss_scale, "f32",
                          StepOptions(smooth_f=True, smooth_g=True, gamma=w.gamma, eta=w.eta, copy_mode="pipe",
                                      order=order))
    for t in range(1, T + 1):
        r0, r1 = recs[t - 1][0], recs[t - 1][1]
        so = r0["state_out"]
        torch.cuda.synchronize()
        for l in range(1, L + 1):
            put(tr.remote_f[l], so.feat_buf[l])
        for l in range(2, L + 1):
            put(tr.remote_g[l], so.grad_buf[l])
        for l in range(L):
            tr.G_peer[l] = torch.from_numpy(r1["G"][l + 1].astype(np.float32)).cuda()
        torch.cuda.synchronize()
        tr.step()
        tr.synchronize()
        exact_decisions(tr, r0, L, w.widths, f"autonomous {order} t={t}")
        compare_step(tr, sim_reference(r0), "f32", L, w.widths, f"autonomous {order} t={t}")


@pytest.mark.parametrize("sf,sg", [(False, False), (True, True)])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("mode", ["pipe", "serial"])
def test_tiny_layer1_cached(sf, sg, dt, mode):
    """Layer 1's aggregate kept across iterations (the input features are constant): the step
    still reproduces the oracle's PipeGCN (or, with serial refills, its synchronous reading)."""
    from oracle.pipegcn import Options as O
    T = 5
    w = configs.TINY
    g = configs.make_graph(w)
    d = configs.make_dense(w, g.n)
    opts = O(mode="pipe" if mode == "pipe" else "vanilla", smooth_f=sf, smooth_g=sg, gamma=w.gamma, eta=w.eta,
             loss=w.loss, loss_scale=w.loss_scale, gemm="bf16" if dt == "bf16" else "f64")
    if mode == "serial":     # refilled before use: the oracle's vanilla mode without smoothing
        if sf or sg:
            pytest.skip("smoothing is defined on stale messages")
    sim, recs = run(g.n, g.rowptr, g.col, g.owner, g.nparts, d.X, d.labels, d.W, T, opts)
    L = w.layers
    tr = PartitionTrainer(g, d.X, d.labels, d.W, w.widths, w.loss, w.loss_scale, dt,
                          StepOptions(smooth_f=sf, smooth_g=sg, gamma=w.gamma, eta=w.eta, copy_mode=mode,
                                      order="auto", cache_layer1=True))
    assert tr.order[1] == B.PGCN_ORDER_AGG
    tol = TOL[dt]
    for t in range(1, T + 1):
        r0, r1 = recs[t - 1][0], recs[t - 1][1]
        src = r0["state_out"]       # pipe: consumed next iteration; vanilla: what this iteration used
        torch.cuda.synchronize()
        for l in range(1, L + 1):
            put(tr.remote_f[l], src.feat_buf[l])
        for l in range(2, L + 1):
            put(tr.remote_g[l], src.grad_buf[l])
        for l in range(L):
            tr.G_peer[l] = torch.from_numpy(r1["G"][l + 1].astype(np.float32)).cuda()
        torch.cuda.synchronize()
        tr.step()
        tr.synchronize()
        # an autonomous run: decisions must agree with the reading exactly (the injected tests certify
        # differing ones); on the bf16 path this run follows the oracle's bf16-operand reading
        exact_decisions(tr, r0, L, w.widths, f"layer-1 cached {dt} {mode} t={t}")
        errs = {"loss": abs(tr.loss.item() - r0["loss"]) / abs(r0["loss"])}
        for l in range(1, L + 1):
            errs[f"H{l}"] = rel_err(host(tr.H[l], w.widths[l]), r0["H"][l])
            errs[f"G{l}"] = rel_err(tr.dW[l - 1].cpu().numpy(), r0["G"][l])
        errs["A1"] = rel_err(host(tr.A1_used, w.widths[0]), r0["A"][1])
        for l in range(L):
            errs[f"W{l + 1}"] = rel_err(tr.W[l].cpu().numpy(), r0["W_out"][l])
        bad = {k: v for k, v in errs.items() if not v <= (tol["grad"] if k.startswith("G") else tol["act"])}
        assert not bad, (t, bad)
