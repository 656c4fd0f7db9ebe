"""GPU parity of GCN layers on partitions built with the symmetric
normalisation D̃^{-1/2} (A + I) D̃^{-1/2} (PGCN_SETUP_SYMMETRIC), against the
oracle's matrix of the same name, through the C ABI: both associations of the
layer product, fp32 and bf16, with and without boundary rows, on the plain,
split-hub and chunked/segmented partitions; and Partition 0's whole step on
the Tiny workload (injected state, both associations; autonomous pipeline)."""
import os

import numpy as np
import pytest
import torch

from gpu_helpers import TOL, dev, host, random_partition_graph, rel_err
from oracle import layers
from oracle.partition import build_partition, propagation_matrix
from oracle.pipegcn import Options, run
from paper_2203_10428_amd import binding as B
from paper_2203_10428_amd import configs
from paper_2203_10428_amd.step import PartitionTrainer, StepOptions, ld_of
from dataclasses import replace

from certify import certified_reference, readings
from test_gpu_pipegcn import compare_step, exact_decisions, inject, put, sim_reference

pytestmark = pytest.mark.gpu


class SymGraph:
    def __init__(self, n_inner=3000, n_pool=1500, nparts=4, mean_deg=12, seed=0, hub_deg=0, env=None):
        self.n, self.rowptr, self.col, self.owner = random_partition_graph(n_inner, n_pool, nparts, mean_deg, seed,
                                                                           hub_deg)
        self.ref = build_partition(self.n, self.rowptr, self.col, self.owner, 0, nparts)
        self.P = propagation_matrix(self.ref, "sym")
        old = {k: os.environ.get(k) for k in (env or {})}
        os.environ.update(env or {})
        try:
            self.part = B.pgcn_partition_setup(self.n, self.rowptr, self.col, self.owner, nparts, 0, symmetric=True)
        finally:
            for k, v in old.items():
                if v is None:
                    os.environ.pop(k, None)
                else:
                    os.environ[k] = v


@pytest.fixture(scope="module")
def graphs():
    return {"plain": SymGraph(), "hub": SymGraph(n_inner=2500, n_pool=900, seed=1, hub_deg=3000),
            "chunked": SymGraph(n_inner=2000, n_pool=1200, seed=2, mean_deg=60, hub_deg=2000,
                                env={"PGCN_AGG_CHUNKS": "3", "PGCN_SEGMENT": "16"})}


def test_symmetric_setup(graphs):
    for g in graphs.values():
        info = B.pgcn_partition_info(g.part)
        assert info["symmetric"] == 1
        assert np.array_equal(B.pgcn_partition_export(g.part)["deg"], g.ref.deg)


ORDERS = {"agg": B.PGCN_ORDER_AGG, "transform": B.PGCN_ORDER_TRANSFORM}


@pytest.mark.parametrize("gname", ["plain", "hub", "chunked"])
@pytest.mark.parametrize("order", list(ORDERS))
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("f_in,f_out", [(41, 47), (602, 256), (256, 41)])
@pytest.mark.parametrize("with_bd", [True, False])
def test_sym_forward(graphs, gname, order, dt, f_in, f_out, with_bd):
    g = graphs[gname]
    rng = np.random.default_rng(f_in + f_out + 5)
    n, b = g.ref.n_inner, g.ref.n_bd
    H_in = rng.standard_normal((n, f_in))
    H_bd = rng.standard_normal((b, f_in)) if with_bd else np.zeros((b, f_in))
    W = rng.uniform(-0.2, 0.2, (f_in, f_out)).astype(np.float32)
    A_ref, _, _ = layers.layer_forward(g.P, np.vstack([H_in, H_bd]), W.astype(np.float64), True, order=order)
    dtype = B.PGCN_BF16 if dt == "bf16" else B.PGCN_F32
    agg = order == "agg"
    A = dev(np.zeros((n, f_in))) if agg and dt == "f32" else None
    A16 = torch.zeros((n, ld_of(f_in)), dtype=torch.bfloat16, device="cuda") if agg and dt == "bf16" else None
    H = dev(np.zeros((n, f_out)))
    nb = B.pgcn_layer_workspace_size(g.part, f_in, f_out, dtype, ORDERS[order])
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    B.pgcn_layer_fwd(g.part, f_in=f_in, f_out=f_out, gemm_dtype=dtype, relu=True, ld_in=ld_of(f_in),
                     ld_out=ld_of(f_out), H_in=dev(H_in), H_bd=dev(H_bd) if with_bd else None,
                     W=torch.from_numpy(W).cuda(), A=A, A_bf16=A16, H_out=H, workspace=ws, workspace_bytes=nb,
                     order=ORDERS[order])
    if A is not None:
        assert rel_err(host(A, f_in), A_ref) < 1e-5
    for gm in readings(dt):             # bf16: the fp64 oracle and its bf16-operand reading
        _, _, H_ref = layers.layer_forward(g.P, np.vstack([H_in, H_bd]), W.astype(np.float64), True, gm, order=order)
        assert rel_err(host(H, f_out), H_ref) < TOL[dt]["act"], gm


@pytest.mark.parametrize("gname", ["plain", "hub", "chunked"])
@pytest.mark.parametrize("order", list(ORDERS))
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("f_in,f_out", [(47, 41), (602, 256), (256, 41)])
def test_sym_backward(graphs, gname, order, dt, f_in, f_out):
    g = graphs[gname]
    rng = np.random.default_rng(f_in * 3 + f_out)
    n, b = g.ref.n_inner, g.ref.n_bd
    H_full = rng.standard_normal((n + b, f_in))
    A = rng.standard_normal((n, f_in))
    Z = rng.standard_normal((n, f_out))
    J = rng.standard_normal((n, f_out)) * 1e-2
    W = rng.uniform(-0.2, 0.2, (f_in, f_out)).astype(np.float32)
    dtype = B.PGCN_BF16 if dt == "bf16" else B.PGCN_F32
    if dt == "bf16" and order == "agg":      # the bf16 path reads A as bf16: the oracle gets the same rounded A
        A = torch.from_numpy(A).to(torch.bfloat16).double().numpy()
    agg = order == "agg"
    dA = dev(A) if agg and dt == "f32" else None
    dA16 = dev(A, dtype=torch.bfloat16) if agg and dt == "bf16" else None
    dG = torch.zeros((f_in, f_out), device="cuda")
    J_in, J_bd = dev(np.zeros((n, f_in))), dev(np.zeros((b, f_in)))
    nb = B.pgcn_layer_workspace_size(g.part, f_in, f_out, dtype, ORDERS[order])
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    B.pgcn_layer_bwd(g.part, f_in=f_in, f_out=f_out, gemm_dtype=dtype, relu=True, ld_in=ld_of(f_in),
                     ld_out=ld_of(f_out), J_out=dev(J), H_out=dev(np.maximum(Z, 0)), A=dA, A_bf16=dA16,
                     W=torch.from_numpy(W).cuda(), dW=dG, J_in=J_in, J_bd_out=J_bd, workspace=ws, workspace_bytes=nb,
                     order=ORDERS[order], H_in=dev(H_full[:n]), H_bd=dev(H_full[n:]))
    tol = TOL[dt]["grad"]
    torch.cuda.synchronize()
    for gm in readings(dt):             # bf16: the fp64 oracle and its bf16-operand reading
        G_ref, Jf_ref = layers.layer_backward(g.P, A, Z, J, W.astype(np.float64), True, True, gm, order=order,
                                              H_full=H_full)
        assert rel_err(dG.cpu().numpy(), G_ref) < tol, gm
        assert rel_err(host(J_in, f_in), Jf_ref[:n]) < tol, gm
        assert rel_err(host(J_bd, f_in), Jf_ref[n:]) < tol, gm


def tiny_setup(T, gemm, order):
    w = configs.TINY
    g = configs.make_graph(w)
    d = configs.make_dense(w, g.n)
    opts = Options(mode="pipe", smooth_f=True, smooth_g=True, gamma=w.gamma, eta=w.eta, loss=w.loss,
                   loss_scale=w.loss_scale, gemm=gemm, order=order, norm="sym")
    sim, recs = run(g.n, g.rowptr, g.col, g.owner, g.nparts, d.X, d.labels, d.W, T, opts)
    return w, g, d, sim, recs


@pytest.mark.parametrize("order", ["agg", "transform"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_tiny_injected_sym(order, dt):
    T = 3
    w, g, d, sim, recs = tiny_setup(T, "f64", order)
    L = w.layers
    tr = PartitionTrainer(g, d.X, d.labels, d.W, w.widths, w.loss, w.loss_scale, dt,
                          StepOptions(gamma=w.gamma, eta=w.eta, copy_mode="none", order=order, norm="sym"))
    assert tr.info["symmetric"] == 1
    for t in range(1, T + 1):
        r0, r1 = recs[t - 1][0], recs[t - 1][1]
        inject(tr, r0, r1, L)
        torch.cuda.synchronize()
        tr.step()
        tr.synchronize()
        H_gpu = {l: host(tr.H[l], w.widths[l]) for l in range(1, L + 1)}
        for gm in readings(dt):
            ref = certified_reference(sim, r0, r1, replace(sim.opts, gemm=gm), H_gpu, dt)
            compare_step(tr, ref, dt, L, w.widths, f"sym {order} {dt} t={t} vs {gm}")


def test_tiny_autonomous_sym():
    T = 4
    w, g, d, sim, recs = tiny_setup(T, "f64", "auto")
    L = w.layers
    tr = PartitionTrainer(g, d.X, d.labels, d.W, w.widths, w.loss, w.loss_scale, "f32",
                          StepOptions(gamma=w.gamma, eta=w.eta, copy_mode="pipe", order="auto", norm="sym"))
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
        exact_decisions(tr, r0, L, w.widths, f"autonomous sym t={t}")
        compare_step(tr, sim_reference(r0), "f32", L, w.widths, f"autonomous sym t={t}")
