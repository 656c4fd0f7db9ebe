"""Whole-step GPU parity at full size, in the bench's configuration.

One injected PipeGCN-GF iteration (Algorithm 1 at t = 2: the stale feature
and gradient buffers received in iteration 1 are consumed and both moving
averages updated; narrowing layers transform-first, as the bench runs them)
of the Reddit-like partition (fp32 update GEMMs) and of the products-like
partition (bf16 update GEMMs), with every output compared element by element
against the oracle's per-partition step (``partition_step``) on the whole
partition: activations of every layer, the loss, the feature gradients of the
inner and boundary rows, the weight gradients, the send buffers, both moving
averages and the updated weights.

The injected inputs are seeded: the stale buffers N(0,1) (features) and
1e-3 N(0,1) (gradient contributions), the moving averages half of that, the
peer's weight gradient (the other AllReduce operand) 1e-3 N(0,1); features,
labels and Glorot weights as the bench draws them.  ReLU decisions that
differ from the oracle's are certified against their rounding bounds before
the oracle's backward takes them (tests/certify.py); the bf16 partition is
held to the plain fp64 oracle and to its bf16-operand reading alike.

One oracle step is an fp64 pass over the whole partition (tens of seconds on
the host), so the work is split into three tests per workload that share a
module cache: the GPU step, the oracle's plain steps, then certification
(with a re-run of the oracle when decisions differ) and the comparison.
"""
from dataclasses import replace
from types import SimpleNamespace

import numpy as np
import pytest
import torch

from certify import certified_step, elem_err, readings
from gpu_helpers import TOL, rel_err
from oracle import layers
from oracle.partition import build_partition, propagation_matrix
from oracle.pipegcn import Options, partition_step
from paper_2203_10428_amd import configs
from paper_2203_10428_amd.step import PartitionTrainer, StepOptions

pytestmark = [pytest.mark.gpu, pytest.mark.slow, pytest.mark.timeout(900)]

NAMES = ["reddit-like-1of4", "products-like-1of8"]
_CACHE = {}


def put(t, x):
    t.zero_()
    t[:, : x.shape[1]] = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(t.device)


def get(t, f):
    return t[:, :f].float().cpu().numpy().astype(np.float64)


def injected_state(w, n_bd, n_send, seed=7):
    rng = np.random.default_rng(seed)
    L, wd = w.layers, w.widths
    feat = {l: rng.standard_normal((n_bd, wd[l - 1])) for l in range(1, L + 1)}
    ema_f = {l: 0.5 * rng.standard_normal((n_bd, wd[l - 1])) for l in range(1, L + 1)}
    grad = {l: 1e-3 * rng.standard_normal((n_send, wd[l - 1])) for l in range(2, L + 1)}
    ema_g = {l: 5e-4 * rng.standard_normal((n_send, wd[l - 1])) for l in range(2, L + 1)}
    G_peer = [1e-3 * rng.standard_normal((wd[l], wd[l + 1])) for l in range(L)]
    return SimpleNamespace(feat_buf=feat, grad_buf=grad, ema_f=ema_f, ema_g=ema_g), G_peer


def oracle_options(w):
    return Options(mode="pipe", smooth_f=True, smooth_g=True, gamma=w.gamma, eta=w.eta, loss=w.loss,
                   loss_scale=w.loss_scale, order="auto")


@pytest.mark.parametrize("name", NAMES)
def test_full_step_1_gpu(name):
    """The GPU step from the injected state; its outputs are kept for the comparison."""
    w = configs.WORKLOADS[name]
    g = configs.make_graph(w)
    d = configs.make_dense(w, g.n)
    p = build_partition(g.n, g.rowptr, g.col, g.owner, 0, g.nparts)
    n, b, s = p.n_inner, p.n_bd, len(p.send_idx)
    state, G_peer = injected_state(w, b, s)
    L, wd = w.layers, w.widths
    print(f"[{name}] GPU step ({n} inner, {b} boundary, {s} sent rows)", flush=True)
    tr = PartitionTrainer(g, d.X, d.labels, d.W, wd, w.loss, w.loss_scale, w.gemm_dtype,
                          StepOptions(smooth_f=True, smooth_g=True, gamma=w.gamma, eta=w.eta, copy_mode="none",
                                      order="auto"))
    assert (tr.n, tr.b, tr.s) == (n, b, s)
    for l in range(L):
        tr.G_peer[l] = torch.from_numpy(G_peer[l].astype(np.float32)).cuda()
    for l in range(1, L + 1):
        put(tr.feat[l][tr.cur], state.feat_buf[l])
        put(tr.ema_f[l], state.ema_f[l])
    for l in range(2, L + 1):
        put(tr.grad[l][tr.cur], state.grad_buf[l])
        put(tr.ema_g[l], state.ema_g[l])
    tr.t = 1
    torch.cuda.synchronize()
    tr.step()
    tr.synchronize()
    got = {"loss": np.array([tr.loss.item()])}
    for l in range(1, L + 1):
        got[f"H{l}"] = get(tr.H[l], wd[l])
        got[f"send_f{l}"] = get(tr.send_f[l], wd[l - 1])
        got[f"G{l}"] = tr.dW[l - 1].cpu().numpy().astype(np.float64)
        got[f"ema_f{l}"] = get(tr.ema_f[l], wd[l - 1])
        got[f"W{l}"] = tr.W[l - 1].cpu().numpy().astype(np.float64)
    for l in range(2, L + 1):
        got[f"J_in{l}"] = get(tr.J_in[l], wd[l - 1])
        got[f"J_bd{l}"] = get(tr.J_bd_out[l], wd[l - 1])
        got[f"ema_g{l}"] = get(tr.ema_g[l], wd[l - 1])
    assert all(np.isfinite(v).all() for v in got.values())
    del tr
    torch.cuda.empty_cache()
    _CACHE[name] = dict(w=w, p=p, P=propagation_matrix(p), X_in=np.asarray(d.X[p.inner_gid], dtype=np.float64),
                        y=d.labels[p.inner_gid], W=[np.asarray(x, dtype=np.float64) for x in d.W], state=state,
                        G_peer=G_peer, got=got, plain={})


@pytest.mark.parametrize("name", NAMES)
def test_full_step_2_oracle(name):
    """The oracle's plain step (each reading) from the same injected state."""
    c = _CACHE.get(name)
    if c is None:
        pytest.skip("the GPU step of this workload did not run")
    w, st = c["w"], c["state"]
    for gm in readings(w.gemm_dtype):
        print(f"[{name}] oracle step, {gm} reading", flush=True)
        cp = lambda dd: {k: v.copy() for k, v in dd.items()}
        ema_f, ema_g = cp(st.ema_f), cp(st.ema_g)
        rec = partition_step(c["p"], c["P"], c["X_in"], c["y"], c["W"], st.feat_buf, st.grad_buf, ema_f, ema_g, 2,
                             replace(oracle_options(w), gemm=gm))
        c["plain"][gm] = (rec, (ema_f, ema_g))


@pytest.mark.parametrize("name", NAMES)
def test_full_step_3_compare(name):
    """ReLU decisions certified (the oracle re-run with them when any differ), then every output
    compared element by element."""
    c = _CACHE.pop(name, None)
    if c is None or not c["plain"]:
        pytest.skip("the GPU step or the oracle step of this workload did not run")
    w, p, got = c["w"], c["p"], c["got"]
    dt, L, n = w.gemm_dtype, w.layers, c["p"].n_inner
    H_gpu = {l: got[f"H{l}"] for l in range(1, L + 1)}
    tol = TOL[dt]
    for gm, plain in c["plain"].items():
        rec, ema_f, ema_g, flips = certified_step(p, c["P"], c["X_in"], c["y"], c["W"], c["state"], 2,
                                                  replace(oracle_options(w), gemm=gm), H_gpu, dt, rec=plain)
        ref = {"loss": np.array([rec["loss"]])}
        for l in range(1, L + 1):
            ref[f"H{l}"] = rec["H"][l]
            ref[f"send_f{l}"] = rec["send_f"][l]
            ref[f"G{l}"] = rec["G"][l]
            ref[f"ema_f{l}"] = ema_f[l]
            ref[f"W{l}"] = layers.sgd(c["W"][l - 1], rec["G"][l] + c["G_peer"][l - 1], w.eta)
        for l in range(2, L + 1):
            ref[f"J_in{l}"] = rec["J_full"][l][:n]
            ref[f"J_bd{l}"] = rec["J_full"][l][n:]
            ref[f"ema_g{l}"] = ema_g[l]
        grad_keys = ("G", "J_in", "J_bd", "ema_g")
        errs = {}
        for k in ref:
            t = tol["grad"] if k.startswith(grad_keys) else tol["act"]
            errs[k] = (rel_err(got[k], ref[k]), elem_err(got[k], ref[k]), t)
        print(f"[{name}] vs {gm}: ReLU flips {flips}; " +
              ", ".join(f"{k} {e:.1e}/{el:.1e}" for k, (e, el, _) in errs.items()), flush=True)
        bad = {k: v for k, v in errs.items() if not v[0] <= v[2]}
        assert not bad, (name, gm, bad)
