"""Staleness diagnostics from the buffers the GPU actually consumes.

Section 3.4 motivates smoothing by the error that one-iteration-stale
boundary features and feature gradients carry.  Here partition 0 of the Tiny
workload runs autonomously on the GPU (its own ping-pong buffers, side-stream
refills and smoothing states; only what partition 1 sends and its weight
gradient are injected), and after every iteration the per-layer errors are
computed from what the GPU used: the boundary rows it aggregated (the stale
buffer, or its moving average) against what partition 1 holds in the same
iteration, and likewise the received gradient contributions it added.  They
must equal the oracle's diagnostics for partition 0
(``oracle.staleness.staleness_errors(parts=(0,))``), for plain PipeGCN and
for PipeGCN-GF at two decays, with a learning rate large enough that the
weights move and the errors are far from zero.
"""
import numpy as np
import pytest
import torch

from oracle.pipegcn import Options, run
from oracle.staleness import staleness_errors
from paper_2203_10428_amd import configs
from paper_2203_10428_amd.step import PartitionTrainer, StepOptions

pytestmark = pytest.mark.gpu

T = 6
ETA = 0.5


def put(t, x):
    t.zero_()
    t[:, : x.shape[1]] = torch.from_numpy(x.astype(np.float32)).cuda()


def get(t, f):
    return t[:, :f].float().cpu().numpy().astype(np.float64)


def frob_rel(used, now):
    return float(np.sqrt(np.sum((used - now) ** 2) / np.sum(now ** 2)))


@pytest.mark.parametrize("smooth,gamma", [(False, 0.95), (True, 0.5), (True, 0.95)])
def test_staleness_errors_of_the_consumed_buffers(smooth, gamma):
    w = configs.TINY
    g = configs.make_graph(w)
    d = configs.make_dense(w, g.n)
    L = w.layers
    opts = Options(mode="pipe", smooth_f=smooth, smooth_g=smooth, gamma=gamma, eta=ETA, loss=w.loss,
                   loss_scale=w.loss_scale)
    graph = (g.n, g.rowptr, g.col, g.owner, g.nparts)
    ref = {r["t"]: r for r in staleness_errors(*graph, d.X, d.labels, d.W, T, opts, vanilla_g=False, parts=(0,))}
    _, recs = run(*graph, d.X, d.labels, d.W, T, opts)
    tr = PartitionTrainer(g, d.X, d.labels, d.W, w.widths, w.loss, w.loss_scale, "f32",
                          StepOptions(smooth_f=smooth, smooth_g=smooth, gamma=gamma, eta=ETA, copy_mode="pipe"))
    for t in range(1, T + 1):
        r0, r1 = recs[t - 1][0], recs[t - 1][1]
        so = r0["state_out"]                 # what partition 1 sends in iteration t
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
        if t == 1:
            continue
        used = 1 - tr.cur                    # the buffer read in iteration t (the other one was refilled)
        errs = {}
        for l in range(1, L + 1):
            H_used = get(tr.ema_f[l] if smooth else tr.feat[l][used], w.widths[l - 1])
            errs[("feat", l)] = frob_rel(H_used, so.feat_buf[l])
        for l in range(2, L + 1):
            C_used = get(tr.ema_g[l] if smooth else tr.grad[l][used], w.widths[l - 1])
            errs[("grad", l)] = frob_rel(C_used, so.grad_buf[l])
        print(f"t={t} smooth={smooth} gamma={gamma}: " +
              ", ".join(f"{k}{l} {e:.4e} (oracle {ref[t][k][l]:.4e})" for (k, l), e in errs.items()))
        for (kind, l), e in errs.items():
            o = ref[t][kind][l]
            # layer 1 exchanges the constant input: exactly zero without smoothing
            assert abs(e - o) <= 1e-4 * o + 1e-6, (t, kind, l, e, o)
        if not smooth:
            assert errs[("feat", 1)] == 0.0 and errs[("feat", 2)] > 1e-3
