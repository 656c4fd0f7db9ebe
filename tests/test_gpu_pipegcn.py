"""End-to-end GPU parity of partition 0's PipeGCN step on the Tiny workload
(2,000-node uniform graph, two halves, 2 layers 32-16-8, softmax-CE) against
the oracle's multi-partition simulation of Algorithm 1.

Two protocols:
* injected: before each iteration the oracle's W_{t-1}, partition 0's stale
  buffers and smoothing states are copied in; every output of the iteration
  is compared (aggregations, activations, loss, feature gradients, outgoing
  buffers, weight gradients, new smoothing states, updated weights);
* autonomous: only what partition 1 sends (features, gradients) and its
  weight gradient (the other AllReduce operand) are injected; the GPU keeps
  its own ping-pong buffers, side-stream refills and smoothing state across
  iterations, and its weights must track the oracle's for 4 iterations.
"""
import numpy as np
import pytest
import torch

from dataclasses import replace

from certify import certified_reference, elem_err, readings
from gpu_helpers import TOL, rel_err
from oracle.pipegcn import Options, run
from paper_2203_10428_amd import configs
from paper_2203_10428_amd.step import PartitionTrainer, StepOptions

pytestmark = pytest.mark.gpu

VARIANTS = {"PipeGCN": (False, False), "PipeGCN-G": (False, True), "PipeGCN-F": (True, False),
            "PipeGCN-GF": (True, True)}


def tiny_setup(T, smooth_f, smooth_g, gemm="f64"):
    w = configs.TINY
    g = configs.make_graph(w)
    d = configs.make_dense(w, g.n)
    opts = Options(mode="pipe", smooth_f=smooth_f, smooth_g=smooth_g, gamma=w.gamma, eta=w.eta,
                   loss=w.loss, loss_scale=w.loss_scale, gemm=gemm)
    sim, recs = run(g.n, g.rowptr, g.col, g.owner, g.nparts, d.X, d.labels, d.W, T, opts)
    return w, g, d, sim, recs


def put(t: torch.Tensor, x: np.ndarray):
    t.zero_()
    if x.size:
        t[:, : x.shape[1]] = torch.from_numpy(x.astype(np.float32)).cuda()


def get(t: torch.Tensor, f: int) -> np.ndarray:
    return t[:, :f].float().cpu().numpy().astype(np.float64)


def compare_step(tr: PartitionTrainer, ref, dt, L, widths, what=""):
    """Every output of partition 0's iteration against a reference dict (``certified_reference``)
    at the path's tolerance; prints both error metrics per tensor."""
    tol = TOL[dt]
    n = tr.n
    pairs = {}
    for l in range(1, L + 1):
        if dt == "f32" and tr.A[l] is not None:          # a transform-first layer keeps no aggregate
            pairs[f"A{l}"] = (get(tr.A[l], widths[l - 1]), ref["A"][l], tol["act"])
        pairs[f"H{l}"] = (get(tr.H[l], widths[l]), ref["H"][l], tol["act"])
        pairs[f"send_f{l}"] = (get(tr.send_f[l], widths[l - 1]), ref["send_f"][l], tol["act"])
        pairs[f"G{l}"] = (tr.dW[l - 1].cpu().numpy(), ref["G"][l], tol["grad"])
        pairs[f"ema_f{l}"] = (get(tr.ema_f[l], widths[l - 1]), ref["ema_f"][l], tol["act"])
    for l in range(2, L + 1):
        pairs[f"J_in{l}"] = (get(tr.J_in[l], widths[l - 1]), ref["J_full"][l][:n], tol["grad"])
        pairs[f"J_bd{l}"] = (get(tr.J_bd_out[l], widths[l - 1]), ref["J_full"][l][n:], tol["grad"])
        pairs[f"ema_g{l}"] = (get(tr.ema_g[l], widths[l - 1]), ref["ema_g"][l], tol["grad"])
    pairs["loss"] = (np.array([tr.loss.item()]), np.array([ref["loss"]]), tol["act"])
    for l in range(L):
        pairs[f"W{l + 1}"] = (tr.W[l].cpu().numpy(), ref["W_out"][l], tol["act"])
    errs = {k: (rel_err(g, o), elem_err(g, o), t) for k, (g, o, t) in pairs.items()}
    print(f"{what}: flips {ref.get('flips')}; " + ", ".join(f"{k} {e:.1e}/{el:.1e}" for k, (e, el, _) in errs.items()))
    bad = {k: v for k, v in errs.items() if not v[0] <= v[2]}
    assert not bad, (what, bad)


def inject(tr, r0, r1, L):
    """The oracle's W_{t-1}, partition 0's stale buffers and smoothing states, and the peer's
    weight gradient (the other AllReduce operand)."""
    si = r0["state_in"]
    for l in range(L):
        tr.W[l].copy_(torch.from_numpy(r0["W_in"][l].astype(np.float32)))
        tr.G_peer[l] = torch.from_numpy(r1["G"][l + 1].astype(np.float32)).cuda()
    for l in range(1, L + 1):
        put(tr.feat[l][tr.cur], si.feat_buf[l])
        put(tr.ema_f[l], si.ema_f[l])
    for l in range(2, L + 1):
        put(tr.grad[l][tr.cur], si.grad_buf[l])
        put(tr.ema_g[l], si.ema_g[l])
    tr.t = r0["t"] - 1


@pytest.mark.parametrize("variant", list(VARIANTS))
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_tiny_injected(variant, dt):
    """bf16 results are held to the plain fp64 oracle and to its bf16-operand reading, at the bf16
    tolerances; ReLU decisions that differ from the oracle's are certified against their rounding
    bounds before the oracle's backward takes them."""
    sf, sg = VARIANTS[variant]
    T = 3
    w, g, d, sim, recs = tiny_setup(T, sf, sg)
    L = w.layers
    tr = PartitionTrainer(g, d.X, d.labels, d.W, w.widths, w.loss, w.loss_scale, dt,
                          StepOptions(smooth_f=sf, smooth_g=sg, gamma=w.gamma, eta=w.eta, copy_mode="none"))
    assert tr.n == sim.parts[0].n_inner and tr.b == sim.parts[0].n_bd
    for t in range(1, T + 1):
        r0, r1 = recs[t - 1][0], recs[t - 1][1]
        inject(tr, r0, r1, L)
        torch.cuda.synchronize()
        tr.step()
        tr.synchronize()
        H_gpu = {l: get(tr.H[l], w.widths[l]) for l in range(1, L + 1)}
        for gm in readings(dt):
            ref = certified_reference(sim, r0, r1, replace(sim.opts, gemm=gm), H_gpu, dt)
            compare_step(tr, ref, dt, L, w.widths, f"{variant} {dt} t={t} vs {gm}")


def exact_decisions(tr, r0, L, widths, what):
    """In an autonomous run the weights run free, so ReLU decisions cannot be re-certified against
    the simulation's: they must agree exactly (the injected tests certify differing decisions)."""
    for l in range(1, L):
        gpu, ref = get(tr.H[l], widths[l]) > 0, r0["Z"][l] > 0
        assert np.array_equal(gpu, ref), f"{what}: layer {l}: {int((gpu != ref).sum())} ReLU decisions differ"


def sim_reference(r0):
    """A simulation record of partition 0 in the reference layout ``compare_step`` reads."""
    return dict(A=r0["A"], H=r0["H"], send_f=r0["send_f"], G=r0["G"], J_full=r0["J_full"], loss=r0["loss"],
                ema_f=r0["state_out"].ema_f, ema_g=r0["state_out"].ema_g, W_out=r0["W_out"])


@pytest.mark.parametrize("refill", ["blit", "dma", "host"])
@pytest.mark.parametrize("variant", list(VARIANTS))
def test_tiny_autonomous_pipeline(variant, refill):
    sf, sg = VARIANTS[variant]
    T = 4
    w, g, d, sim, recs = tiny_setup(T, sf, sg)
    L = w.layers
    tr = PartitionTrainer(g, d.X, d.labels, d.W, w.widths, w.loss, w.loss_scale, "f32",
                          StepOptions(smooth_f=sf, smooth_g=sg, gamma=w.gamma, eta=w.eta, copy_mode="pipe",
                                      refill_dma=refill == "dma", remote="host" if refill == "host" else "device"))
    if refill == "host":
        assert tr.remote_f[1].is_pinned() and not tr.remote_f[1].is_cuda
    for t in range(1, T + 1):
        r0, r1 = recs[t - 1][0], recs[t - 1][1]
        so = r0["state_out"]
        torch.cuda.synchronize()
        # what partition 1 sends in iteration t (consumed by partition 0 in t+1)
        for l in range(1, L + 1):
            put(tr.remote_f[l], so.feat_buf[l])
        for l in range(2, L + 1):
            put(tr.remote_g[l], so.grad_buf[l])
        for l in range(L):
            tr.G_peer[l] = torch.from_numpy(r1["G"][l + 1].astype(np.float32)).cuda()
        torch.cuda.synchronize()
        tr.step()
        tr.synchronize()
        exact_decisions(tr, r0, L, w.widths, f"autonomous {variant} {refill} t={t}")
        compare_step(tr, sim_reference(r0), "f32", L, w.widths, f"autonomous {variant} {refill} t={t}")


@pytest.mark.parametrize("refill_dma", [False, True])
def test_tiny_stale_buffers_never_read_before_refill(refill_dma):
    """A NaN sentinel in the buffer being refilled must never reach an output."""
    w, g, d, sim, recs = tiny_setup(1, True, True)
    tr = PartitionTrainer(g, d.X, d.labels, d.W, w.widths, w.loss, w.loss_scale, "f32",
                          StepOptions(copy_mode="pipe", refill_dma=refill_dma))
    for _ in range(3):
        torch.cuda.synchronize()
        nxt = 1 - tr.cur
        for l in tr.feat:
            tr.feat[l][nxt].fill_(float("nan"))
        for l in tr.grad:
            tr.grad[l][nxt].fill_(float("nan"))
        torch.cuda.synchronize()
        before = {l: tr.feat[l][tr.cur].clone() for l in tr.feat}
        cur = tr.cur
        tr.step()
        tr.synchronize()
        assert np.isfinite(tr.loss.item())
        for l in range(1, w.layers + 1):
            assert torch.isfinite(tr.H[l]).all()
            assert torch.equal(tr.feat[l][cur], before[l])        # the buffer being read is not written
        for W in tr.W:
            assert torch.isfinite(W).all()


def test_refill_from_host_needs_pinned_memory():
    from paper_2203_10428_amd import binding as B
    dst = torch.zeros(1024, device="cuda")
    pinned = torch.arange(1024, dtype=torch.float32).pin_memory()
    B.pgcn_refill_async(dst, pinned, 4096, B.PGCN_REFILL_FROM_HOST)
    torch.cuda.synchronize()
    assert torch.equal(dst.cpu(), pinned)
    with pytest.raises(B.PgcnError, match="pinned host"):
        B.pgcn_refill_async(dst, torch.zeros(1024), 4096, B.PGCN_REFILL_FROM_HOST)
    with pytest.raises(B.PgcnError, match="unknown flags"):
        B.pgcn_refill_async(dst, pinned, 4096, 8)


@pytest.mark.parametrize("nbytes,offset,flags", [
    (16, 0, 0), (4096, 0, 0),                                        # small: the runtime's copy
    (4 << 20, 0, 0), (2048 * 256 * 16 * 2 + 48, 0, 0),               # the copy kernel: whole and partial last block
    (4100, 0, 0), (4096, 4, 0), ((4 << 20) + 4, 0, 0), (4 << 20, 4, 0),   # size or address not 16-byte aligned
    (4096, 0, 1), (4100, 4, 1)])                                     # the DMA engines
def test_device_refill_copies_exactly(nbytes, offset, flags):
    from paper_2203_10428_amd import binding as B
    guard = 256
    src = torch.randint(0, 256, (nbytes + offset + guard,), dtype=torch.uint8, device="cuda")
    dst = torch.full((nbytes + offset + guard,), 0xA5, dtype=torch.uint8, device="cuda")
    B.pgcn_refill_async(dst[offset:], src[offset:], nbytes, flags)
    torch.cuda.synchronize()
    assert torch.equal(dst[offset:offset + nbytes], src[offset:offset + nbytes])
    assert (dst[:offset] == 0xA5).all() and (dst[offset + nbytes:] == 0xA5).all()
