"""Full-size GPU parity of the GraphSAGE layer (the experiments' model:
Section 2's CONCAT update, mean over N(v) without a self loop) on the
Reddit-like (fp32) and products-like (bf16) partitions, in the bench's launch
configuration.  Sampled outputs are computed one by one from the definitions,
straight from the global graph (the oracle cannot afford whole fp64 layers):

* forward row v:  z[v] = mean_{u in N(v)} X[u] (0 without neighbours),
                  H[v] = relu([z[v], X[v]] W);
* weight-gradient columns: G[:, c] = [z, X]^T M[:, c] over all inner rows;
* transposed row u: sum over inner v adjacent to u of (M W_top^T)[v] / |N(v)|,
  plus (M W_bot^T)[u] when u is inner.

The dropout mask of the bench's setting is checked on sampled rows of a
full-size input against the oracle's Philox4x32-10.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import TOL
from oracle.layers import round_bf16
from oracle.philox import dropout_mask_rows
from paper_2203_10428_amd import binding as B
from paper_2203_10428_amd import configs
from paper_2203_10428_amd.step import ld_of

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]

WORKLOADS = ["reddit-like-1of4", "products-like-1of8"]
_CACHE = {}


class FullSage:
    def __init__(self, name):
        self.w = configs.WORKLOADS[name]
        g = configs.make_graph(self.w)
        self.g = g
        self.inner = np.flatnonzero(g.owner == 0)
        starts, ends = g.rowptr[self.inner], g.rowptr[self.inner + 1]
        lens = ends - starts
        idx = np.repeat(starts - np.concatenate([[0], np.cumsum(lens)[:-1]]), lens) + np.arange(lens.sum())
        nb = np.unique(g.col[idx])
        nb = nb[g.owner[nb] != 0]
        self.bd = nb[np.lexsort((nb, g.owner[nb]))]
        self.n, self.b = len(self.inner), len(self.bd)
        self.deg = np.diff(g.rowptr)                     # generator output: no self loops, no duplicates
        self.part = B.pgcn_partition_setup(g.n, g.rowptr, g.col, g.owner, g.nparts, 0, self_loop=False)
        info = B.pgcn_partition_info(self.part)
        assert (info["n_inner"], info["n_bd"]) == (self.n, self.b)
        self.local_inner = np.full(g.n, -1, np.int64)
        self.local_inner[self.inner] = np.arange(self.n)

    def neighbours(self, gid):
        return self.g.col[self.g.rowptr[gid]:self.g.rowptr[gid + 1]].astype(np.int64)

    def sample_inner(self, k, seed):
        rng = np.random.default_rng(seed)
        heavy = np.argsort(-self.deg[self.inner])[:4]
        return np.unique(np.concatenate([heavy, rng.choice(self.n, k, replace=False)]))


def full(name):
    if name not in _CACHE:
        _CACHE.clear()
        torch.cuda.empty_cache()
        _CACHE[name] = FullSage(name)
    return _CACHE[name]


def upload(x, dtype=torch.float32):
    rows, f = x.shape
    t = torch.zeros((rows, ld_of(f)), dtype=dtype, device="cuda")
    t[:, :f] = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda").to(dtype)
    return t


def rel(gpu, ref):
    return float(np.abs(gpu - ref).max() / max(np.abs(ref).max(), 1e-30))


@pytest.mark.parametrize("name", WORKLOADS)
def test_sage_forward_full_size(name):
    F = full(name)
    w = F.w
    bf16 = w.gemm_dtype == "bf16"
    dt = B.PGCN_BF16 if bf16 else B.PGCN_F32
    rng = np.random.default_rng(1)
    f_in, f_out = w.widths[0], w.widths[1]
    Xg = rng.standard_normal((F.g.n, f_in)).astype(np.float32)
    W = rng.uniform(-0.1, 0.1, (2 * f_in, f_out)).astype(np.float32)
    dX, dXbd = upload(Xg[F.inner]), upload(Xg[F.bd])
    dX16 = upload(Xg[F.inner], torch.bfloat16) if bf16 else None
    A = None if bf16 else torch.zeros((F.n, ld_of(f_in)), device="cuda")
    A16 = torch.zeros((F.n, ld_of(f_in)), dtype=torch.bfloat16, device="cuda") if bf16 else None
    H = torch.zeros((F.n, ld_of(f_out)), device="cuda")
    nb = max(B.pgcn_workspace_size(F.part, f_in, f_out, dt), 256)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    B.pgcn_sage_layer_fwd(F.part, f_in=f_in, f_out=f_out, gemm_dtype=dt, relu=True, ld_in=ld_of(f_in),
                          ld_out=ld_of(f_out), X_in=dX, X_in_bf16=dX16, X_bd=dXbd, W=torch.from_numpy(W).cuda(),
                          A=A, A_bf16=A16, H_out=H, workspace=ws, workspace_bytes=nb)
    torch.cuda.synchronize()
    rows = F.sample_inner(48, 3)
    ri = torch.from_numpy(rows).cuda()
    z_gpu = (A if A is not None else A16)[ri, :f_in].float().cpu().numpy()
    H_gpu = H[ri, :f_out].cpu().numpy()
    z_ref = np.zeros((len(rows), f_in))
    for k, r in enumerate(rows):
        nbrs = F.neighbours(F.inner[r])
        if len(nbrs):
            z_ref[k] = Xg[nbrs].astype(np.float64).mean(0)
    Xc = np.hstack([z_ref, Xg[F.inner[rows]].astype(np.float64)])
    Wd = W.astype(np.float64)
    if bf16:
        Z_ref = round_bf16(Xc) @ round_bf16(Wd)
        assert rel(z_gpu, z_ref) < 1e-2
    else:
        Z_ref = Xc @ Wd
        assert rel(z_gpu, z_ref) < 1e-5
    assert rel(H_gpu, np.maximum(Z_ref, 0)) < TOL["bf16" if bf16 else "f32"]["act"], name
    if bf16:                                             # and the plain fp64 oracle, same tolerance
        assert rel(H_gpu, np.maximum(Xc @ Wd, 0)) < TOL["bf16"]["act"], (name, "fp64")


@pytest.mark.parametrize("name", WORKLOADS)
def test_sage_backward_full_size(name):
    F = full(name)
    w = F.w
    bf16 = w.gemm_dtype == "bf16"
    dt = B.PGCN_BF16 if bf16 else B.PGCN_F32
    tol = TOL["bf16" if bf16 else "f32"]["grad"]
    rng = np.random.default_rng(2)
    f_in, f_out = w.widths[1], w.widths[2]
    z = rng.standard_normal((F.n, f_in)).astype(np.float32)
    X = rng.standard_normal((F.n, f_in)).astype(np.float32)
    if bf16:
        z, X = round_bf16(z).astype(np.float32), round_bf16(X).astype(np.float32)
    J = (rng.standard_normal((F.n, f_out)) * 1e-3).astype(np.float32)
    Hout = rng.standard_normal((F.n, f_out)).astype(np.float32)
    W = rng.uniform(-0.1, 0.1, (2 * f_in, f_out)).astype(np.float32)
    dG = torch.zeros((2 * f_in, f_out), device="cuda")
    J_in = torch.zeros((F.n, ld_of(f_in)), device="cuda")
    J_bd = torch.zeros((F.b, ld_of(f_in)), device="cuda")
    nb = max(B.pgcn_workspace_size(F.part, f_in, f_out, dt), 256)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    B.pgcn_sage_layer_bwd(F.part, f_in=f_in, f_out=f_out, gemm_dtype=dt, relu=True, ld_in=ld_of(f_in),
                          ld_out=ld_of(f_out), J_out=upload(J), H_out=upload(Hout),
                          A=None if bf16 else upload(z), A_bf16=upload(z, torch.bfloat16) if bf16 else None,
                          X_in=None if bf16 else upload(X), X_in_bf16=upload(X, torch.bfloat16) if bf16 else None,
                          W=torch.from_numpy(W).cuda(), dW=dG, J_in=J_in, J_bd_out=J_bd, workspace=ws,
                          workspace_bytes=nb)
    torch.cuda.synchronize()
    M0 = J.astype(np.float64) * (Hout > 0)
    W0 = W.astype(np.float64)
    cols = rng.choice(f_out, 6, replace=False)
    Xc = np.hstack([z.astype(np.float64), X.astype(np.float64)])
    d_inner = F.deg[F.inner]
    rows_in = F.sample_inner(24, 5)
    rows_bd = np.unique(np.concatenate([rng.choice(F.b, 24, replace=False), np.argsort(-F.deg[F.bd])[:2]]))
    got_G = dG.cpu().numpy()[:, cols]
    got_in = J_in[torch.from_numpy(rows_in).cuda(), :f_in].cpu().numpy()
    got_bd = J_bd[torch.from_numpy(rows_bd).cuda(), :f_in].cpu().numpy()
    # bf16: the bf16-operand reading (M and W rounded) and the plain fp64 oracle, same tolerance
    for rounded in ((True, False) if bf16 else (False,)):
        M, Wd = (round_bf16(M0), round_bf16(W0)) if rounded else (M0, W0)
        assert rel(got_G, Xc.T @ M[:, cols]) < tol, (name, rounded)

        def top(local):                                  # (M W_top^T)[v] / |N(v)|
            return (M[local] @ Wd[:f_in].T) / d_inner[local][:, None]

        ref_in = np.zeros((len(rows_in), f_in))
        for k, r in enumerate(rows_in):
            vs = F.local_inner[F.neighbours(F.inner[r])]
            vs = vs[vs >= 0]
            ref_in[k] = (top(vs).sum(0) if len(vs) else 0.0) + M[r] @ Wd[f_in:].T
        assert rel(got_in, ref_in) < tol, (name, rounded)
        ref_bd = np.zeros((len(rows_bd), f_in))
        for k, r in enumerate(rows_bd):
            vs = F.local_inner[F.neighbours(F.bd[r])]
            ref_bd[k] = top(vs[vs >= 0]).sum(0)
        assert rel(got_bd, ref_bd) < tol, (name, rounded)


@pytest.mark.parametrize("name", WORKLOADS)
def test_dropout_full_size_rows_are_the_oracles(name):
    F = full(name)
    w = F.w
    f = w.widths[0]
    rng = np.random.default_rng(4)
    rows = F.n + F.b
    x = torch.randn((rows, ld_of(f)), device="cuda")
    out = torch.empty_like(x)
    B.pgcn_dropout(out, x, rows, f, ld_of(f), 0, w.sage_dropout, 0, 0, 1, 7)
    torch.cuda.synchronize()
    sample = np.unique(np.concatenate([rng.choice(rows, 64, replace=False), [0, rows - 1]]))
    keep = dropout_mask_rows(sample, f, w.sage_dropout, 0, 0, 1, 7) != 0
    got = out[torch.from_numpy(sample).cuda(), :f].cpu().numpy()
    xs = x[torch.from_numpy(sample).cuda(), :f].cpu().numpy()
    assert np.array_equal(got != 0, keep & (xs != 0))
    scale = np.float32(1.0 / (1.0 - w.sage_dropout))
    assert np.array_equal(got[keep], xs[keep] * scale)
