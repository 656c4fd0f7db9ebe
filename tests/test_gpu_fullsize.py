"""Full-size GPU parity on the four large workloads, in the launch
configuration the bench uses (same partition, widths, dtypes and kernels).

The oracle cannot afford whole fp64 layers here, so each test feeds seeded
synthetic inputs to one layer call and checks sampled outputs that the test
computes one by one from the definitions, straight from the global graph:

* forward row v:  A[v] = (H[v] + sum_{u in N(v)} H[u]) / (|N(v)| + 1),
                  H_out[v] = relu(A[v] W)  (bf16 reading on bf16 workloads);
* weight-gradient columns: G[:, c] = A^T M[:, c] over all inner rows;
* transposed row u (inner or boundary): sum over inner v adjacent to u (and
  u itself when inner) of (M W^T)[v] / d_v.

Sampled rows include random rows, the longest rows (split into segments) and
boundary rows.  Local numbering is recomputed here from its definition (rank
of the global id; boundary by (owner, id)), independent of the library.

The transform-first layers the bench runs (every narrowing layer: the last
one, and the first on the Reddit-like workload) are checked the same way:
forward rows from (sum of the neighbourhood's H rows) W / d_v, and the
backward from T = P_i^T M built here as a sparse matrix from the global
graph (G columns = H_full^T T, sampled rows of J = T W^T).
"""
import numpy as np
import pytest
import scipy.sparse as sp
import torch

from gpu_helpers import TOL
from oracle.layers import round_bf16
from paper_2203_10428_amd import binding as B
from paper_2203_10428_amd import configs
from paper_2203_10428_amd.step import ld_of

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]

WORKLOADS = ["reddit-like-1of4", "products-like-1of8", "yelp-like-1of3", "stress-rmat-2M"]
_CACHE = {}


class Full:
    def __init__(self, name):
        self.w = configs.WORKLOADS[name]
        g = configs.make_graph(self.w)
        self.g = g
        self.inner = np.flatnonzero(g.owner == 0)
        # boundary: distinct non-inner neighbours of inner rows, by (owner, global id)
        starts, ends = g.rowptr[self.inner], g.rowptr[self.inner + 1]
        lens = ends - starts
        idx = np.repeat(starts - np.concatenate([[0], np.cumsum(lens)[:-1]]), lens) + np.arange(lens.sum())
        nb = np.unique(g.col[idx])
        nb = nb[g.owner[nb] != 0]
        self.bd = nb[np.lexsort((nb, g.owner[nb]))]
        self.n, self.b = len(self.inner), len(self.bd)
        self.deg = np.diff(g.rowptr)                     # generator output: no self loops, no duplicates
        self.part = B.pgcn_partition_setup(g.n, g.rowptr, g.col, g.owner, g.nparts, 0)
        self.info = B.pgcn_partition_info(self.part)
        assert (self.info["n_inner"], self.info["n_bd"]) == (self.n, self.b)
        self.local_inner = np.full(g.n, -1, np.int64)
        self.local_inner[self.inner] = np.arange(self.n)

    def local_ids(self):
        """Local id of every global node (inner by rank, boundary after them by (owner, id)); -1 elsewhere."""
        loc = np.full(self.g.n, -1, np.int64)
        loc[self.inner] = np.arange(self.n)
        loc[self.bd] = self.n + np.arange(self.b)
        return loc

    def propagation_t(self):
        """P_i^T as a sparse [(n + b) x n] matrix: entry (u, v) = 1 / d_v for u in N(v) or u = v."""
        g = self.g
        starts, lens = g.rowptr[self.inner], self.deg[self.inner]
        idx = np.repeat(starts - np.concatenate([[0], np.cumsum(lens)[:-1]]), lens) + np.arange(lens.sum())
        rows = np.repeat(np.arange(self.n), lens)
        cols = self.local_ids()[g.col[idx]]
        assert (cols >= 0).all()
        d = (lens + 1).astype(np.float64)
        vals = np.concatenate([1.0 / d[rows], 1.0 / d])
        r = np.concatenate([cols, np.arange(self.n)])
        c = np.concatenate([rows, np.arange(self.n)])
        return sp.csr_matrix((vals, (r, c)), shape=(self.n + self.b, self.n))

    def neighbours(self, gid):
        return self.g.col[self.g.rowptr[gid]:self.g.rowptr[gid + 1]].astype(np.int64)

    def sample_inner(self, k, seed):
        rng = np.random.default_rng(seed)
        lens = self.deg[self.inner]
        heavy = np.argsort(-lens)[:4]                    # longest rows: split into segments
        return np.unique(np.concatenate([heavy, rng.choice(self.n, k, replace=False)]))


def full(name) -> Full:
    if name not in _CACHE:                               # the four partitions stay resident (a few GB)
        _CACHE[name] = Full(name)
    return _CACHE[name]


def upload(x, dtype=torch.float32):
    rows, f = x.shape
    t = torch.zeros((rows, ld_of(f)), dtype=dtype, device="cuda")
    t[:, :f] = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda").to(dtype)
    return t


def rel(gpu, ref):
    return float(np.abs(gpu - ref).max() / max(np.abs(ref).max(), 1e-30))


@pytest.mark.parametrize("name", WORKLOADS)
def test_forward_layers_full_size(name):
    F = full(name)
    w = F.w
    dt = B.PGCN_BF16 if w.gemm_dtype == "bf16" else B.PGCN_F32
    tol = TOL["bf16" if dt == B.PGCN_BF16 else "f32"]["act"]
    rng = np.random.default_rng(1)
    for layer in (1, 2):                                 # the input width and a hidden width
        f_in, f_out = w.widths[layer - 1], w.widths[layer]
        Hg = rng.standard_normal((F.g.n, f_in)).astype(np.float32)   # one row per global node
        W = rng.uniform(-0.1, 0.1, (f_in, f_out)).astype(np.float32)
        dH_in, dH_bd = upload(Hg[F.inner]), upload(Hg[F.bd])
        A = torch.zeros((F.n, ld_of(f_in)), device="cuda") if dt == B.PGCN_F32 else None
        A16 = torch.zeros((F.n, ld_of(f_in)), dtype=torch.bfloat16, device="cuda") if dt == B.PGCN_BF16 else None
        H = torch.zeros((F.n, ld_of(f_out)), device="cuda")
        nb = max(B.pgcn_workspace_size(F.part, f_in, f_out, dt), 256)
        ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
        B.pgcn_layer_fwd(F.part, f_in=f_in, f_out=f_out, gemm_dtype=dt, relu=True, ld_in=ld_of(f_in),
                         ld_out=ld_of(f_out), H_in=dH_in, H_bd=dH_bd, W=torch.from_numpy(W).cuda(), A=A,
                         A_bf16=A16, H_out=H, workspace=ws, workspace_bytes=nb)
        torch.cuda.synchronize()
        rows = F.sample_inner(48, layer)
        A_gpu = (A if A is not None else A16)[torch.from_numpy(rows).cuda(), :f_in].float().cpu().numpy()
        H_gpu = H[torch.from_numpy(rows).cuda(), :f_out].cpu().numpy()
        A_ref = np.zeros((len(rows), f_in))
        for k, r in enumerate(rows):
            gid = F.inner[r]
            nbrs = F.neighbours(gid)
            A_ref[k] = (Hg[gid].astype(np.float64) + Hg[nbrs].astype(np.float64).sum(0)) / (len(nbrs) + 1)
        Wd = W.astype(np.float64)
        if dt == B.PGCN_BF16:
            Z_ref = round_bf16(A_ref) @ round_bf16(Wd)
            assert rel(A_gpu, A_ref) < 1e-2
        else:
            Z_ref = A_ref @ Wd
            assert rel(A_gpu, A_ref) < 1e-5
        assert rel(H_gpu, np.maximum(Z_ref, 0)) < tol, (name, layer)
        if dt == B.PGCN_BF16:                            # and the plain fp64 oracle, same tolerance
            assert rel(H_gpu, np.maximum(A_ref @ Wd, 0)) < tol, (name, layer, "fp64")
        del dH_in, dH_bd, A, A16, H, ws


@pytest.mark.parametrize("name", WORKLOADS)
def test_backward_layer_full_size(name):
    F = full(name)
    w = F.w
    dt = B.PGCN_BF16 if w.gemm_dtype == "bf16" else B.PGCN_F32
    tol = TOL["bf16" if dt == B.PGCN_BF16 else "f32"]["grad"]
    rng = np.random.default_rng(2)
    f_in, f_out = w.widths[1], w.widths[2]              # a hidden layer (has an input gradient)
    A = rng.standard_normal((F.n, f_in)).astype(np.float32)
    if dt == B.PGCN_BF16:
        A = round_bf16(A).astype(np.float32)             # the bf16 path stores A as bf16
    J = (rng.standard_normal((F.n, f_out)) * 1e-3).astype(np.float32)
    Hout = rng.standard_normal((F.n, f_out)).astype(np.float32)
    W = rng.uniform(-0.1, 0.1, (f_in, f_out)).astype(np.float32)
    dA = upload(A) if dt == B.PGCN_F32 else None
    dA16 = upload(A, torch.bfloat16) if dt == B.PGCN_BF16 else None
    dG = torch.zeros((f_in, f_out), device="cuda")
    J_in = torch.zeros((F.n, ld_of(f_in)), device="cuda")
    J_bd = torch.zeros((F.b, ld_of(f_in)), device="cuda")
    nb = max(B.pgcn_workspace_size(F.part, f_in, f_out, dt), 256)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    B.pgcn_layer_bwd(F.part, f_in=f_in, f_out=f_out, gemm_dtype=dt, relu=True, ld_in=ld_of(f_in),
                     ld_out=ld_of(f_out), J_out=upload(J), H_out=upload(Hout), A=dA, A_bf16=dA16,
                     W=torch.from_numpy(W).cuda(), dW=dG, J_in=J_in, J_bd_out=J_bd, workspace=ws,
                     workspace_bytes=nb)
    torch.cuda.synchronize()
    M0 = J.astype(np.float64) * (Hout > 0)
    W0 = W.astype(np.float64)
    Ad = A.astype(np.float64)
    cols = rng.choice(f_out, 6, replace=False)
    d_inner = F.deg[F.inner] + 1
    rows_in = F.sample_inner(24, 5)
    rows_bd = np.unique(np.concatenate([rng.choice(F.b, 24, replace=False),
                                        np.argsort(-F.deg[F.bd])[:2]]))
    got_G = dG.cpu().numpy()[:, cols]
    got_in = J_in[torch.from_numpy(rows_in).cuda(), :f_in].cpu().numpy()
    got_bd = J_bd[torch.from_numpy(rows_bd).cuda(), :f_in].cpu().numpy()
    # bf16: the bf16-operand reading (M and W rounded) and the plain fp64 oracle, same tolerance
    for rounded in ((True, False) if dt == B.PGCN_BF16 else (False,)):
        M, Wd = (round_bf16(M0), round_bf16(W0)) if rounded else (M0, W0)
        assert rel(got_G, Ad.T @ M[:, cols]) < tol, (name, rounded)

        def D_rows(local):                               # (M W^T)[v] / d_v for inner local rows
            return (M[local] @ Wd.T) / d_inner[local][:, None]

        # transposed aggregation on sampled inner and boundary rows
        ref_in = np.zeros((len(rows_in), f_in))
        for k, r in enumerate(rows_in):
            gid = F.inner[r]
            vs = F.local_inner[F.neighbours(gid)]
            vs = np.concatenate([vs[vs >= 0], [r]])
            ref_in[k] = D_rows(vs).sum(0)
        assert rel(got_in, ref_in) < tol, (name, rounded)
        ref_bd = np.zeros((len(rows_bd), f_in))
        for k, r in enumerate(rows_bd):
            vs = F.local_inner[F.neighbours(F.bd[r])]
            ref_bd[k] = D_rows(vs[vs >= 0]).sum(0)
        assert rel(got_bd, ref_bd) < tol, (name, rounded)


@pytest.mark.parametrize("order", ["agg", "auto"])
@pytest.mark.parametrize("name", WORKLOADS)
def test_full_step_is_finite_and_deterministic(name, order):
    """Three PipeGCN-GF iterations of the bench configuration, run twice: finite and bitwise equal."""
    from paper_2203_10428_amd.step import PartitionTrainer, StepOptions
    F = full(name)
    w = F.w
    d = configs.make_dense(w, F.g.n)
    outs = []
    for _ in range(2):
        tr = PartitionTrainer(F.g, d.X, d.labels, d.W, w.widths, w.loss, w.loss_scale, w.gemm_dtype,
                              StepOptions(smooth_f=True, smooth_g=True, gamma=w.gamma, eta=w.eta, copy_mode="pipe",
                                          order=order))
        losses = []
        for _ in range(3):
            tr.step()
            losses.append(tr.loss.item())
        tr.synchronize()
        assert all(np.isfinite(losses)), losses
        outs.append((losses, [x.cpu() for x in tr.W]))
        del tr
        torch.cuda.empty_cache()
    assert outs[0][0] == outs[1][0]
    for a, b in zip(outs[0][1], outs[1][1]):
        assert torch.equal(a, b)


def narrowing_layers(w):
    return [l for l in range(1, len(w.widths)) if w.widths[l] < w.widths[l - 1]]


@pytest.mark.parametrize("name", WORKLOADS)
def test_transform_forward_full_size(name):
    F = full(name)
    w = F.w
    dt = B.PGCN_BF16 if w.gemm_dtype == "bf16" else B.PGCN_F32
    tol = TOL["bf16" if dt == B.PGCN_BF16 else "f32"]["act"]
    rng = np.random.default_rng(11)
    L = len(w.widths) - 1
    for layer in narrowing_layers(w):
        f_in, f_out = w.widths[layer - 1], w.widths[layer]
        relu = layer < L
        Hg = rng.standard_normal((F.g.n, f_in)).astype(np.float32)
        W = rng.uniform(-0.1, 0.1, (f_in, f_out)).astype(np.float32)
        H = torch.zeros((F.n, ld_of(f_out)), device="cuda")
        nb = B.pgcn_layer_workspace_size(F.part, f_in, f_out, dt, B.PGCN_ORDER_TRANSFORM)
        ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
        B.pgcn_layer_fwd(F.part, f_in=f_in, f_out=f_out, gemm_dtype=dt, relu=relu, ld_in=ld_of(f_in),
                         ld_out=ld_of(f_out), H_in=upload(Hg[F.inner]), H_bd=upload(Hg[F.bd]),
                         W=torch.from_numpy(W).cuda(), A=None, A_bf16=None, H_out=H, workspace=ws,
                         workspace_bytes=nb, order=B.PGCN_ORDER_TRANSFORM)
        torch.cuda.synchronize()
        rows = F.sample_inner(48, layer + 7)
        H_gpu = H[torch.from_numpy(rows).cuda(), :f_out].cpu().numpy()
        # bf16: the bf16-operand reading (H and W rounded) and the plain fp64 oracle, same tolerance
        for rounded in ((True, False) if dt == B.PGCN_BF16 else (False,)):
            Hd = round_bf16(Hg) if rounded else Hg.astype(np.float64)
            Wd = round_bf16(W) if rounded else W.astype(np.float64)
            Z_ref = np.zeros((len(rows), f_out))
            for k, r in enumerate(rows):
                gid = F.inner[r]
                nbrs = F.neighbours(gid)
                Z_ref[k] = ((Hd[gid] + Hd[nbrs].sum(0)) @ Wd) / (len(nbrs) + 1)
            ref = np.maximum(Z_ref, 0) if relu else Z_ref
            assert rel(H_gpu, ref) < tol, (name, layer, rounded)
        del H, ws


@pytest.mark.parametrize("name", WORKLOADS)
def test_transform_backward_full_size(name):
    F = full(name)
    w = F.w
    dt = B.PGCN_BF16 if w.gemm_dtype == "bf16" else B.PGCN_F32
    tol = TOL["bf16" if dt == B.PGCN_BF16 else "f32"]["grad"]
    rng = np.random.default_rng(12)
    L = len(w.widths) - 1
    f_in, f_out = w.widths[L - 1], w.widths[L]           # the last layer: narrowing, with an input gradient
    H_full = rng.standard_normal((F.n + F.b, f_in)).astype(np.float32)
    J = (rng.standard_normal((F.n, f_out)) * 1e-3).astype(np.float32)
    W = rng.uniform(-0.1, 0.1, (f_in, f_out)).astype(np.float32)
    dG = torch.zeros((f_in, f_out), device="cuda")
    J_in = torch.zeros((F.n, ld_of(f_in)), device="cuda")
    J_bd = torch.zeros((F.b, ld_of(f_in)), device="cuda")
    nb = B.pgcn_layer_workspace_size(F.part, f_in, f_out, dt, B.PGCN_ORDER_TRANSFORM)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    B.pgcn_layer_bwd(F.part, f_in=f_in, f_out=f_out, gemm_dtype=dt, relu=False, ld_in=ld_of(f_in),
                     ld_out=ld_of(f_out), J_out=upload(J), H_out=None, A=None, A_bf16=None,
                     W=torch.from_numpy(W).cuda(), dW=dG, J_in=J_in, J_bd_out=J_bd, workspace=ws,
                     workspace_bytes=nb, order=B.PGCN_ORDER_TRANSFORM, H_in=upload(H_full[:F.n]),
                     H_bd=upload(H_full[F.n:]))
    torch.cuda.synchronize()
    T0 = F.propagation_t() @ J.astype(np.float64)         # no ReLU on the last layer: M = J
    cols = rng.choice(f_out, 6, replace=False)
    rows_in = F.sample_inner(24, 13)
    rows_bd = np.unique(np.concatenate([rng.choice(F.b, 24, replace=False), np.argsort(-F.deg[F.bd])[:2]]))
    got_G = dG.cpu().numpy()[:, cols]
    got_in = J_in[torch.from_numpy(rows_in).cuda(), :f_in].cpu().numpy()
    got_bd = J_bd[torch.from_numpy(rows_bd).cuda(), :f_in].cpu().numpy()
    # bf16: the bf16-operand reading (T, H, W rounded) and the plain fp64 oracle, same tolerance
    for rounded in ((True, False) if dt == B.PGCN_BF16 else (False,)):
        T, Hd, Wd = T0, H_full.astype(np.float64), W.astype(np.float64)
        if rounded:
            T, Hd, Wd = round_bf16(T), round_bf16(Hd), round_bf16(Wd)
        assert rel(got_G, Hd.T @ T[:, cols]) < tol, (name, rounded)
        assert rel(got_in, T[rows_in] @ Wd.T) < tol, (name, rounded)
        assert rel(got_bd, T[F.n + rows_bd] @ Wd.T) < tol, (name, rounded)
