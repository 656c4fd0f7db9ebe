"""The layer forward that allocates nothing (pgcn_layer_fwd_noalloc, for
callers that cannot allocate: graph capture, serving loops) against
pgcn_layer_fwd with a caller-owned workspace.  Both run the same kernels, so
every output must agree bit for bit; the outputs are also held to the fp64
oracle at the path's tolerance.  Two calls in a row share the library's fixed
scratch array: the first on a partition with column chunks, split rows and a
dense block (partial sums, block sums and block images in the scratch), the
second on a smaller partition with
narrower layers, in both associations and both GEMM precisions.  Arguments the
entry point must refuse (a workspace given, a layer whose workspace exceeds
the fixed array) are refused before any launch."""
import os

import numpy as np
import pytest
import torch

from gpu_helpers import TOL, dev, host, random_partition_graph, rel_err
from oracle import layers
from oracle.partition import build_partition, propagation_matrix
from paper_2203_10428_amd import binding as B
from paper_2203_10428_amd.step import ld_of

pytestmark = pytest.mark.gpu

ORDER = {"agg": B.PGCN_ORDER_AGG, "transform": B.PGCN_ORDER_TRANSFORM}


class Part:
    def __init__(self, n_inner, n_pool, mean_deg, seed, hub_deg=0, env=None):
        self.n, self.rowptr, self.col, self.owner = random_partition_graph(n_inner, n_pool, 3, mean_deg, seed,
                                                                           hub_deg)
        self.ref = build_partition(self.n, self.rowptr, self.col, self.owner, 0, 3)
        self.P = propagation_matrix(self.ref)
        old = {k: os.environ.get(k) for k in (env or {})}
        os.environ.update(env or {})           # set-up tuning knobs: column chunks, segment length
        try:
            self.part = B.pgcn_partition_setup(self.n, self.rowptr, self.col, self.owner, 3, 0)
        finally:
            for k, v in old.items():
                if v is None:
                    os.environ.pop(k, None)
                else:
                    os.environ[k] = v
        self.info = B.pgcn_partition_info(self.part)
        self.n_in, self.n_bd = self.ref.n_inner, self.ref.n_bd


@pytest.fixture(scope="module")
def parts():
    # 3 column chunks, rows split every 64 non-zeros and a 600 x 1000 dense block on the matrix cores:
    # the forward keeps partial sums, block sums and block images in its workspace
    big = Part(3000, 1500, 12, 0, hub_deg=3000, env={"PGCN_AGG_CHUNKS": "3", "PGCN_SEGMENT": "64",
                                                     "PGCN_HUB_ROWS": "600", "PGCN_HUB_COLS": "1000"})
    small = Part(1000, 400, 8, 1)
    assert big.info["spmm_chunks"] == 3 and big.info["spmm_split_slots"] > 0
    assert (big.info["spmm_hub_rows"], big.info["spmm_hub_cols"]) == (600, 1000) and big.info["spmm_hub_nnz"] > 0
    assert small.info["spmm_hub_rows"] == 0
    return big, small


def outputs(g, f_in, f_out, order, dt):
    n = g.n_in
    agg = order == "agg"
    return dict(A=dev(np.zeros((n, f_in))) if agg else None,
                A_bf16=torch.zeros((n, ld_of(f_in)), dtype=torch.bfloat16, device="cuda") if agg and dt == "bf16"
                else None,
                H_out=dev(np.zeros((n, f_out))),
                send_out=dev(np.zeros((g.info["n_send"], f_out))))


def one_call(g, f_in, f_out, order, dt, seed):
    """Runs the layer through both entry points; returns both output sets and the oracle's H."""
    rng = np.random.default_rng(seed)
    n, b = g.n_in, g.n_bd
    X = rng.standard_normal((n + b, f_in))
    W = rng.uniform(-0.3, 0.3, (f_in, f_out)).astype(np.float32)
    dtype = B.PGCN_BF16 if dt == "bf16" else B.PGCN_F32
    common = dict(f_in=f_in, f_out=f_out, gemm_dtype=dtype, relu=True, ld_in=ld_of(f_in), ld_out=ld_of(f_out),
                  H_in=dev(X[:n]), H_bd=dev(X[n:]), W=torch.from_numpy(W).cuda(), order=ORDER[order])
    need = B.pgcn_layer_workspace_size(g.part, f_in, f_out, dtype, ORDER[order])
    assert need <= B.PGCN_NOALLOC_SCRATCH_BYTES
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device="cuda")
    ref_out, na_out = outputs(g, f_in, f_out, order, dt), outputs(g, f_in, f_out, order, dt)
    B.pgcn_layer_fwd(g.part, workspace=ws, workspace_bytes=ws.numel(), **common, **ref_out)
    B.pgcn_layer_fwd_noalloc(g.part, **common, **na_out)
    torch.cuda.synchronize()
    _, _, H_ref = layers.layer_forward(g.P, X, W.astype(np.float64), True, "f64", order=order)
    return ref_out, na_out, H_ref


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("order", ["agg", "transform"])
def test_noalloc_forward_equals_workspace_forward(parts, order, dt):
    big, small = parts
    # two calls in a row on the shared scratch: a large layer, then a smaller partition and narrower layer
    for g, f_in, f_out, seed in ((big, 96, 80, 11), (small, 40, 24, 12)):
        ref_out, na_out, H_ref = one_call(g, f_in, f_out, order, dt, seed)
        print(f"noalloc {order} {dt}: {g.n_in} inner rows, {f_in} -> {f_out}", flush=True)
        for k, v in ref_out.items():
            if v is not None:
                assert torch.equal(v, na_out[k]), (k, g.n_in)
        assert rel_err(host(na_out["H_out"], f_out), H_ref) < TOL[dt]["act"]


def test_noalloc_rejects_a_workspace_and_oversized_layers(parts):
    big, _ = parts
    n, b = big.n_in, big.n_bd
    f_in, f_out = 8, 2048                  # transform first: Y alone is (n + b) x 2048 floats, above 32 MiB
    need = B.pgcn_layer_workspace_size(big.part, f_in, f_out, B.PGCN_F32, B.PGCN_ORDER_TRANSFORM)
    assert need > B.PGCN_NOALLOC_SCRATCH_BYTES
    z = lambda r, c: torch.zeros((max(r, 1), c), device="cuda")
    common = dict(f_in=f_in, f_out=f_out, gemm_dtype=B.PGCN_F32, relu=True, ld_in=8, ld_out=f_out, H_in=z(n, 8),
                  H_bd=z(b, 8), W=z(f_in, f_out), A=None, A_bf16=None, H_out=z(n, f_out))
    with pytest.raises(B.PgcnError, match="PGCN_NOALLOC_SCRATCH_BYTES") as e:
        B.pgcn_layer_fwd_noalloc(big.part, order=B.PGCN_ORDER_TRANSFORM, **common)
    assert e.value.code == B.PGCN_EWORKSPACE
    ws = torch.empty(256, dtype=torch.uint8, device="cuda")
    with pytest.raises(B.PgcnError, match="workspace must be NULL") as e:
        B.pgcn_layer_fwd_noalloc(big.part, workspace=ws, workspace_bytes=256, **common)
    assert e.value.code == B.PGCN_EINVAL
