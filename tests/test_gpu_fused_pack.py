"""The send rows a layer's output kernel writes (pgcn_fwd_args.send_out,
pgcn_sage_fwd_args.send_out) against pgcn_pack_boundary of the same output,
bit for bit, for every kernel that can produce a layer output: the update
GEMM (aggregate first, GCN and GraphSAGE, fp32 and bf16, with a given
aggregate), the aggregation's last pass (transform-first GCN, with split rows
and column chunks) and the accumulating GEMM of the transform-first
GraphSAGE layer.  Send rows hold duplicates (an inner row sent to several
peers) and follow send_idx order."""
import os

import numpy as np
import pytest
import torch

from gpu_helpers import dev, random_partition_graph
from paper_2203_10428_amd import binding as B
from paper_2203_10428_amd.step import ld_of

pytestmark = pytest.mark.gpu

GRAPHS = {"plain": dict(args=(3000, 1500, 4, 12, 0, 0)),
          "split": dict(args=(2500, 900, 4, 12, 1, 3000)),
          "chunked": dict(args=(2000, 1200, 4, 60, 2, 2000), env={"PGCN_AGG_CHUNKS": "3", "PGCN_SEGMENT": "16"}),
          "tall": dict(args=(5000, 1500, 5, 10, 3, 0))}
_PARTS = {}


def part_for(gname, sage, sym):
    key = (gname, sage, sym)
    if key not in _PARTS:
        spec = GRAPHS[gname]
        n, rowptr, col, owner = random_partition_graph(*spec["args"])
        old = {k: os.environ.get(k) for k in spec.get("env", {})}
        os.environ.update(spec.get("env", {}))
        try:
            _PARTS[key] = B.pgcn_partition_setup(n, rowptr, col, owner, spec["args"][2], 0, self_loop=not sage,
                                                 symmetric=sym)
        finally:
            for k, v in old.items():
                if v is None:
                    os.environ.pop(k, None)
                else:
                    os.environ[k] = v
    return _PARTS[key]


FORMS = [("gcn", "agg", False), ("gcn", "transform", False), ("gcn", "agg", True), ("gcn", "transform", True),
         ("sage", "agg", False), ("sage", "transform", False)]
ORDER = {"agg": B.PGCN_ORDER_AGG, "transform": B.PGCN_ORDER_TRANSFORM}


@pytest.mark.parametrize("gname", list(GRAPHS))
@pytest.mark.parametrize("model,order,sym", FORMS)
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("f_in,f_out", [(41, 47), (300, 512), (602, 256), (256, 41)])
def test_fused_send_rows_equal_pack(gname, model, order, sym, dt, f_in, f_out):
    sage = model == "sage"
    part = part_for(gname, sage, sym)
    info = B.pgcn_partition_info(part)
    n, b, s = info["n_inner"], info["n_bd"], info["n_send"]
    assert s > n // 2                                       # rows are sent, several of them to more than one peer
    rng = np.random.default_rng(f_in + 7 * f_out)
    dtype = B.PGCN_BF16 if dt == "bf16" else B.PGCN_F32
    k = 2 if sage else 1
    li, lo = ld_of(f_in), ld_of(f_out)
    X, Xbd = dev(rng.standard_normal((n, f_in))), dev(rng.standard_normal((b, f_in)))
    W = torch.from_numpy(rng.uniform(-0.2, 0.2, (k * f_in, f_out)).astype(np.float32)).cuda()
    agg = order == "agg"
    A = dev(np.zeros((n, f_in))) if agg else None
    A16 = torch.zeros((n, li), dtype=torch.bfloat16, device="cuda") if agg and dt == "bf16" else None
    X16 = X.to(torch.bfloat16) if sage and dt == "bf16" else None
    H = dev(np.zeros((n, f_out)))
    send = torch.full((s, lo), -7.0, device="cuda")        # must be overwritten in columns [0, f_out)
    nb = max(B.pgcn_layer_workspace_size(part, f_in, f_out, dtype, ORDER[order]), 256)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    common = dict(f_in=f_in, f_out=f_out, gemm_dtype=dtype, relu=f_out != 41, ld_in=li, ld_out=lo, W=W, A=A,
                  A_bf16=A16, H_out=H, workspace=ws, workspace_bytes=nb, order=ORDER[order], send_out=send)
    if sage:
        B.pgcn_sage_layer_fwd(part, X_in=X, X_in_bf16=X16, X_bd=Xbd, **common)
    else:
        B.pgcn_layer_fwd(part, H_in=X, H_bd=Xbd, **common)
    ref = torch.zeros((s, lo), device="cuda")
    B.pgcn_pack_boundary(part, B.PGCN_PACK_FEAT, H, ref, f_out, lo)
    torch.cuda.synchronize()
    assert torch.equal(send[:, :f_out], ref[:, :f_out])
    assert torch.count_nonzero(H[:, :f_out]) > 0


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_fused_send_rows_with_given_aggregate(dt):
    part = part_for("plain", False, False)
    info = B.pgcn_partition_info(part)
    n, s = info["n_inner"], info["n_send"]
    f_in, f_out = 100, 128
    rng = np.random.default_rng(5)
    dtype = B.PGCN_BF16 if dt == "bf16" else B.PGCN_F32
    H, send = dev(np.zeros((n, f_out))), torch.zeros((s, ld_of(f_out)), device="cuda")
    nb = max(B.pgcn_layer_workspace_size(part, f_in, f_out, dtype, B.PGCN_ORDER_AGG), 256)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    B.pgcn_layer_fwd(part, f_in=f_in, f_out=f_out, gemm_dtype=dtype, relu=True, ld_in=ld_of(f_in),
                     ld_out=ld_of(f_out), H_in=None, H_bd=None,
                     W=torch.from_numpy(rng.uniform(-0.2, 0.2, (f_in, f_out)).astype(np.float32)).cuda(),
                     A=dev(rng.standard_normal((n, f_in))), A_bf16=None, H_out=H, workspace=ws, workspace_bytes=nb,
                     a_given=True, send_out=send)
    ref = torch.zeros_like(send)
    B.pgcn_pack_boundary(part, B.PGCN_PACK_FEAT, H, ref, f_out, ld_of(f_out))
    torch.cuda.synchronize()
    assert torch.equal(send[:, :f_out], ref[:, :f_out])


def test_send_out_must_be_aligned():
    part = part_for("plain", False, False)
    info = B.pgcn_partition_info(part)
    n, b, s = info["n_inner"], info["n_bd"], info["n_send"]
    buf = torch.zeros((s + 1) * 48, device="cuda")
    x = dev(np.zeros((n, 48)))
    nb = max(B.pgcn_layer_workspace_size(part, 48, 48, B.PGCN_F32, B.PGCN_ORDER_AGG), 256)
    with pytest.raises(B.PgcnError) as e:
        B.pgcn_layer_fwd(part, f_in=48, f_out=48, gemm_dtype=B.PGCN_F32, relu=True, ld_in=48, ld_out=48, H_in=x,
                         H_bd=dev(np.zeros((b, 48))), W=torch.zeros((48, 48), device="cuda"), A=dev(np.zeros((n, 48))),
                         A_bf16=None, H_out=dev(np.zeros((n, 48))),
                         workspace=torch.empty(nb, dtype=torch.uint8, device="cuda"), workspace_bytes=nb,
                         send_out=buf[1:])                 # 4 bytes past a 16-byte boundary
    assert e.value.code == B.PGCN_EINVAL
