"""The fp32 update GEMMs by bf16 parts (the default fp32 path: both operands
split exactly into three bf16 parts, six part products on the bf16 matrix
cores, fp32 accumulation) against the fp64 oracle and against the plain fp32
matrix-core kernels (PGCN_GEMM_F32=native) on the same inputs: every element
within the certified rounding bound (tests/certify.py), and the largest error
no more than twice the plain kernel's (or 2^-20 of the output's scale).
Forward (plain) GEMM, feature gradient (masked, row-scaled operand) and
weight gradient (node-split, masked right operand); ragged widths and row
tiles."""
import os
from contextlib import contextmanager

import numpy as np
import pytest
import torch

from certify import input_rounding, z_bound
from gpu_helpers import dev, host, random_partition_graph
from oracle import layers
from oracle.partition import build_partition, propagation_matrix
from paper_2203_10428_amd import binding as B
from paper_2203_10428_amd.step import ld_of

pytestmark = pytest.mark.gpu


@contextmanager
def gemm_f32(mode):
    old = os.environ.get("PGCN_GEMM_F32")
    if mode == "native":
        os.environ["PGCN_GEMM_F32"] = "native"
    else:
        os.environ.pop("PGCN_GEMM_F32", None)
    try:
        yield
    finally:
        if old is None:
            os.environ.pop("PGCN_GEMM_F32", None)
        else:
            os.environ["PGCN_GEMM_F32"] = old


@pytest.fixture(scope="module")
def graph():
    n_g, rowptr, col, owner = random_partition_graph(5000, 1500, 4, 10, 11)
    ref = build_partition(n_g, rowptr, col, owner, 0, 4)
    part = B.pgcn_partition_setup(n_g, rowptr, col, owner, 4, 0)
    return ref, propagation_matrix(ref), part


def max_rel(got, ref):
    return float(np.abs(got - ref).max() / max(np.abs(ref).max(), 1e-30))


@pytest.mark.parametrize("f_in,f_out", [(41, 47), (300, 512), (602, 256), (1100, 16), (2048, 64), (7, 130)])
def test_forward_by_parts(graph, f_in, f_out):
    ref, P, part = graph
    n, b = ref.n_inner, ref.n_bd
    rng = np.random.default_rng(f_in * 3 + f_out)
    X = rng.standard_normal((n + b, f_in))
    W = rng.uniform(-0.2, 0.2, (f_in, f_out)).astype(np.float32)
    _, Z_ref, _ = layers.layer_forward(P, X, W.astype(np.float64), False)
    nb = max(B.pgcn_workspace_size(part, f_in, f_out, B.PGCN_F32), 256)
    out = {}
    for mode in ("parts", "native"):
        ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
        A, H = dev(np.zeros((n, f_in))), dev(np.zeros((n, f_out)))
        with gemm_f32(mode):
            B.pgcn_layer_fwd(part, f_in=f_in, f_out=f_out, gemm_dtype=B.PGCN_F32, relu=False, ld_in=ld_of(f_in),
                             ld_out=ld_of(f_out), H_in=dev(X[:n]), H_bd=dev(X[n:]), W=torch.from_numpy(W).cuda(),
                             A=A, A_bf16=None, H_out=H, workspace=ws, workspace_bytes=nb)
        torch.cuda.synchronize()
        out[mode] = host(H, f_out)
    bound = z_bound(P, X, input_rounding(X), W.astype(np.float64), "f32")
    for mode, Z in out.items():
        over = np.abs(Z - Z_ref) > bound
        assert not over.any(), (mode, int(over.sum()))
    e_parts, e_native = max_rel(out["parts"], Z_ref), max_rel(out["native"], Z_ref)
    print(f"forward {f_in}x{f_out}: max rel err by parts {e_parts:.2e}, native {e_native:.2e}")
    assert e_parts <= max(2.0 * e_native, 2.0 ** -20)


@pytest.mark.parametrize("f_in,f_out", [(47, 41), (512, 300), (256, 256), (130, 1100), (1000, 200)])
def test_feature_gradient_by_parts(graph, f_in, f_out):
    ref, P, part = graph
    n, b = ref.n_inner, ref.n_bd
    rng = np.random.default_rng(f_in * 5 + f_out)
    A = rng.standard_normal((n, f_in))
    Z = rng.standard_normal((n, f_out))
    J = rng.standard_normal((n, f_out)) * 1e-2
    W = rng.uniform(-0.2, 0.2, (f_in, f_out)).astype(np.float32)
    G_ref, Jf_ref = layers.layer_backward(P, A, Z, J, W.astype(np.float64), True, True)
    nb = max(B.pgcn_workspace_size(part, f_in, f_out, B.PGCN_F32), 256)
    out, outG = {}, {}
    for mode in ("parts", "native"):
        ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
        J_in, J_bd = dev(np.zeros((n, f_in))), dev(np.zeros((b, f_in)))
        dG = torch.zeros((f_in, f_out), device="cuda")
        with gemm_f32(mode):
            B.pgcn_layer_bwd(part, f_in=f_in, f_out=f_out, gemm_dtype=B.PGCN_F32, relu=True, ld_in=ld_of(f_in),
                             ld_out=ld_of(f_out), J_out=dev(J), H_out=dev(np.maximum(Z, 0)), A=dev(A), A_bf16=None,
                             W=torch.from_numpy(W).cuda(), dW=dG, J_in=J_in, J_bd_out=J_bd, workspace=ws,
                             workspace_bytes=nb)
        torch.cuda.synchronize()
        out[mode] = np.vstack([host(J_in, f_in), host(J_bd, f_in)])
        outG[mode] = dG.cpu().numpy().astype(np.float64)
    e_parts, e_native = max_rel(out["parts"], Jf_ref), max_rel(out["native"], Jf_ref)
    g_parts, g_native = max_rel(outG["parts"], G_ref), max_rel(outG["native"], G_ref)
    print(f"feature gradient {f_in}x{f_out}: max rel err by parts {e_parts:.2e}, native {e_native:.2e}; "
          f"weight gradient by parts {g_parts:.2e}, native {g_native:.2e}")
    assert e_parts <= max(2.0 * e_native, 2.0 ** -20)
    assert e_parts < 1e-5
    assert g_parts <= max(2.0 * g_native, 2.0 ** -20)
    assert g_parts < 1e-5


def test_non_finite_operands_stay_non_finite(graph):
    ref, P, part = graph
    n, b = ref.n_inner, ref.n_bd
    f_in, f_out = 64, 64
    rng = np.random.default_rng(9)
    X = rng.standard_normal((n + b, f_in))
    bad = [10, 200]                              # inner rows whose features are NaN / Inf
    X[bad[0], 3] = np.nan
    X[bad[1], 5] = np.inf
    W = rng.uniform(-0.2, 0.2, (f_in, f_out)).astype(np.float32)
    nb = max(B.pgcn_workspace_size(part, f_in, f_out, B.PGCN_F32), 256)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    A, H = dev(np.zeros((n, f_in))), dev(np.zeros((n, f_out)))
    B.pgcn_layer_fwd(part, f_in=f_in, f_out=f_out, gemm_dtype=B.PGCN_F32, relu=False, ld_in=f_in, ld_out=f_out,
                     H_in=dev(X[:n]), H_bd=dev(X[n:]), W=torch.from_numpy(W).cuda(), A=A, A_bf16=None, H_out=H,
                     workspace=ws, workspace_bytes=nb)
    torch.cuda.synchronize()
    Ah, Hh = host(A, f_in), host(H, f_out)
    rows_bad = ~np.isfinite(Ah).all(axis=1)      # rows whose aggregation met a non-finite input
    assert rows_bad.any()
    assert not np.isfinite(Hh[rows_bad]).all(axis=1).any()
    assert np.isfinite(Hh[~rows_bad]).all()
