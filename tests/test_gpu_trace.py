"""Kernel tracing through the C ABI (the per-launch durations bench.py reads):
every traced launch is counted exactly once, with a positive duration (the
chunk launches of one aggregation column range share one record that says
how many launches it spans), the kind filter holds, and nothing is recorded
once tracing is off."""
import os

import numpy as np
import pytest
import torch

from gpu_helpers import dev, random_partition_graph
from paper_2203_10428_amd import binding as B
from paper_2203_10428_amd.step import ld_of

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def part():
    n, rowptr, col, owner = random_partition_graph(2000, 1200, 3, 60, 2, 2000)
    old = {k: os.environ.get(k) for k in ("PGCN_AGG_CHUNKS", "PGCN_SEGMENT")}
    os.environ.update({"PGCN_AGG_CHUNKS": "3", "PGCN_SEGMENT": "16"})
    try:
        p = B.pgcn_partition_setup(n, rowptr, col, owner, 3, 0)
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    return p


def forward(part, f_in=300, f_out=128):
    info = B.pgcn_partition_info(part)
    n, b = info["n_inner"], info["n_bd"]
    rng = np.random.default_rng(0)
    nb = B.pgcn_workspace_size(part, f_in, f_out, B.PGCN_F32)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    H = dev(np.zeros((n, f_out)))
    B.pgcn_layer_fwd(part, f_in=f_in, f_out=f_out, gemm_dtype=B.PGCN_F32, relu=True, ld_in=ld_of(f_in),
                     ld_out=ld_of(f_out), H_in=dev(rng.standard_normal((n, f_in))),
                     H_bd=dev(rng.standard_normal((b, f_in))),
                     W=torch.from_numpy(rng.uniform(-0.2, 0.2, (f_in, f_out)).astype(np.float32)).cuda(),
                     A=dev(np.zeros((n, f_in))), A_bf16=None, H_out=H, workspace=ws, workspace_bytes=nb)
    torch.cuda.synchronize()


def test_trace_records_every_launch(part):
    info = B.pgcn_partition_info(part)
    assert info["spmm_chunks"] == 3 and info["spmm_split_slots"] > 0
    B.pgcn_trace_enable(256)
    try:
        forward(part)
        rec = B.pgcn_trace_collect()
    finally:
        B.pgcn_trace_disable()
    # 300 columns = 75 float4: one 64-float4 slice and one 11-float4 remainder; per column range
    # one record for its 3 chunk launches, then its fix-up pass; then the GEMM packs its
    # weights and runs
    assert [(k, n) for k, _, n in rec] == [("agg_fwd", 3), ("agg_fixup", 1), ("agg_fwd", 3), ("agg_fixup", 1),
                                           ("gemm_pack", 1), ("gemm_fwd", 1)]
    assert all(ms > 0 for _, ms, _ in rec)


def test_trace_filter_and_disable(part):
    B.pgcn_trace_enable(256)
    try:
        B.pgcn_trace_filter(["gemm_fwd"])
        forward(part)
        rec = B.pgcn_trace_collect()
        assert [(k, n) for k, _, n in rec] == [("gemm_fwd", 1)] and rec[0][1] > 0
        B.pgcn_trace_filter(["agg_fwd"])
        forward(part)
        forward(part)
        rec = B.pgcn_trace_collect()
        assert [(k, n) for k, _, n in rec] == [("agg_fwd", 3)] * 4 and all(ms > 0 for _, ms, _ in rec)
    finally:
        B.pgcn_trace_disable()
    forward(part)                                     # nothing traced once disabled
    B.pgcn_trace_enable(16)
    try:
        assert B.pgcn_trace_collect() == []
    finally:
        B.pgcn_trace_disable()
