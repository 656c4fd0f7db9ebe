"""CPU checks of bench.py: it refuses runs on more than one GPU, and its
per-step algorithmic work (the roofline's numerator) counts exactly the
matrix products each layer forms.  The expected flops are listed product by
product from the layer algebra (GCN: Z = (P H) W or P (H W); GraphSAGE:
CONCAT(P X, X) W, or P (X W_top) + X_in W_bot; backward: the weight gradient
and, above layer 1, the feature gradient of each product).  The counter-based
traffic figure is reported only while the sources it was measured with are
unchanged."""
import importlib.util
import os
import subprocess
import sys
from types import SimpleNamespace

import pytest

from paper_2203_10428_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def load_bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def products(model, order, l, n, b, f, fo):
    """(rows, inner dim, cols) of every dense product of layer l: forward, weight gradient, feature gradient."""
    if order == B.PGCN_ORDER_TRANSFORM:
        fwd = [(n + b, f, fo)]                          # Y = [H; H_bd] W (W_top for GraphSAGE)
        wgrad = [(f, n + b, fo)]                        # G = H_full^T (P^T M)
        dgrad = [(n + b, fo, f)]                        # J = (P^T M) W^T
        if model == "sage":
            fwd.append((n, f, fo))                      # X_in W_bot
            wgrad.append((f, n, fo))                    # X_in^T M
            dgrad.append((n, fo, f))                    # M W_bot^T
    else:
        k = 2 * f if model == "sage" else f
        fwd = [(n, k, fo)]                              # A W with A = P H (CONCAT(P X, X) for GraphSAGE)
        wgrad = [(k, n, fo)]                            # A^T M
        dgrad = [(n, fo, k)]                            # M W^T
    return fwd, wgrad, dgrad if l > 1 else []


@pytest.mark.parametrize("model", ["gcn", "sage"])
@pytest.mark.parametrize("orders", [("agg", "agg", "agg"), ("transform", "agg", "transform"),
                                    ("transform", "transform", "transform")])
def test_gemm_flops_match_layer_products(model, orders):
    bench = load_bench()
    n, b, e = 1000, 300, 12000
    widths = [40, 24, 24, 7]
    order = {l + 1: (B.PGCN_ORDER_TRANSFORM if o == "transform" else B.PGCN_ORDER_AGG) for l, o in enumerate(orders)}
    tr = SimpleNamespace(info=dict(n_inner=n, n_bd=b, nnz=e, n_send=280, spmm_items=1100, spmmt_items=1400), L=3,
                         widths=widths, order=order)
    w = SimpleNamespace(gemm_dtype="f32")
    got = bench.algorithmic_work(tr, w, model)
    want = {"gemm_fwd": 0.0, "gemm_wgrad": 0.0, "gemm_dgrad": 0.0}
    for l in range(1, 4):
        fwd, wgrad, dgrad = products(model, order[l], l, n, b, widths[l - 1], widths[l])
        for key, prods in (("gemm_fwd", fwd), ("gemm_wgrad", wgrad), ("gemm_dgrad", dgrad)):
            want[key] += sum(2.0 * r * k * c for r, k, c in prods)
    for key, v in want.items():
        assert got[key] == v, key
    # every aggregation model moves at least the compulsory bytes
    assert got["agg_fwd_gather"] >= got["agg_fwd"] > 0 and got["agg_bwd_gather"] >= got["agg_bwd"] > 0
    # a GEMM's compulsory bytes cover at least its operands' and output's fp32-or-bf16 elements once
    for key in ("gemm_fwd", "gemm_wgrad", "gemm_dgrad"):
        assert got[key + "_bytes"] > 0 and got[key] / got[key + "_bytes"] < 64


def test_measured_traffic_is_void_once_a_source_changes(tmp_path, monkeypatch):
    # roofline.traffic comes from committed counter runs only while the sources
    # they were taken with hash the same
    import hashlib
    import json
    bench = load_bench()
    csrc = tmp_path / "paper_2203_10428_amd" / "csrc"
    csrc.mkdir(parents=True)
    (csrc / "aggregate.hip").write_text("kernel, first version")
    (tmp_path / "profiles").mkdir()
    digest = hashlib.sha256(b"kernel, first version").hexdigest()
    rec = {"sources": {"aggregate.hip": digest}, "kernels": {"agg_fwd": 123.0}}
    (tmp_path / "profiles" / "traffic_w.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("w", "agg_fwd") == 123.0
    assert bench.measured_traffic("w", "agg_bwd") is None
    assert bench.measured_traffic("other", "agg_fwd") is None
    (csrc / "aggregate.hip").write_text("kernel, second version")
    assert bench.measured_traffic("w", "agg_fwd") is None


def test_committed_traffic_records_name_existing_sources():
    import json
    for wl in ("reddit-like-1of4", "yelp-like-1of3"):
        rec = json.load(open(os.path.join(ROOT, "profiles", f"traffic_{wl}.json")))
        assert {"aggregate.hip", "setup.cpp", "api.cpp"} <= set(rec["sources"])
        for name in rec["sources"]:
            assert os.path.exists(os.path.join(ROOT, "paper_2203_10428_amd", "csrc", name))
        assert rec["kernels"]["agg_fwd"] > 0 and rec["kernels"]["agg_bwd"] > 0


def test_cpu_baseline_times_short_steps_as_a_mean():
    """One oracle step shorter than a second is dominated by first-call costs: the baseline
    times further steps after it (at most 200) and reports their mean."""
    from paper_2203_10428_amd import configs
    bench = load_bench()
    sec, n_inner, nnz, threads, reps = bench.cpu_baseline(configs.WORKLOADS["tiny-2k-2parts"], 1.0)
    assert reps > 1 and reps <= 200
    assert 0 < sec < 1.0 and n_inner > 0 and nnz > 0 and threads >= 1


def test_f32_gemm_method_follows_the_override(monkeypatch):
    bench = load_bench()
    monkeypatch.delenv("PGCN_GEMM_F32", raising=False)
    assert bench.f32_gemm_method() == "bf16-parts-x6"
    monkeypatch.setenv("PGCN_GEMM_F32", "native")
    assert bench.f32_gemm_method() == "fp32-matrix-cores"
    assert bench.F32_PARTS_CEILING_TFLOPS == bench.MFMA_PEAK_TFLOPS["bf16"] / 6
