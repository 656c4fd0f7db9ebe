"""Pins of the staleness-error diagnostics (oracle.staleness)."""
import numpy as np
import pytest

from oracle.pipegcn import Options
from oracle.staleness import staleness_errors
from paper_2203_10428_amd import configs, synth
from test_oracle_sage_pins import sage_problem


def tiny():
    g = synth.tiny_uniform()
    return (g.n, g.rowptr, g.col, g.owner, g.nparts)


def test_constant_input_layer_has_no_feature_staleness():
    graph = tiny()
    w = configs.TINY
    d = configs.make_dense(w, graph[0])
    rows = staleness_errors(*graph, d.X, d.labels, d.W, 4, Options(eta=0.1, loss_scale=1.0 / graph[0]))
    assert all(r["feat"][1] == 0.0 for r in rows)          # layer 1 exchanges X, which never changes
    assert all(r["feat"][2] > 0.0 for r in rows[1:])         # hidden features move with the weights


def test_zero_learning_rate_has_no_staleness_after_warm_up():
    graph = tiny()
    w = configs.TINY
    d = configs.make_dense(w, graph[0])
    rows = staleness_errors(*graph, d.X, d.labels, d.W, 6, Options(eta=0.0, loss_scale=1.0 / graph[0]))
    last = rows[-1]
    assert last["feat"][2] == 0.0 and last["grad"][2] == 0.0 and last["G"] < 1e-13


def test_gamma_zero_smoothing_is_plain_pipegcn():
    graph = tiny()
    w = configs.TINY
    d = configs.make_dense(w, graph[0])
    kw = dict(eta=0.2, loss_scale=1.0 / graph[0])
    a = staleness_errors(*graph, d.X, d.labels, d.W, 5, Options(**kw), vanilla_g=False)
    b = staleness_errors(*graph, d.X, d.labels, d.W, 5, Options(smooth_f=True, smooth_g=True, gamma=0.0, **kw),
                         vanilla_g=False)
    for ra, rb in zip(a, b):
        assert ra["feat"] == rb["feat"] and ra["grad"] == rb["grad"]


@pytest.mark.parametrize("model", ["gcn", "sage"])
def test_weight_gradient_error_scales_with_the_learning_rate(model):
    """The gradient error bound of the convergence analysis is proportional to eta."""
    graph = tiny()
    w = configs.TINY
    if model == "sage":
        X, W, y = sage_problem(graph[:4], list(w.widths))
    else:
        d = configs.make_dense(w, graph[0])
        X, W, y = d.X, d.W, d.labels
    errs = []
    for eta in (1e-3, 1e-2, 1e-1):
        rows = staleness_errors(*graph, X, y, W, 6, Options(model=model, eta=eta, loss_scale=1.0 / graph[0]))
        errs.append(np.mean([r["G"] for r in rows if r["t"] >= 4]))
    assert 5.0 < errs[1] / errs[0] < 20.0, errs
    assert 5.0 < errs[2] / errs[1] < 20.0, errs


def test_per_partition_errors_combine_into_the_total():
    """The error over all partitions is the root of the den-weighted mean of the per-partition squared
    errors, so it lies between them; both partitions together give the default."""
    graph = tiny()
    w = configs.TINY
    d = configs.make_dense(w, graph[0])
    o = Options(smooth_f=True, smooth_g=True, gamma=0.5, eta=0.2, loss_scale=1.0 / graph[0])
    all_ = staleness_errors(*graph, d.X, d.labels, d.W, 4, o, vanilla_g=False)
    both = staleness_errors(*graph, d.X, d.labels, d.W, 4, o, vanilla_g=False, parts=(0, 1))
    p0 = staleness_errors(*graph, d.X, d.labels, d.W, 4, o, vanilla_g=False, parts=(0,))
    p1 = staleness_errors(*graph, d.X, d.labels, d.W, 4, o, vanilla_g=False, parts=(1,))
    for ra, rb, r0, r1 in zip(all_, both, p0, p1):
        assert ra["feat"] == rb["feat"] and ra["grad"] == rb["grad"]
        for kind in ("feat", "grad"):
            for l, e in ra[kind].items():
                lo, hi = sorted((r0[kind][l], r1[kind][l]))
                assert lo - 1e-15 <= e <= hi + 1e-15, (kind, l, lo, e, hi)
