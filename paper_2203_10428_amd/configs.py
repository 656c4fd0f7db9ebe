"""Workload definitions: synthetic partitions shaped like the paper's setups.

The layer widths, layer counts and partition counts follow the paper's
experiment setup table (Reddit: 4 layers, 256 hidden, 602 features;
ogbn-products: 3 layers, 128 hidden, 100 features; Yelp: 4 layers, 512 hidden,
300 features).  The graphs themselves are synthetic (see ``synth``); the
datasets are not used.  Nothing here performs any of the method's arithmetic.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from functools import lru_cache

import numpy as np

from . import synth


@dataclass(frozen=True)
class Workload:
    name: str
    widths: tuple            # f_0 .. f_L
    loss: str                # "softmax_ce" or "sigmoid_bce"
    gemm_dtype: str          # "f32" or "bf16"
    n_global_labels: int     # node count the loss is normalised by (global graph)
    graph_kind: str
    graph_args: tuple
    gamma: float = 0.95
    eta: float = 0.01
    seed: int = 0
    # the experiments' GraphSAGE training (setup table): dropout rate and Adam learning rate
    sage_dropout: float = 0.0
    sage_lr: float = 0.01

    @property
    def layers(self) -> int:
        return len(self.widths) - 1

    @property
    def classes(self) -> int:
        return self.widths[-1]

    @property
    def loss_scale(self) -> float:
        # softmax-CE: sum over labelled nodes / N_global; BCE: mean over nodes x classes
        if self.loss == "softmax_ce":
            return 1.0 / self.n_global_labels
        return 1.0 / (self.n_global_labels * self.classes)


TINY = Workload(
    name="tiny-2k-2parts", widths=(32, 16, 8), loss="softmax_ce", gemm_dtype="f32",
    n_global_labels=2000, graph_kind="tiny_uniform", graph_args=(2000, 10000, 2), sage_dropout=0.3)

REDDIT = Workload(
    name="reddit-like-1of4", widths=(602, 256, 256, 256, 41), loss="softmax_ce", gemm_dtype="f32",
    n_global_labels=233000, graph_kind="chung_lu",
    graph_args=(58000, 30000, 4, 491.0, 26000.0, 2.3, 0.5, 1.07), sage_dropout=0.5, sage_lr=0.01)

PRODUCTS = Workload(
    name="products-like-1of8", widths=(100, 128, 128, 47), loss="softmax_ce", gemm_dtype="bf16",
    n_global_labels=2449000, graph_kind="chung_lu",
    graph_args=(306000, 150000, 8, 51.0, 5000.0, 2.3, 0.7, 1.0), sage_dropout=0.3, sage_lr=0.003)

YELP = Workload(
    name="yelp-like-1of3", widths=(300, 512, 512, 512, 100), loss="sigmoid_bce", gemm_dtype="f32",
    n_global_labels=717000, graph_kind="er_hubs",
    graph_args=(239000, 100000, 3, 19.0, 2000, 0.05, 0.6), sage_dropout=0.1, sage_lr=0.001)

STRESS = Workload(
    name="stress-rmat-2M", widths=(128,) + (256,) * 7 + (64,), loss="softmax_ce", gemm_dtype="bf16",
    n_global_labels=2000000 * 8, graph_kind="rmat",
    graph_args=(2000000, 21, 8, 33.0, 0.5, 1.0))

WORKLOADS = {w.name: w for w in (TINY, REDDIT, PRODUCTS, YELP, STRESS)}


def with_inner_scale(w: Workload, scale: float) -> Workload:
    """The same graph law with the inner and pool node counts scaled (a bounded sample)."""
    a = list(w.graph_args)
    if w.graph_kind in ("chung_lu", "er_hubs"):
        a[0] = max(16, int(a[0] * scale))
        a[1] = max(16, int(a[1] * scale))
        if w.graph_kind == "chung_lu":
            a[4] = a[4] * scale ** 0.5
    elif w.graph_kind == "rmat":
        a[0] = max(16, int(a[0] * scale))
        a[1] = max(4, a[1] + int(np.round(np.log2(scale))))
    else:
        raise ValueError("bounded samples are defined for partition-local graphs only")
    return Workload(**{**w.__dict__, "name": f"{w.name}@{scale:g}", "graph_args": tuple(a)})


def make_graph(w: Workload) -> synth.GlobalGraph:
    a = w.graph_args
    if w.graph_kind == "tiny_uniform":
        return synth.tiny_uniform(a[0], a[1], a[2], seed=w.seed)
    if w.graph_kind == "chung_lu":
        return synth.chung_lu_partition(a[0], a[1], a[2], a[3], a[4], a[5], a[6], w.seed, oversample=a[7])
    if w.graph_kind == "er_hubs":
        return synth.er_hubs_partition(a[0], a[1], a[2], a[3], a[4], a[5], a[6], w.seed)
    if w.graph_kind == "rmat":
        return synth.rmat_partition(a[0], a[1], a[2], a[3], a[4], w.seed, oversample=a[5])
    raise ValueError(w.graph_kind)


@dataclass
class DenseInputs:
    X: np.ndarray                    # [n_global_or_local, f_0] features of every global node
    W: list                          # Glorot weights per layer [f_{l-1}, f_l] ([2 f_{l-1}, f_l] for GraphSAGE)
    labels: np.ndarray               # int32 [n] or float32 [n, C]


def make_dense(w: Workload, n_nodes: int, model: str = "gcn") -> DenseInputs:
    """Features for every global node, initial weights and labels (all seeded).

    GraphSAGE weights are [2 f_{l-1}, f_l] (they act on CONCAT(z, h))."""
    rx, rw, ry = synth.dense_streams(w.seed, 3)
    X = synth.features(rx, n_nodes, w.widths[0])
    k = 2 if model == "sage" else 1
    W = [synth.glorot_uniform(rw, k * w.widths[l], w.widths[l + 1]) for l in range(w.layers)]
    if w.loss == "softmax_ce":
        y = synth.labels_single(ry, n_nodes, w.classes)
    else:
        y = synth.labels_multi(ry, n_nodes, w.classes, 0.05)
    return DenseInputs(X, W, y)
