"""Multi-partition simulation of Algorithm 1 (PipeGCN), float64.

Every partition of the global graph is simulated in one process.  Two modes:

* ``pipe``    — PipeGCN.  A message sent in iteration t (boundary features in
  the forward, boundary feature gradients in the backward) is consumed in
  iteration t+1 (Algorithm 1; the forward and backward equations of
  Section 3.2).  At t = 1 no message has arrived: boundary features are zero
  (Algorithm 1's initialisation of H⁽⁰⁾) and no gradient is accumulated.
* ``vanilla`` — vanilla partition-parallel training (Section 3.1): every
  message is delivered before the layer that needs it, so the result equals
  full-graph GCN training.

Optional moving-average smoothing (Section 3.4), independently for the
received boundary features (``smooth_f``, PipeGCN-F) and the received
boundary feature gradients (``smooth_g``, PipeGCN-G); decay ``gamma``.

Readings of points the paper leaves open (each is a keyword here):

* ``relu_last``     Algorithm 1 applies σ at every layer; by default the last
                    layer returns logits (``relu_last=False``).
* ``x_bd_preload``  Algorithm 1 starts every boundary row at zero, including
                    the input features; ``True`` loads X_bd at set-up.
* ``ema_init``      the smoothing state starts at zero (``"zero"``) and is
                    updated only when a message is consumed; ``"first"``
                    sets it to the first consumed message.
* gradient smoothing is applied at the receiver, on the received per-row
  contributions C_j, which equals smoothing each remote node's δz before the
  1/d_v weighting because the weighting is fixed across iterations.
* the received gradients are added for ascending peer j (Algorithm 1's loop).
* the AllReduce is a sum; the optimiser is Algorithm 1's SGD, or Adam (the
  experiments' optimiser) with ``optimizer="adam"``.
* ``model="sage"`` trains the experiments' GraphSAGE layer (Section 2's
  CONCAT update; mean over N(v) without a self loop) instead of the GCN
  layer of Algorithm 1.
* ``dropout`` p drops each layer's whole input (inner and received boundary
  rows, after smoothing) with one mask for the forward and the backward, as
  the paper's implementation notes require; the mask is drawn from
  Philox4x32-10 keyed by (``seed``, partition) and counted by (element,
  layer, iteration) (``oracle.philox``).  The input gradient is multiplied
  by the same mask before it is sent or accumulated.

Pinned by: reduction to full-graph GCN in vanilla mode, equality of the
modes with one partition, the η = 0 / γ = 0 staleness-timing fixed point, and
the moving-average closed form (tests).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import layers
from .partition import Partition, build_partition, propagation_matrix
from .philox import dropout_mask


@dataclass
class Options:
    mode: str = "pipe"              # "pipe" | "vanilla"
    smooth_f: bool = False
    smooth_g: bool = False
    gamma: float = 0.95
    eta: float = 0.01
    loss: str = "softmax_ce"        # "softmax_ce" | "sigmoid_bce"
    loss_scale: float = 1.0
    relu_last: bool = False
    x_bd_preload: bool = False
    ema_init: str = "zero"          # "zero" | "first"
    gemm: str = "f64"               # "f64" | "bf16" (operands of the update products rounded to bf16)
    order: str = "agg"              # GCN layer association: "agg" (P H) W, "transform" P (H W), "auto": transform if f_out < f_in
    norm: str = "mean"              # GCN propagation matrix: "mean" D̃⁻¹Ã, "sym" D̃^{-1/2} Ã D̃^{-1/2}
    model: str = "gcn"              # "gcn" | "sage"
    dropout: float = 0.0
    seed: int = 0
    optimizer: str = "sgd"          # "sgd" | "adam" (learning rate eta)
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8


def layer_order(o: Options, W: np.ndarray, sage: bool = False) -> str:
    """The association a layer is evaluated in; W is [f_in, f_out] (GCN) or [2 f_in, f_out] (GraphSAGE,
    whose aggregated half is f_in wide)."""
    if o.order == "auto":
        f_in = W.shape[0] // 2 if sage else W.shape[0]
        return "transform" if W.shape[1] < f_in else "agg"
    assert o.order in ("agg", "transform")
    return o.order


@dataclass
class PartState:
    """What partition i holds between iterations."""
    feat_buf: dict                  # layer -> [b, f_{l-1}]   received features (consumed next step)
    grad_buf: dict                  # layer -> [s, f_{l-1}]   received gradient contributions
    ema_f: dict                     # layer -> [b, f_{l-1}]
    ema_g: dict                     # layer -> [s, f_{l-1}]
    ema_seen_f: dict = field(default_factory=dict)
    ema_seen_g: dict = field(default_factory=dict)

    def copy(self):
        c = lambda d: {k: v.copy() for k, v in d.items()}
        return PartState(c(self.feat_buf), c(self.grad_buf), c(self.ema_f), c(self.ema_g),
                         dict(self.ema_seen_f), dict(self.ema_seen_g))


class Simulation:
    def __init__(self, n, rowptr, col, owner, nparts, X, labels, W0, opts: Options):
        self.opts = opts
        self.nparts = nparts
        self.parts: list[Partition] = [build_partition(n, rowptr, col, owner, i, nparts,
                                                       self_loop=opts.model == "gcn")
                                       for i in range(nparts)]
        self.P = [propagation_matrix(p, opts.norm) for p in self.parts]
        self.X = np.asarray(X, dtype=np.float64)
        self.labels = labels
        self.W = [np.asarray(w, dtype=np.float64).copy() for w in W0]
        self.L = len(self.W)
        self.widths = [self.W[0].shape[0] // (2 if opts.model == "sage" else 1)] + [w.shape[1] for w in self.W]
        self.adam_m = [np.zeros_like(w) for w in self.W]
        self.adam_v = [np.zeros_like(w) for w in self.W]
        self.t = 0
        self.state = []
        for p in self.parts:
            fb = {l: np.zeros((p.n_bd, self.widths[l - 1])) for l in range(1, self.L + 1)}
            gb = {l: np.zeros((len(p.send_idx), self.widths[l - 1])) for l in range(2, self.L + 1)}
            if opts.x_bd_preload:
                fb[1] = self.X[p.bd_gid].copy()
            self.state.append(PartState(fb, gb, {l: np.zeros_like(v) for l, v in fb.items()},
                                        {l: np.zeros_like(v) for l, v in gb.items()}))

    # -- helpers ----------------------------------------------------------
    def _relu(self, l):
        return l < self.L or self.opts.relu_last

    def _order(self, l):
        return layer_order(self.opts, self.W[l - 1], self.opts.model == "sage")

    def _use_features(self, i, l, t):
        """Boundary rows that layer l of partition i reads at iteration t."""
        st, p, o = self.state[i], self.parts[i], self.opts
        available = t > 1 or (l == 1 and o.x_bd_preload)
        if not available:
            return np.zeros((p.n_bd, self.widths[l - 1]))
        B = st.feat_buf[l]
        if not o.smooth_f:
            return B
        if o.ema_init == "first" and not st.ema_seen_f.get(l, False):
            st.ema_f[l] = B.copy()
        else:
            st.ema_f[l] = layers.ema(st.ema_f[l], B, o.gamma)
        st.ema_seen_f[l] = True
        return st.ema_f[l]

    def _use_gradients(self, i, l):
        st, o = self.state[i], self.opts
        C = st.grad_buf[l]
        if not o.smooth_g:
            return C
        if o.ema_init == "first" and not st.ema_seen_g.get(l, False):
            st.ema_g[l] = C.copy()
        else:
            st.ema_g[l] = layers.ema(st.ema_g[l], C, o.gamma)
        st.ema_seen_g[l] = True
        return st.ema_g[l]

    def _loss(self, i, out):
        p, o = self.parts[i], self.opts
        y = self.labels[p.inner_gid]
        if o.loss == "softmax_ce":
            return layers.softmax_ce(out, y, o.loss_scale)
        return layers.sigmoid_bce(out, y, o.loss_scale)

    # -- one iteration of Algorithm 1 for every partition ------------------
    def step(self):
        o = self.opts
        self.t += 1
        t = self.t
        pipe = o.mode == "pipe"
        rec = [dict(t=t, W_in=[w.copy() for w in self.W], state_in=self.state[i].copy(),
                    adam_in=([m.copy() for m in self.adam_m], [v.copy() for v in self.adam_v]),
                    A={}, Z={}, H={}, H_bd_used={}, C_used={}, J_full={}, G={}, X_in={}, X_full={}, mask={},
                    send_f={}, send_g={}) for i in range(self.nparts)]
        H_prev = [self.X[p.inner_gid] for p in self.parts]

        # forward, layer by layer
        for l in range(1, self.L + 1):
            sends = [[H_prev[i][p.send_idx[p.send_ptr[j]:p.send_ptr[j + 1]]] for j in range(self.nparts)]
                     for i, p in enumerate(self.parts)]
            for i in range(self.nparts):
                rec[i]["send_f"][l] = np.concatenate(sends[i], axis=0)
            if not pipe:
                for j, pj in enumerate(self.parts):
                    self.state[j].feat_buf[l] = self._gather_features(j, l, sends)
            for i, p in enumerate(self.parts):
                if pipe:
                    Hbd = self._use_features(i, l, t)
                else:
                    Hbd = self.state[i].feat_buf[l]
                rec[i]["H_bd_used"][l] = Hbd.copy()
                X, mask = self._dropped_input(i, l, t, H_prev[i], Hbd)
                rec[i]["X_in"][l], rec[i]["mask"][l] = X[: p.n_inner], mask
                if o.model == "sage":
                    A, Z, H = layers.sage_forward(self.P[i], X, p.n_inner, self.W[l - 1], self._relu(l), o.gemm,
                                                  self._order(l))
                else:
                    A, Z, H = layers.layer_forward(self.P[i], X, self.W[l - 1], self._relu(l), o.gemm,
                                                   self._order(l))
                rec[i]["A"][l], rec[i]["Z"][l], rec[i]["H"][l] = A, Z, H
                rec[i]["X_full"][l] = X
                H_prev[i] = H
            if pipe:
                # messages sent in this iteration are consumed in the next one
                for j in range(self.nparts):
                    self.state[j].feat_buf[l] = self._gather_features(j, l, sends)

        # loss
        J = []
        for i in range(self.nparts):
            loss, Jl = self._loss(i, H_prev[i])
            rec[i]["loss"] = loss
            J.append(Jl)

        # backward
        G_sum = [None] * self.L
        for l in range(self.L, 0, -1):
            J_full = [None] * self.nparts
            for i, p in enumerate(self.parts):
                if o.model == "sage":
                    G, Jf = layers.sage_backward(self.P[i], rec[i]["A"][l], rec[i]["X_in"][l], rec[i]["Z"][l], J[i],
                                                 self.W[l - 1], self._relu(l), l > 1, o.gemm, self._order(l),
                                                 rec[i]["X_full"][l])
                else:
                    G, Jf = layers.layer_backward(self.P[i], rec[i]["A"][l], rec[i]["Z"][l], J[i],
                                                  self.W[l - 1], self._relu(l), l > 1, o.gemm,
                                                  self._order(l), rec[i]["X_full"][l])
                if Jf is not None:
                    Jf = Jf * rec[i]["mask"][l]
                rec[i]["G"][l] = G
                G_sum[l - 1] = G if G_sum[l - 1] is None else G_sum[l - 1] + G
                J_full[i] = Jf
            if l == 1:
                break
            gsends = [[J_full[i][p.n_inner + p.recv_ptr[j]: p.n_inner + p.recv_ptr[j + 1]]
                       for j in range(self.nparts)] for i, p in enumerate(self.parts)]
            if not pipe:
                for i in range(self.nparts):
                    self.state[i].grad_buf[l] = self._gather_gradients(i, l, gsends)
            for i, p in enumerate(self.parts):
                if (not pipe) or t > 1:
                    C = self._use_gradients(i, l) if pipe else self.state[i].grad_buf[l]
                    rec[i]["C_used"][l] = C.copy()
                    for j in range(self.nparts):
                        a, b = p.send_ptr[j], p.send_ptr[j + 1]
                        J_full[i][p.send_idx[a:b]] += C[a:b]
                rec[i]["J_full"][l] = J_full[i].copy()
                rec[i]["send_g"][l] = J_full[i][p.n_inner:].copy()
                J[i] = J_full[i][:p.n_inner]
            if pipe:
                for i in range(self.nparts):
                    self.state[i].grad_buf[l] = self._gather_gradients(i, l, gsends)

        # AllReduce (sum) and the update
        for l in range(self.L):
            if o.optimizer == "adam":
                self.W[l], self.adam_m[l], self.adam_v[l] = layers.adam(
                    self.W[l], G_sum[l], self.adam_m[l], self.adam_v[l], t, o.eta, o.beta1, o.beta2, o.eps)
            else:
                self.W[l] = layers.sgd(self.W[l], G_sum[l], o.eta)
        for i in range(self.nparts):
            rec[i]["G_sum"] = [g.copy() for g in G_sum]
            rec[i]["W_out"] = [w.copy() for w in self.W]
            rec[i]["state_out"] = self.state[i].copy()
        return rec

    def _dropped_input(self, i, l, t, H_inner, H_bd):
        """Layer l's input of partition i after dropout, and the mask (ones without dropout)."""
        o, p = self.opts, self.parts[i]
        X = np.vstack([H_inner, H_bd])
        mask = dropout_mask(X.shape[0], X.shape[1], o.dropout, o.seed, p.part, l, t)
        return X * mask, mask

    def _gather_features(self, j, l, sends):
        """Boundary block of partition j owned by i is what i sent to j."""
        pj = self.parts[j]
        out = np.zeros((pj.n_bd, self.widths[l - 1]))
        for i in range(self.nparts):
            a, b = pj.recv_ptr[i], pj.recv_ptr[i + 1]
            if b > a:
                out[a:b] = sends[i][j]
        return out

    def _gather_gradients(self, i, l, gsends):
        """Block j of partition i's send list receives j's boundary rows owned by i."""
        p = self.parts[i]
        out = np.zeros((len(p.send_idx), self.widths[l - 1]))
        for j in range(self.nparts):
            a, b = p.send_ptr[j], p.send_ptr[j + 1]
            if b > a:
                out[a:b] = gsends[j][i]
        return out


def run(n, rowptr, col, owner, nparts, X, labels, W0, T, opts: Options):
    """Simulate T iterations; returns the simulation and the per-iteration records."""
    sim = Simulation(n, rowptr, col, owner, nparts, X, labels, W0, opts)
    return sim, [sim.step() for _ in range(T)]


def partition_step(p: Partition, P, X_in, y, W, received_f: dict, received_g: dict, ema_f: dict, ema_g: dict,
                   t: int, opts: Options, relu_masks: dict = None):
    """One iteration of Algorithm 1 for one partition, given what it received.

    ``received_f[l]`` ([b, f_{l-1}]) and ``received_g[l]`` ([s, f_{l-1}], l >= 2)
    are the messages of iteration t-1 (ignored at t = 1); ``ema_f`` / ``ema_g``
    are the smoothing states, updated in place when a message is consumed.
    Returns a record with the same keys as a Simulation record (A, Z, H, loss,
    J_full, G, send_f, X_in, mask) and the partition's weight gradients,
    without applying the update.  Pipelined mode; ``ema_init`` "zero"; no
    boundary preload.  ``P`` must match ``opts.model`` (self loops for GCN).
    ``relu_masks[l]`` (bool [n, f_l]), where given, is layer l's ReLU
    decision in the backward instead of Z > 0 (``layers.relu_mask``).
    """
    relu_masks = relu_masks or {}
    o = opts
    L = len(W)
    sage = o.model == "sage"
    rec = dict(A={}, Z={}, H={}, J_full={}, G={}, send_f={}, X_in={}, X_full={}, mask={})
    H = np.asarray(X_in, dtype=np.float64)
    for l in range(1, L + 1):
        rec["send_f"][l] = H[p.send_idx]
        if t > 1:
            Hbd = received_f[l]
            if o.smooth_f:
                ema_f[l] = layers.ema(ema_f[l], Hbd, o.gamma)
                Hbd = ema_f[l]
        else:
            Hbd = np.zeros((p.n_bd, H.shape[1]))
        relu = l < L or o.relu_last
        X = np.vstack([H, Hbd])
        mask = dropout_mask(X.shape[0], X.shape[1], o.dropout, o.seed, p.part, l, t)
        X = X * mask
        rec["X_in"][l], rec["mask"][l] = X[: p.n_inner], mask
        if sage:
            A, Z, H = layers.sage_forward(P, X, p.n_inner, W[l - 1], relu, o.gemm, layer_order(o, W[l - 1], sage))
        else:
            A, Z, H = layers.layer_forward(P, X, W[l - 1], relu, o.gemm, layer_order(o, W[l - 1], sage))
        rec["A"][l], rec["Z"][l], rec["H"][l] = A, Z, H
        rec["X_full"][l] = X
    f = layers.softmax_ce if o.loss == "softmax_ce" else layers.sigmoid_bce
    rec["loss"], J = f(H, y, o.loss_scale)
    for l in range(L, 0, -1):
        relu = l < L or o.relu_last
        if sage:
            G, Jf = layers.sage_backward(P, rec["A"][l], rec["X_in"][l], rec["Z"][l], J, W[l - 1], relu, l > 1,
                                         o.gemm, layer_order(o, W[l - 1], sage), rec["X_full"][l],
                                         mask=relu_masks.get(l))
        else:
            G, Jf = layers.layer_backward(P, rec["A"][l], rec["Z"][l], J, W[l - 1], relu, l > 1, o.gemm,
                                          layer_order(o, W[l - 1], sage), rec["X_full"][l],
                                          mask=relu_masks.get(l))
        rec["G"][l] = G
        if l == 1:
            break
        Jf = Jf * rec["mask"][l]
        if t > 1:
            C = received_g[l]
            if o.smooth_g:
                ema_g[l] = layers.ema(ema_g[l], C, o.gamma)
                C = ema_g[l]
            for j in range(len(p.send_ptr) - 1):
                a, b = p.send_ptr[j], p.send_ptr[j + 1]
                Jf[p.send_idx[a:b]] += C[a:b]
        rec["J_full"][l] = Jf
        J = Jf[: p.n_inner]
    return rec
