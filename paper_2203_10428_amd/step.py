"""One partition's PipeGCN training step on one GPU (Algorithm 1, per-partition view).

Every computation is a libpgcn call (``binding``); torch provides device
memory, streams and events only.

Pipeline emulation on one GPU: Algorithm 1 exchanges boundary features and
boundary feature gradients with the peer partitions in background threads
and consumes what arrived in the previous iteration.  Here each stale buffer
is double-buffered: in iteration t the compute stream reads ``cur`` while a
side stream refills ``next`` from an emulated peer source, ordered after this
iteration's send (pack) by an event; the compute stream waits for that refill
only in iteration t+1 (the paper batches all layers' communication on a
second stream, as here).  Copy modes for measurement:

* ``"pipe"``   refills on the side stream (PipeGCN);
* ``"serial"`` refills on the compute stream before the layer that needs them
  (the synchronous exchange of vanilla partition-parallel training);
* ``"none"``   no refills (compute only).

Smoothing (Section 3.4): ``smooth_f`` and ``smooth_g`` keep a moving average
of the received boundary features / gradients, updated when a message is
consumed (iteration 2 on), starting from zero.

Model: ``"gcn"`` (Algorithm 1's layer) or ``"sage"`` (the experiments'
GraphSAGE layer, Section 2's CONCAT update; the partition is built without
self loops).  ``dropout`` p drops each layer's whole input after the receive
and smoothing, and the same mask multiplies the input gradient before it is
sent or accumulated (the paper's implementation notes); the mask comes from
the library's counter-based generator keyed by (``seed``, partition) and
counted by (layer, iteration).  ``optimizer``: Algorithm 1's SGD or Adam.

``order`` picks the association of each GCN layer's product P H W:
``"agg"`` (P H) W, ``"transform"`` P (H W), ``"auto"`` transform-first where
the layer narrows (f_out < f_in), which aggregates fewer columns.

``cache_layer1`` keeps layer 1's aggregate across iterations (GCN, no
dropout): its input X never changes, so after the peers' rows have arrived
once, A_full = P [X_in; X_bd] is fixed, and with feature smoothing the
aggregate the layer uses is the moving average of A_full started at
P [X_in; 0] (the smoothing is linear).  Layer 1 then runs aggregate-first
without a gather, and its boundary rows are exchanged once.  It reuses
outputs across iterations, so it is a variant, not the measured step.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

from . import binding as B


def ld_of(f: int) -> int:
    """Row stride used for every activation matrix: a multiple of 8 elements."""
    return (f + 7) // 8 * 8


@dataclass
class StepOptions:
    smooth_f: bool = True
    smooth_g: bool = True
    gamma: float = 0.95
    eta: float = 0.01
    relu_last: bool = False
    copy_mode: str = "pipe"          # "pipe" | "serial" | "none"
    refill_dma: bool = False         # refills by the DMA engines instead of a blit kernel
    fuse_pack: bool = True           # a layer's output kernel also writes the next layer's send rows
    remote: str = "device"           # emulated peers' data in "device" memory or pinned "host" memory
    model: str = "gcn"               # "gcn" | "sage"
    dropout: float = 0.0
    seed: int = 0
    optimizer: str = "sgd"           # "sgd" | "adam" (learning rate eta)
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    order: str = "agg"               # "agg" | "transform" | "auto" (GCN layers)
    norm: str = "mean"               # GCN propagation: "mean" D̃⁻¹Ã or "sym" D̃^{-1/2} Ã D̃^{-1/2}
    cache_layer1: bool = False       # keep layer 1's aggregate across iterations (see the module notes)


def layer_order(order: str, f_in: int, f_out: int) -> int:
    """libpgcn order of a GCN layer f_in -> f_out under the option ``order``."""
    assert order in ("agg", "transform", "auto"), order
    tf = order == "transform" or (order == "auto" and f_out < f_in)
    return B.PGCN_ORDER_TRANSFORM if tf else B.PGCN_ORDER_AGG


class PartitionTrainer:
    """Device state of one partition and its training step."""

    def __init__(self, graph, X_global: np.ndarray, labels_global: np.ndarray, W0: list, widths, loss: str,
                 loss_scale: float, gemm_dtype: str, opts: StepOptions, device="cuda:0",
                 remote_seed: int = 1234):
        self.dev = torch.device(device)
        self.opts = opts
        self.widths = list(widths)
        self.L = len(widths) - 1
        self.loss_kind = B.PGCN_SOFTMAX_CE if loss == "softmax_ce" else B.PGCN_SIGMOID_BCE
        self.loss_scale = float(loss_scale)
        self.dtype = B.PGCN_BF16 if gemm_dtype == "bf16" else B.PGCN_F32
        self.sage = opts.model == "sage"
        self.self_part = graph.self_part
        with torch.cuda.device(self.dev):
            assert opts.norm in ("mean", "sym") and not (self.sage and opts.norm == "sym"), opts.norm
            self.part = B.pgcn_partition_setup(graph.n, graph.rowptr, graph.col, graph.owner, graph.nparts,
                                               graph.self_part, self_loop=not self.sage, symmetric=opts.norm == "sym")
        self.info = B.pgcn_partition_info(self.part)
        n, b, s = self.info["n_inner"], self.info["n_bd"], self.info["n_send"]
        self.n, self.b, self.s = n, b, s
        ex = B.pgcn_partition_export(self.part)
        self.inner_gid, self.bd_gid = ex["inner_gid"], ex["bd_gid"]
        self.send_idx = ex["send_idx"]

        z = lambda r, f, dt=torch.float32: torch.zeros((r, ld_of(f)), dtype=dt, device=self.dev)
        L, wd = self.L, self.widths
        f32 = self.dtype == B.PGCN_F32
        # inputs
        self.X = z(n, wd[0])
        self.X[:, : wd[0]] = torch.from_numpy(np.ascontiguousarray(X_global[self.inner_gid])).to(self.dev)
        if self.loss_kind == B.PGCN_SOFTMAX_CE:
            self.labels = torch.from_numpy(labels_global[self.inner_gid].astype(np.int32)).to(self.dev)
            self.targets = None
        else:
            self.labels = None
            self.targets = z(n, wd[-1])
            self.targets[:, : wd[-1]] = torch.from_numpy(labels_global[self.inner_gid]).to(self.dev)
        self.W = [torch.from_numpy(np.ascontiguousarray(w, dtype=np.float32)).to(self.dev) for w in W0]
        k = 2 if self.sage else 1
        for l, w in enumerate(self.W):
            assert tuple(w.shape) == (k * wd[l], wd[l + 1]), (l, tuple(w.shape))
        self.dW = [torch.zeros_like(w) for w in self.W]
        self.adam_m = [torch.zeros_like(w) for w in self.W] if opts.optimizer == "adam" else None
        self.adam_v = [torch.zeros_like(w) for w in self.W] if opts.optimizer == "adam" else None
        # dropped layer inputs (dropout, or the bf16 copy of the GraphSAGE self operand)
        self.use_drop = opts.dropout > 0.0 or (self.sage and not f32)
        self.Xd_in = {l: z(n, wd[l - 1]) for l in range(1, L + 1)} if self.use_drop else {}
        self.Xd_bd = {l: z(b, wd[l - 1]) for l in range(1, L + 1)} if self.use_drop else {}
        self.Xd_16 = {l: z(n, wd[l - 1], torch.bfloat16) for l in range(1, L + 1)} \
            if (self.sage and not f32) else {}
        self.G_peer = [None] * L
        self.order = {l: layer_order(opts.order, wd[l - 1], wd[l]) for l in range(1, L + 1)}
        self.cache1 = opts.cache_layer1
        if self.cache1:
            assert not self.sage and opts.dropout == 0.0, "layer-1 caching needs a constant layer input"
            self.order[1] = B.PGCN_ORDER_AGG
        # activations, indexed by layer 1..L (a transform-first layer keeps no aggregate)
        agg = {l: self.order[l] == B.PGCN_ORDER_AGG for l in range(1, L + 1)}
        self.A = {l: (z(n, wd[l - 1]) if f32 and agg[l] else None) for l in range(1, L + 1)}
        self.A16 = {l: (None if f32 or not agg[l] else z(n, wd[l - 1], torch.bfloat16)) for l in range(1, L + 1)}
        if self.cache1:   # fp32 aggregates of layer 1 on both paths: the running one and A_full
            self.A[1], self.A16[1] = z(n, wd[0]), None
            self.A1_full = z(n, wd[0])
            self.H1_scratch = z(n, wd[1])
            self.A1_ready = self.A1_started = False
            self.A1_used = self.A[1]
        self.H = {l: z(n, wd[l]) for l in range(1, L + 1)}
        self.J_top = z(n, wd[L])
        self.J_in = {l: z(n, wd[l - 1]) for l in range(2, L + 1)}
        self.J_bd_out = {l: z(b, wd[l - 1]) for l in range(2, L + 1)}
        # stale feature buffers (layer l reads boundary rows of H^(l-1)), gradient buffers for l >= 2
        self.feat = {l: [z(b, wd[l - 1]), z(b, wd[l - 1])] for l in range(1, L + 1)}
        self.ema_f = {l: z(b, wd[l - 1]) for l in range(1, L + 1)}
        self.send_f = {l: z(s, wd[l - 1]) for l in range(1, L + 1)}
        self.grad = {l: [z(s, wd[l - 1]), z(s, wd[l - 1])] for l in range(2, L + 1)}
        self.ema_g = {l: z(s, wd[l - 1]) for l in range(2, L + 1)}
        # emulated peers: what the other partitions send each iteration
        g = torch.Generator(device="cpu").manual_seed(remote_seed)
        if opts.remote == "host":          # pinned host memory: refills cross the host link (CPU-staged exchange)
            zr = lambda r, f: torch.zeros((r, ld_of(f)), dtype=torch.float32, pin_memory=True)
        else:
            zr = z
        self.remote_f = {l: zr(b, wd[l - 1]) for l in range(1, L + 1)}
        self.remote_g = {l: zr(s, wd[l - 1]) for l in range(2, L + 1)}
        for l in range(1, L + 1):
            self.remote_f[l][:, : wd[l - 1]] = torch.randn((b, wd[l - 1]), generator=g).to(self.remote_f[l].device)
        for l in range(2, L + 1):
            self.remote_g[l][:, : wd[l - 1]] = (1e-3 * torch.randn((s, wd[l - 1]), generator=g)).to(
                self.remote_g[l].device)
        self.refill_bytes = sum(t.numel() * 4 for t in self.remote_f.values()) + \
            sum(t.numel() * 4 for t in self.remote_g.values())
        self.X_used = {}                  # layer input the forward used (the GraphSAGE self operand)
        self.X_bd_used = {}               # boundary rows the forward used (transform-first backward)
        self.cur = 0                      # index of the buffer read in this iteration
        self.t = 0
        self.loss = torch.zeros(1, dtype=torch.float32, device=self.dev)
        ws = max(B.pgcn_layer_workspace_size(self.part, wd[l - 1], wd[l], self.dtype, self.order[l])
                 for l in range(1, L + 1))
        self.ws_bytes = max(ws, 256)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.dev)
        self.stream = torch.cuda.Stream(device=self.dev)
        self.side = torch.cuda.Stream(device=self.dev)
        self.ev_pack = {l: torch.cuda.Event() for l in range(1, L + 1)}
        self.ev_feat = {l: torch.cuda.Event() for l in range(1, L + 1)}
        self.ev_bwd = {l: torch.cuda.Event() for l in range(2, L + 1)}
        self.ev_grad = {l: torch.cuda.Event() for l in range(2, L + 1)}
        torch.cuda.synchronize(self.dev)

    # ------------------------------------------------------------------
    def _relu(self, l):
        return l < self.L or self.opts.relu_last

    def _refill(self, dst, src, stream):
        if self.opts.remote == "host":
            flags = B.PGCN_REFILL_FROM_HOST
        else:
            flags = B.PGCN_REFILL_DMA if self.opts.refill_dma else 0
        B.pgcn_refill_async(dst, src, dst.numel() * dst.element_size(), flags, stream)

    def _dropout(self, out, inp, rows, l, row0, out16, st):
        o, f = self.opts, self.widths[l - 1]
        B.pgcn_dropout(out, inp, rows, f, ld_of(f), row0, o.dropout, o.seed, self.self_part, l, self.t, out16,
                       ld_of(f) if out16 is not None else 0, st)

    def _forward_layer1_cached(self, H_bd, st):
        """Layer 1 from the kept aggregate: A_full once the peers' rows are in, then the moving
        average of A_full (smoothing) or A_full itself; iteration 1 aggregates with zero
        boundary rows straight into the running aggregate."""
        o, wd, f = self.opts, self.widths, self.widths[0]
        common = dict(f_in=f, f_out=wd[1], gemm_dtype=self.dtype, relu=self._relu(1), ld_in=ld_of(f),
                      ld_out=ld_of(wd[1]), W=self.W[0], A_bf16=None, workspace=self.ws,
                      workspace_bytes=self.ws_bytes, stream=st)
        send = self._send_out(1)
        if not self.A1_ready:
            if not self.A1_started:        # the running aggregate starts at P [X_in; 0]
                B.pgcn_layer_fwd(self.part, H_in=self.X, H_bd=None, A=self.A[1], H_out=self.H[1], send_out=send,
                                 **common)
                self.A1_started = True
                if H_bd is None:
                    self.A1_used = self.A[1]
                    return
            B.pgcn_layer_fwd(self.part, H_in=self.X, H_bd=H_bd, A=self.A1_full, H_out=self.H1_scratch, **common)
            self.A1_ready = True
        if o.smooth_f:
            B.pgcn_smooth_ema(self.A[1], self.A1_full, self.n, f, ld_of(f), o.gamma, st)
            A1 = self.A[1]
        else:
            A1 = self.A1_full
        B.pgcn_layer_fwd(self.part, H_in=None, H_bd=None, A=A1, H_out=self.H[1], a_given=True, send_out=send,
                         **common)
        self.A1_used = A1

    def _send_out(self, l):
        """Send rows of layer l's output (the next layer's input), written by the layer's own output
        kernel when packs are fused; None for the last layer or without fusion."""
        return self.send_f[l + 1] if self.opts.fuse_pack and l < self.L else None

    def _forward_layer(self, l, H_in, H_bd, st):
        """Dropout of the layer input (after the receive), then the GCN or GraphSAGE layer."""
        wd, f = self.widths, self.widths[l - 1]
        X_in, X_bd, X16 = H_in, H_bd, None
        if self.use_drop:
            X16 = self.Xd_16.get(l)
            self._dropout(self.Xd_in[l], H_in, self.n, l, 0, X16, st)
            X_in = self.Xd_in[l]
            if H_bd is not None:
                self._dropout(self.Xd_bd[l], H_bd, self.b, l, self.n, None, st)
                X_bd = self.Xd_bd[l]
        common = dict(f_in=f, f_out=wd[l], gemm_dtype=self.dtype, relu=self._relu(l), ld_in=ld_of(f),
                      ld_out=ld_of(wd[l]), W=self.W[l - 1], A=self.A[l], A_bf16=self.A16[l], H_out=self.H[l],
                      workspace=self.ws, workspace_bytes=self.ws_bytes, stream=st)
        send = self._send_out(l)
        if self.sage:
            B.pgcn_sage_layer_fwd(self.part, X_in=X_in, X_in_bf16=X16, X_bd=X_bd, order=self.order[l], send_out=send,
                                  **common)
        else:
            B.pgcn_layer_fwd(self.part, H_in=X_in, H_bd=X_bd, order=self.order[l], send_out=send, **common)
        self.X_used[l] = X_in
        self.X_bd_used[l] = X_bd

    def _backward_layer(self, l, J_out, st):
        """Layer gradients; the input gradient then takes the forward's dropout mask."""
        wd, f = self.widths, self.widths[l - 1]
        A = self.A1_used if (self.cache1 and l == 1) else self.A[l]
        common = dict(f_in=f, f_out=wd[l], gemm_dtype=self.dtype, relu=self._relu(l), ld_in=ld_of(f),
                      ld_out=ld_of(wd[l]), J_out=J_out, H_out=self.H[l], A=A, A_bf16=self.A16[l],
                      W=self.W[l - 1], dW=self.dW[l - 1], J_in=self.J_in.get(l), J_bd_out=self.J_bd_out.get(l),
                      workspace=self.ws, workspace_bytes=self.ws_bytes, stream=st)
        if self.sage:
            B.pgcn_sage_layer_bwd(self.part, X_in=self.X_used[l], X_in_bf16=self.Xd_16.get(l), order=self.order[l],
                                  X_bd=self.X_bd_used.get(l), **common)
        else:
            B.pgcn_layer_bwd(self.part, order=self.order[l], H_in=self.X_used.get(l), H_bd=self.X_bd_used.get(l),
                             **common)
        if l > 1 and self.opts.dropout > 0.0:
            self._dropout(self.J_in[l], self.J_in[l], self.n, l, 0, None, st)
            self._dropout(self.J_bd_out[l], self.J_bd_out[l], self.b, l, self.n, None, st)

    def step(self):
        o, L, wd = self.opts, self.L, self.widths
        n, b, s = self.n, self.b, self.s
        st, side = self.stream, self.side
        self.t += 1
        t = self.t
        cur, nxt = self.cur, 1 - self.cur
        mode = o.copy_mode
        caller = torch.cuda.current_stream(self.dev)
        st.wait_stream(caller)          # inputs written by the caller's stream are visible

        # ---- forward --------------------------------------------------
        for l in range(1, L + 1):
            f = wd[l - 1]
            H_in = self.X if l == 1 else self.H[l - 1]
            H_bd = None
            if self.cache1 and l == 1:
                # the constant layer input: its boundary rows are exchanged once (iteration 1's send,
                # received in iteration 2) and the smoothing acts on the kept aggregate
                if self.A1_ready:
                    self._forward_layer1_cached(None, st)
                    continue
                if mode == "serial":
                    self._refill(self.feat[1][cur], self.remote_f[1], st)
                if t > 1 or mode == "serial":
                    if mode == "pipe":
                        st.wait_event(self.ev_feat[1])
                    H_bd = self.feat[1][cur]
                if t == 1:
                    B.pgcn_pack_boundary(self.part, B.PGCN_PACK_FEAT, H_in, self.send_f[1], f, ld_of(f), st)
                    if mode == "pipe":
                        self.ev_pack[1].record(st)
                        side.wait_event(self.ev_pack[1])
                        self._refill(self.feat[1][nxt], self.remote_f[1], side)
                        self.ev_feat[1].record(side)
                self._forward_layer1_cached(H_bd, st)
                continue
            if mode == "serial":
                self._refill(self.feat[l][cur], self.remote_f[l], st)
            if t > 1 or mode == "serial":
                if mode == "pipe":
                    st.wait_event(self.ev_feat[l])
                H_bd = self.feat[l][cur]
                if o.smooth_f:
                    B.pgcn_smooth_ema(self.ema_f[l], H_bd, b, f, ld_of(f), o.gamma, st)
                    H_bd = self.ema_f[l]
            if l == 1 or not o.fuse_pack:      # fused: layer l - 1's output kernel wrote these rows
                B.pgcn_pack_boundary(self.part, B.PGCN_PACK_FEAT, H_in, self.send_f[l], f, ld_of(f), st)
            if mode == "pipe":
                self.ev_pack[l].record(st)
                side.wait_event(self.ev_pack[l])
                self._refill(self.feat[l][nxt], self.remote_f[l], side)
                self.ev_feat[l].record(side)
            self._forward_layer(l, H_in, H_bd, st)

        # ---- loss -----------------------------------------------------
        C_ = wd[L]
        B.pgcn_loss_fwd_bwd(self.loss_kind, self.H[L], n, C_, ld_of(C_), self.labels, self.targets, ld_of(C_),
                            self.loss_scale, self.J_top, self.loss, self.ws, self.ws_bytes, st)

        # ---- backward -------------------------------------------------
        for l in range(L, 0, -1):
            f = wd[l - 1]
            J_out = self.J_top if l == L else self.J_in[l + 1]
            self._backward_layer(l, J_out, st)
            if l == 1:
                break
            if mode == "serial":
                self._refill(self.grad[l][cur], self.remote_g[l], st)
            if t > 1 or mode == "serial":
                if mode == "pipe":
                    st.wait_event(self.ev_grad[l])
                C = self.grad[l][cur]
                if o.smooth_g:      # smoothing of the received rows fused with their accumulation
                    B.pgcn_accum_smoothed(self.part, C, self.ema_g[l], o.gamma, self.J_in[l], f, ld_of(f), st)
                else:
                    B.pgcn_pack_boundary(self.part, B.PGCN_ACCUM_GRAD, C, self.J_in[l], f, ld_of(f), st)
            if mode == "pipe":
                self.ev_bwd[l].record(st)
                side.wait_event(self.ev_bwd[l])
                self._refill(self.grad[l][nxt], self.remote_g[l], side)
                self.ev_grad[l].record(side)

        # ---- AllReduce (identity on one partition, or + the injected peer sum) and the update
        for l in range(L):
            if o.optimizer == "adam":
                B.pgcn_adam_update(self.W[l], self.dW[l], self.G_peer[l], self.adam_m[l], self.adam_v[l],
                                   self.W[l].numel(), o.eta, o.beta1, o.beta2, o.eps, t, st)
            else:
                B.pgcn_sgd_update(self.W[l], self.dW[l], self.G_peer[l], self.W[l].numel(), o.eta, st)
        if mode == "pipe":
            self.cur = nxt
        caller.wait_stream(st)          # results are ordered before the caller's next work
        return self.loss

    def synchronize(self):
        self.stream.synchronize()
        self.side.synchronize()
