"""Two-layer GCN training on the libgcn C ABI.

This module only allocates device buffers (through torch) and sequences the
library calls; every arithmetic step runs in the HIP kernels.  One training
step is (Section "Graph Convolutions", Eq. (1), two stacked layers; O2 mixed
precision of Section "Background and Motivation"):

    H1 = dropout(ReLU(A_hat (X W1) + b1))        gcn_layer_fwd, layer 0
    Z2 = A_hat (H1 W2) + b2                       gcn_layer_fwd, layer 1
    loss, dZ2 = softmax-CE(Z2) * S                gcn_loss (S = loss scale)
    dW2, db2, dZ1 = backward of layer 1           gcn_layer_bwd
    dW1, db1      = backward of layer 0           gcn_layer_bwd
    Adam on fp32 masters + dynamic loss scale     gcn_optimizer_step
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass

import numpy as np
import torch

from . import gcn as G


def round8(x: int) -> int:
    return (x + 7) // 8 * 8


def _nullctx():
    import contextlib
    return contextlib.nullcontext()


class DeviceGraph:
    """A_hat on the device, built by gcn_normalize (+ gcn_schedule for CSR)."""

    def __init__(self, n, src, dst, prec=G.GCN_F16, index=G.GCN_I32, dense=False, values=True,
                 schedule=True, device="cuda", heavy_threshold=0, chunk_nnz=0, stream=None, tiled=None,
                 col_parts=0):
        """dense=True stores A_hat densely: in the tiled operand order by
        default (tiled=None or True), row-major when tiled=False.
        heavy_threshold, chunk_nnz, col_parts: gcn_schedule's arguments
        (0 = the library's defaults)."""
        self.n = int(n)
        self.prec = prec
        dev = torch.device(device)
        if isinstance(src, torch.Tensor):   # device-drawn edges (large graphs)
            src_t, dst_t = src.to(dev, torch.int32), dst.to(dev, torch.int32)
        else:
            src_t = torch.as_tensor(np.ascontiguousarray(src, dtype=np.int32)).to(dev)
            dst_t = torch.as_tensor(np.ascontiguousarray(dst, dtype=np.int32)).to(dev)
        ne = src_t.numel()
        cap = 2 * ne + self.n
        itype = torch.int64 if index == G.GCN_I64 else torch.int32
        self.rowptr = torch.empty(self.n + 1, dtype=itype, device=dev)
        self.colidx = torch.empty(cap, dtype=torch.int32, device=dev)
        self.deg = torch.empty(self.n, dtype=torch.int32, device=dev)
        self.dinv = torch.empty(self.n, dtype=torch.float32, device=dev)
        vdt = G.torch_dtype(prec)
        self.tiled = bool(dense) and (tiled is None or tiled)
        self.values = torch.empty(cap, dtype=vdt, device=dev) if (values and not dense) else None
        self.ld_dense = round8(self.n) if (dense and not self.tiled) else 0
        if not dense:
            self.dense = None
        elif self.tiled:
            self.dense = torch.empty(G.gcn_dense_tiled_elems(self.n, prec), dtype=vdt, device=dev)
        else:
            self.dense = torch.empty((self.n, self.ld_dense), dtype=vdt, device=dev)
        ws = torch.empty(G.gcn_normalize_workspace_size(self.n, ne), dtype=torch.uint8, device=dev)
        self.nnz = G.gcn_normalize(self.n, src_t if ne else None, dst_t if ne else None, index, self.rowptr,
                                   self.colidx, self.deg, self.dinv, prec, self.values,
                                   None if self.tiled else self.dense, self.ld_dense, ws, stream)
        del ws, src_t, dst_t
        self.adj = G.GcnAdj()
        a = self.adj
        a.n = self.n
        a.nnz = self.nnz
        a.format = G.GCN_CSR
        a.index = index
        a.value_prec = prec
        a.rowptr = self.rowptr.data_ptr()
        a.colidx = self.colidx.data_ptr()
        a.values = self.values.data_ptr() if self.values is not None else None
        a.dinv = self.dinv.data_ptr()
        if self.tiled:   # the CSR (values from dinv) is the source of the tiled copy
            G.gcn_densify(a, G.GCN_DENSE_TILED, prec, self.dense, 0, stream)
        if dense:
            a.format = G.GCN_DENSE_TILED if self.tiled else G.GCN_DENSE
            a.dense = self.dense.data_ptr()
            a.ld_dense = self.ld_dense
        self.sched = None
        if schedule and not dense:
            nbytes = G.gcn_schedule_size(self.n, self.nnz, heavy_threshold, chunk_nnz, col_parts)
            self.sched = torch.empty(nbytes, dtype=torch.uint8, device=dev)
            G.gcn_schedule(a, self.sched, heavy_threshold, chunk_nnz, col_parts, stream)

    def csr_host(self):
        rp = self.rowptr.cpu().numpy().astype(np.int64)
        return rp, self.colidx[: self.nnz].cpu().numpy()


@dataclass
class AdamConfig:
    lr: float = 0.01
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    backoff: float = 0.5
    growth: float = 2.0
    interval: int = 2000
    min_scale: float = 1.0
    max_scale: float = 16777216.0

    def c(self):
        return G.GcnAdamConfig(self.lr, self.beta1, self.beta2, self.eps, self.backoff, self.growth,
                               self.interval, self.min_scale, self.max_scale)


LEVELS = ("O0", "O1", "O2", "O3")


class GCN2:
    """Two-layer GCN for vertex classification with device-resident state.

    ``level`` selects the optimisation level of Section "Background and
    Motivation" (default: O0 for prec = GCN_F32, else O2):

    * O0: everything in fp32.
    * O2: 16-bit weights, activations and gradients; fp32 master weights
      and Adam moments; dynamic loss scaling.
    * O1: the cast-list policy.  The model's inputs (X and A_hat) and its
      parameters stay fp32; the GEMM-class operations (the transform, the
      aggregation and their backward products) run on 16-bit copies made by
      gcn_cast at every forward pass (the weights' copy is cached per step:
      it is the optimiser's working copy), and the loss runs in fp32 on an
      fp32 copy of the logits; dynamic loss scaling.  ``graph`` must then
      hold A_hat in fp32, CSR or row-major dense.
    * O3: every tensor in 16 bits, the weights and the Adam moments
      included (gcn_optimizer_step_half); no master copy and no loss scale.
    """

    def __init__(self, graph: DeviceGraph, X, labels, mask, W1, W2, b1=None, b2=None, prec=G.GCN_F16,
                 dropout=0.5, seed=0, loss_scale=65536.0, adam: AdamConfig | None = None, device="cuda",
                 level: str | None = None, device_epoch: bool = False):
        """device_epoch: the dropout counter of an epoch is read on the device
        from the loss-scale state (optimiser calls so far) instead of being
        passed by the host, so that one captured epoch (capture()) can be
        replayed; the epoch argument of step() is then ignored, and epochs
        count from 0 at construction."""
        dev = torch.device(device)
        if level is None:
            level = "O0" if prec == G.GCN_F32 else "O2"
        if level not in LEVELS:
            raise ValueError(f"level must be one of {LEVELS}")
        if (level == "O0") != (prec == G.GCN_F32):
            raise ValueError("O0 computes in fp32 (prec = GCN_F32); O1-O3 need a 16-bit prec")
        self.level = level
        self.g = graph
        self.prec = prec
        self.dt = G.torch_dtype(prec)
        n = graph.n
        self.n = n
        # the adjacency the layers read: for O1 a 16-bit copy of the fp32
        # input, refreshed by every forward pass
        self.adj = graph.adj
        self.A16 = None
        if level == "O1":
            a = graph.adj
            if a.value_prec != G.GCN_F32 or a.format == G.GCN_DENSE_TILED:
                raise ValueError("O1 casts an fp32 A_hat: build the graph with prec=GCN_F32 and tiled=False")
            self.adj = G.GcnAdj.from_buffer_copy(a)
            self.adj.value_prec = prec
            if a.format == G.GCN_DENSE:
                self.A16 = torch.empty(graph.dense.shape, dtype=self.dt, device=dev)
                self.adj.dense = self.A16.data_ptr()
            elif graph.values is not None:
                self.A16 = torch.empty(graph.nnz, dtype=self.dt, device=dev)
                self.adj.values = self.A16.data_ptr()
        self.f_in, self.f_h = W1.shape
        self.C = W2.shape[1]
        assert W2.shape[0] == self.f_h
        self.ld_x, self.ld_h, self.ld_c = round8(self.f_in), round8(self.f_h), round8(self.C)
        self.p = float(dropout)
        self.seed = int(seed)
        self.adam = adam or AdamConfig()
        # inputs (padding columns zero); a device tensor already in the
        # storage layout (n x round8(f_in), storage dtype) is used in place
        self.X32 = None
        # X = None: the featureless input X = I (f_in = n, W1 is n x f_h)
        self.featureless = X is None
        if self.featureless:
            assert self.f_in == n, "featureless input: W1 must have n rows"
            self.X = None
        elif level == "O1":     # fp32 input plus the 16-bit copy its GEMM reads
            self.X32 = torch.zeros((n, self.ld_x), dtype=torch.float32, device=dev)
            self.X32[:, : self.f_in] = torch.as_tensor(np.asarray(X, np.float32)).to(dev)
            self.X = torch.zeros((n, self.ld_x), dtype=self.dt, device=dev)
        elif isinstance(X, torch.Tensor) and X.is_cuda and X.dtype == self.dt and tuple(X.shape) == (n, self.ld_x):
            self.X = X
        else:
            self.X = torch.zeros((n, self.ld_x), dtype=self.dt, device=dev)
            self.X[:, : self.f_in] = torch.as_tensor(np.asarray(X, np.float32)).to(dev).to(self.dt)
        if isinstance(labels, torch.Tensor):
            self.labels = labels.to(dev, torch.int32)
            self.mask = mask.to(dev, torch.uint8)
            self.n_mask = int(self.mask.sum().item())
        else:
            self.labels = torch.as_tensor(np.asarray(labels, np.int32)).to(dev)
            mask = np.asarray(mask, np.uint8)
            self.mask = torch.as_tensor(mask).to(dev)
            self.n_mask = int(mask.sum())
        # flat parameters: [W1 (f_in x ld_h), b1 (ld_h), W2 (f_h x ld_c), b2 (ld_c)]
        sizes = [self.f_in * self.ld_h, self.ld_h, self.f_h * self.ld_c, self.ld_c]
        offs = np.cumsum([0] + sizes)
        self.P = int(offs[-1])
        self.offs = offs
        master = np.zeros(self.P, np.float32)
        w1 = np.zeros((self.f_in, self.ld_h), np.float32)
        w1[:, : self.f_h] = W1
        w2 = np.zeros((self.f_h, self.ld_c), np.float32)
        w2[:, : self.C] = W2
        master[offs[0]:offs[1]] = w1.ravel()
        if b1 is not None:
            master[offs[1]:offs[1] + self.f_h] = b1
        master[offs[2]:offs[3]] = w2.ravel()
        if b2 is not None:
            master[offs[3]:offs[3] + self.C] = b2
        self.master = torch.as_tensor(master).to(dev)
        self.working = self.master.to(self.dt)
        self.grad = torch.zeros(self.P, dtype=torch.float32, device=dev)
        # Adam moments: fp32 next to the masters, 16-bit in O3 (where
        # `master` only holds the fp32 widening of the 16-bit parameters that
        # the bias epilogue reads)
        mdt = self.dt if level == "O3" else torch.float32
        if level == "O3":
            self.master = self.working.float()
        self.m = torch.zeros(self.P, dtype=mdt, device=dev)
        self.v = torch.zeros(self.P, dtype=mdt, device=dev)
        self.scaler = torch.zeros(4, dtype=torch.int32, device=dev)   # gcn_scaler (16 bytes)
        self.scaler.view(torch.float32)[0] = loss_scale if level in ("O1", "O2") else 1.0
        self.overflow = torch.zeros(1, dtype=torch.int32, device=dev)
        self.loss = torch.zeros(1, dtype=torch.float32, device=dev)
        self.n_correct = torch.zeros(1, dtype=torch.int32, device=dev)
        # activations
        self.H1 = torch.empty((n, self.ld_h), dtype=self.dt, device=dev)
        self.SG1 = torch.empty((n, self.ld_h), dtype=self.dt, device=dev)   # S1, later G_S1
        self.dZ1 = torch.empty((n, self.ld_h), dtype=self.dt, device=dev)
        self.Z2 = torch.empty((n, self.ld_c), dtype=self.dt, device=dev)
        self.SG2 = torch.empty((n, self.ld_c), dtype=self.dt, device=dev)   # S2, later G_S2
        self.dZ2 = torch.empty((n, self.ld_c), dtype=self.dt, device=dev)
        if level == "O1":     # the loss's fp32 copies of the logits and of their gradient
            self.Z2f = torch.empty((n, self.ld_c), dtype=torch.float32, device=dev)
            self.dZ2f = torch.empty((n, self.ld_c), dtype=torch.float32, device=dev)
        # layers
        self.L1 = G.GcnLayer(self.f_in, self.f_h, self.ld_x, self.ld_h, G.GCN_ACT_RELU, self.p, 0,
                             1 if self.featureless else 0)
        self.L2 = G.GcnLayer(self.f_h, self.C, self.ld_h, self.ld_c, G.GCN_ACT_NONE, 0.0, 1, 0)
        self.device_epoch = bool(device_epoch)
        if self.device_epoch:
            self.L1.epoch_from = self.scaler.data_ptr()
            self.L2.epoch_from = self.scaler.data_ptr()
        self.graph = None
        ws = max(G.gcn_layer_workspace_size(self.adj, self.L1, prec),
                 G.gcn_layer_workspace_size(self.adj, self.L2, prec),
                 G.gcn_loss_workspace_size(n, self.C),
                 0 if self.featureless else G.gcn_transform_workspace_size(n, self.f_in, self.f_h, prec),
                 G.gcn_transform_workspace_size(n, self.f_h, self.C, prec),
                 G.gcn_aggregate_workspace_size(self.adj, self.f_h, prec),
                 G.gcn_aggregate_workspace_size(self.adj, self.C, prec))
        self.ws = torch.empty(ws // 4 + 64, dtype=torch.float32, device=dev)
        self.adam_c = self.adam.c()

    # parameter views
    def _view(self, buf, k, shape):
        return buf[self.offs[k]:self.offs[k + 1]].view(*shape)

    def W1w(self): return self._view(self.working, 0, (self.f_in, self.ld_h))
    def W2w(self): return self._view(self.working, 2, (self.f_h, self.ld_c))
    def b1m(self): return self._view(self.master, 1, (self.ld_h,))
    def b2m(self): return self._view(self.master, 3, (self.ld_c,))
    def dW1(self): return self._view(self.grad, 0, (self.f_in, self.ld_h))
    def db1(self): return self._view(self.grad, 1, (self.ld_h,))
    def dW2(self): return self._view(self.grad, 2, (self.f_h, self.ld_c))
    def db2(self): return self._view(self.grad, 3, (self.ld_c,))

    def scale_ptr(self):
        return self.scaler.data_ptr()   # first field of gcn_scaler is the float scale

    def forward(self, epoch: int, training: bool = True, stream=None, agg_timer=None, gemm_timer=None):
        """Both layers.  With ``agg_timer`` (a callable returning a context
        manager), each layer runs as gcn_transform + gcn_aggregate and the
        aggregation call is bracketed by the timer (the transform by
        ``gemm_timer`` if given); the arithmetic is the same as
        gcn_layer_fwd."""
        a = self.adj
        if self.device_epoch:
            if agg_timer is not None or gemm_timer is not None:
                raise ValueError("timed split calls take the epoch from the host; use device_epoch=False")
            epoch = 0         # the device counter supplies the epoch
        if self.level == "O1":
            self.cast_inputs(stream)
        if agg_timer is None:
            G.gcn_layer_fwd(a, self.L1, self.prec, training, self.X, self.W1w(), self.b1m(), self.seed, epoch,
                            self.SG1, self.H1, self.overflow, self.ws, stream)
            G.gcn_layer_fwd(a, self.L2, self.prec, training, self.H1, self.W2w(), self.b2m(), self.seed, epoch,
                            self.SG2, self.Z2, self.overflow, self.ws, stream)
            return
        for L, H, W, b, S, out in ((self.L1, self.X, self.W1w(), self.b1m(), self.SG1, self.H1),
                                   (self.L2, self.H1, self.W2w(), self.b2m(), self.SG2, self.Z2)):
            if L.identity_input:      # S = I W = W
                S = W
            else:
                with (gemm_timer() if gemm_timer is not None else _nullctx()):
                    G.gcn_transform(self.n, L.f_in, L.f_out, self.prec, H, L.ld_in, W, L.ld_out, S, L.ld_out,
                                    self.overflow, self.ws, stream)
            with agg_timer():
                G.gcn_aggregate(a, L.f_out, self.prec, S, L.ld_out, b, L.act, L.dropout_p, training, self.seed,
                                L.layer_id, epoch, out, L.ld_out, self.overflow, self.ws, stream)

    def cast_inputs(self, stream=None):
        """O1: the 16-bit copies of X and A_hat that this forward pass's
        GEMM-class operations read."""
        if self.X32 is not None:
            G.gcn_cast(self.n, self.f_in, G.GCN_F32, self.X32, self.ld_x, self.prec, self.X, self.ld_x,
                       self.overflow, stream)
        g = self.g
        if g.adj.format == G.GCN_DENSE:
            G.gcn_cast(self.n, self.n, G.GCN_F32, g.dense, g.ld_dense, self.prec, self.A16, g.ld_dense,
                       self.overflow, stream)
        elif self.A16 is not None:
            G.gcn_cast(1, g.nnz, G.GCN_F32, g.values, 0, self.prec, self.A16, 0, self.overflow, stream)

    def loss_and_backward(self, stream=None):
        a = self.adj
        if self.level == "O1":     # the loss is on the fp32 list
            G.gcn_cast(self.n, self.C, self.prec, self.Z2, self.ld_c, G.GCN_F32, self.Z2f, self.ld_c, None, stream)
            G.gcn_loss(self.n, self.C, self.ld_c, G.GCN_F32, self.Z2f, self.labels, self.mask, self.n_mask,
                       self.scale_ptr(), self.loss, self.dZ2f, self.n_correct, self.overflow, self.ws, stream)
            G.gcn_cast(self.n, self.C, G.GCN_F32, self.dZ2f, self.ld_c, self.prec, self.dZ2, self.ld_c,
                       self.overflow, stream)
            db2 = self.db2()
        else:
            # db2 (the column sums of dZ2) comes from the loss kernel
            G.gcn_loss(self.n, self.C, self.ld_c, self.prec, self.Z2, self.labels, self.mask, self.n_mask,
                       self.scale_ptr(), self.loss, self.dZ2, self.n_correct, self.overflow, self.ws, stream,
                       dlogits_colsum=self.db2())
            db2 = None
        # db1 (the column sums of dZ1) comes from the call that writes dZ1
        G.gcn_layer_bwd(a, self.L2, self.prec, self.H1, self.W2w(), self.dZ2, G.GCN_ACT_RELU, self.p,
                        self.dW2(), db2, self.dZ1, self.SG2, self.overflow, self.ws, stream,
                        dbias_below=self.db1())
        G.gcn_layer_bwd(a, self.L1, self.prec, self.X, self.W1w(), self.dZ1, G.GCN_ACT_NONE, 0.0,
                        self.dW1(), None, None, self.SG1, self.overflow, self.ws, stream)

    def optimizer_step(self, stream=None):
        if self.level == "O3":
            G.gcn_optimizer_step_half(self.P, self.working, self.grad, self.m, self.v, self.master, self.prec,
                                      self.adam_c, self.scaler, self.overflow, stream)
            return
        G.gcn_optimizer_step(self.P, self.master, self.grad, self.m, self.v, self.working, self.prec,
                             self.adam_c, self.scaler, self.overflow, stream)

    def step(self, epoch: int, stream=None, agg_timer=None, gemm_timer=None):
        """One full training step; asynchronous (no host synchronisation)."""
        self.forward(epoch, True, stream, agg_timer, gemm_timer)
        self.loss_and_backward(stream)
        self.optimizer_step(stream)

    def capture(self):
        """Record one training epoch (forward, loss, backward, optimiser)
        into a HIP graph; replay() then runs it.  Needs device_epoch=True
        (the graph reads its dropout epoch on the device).  Nothing runs
        while capturing: the model's state is unchanged."""
        if not self.device_epoch:
            raise ValueError("capture() needs device_epoch=True")
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.step(0)
        self.graph = g
        return g

    def replay(self):
        """One training epoch from the captured graph; asynchronous."""
        self.graph.replay()

    def scaler_state(self):
        s = self.scaler.cpu()
        return dict(scale=float(s.view(torch.float32)[0]), good_steps=int(s[1]), step=int(s[2]),
                    skipped=int(s[3]))


class GAE2:
    """Graph auto-encoder for link prediction (Section "Graph Auto-Encoders",
    Eq. (2)): Z = GCN(A_hat, X) with two layers (ReLU on the hidden layer, no
    dropout, linear embedding layer), A' = sigmoid(Z Z^T) evaluated on the
    pairs of each epoch: n_pos training edges and n_neg uniform pairs drawn
    by gcn_sample_pairs, logistic loss by gcn_pair_loss, its gradient into Z
    by gcn_pair_backward, then the encoder's backward pass and Adam with
    dynamic loss scaling as in GCN2."""

    def __init__(self, graph: DeviceGraph, X, W1, W2, train_u, train_v, b1=None, b2=None, prec=G.GCN_F16,
                 n_pos=1 << 20, n_neg=1 << 20, seed=0, loss_scale=65536.0, adam: AdamConfig | None = None,
                 device="cuda"):
        dev = torch.device(device)
        self.g = graph
        self.prec = prec
        self.dt = G.torch_dtype(prec)
        n = graph.n
        self.n = n
        self.f_in, self.f_h = W1.shape
        self.f_e = W2.shape[1]
        self.ld_x, self.ld_h, self.ld_e = round8(self.f_in), round8(self.f_h), round8(self.f_e)
        self.n_pos, self.n_neg = int(n_pos), int(n_neg)
        self.K = self.n_pos + self.n_neg
        self.seed = int(seed)
        self.adam = adam or AdamConfig()
        if isinstance(X, torch.Tensor) and X.is_cuda and X.dtype == self.dt and tuple(X.shape) == (n, self.ld_x):
            self.X = X
        else:
            self.X = torch.zeros((n, self.ld_x), dtype=self.dt, device=dev)
            self.X[:, : self.f_in] = torch.as_tensor(np.asarray(X, np.float32)).to(dev).to(self.dt)
        self.train_u = torch.as_tensor(np.asarray(train_u, np.int32)).to(dev)
        self.train_v = torch.as_tensor(np.asarray(train_v, np.int32)).to(dev)
        sizes = [self.f_in * self.ld_h, self.ld_h, self.f_h * self.ld_e, self.ld_e]
        offs = np.cumsum([0] + sizes)
        self.P = int(offs[-1])
        self.offs = offs
        master = np.zeros(self.P, np.float32)
        w1 = np.zeros((self.f_in, self.ld_h), np.float32)
        w1[:, : self.f_h] = W1
        w2 = np.zeros((self.f_h, self.ld_e), np.float32)
        w2[:, : self.f_e] = W2
        master[offs[0]:offs[1]] = w1.ravel()
        if b1 is not None:
            master[offs[1]:offs[1] + self.f_h] = b1
        master[offs[2]:offs[3]] = w2.ravel()
        if b2 is not None:
            master[offs[3]:offs[3] + self.f_e] = b2
        self.master = torch.as_tensor(master).to(dev)
        self.working = self.master.to(self.dt)
        self.grad = torch.zeros(self.P, dtype=torch.float32, device=dev)
        self.m = torch.zeros(self.P, dtype=torch.float32, device=dev)
        self.v = torch.zeros(self.P, dtype=torch.float32, device=dev)
        self.scaler = torch.zeros(4, dtype=torch.int32, device=dev)
        self.scaler.view(torch.float32)[0] = loss_scale if prec != G.GCN_F32 else 1.0
        self.overflow = torch.zeros(1, dtype=torch.int32, device=dev)
        self.loss = torch.zeros(1, dtype=torch.float32, device=dev)
        self.H1 = torch.empty((n, self.ld_h), dtype=self.dt, device=dev)
        self.SG1 = torch.empty((n, self.ld_h), dtype=self.dt, device=dev)
        self.dZ1 = torch.empty((n, self.ld_h), dtype=self.dt, device=dev)
        self.Z = torch.empty((n, self.ld_e), dtype=self.dt, device=dev)
        self.SG2 = torch.empty((n, self.ld_e), dtype=self.dt, device=dev)
        self.dZ = torch.empty((n, self.ld_e), dtype=self.dt, device=dev)
        self.pair_u = torch.empty(self.K, dtype=torch.int32, device=dev)
        self.pair_v = torch.empty(self.K, dtype=torch.int32, device=dev)
        self.pair_g = torch.empty(self.K, dtype=torch.float32, device=dev)
        self.L1 = G.GcnLayer(self.f_in, self.f_h, self.ld_x, self.ld_h, G.GCN_ACT_RELU, 0.0, 0, 0)
        self.L2 = G.GcnLayer(self.f_h, self.f_e, self.ld_h, self.ld_e, G.GCN_ACT_NONE, 0.0, 1, 0)
        ws = max(G.gcn_layer_workspace_size(graph.adj, self.L1, prec),
                 G.gcn_layer_workspace_size(graph.adj, self.L2, prec),
                 G.gcn_pair_loss_workspace_size(self.K),
                 G.gcn_pair_backward_workspace_size(n, self.K, self.f_e))
        self.ws = torch.empty(ws // 4 + 64, dtype=torch.float32, device=dev)
        self.adam_c = self.adam.c()

    def _view(self, buf, k, shape):
        return buf[self.offs[k]:self.offs[k + 1]].view(*shape)

    def W1w(self): return self._view(self.working, 0, (self.f_in, self.ld_h))
    def W2w(self): return self._view(self.working, 2, (self.f_h, self.ld_e))
    def b1m(self): return self._view(self.master, 1, (self.ld_h,))
    def b2m(self): return self._view(self.master, 3, (self.ld_e,))
    def dW1(self): return self._view(self.grad, 0, (self.f_in, self.ld_h))
    def db1(self): return self._view(self.grad, 1, (self.ld_h,))
    def dW2(self): return self._view(self.grad, 2, (self.f_h, self.ld_e))
    def db2(self): return self._view(self.grad, 3, (self.ld_e,))

    def encode(self, stream=None):
        a = self.g.adj
        G.gcn_layer_fwd(a, self.L1, self.prec, True, self.X, self.W1w(), self.b1m(), 0, 0, self.SG1, self.H1,
                        self.overflow, self.ws, stream)
        G.gcn_layer_fwd(a, self.L2, self.prec, True, self.H1, self.W2w(), self.b2m(), 0, 0, self.SG2, self.Z,
                        self.overflow, self.ws, stream)

    def loss_and_backward(self, epoch: int, stream=None):
        a = self.g.adj
        G.gcn_sample_pairs(self.n, self.train_u, self.train_v, self.n_pos, self.n_neg, self.seed, epoch,
                           self.pair_u, self.pair_v, stream)
        G.gcn_pair_loss(self.n, self.f_e, self.ld_e, self.prec, self.Z, self.pair_u, self.pair_v, self.n_pos,
                        self.n_neg, self.scaler, self.loss, None, self.pair_g, self.overflow, self.ws, stream)
        G.gcn_pair_backward(self.n, self.f_e, self.ld_e, self.prec, self.Z, self.pair_u, self.pair_v, self.K,
                            self.pair_g, self.dZ, self.ld_e, self.overflow, self.ws, stream)
        G.gcn_layer_bwd(a, self.L2, self.prec, self.H1, self.W2w(), self.dZ, G.GCN_ACT_RELU, 0.0,
                        self.dW2(), self.db2(), self.dZ1, self.SG2, self.overflow, self.ws, stream,
                        dbias_below=self.db1())
        G.gcn_layer_bwd(a, self.L1, self.prec, self.X, self.W1w(), self.dZ1, G.GCN_ACT_NONE, 0.0,
                        self.dW1(), None, None, self.SG1, self.overflow, self.ws, stream)

    def optimizer_step(self, stream=None):
        G.gcn_optimizer_step(self.P, self.master, self.grad, self.m, self.v, self.working, self.prec,
                             self.adam_c, self.scaler, self.overflow, stream)

    def step(self, epoch: int, stream=None):
        """One training epoch; asynchronous."""
        self.encode(stream)
        self.loss_and_backward(epoch, stream)
        self.optimizer_step(stream)

    def evaluate(self, test_u, test_v, n_test_pos, stream=None):
        """AUC and AP of held-out pairs (positives first) on the current
        embeddings; one host synchronisation."""
        dev = self.Z.device
        tu = torch.as_tensor(np.asarray(test_u, np.int32)).to(dev)
        tv = torch.as_tensor(np.asarray(test_v, np.int32)).to(dev)
        k = tu.numel()
        self.encode(stream)
        scores = torch.empty(k, dtype=torch.float32, device=dev)
        g = torch.empty(k, dtype=torch.float32, device=dev)
        loss = torch.empty(1, dtype=torch.float32, device=dev)
        flag = torch.zeros(1, dtype=torch.int32, device=dev)
        ws = torch.empty(G.gcn_pair_loss_workspace_size(k) // 4 + 64, dtype=torch.float32, device=dev)
        G.gcn_pair_loss(self.n, self.f_e, self.ld_e, self.prec, self.Z, tu, tv, n_test_pos, k - n_test_pos, None,
                        loss, scores, g, flag, ws, stream)
        out = torch.empty(2, dtype=torch.float64, device=dev)
        mws = torch.empty(G.gcn_pair_metrics_workspace_size(n_test_pos, k - n_test_pos), dtype=torch.uint8, device=dev)
        G.gcn_pair_metrics(scores, n_test_pos, k - n_test_pos, out, mws, stream)
        auc, ap = out.cpu().tolist()
        return auc, ap, float(loss.item())

    def scaler_state(self):
        s = self.scaler.cpu()
        return dict(scale=float(s.view(torch.float32)[0]), good_steps=int(s[1]), step=int(s[2]),
                    skipped=int(s[3]))
