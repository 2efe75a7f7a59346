"""Device-side objects for running layers through the C ABI.

DeviceGraph uploads a sampled subgraph's CSR and runs the per-subgraph
preparation (transposed values, aggregation plan).  SageStack holds the
weights and activations of an L-layer GraphSAGE stack and chains the
layers (Algorithm 1's layer loop: forward l = 1..L, backward l = L..1 with
each layer's dX feeding the layer below).  Only buffer management and calls
into libgnnprop happen here.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import numpy as np
import torch

from . import gnnprop as G


def _round_up(a: int, b: int) -> int:
    return (a + b - 1) // b * b


def padded(t: torch.Tensor, ld: int) -> torch.Tensor:
    """Copy a (rows, cols) tensor into a (rows, ld) buffer; returns the
    (rows, cols) view with row stride ld."""
    rows, cols = t.shape
    buf = torch.zeros((rows, ld), dtype=t.dtype, device=t.device)
    buf[:, :cols] = t
    return buf[:, :cols]


class DeviceGraph:
    def __init__(self, csr, device: str = "cuda"):
        self.n = int(csr.n)
        self.nnz = int(csr.nnz)
        self.device = device
        self.indptr = torch.from_numpy(np.ascontiguousarray(csr.indptr)).to(device)
        self.indices = torch.from_numpy(np.ascontiguousarray(csr.indices)).to(device)
        self.values = torch.from_numpy(np.ascontiguousarray(csr.values, np.float32)).to(device)
        # at least one element so that data pointers are never NULL
        self.values_t = torch.empty(max(self.nnz, 1), dtype=torch.float32, device=device)
        if self.nnz == 0:
            self.indices = torch.empty(1, dtype=torch.int32, device=device)
            self.values = torch.empty(1, dtype=torch.float32, device=device)
        self.plan = torch.empty(max(G.gnn_plan_bytes(self.n, self.nnz), 256),
                                dtype=torch.uint8, device=device)

    @classmethod
    def on_device(cls, n: int, indptr: torch.Tensor, indices: torch.Tensor,
                  values: torch.Tensor) -> "DeviceGraph":
        """Wraps a CSR already in device memory (int32 indptr of n + 1,
        int32 indices and float32 values of nnz entries, nnz >= 1)."""
        g = cls.__new__(cls)
        g.n, g.nnz = int(n), int(indices.numel())
        g.device = indptr.device
        g.indptr, g.indices, g.values = indptr, indices, values
        g.values_t = torch.empty(max(g.nnz, 1), dtype=torch.float32, device=g.device)
        g.plan = torch.empty(max(G.gnn_plan_bytes(g.n, g.nnz), 256), dtype=torch.uint8,
                             device=g.device)
        return g

    def struct(self) -> G.gnn_csr:
        return G.make_csr(self.n, self.nnz, self.indptr, self.indices, self.values,
                          self.values_t, self.plan)

    def prepare(self, stream=None):
        """Per-subgraph preparation: (A_s)^T values and the work plan."""
        c = self.struct()
        G.gnn_csr_build_plan(c, self.plan, stream)
        G.gnn_csr_transpose_values(c, self.values_t, stream)

    def validate(self, symmetric: bool = True) -> int:
        return G.gnn_csr_validate(self.struct(), symmetric)


class FullGraphDevice:
    """A full training graph resident in device memory with its features
    and labels; builds minibatch subgraphs from host node lists (the
    induction of Algorithms 2 / 3 and Algorithm 1's feature and label
    lookup, all in libgnnprop)."""

    def __init__(self, full, X: Optional[np.ndarray] = None,
                 labels: Optional[np.ndarray] = None, norm: int = G.GNN_NORM_ROW,
                 device: str = "cuda"):
        self.n, self.nnz = int(full.n), int(full.nnz)
        self.deg = np.asarray(full.degrees(), np.int64)
        self.device, self.norm = device, norm
        self.indptr = torch.from_numpy(np.ascontiguousarray(full.indptr, np.int64)).to(device)
        self.indices = torch.from_numpy(np.ascontiguousarray(full.indices, np.int32)).to(device)
        if self.nnz == 0:
            self.indices = torch.empty(1, dtype=torch.int32, device=device)
        self.map = torch.full((max(self.n, 1),), -1, dtype=torch.int32, device=device)
        self.X = None if X is None else \
            torch.from_numpy(np.ascontiguousarray(X, np.float32)).to(device)
        self.labels = None if labels is None else \
            torch.from_numpy(np.ascontiguousarray(labels, np.float32)).to(device)
        self.nnz_out = torch.zeros(1, dtype=torch.int64, device=device)
        self.status = torch.zeros(1, dtype=torch.int32, device=device)

    def capacity(self, nodes: np.ndarray) -> int:
        """Entries the induced subgraph of `nodes` can hold at most."""
        return int(self.deg[nodes].sum()) + len(nodes)

    def induce(self, nodes: np.ndarray, stream=None, pad: int = 16):
        """Subgraph on the sorted, distinct host node list `nodes`: returns
        (DeviceGraph prepared for propagation, X_s, labels_s).  Reads the
        entry count back (one synchronisation)."""
        nodes = np.ascontiguousarray(nodes, np.int32)
        n_s = len(nodes)
        cap = self.capacity(nodes) if n_s else 0
        nd = torch.from_numpy(nodes).to(self.device) if n_s else \
            torch.empty(1, dtype=torch.int32, device=self.device)
        ip = torch.empty(n_s + 1, dtype=torch.int32, device=self.device)
        ix = torch.empty(max(cap, 1), dtype=torch.int32, device=self.device)
        vals = torch.empty(max(cap, 1), dtype=torch.float32, device=self.device)
        ws = torch.empty(max(G.gnn_induce_workspace_bytes(n_s), 256), dtype=torch.uint8,
                         device=self.device)
        G.gnn_induce_subgraph(self.n, self.nnz, self.indptr, self.indices, n_s, nd,
                              self.norm, self.map, cap, ip, ix, vals, self.nnz_out,
                              self.status, ws, stream)
        Xs = Ts = None
        if self.X is not None:
            f = self.X.shape[1]
            Xs = torch.empty((max(n_s, 1), _round_up(f, pad)), device=self.device)[:n_s, :f]
            G.gnn_gather_rows(n_s, nd, f, self.X, self.X.stride(0), self.n, Xs,
                              Xs.stride(0), stream)
        if self.labels is not None:
            C = self.labels.shape[1]
            Ts = torch.empty((n_s, C), device=self.device)
            G.gnn_gather_rows(n_s, nd, C, self.labels, self.labels.stride(0), self.n, Ts,
                              C, stream)
        st, nnz = int(self.status.item()), int(self.nnz_out.item())
        if st:
            raise ValueError("gnn_induce_subgraph status %d (1: id out of range, 2: ids "
                             "not ascending, 4: over capacity)" % st)
        dg = DeviceGraph.on_device(n_s, ip, ix[: max(nnz, 1)], vals[: max(nnz, 1)])
        dg.nnz = nnz
        dg.nodes = nd
        dg.prepare(stream)
        return dg, Xs, Ts


class SageStack:
    """Weights, activations and gradients of an L-layer stack on one graph."""

    def __init__(self, graph: DeviceGraph, params: Sequence, f_in: int,
                 order: int = 0, flags: int = 0, pad: int = 16,
                 fuse_masks: bool = False, device: str = "cuda"):
        """fuse_masks: in the backward pass layer l > 0 writes its dX already
        masked by its input's sign (the ReLU mask of layer l - 1), which layer
        l - 1 then takes as its masked dY, so no separate masking pass runs
        below the top layer.  The dX buffers of layers l > 0 then hold those
        masked gradients; the first layer's dX is always the plain one.  Off
        by default: the mask read lands in the tail of the dX product, where
        it costs about what the masking pass it replaces does."""
        self.g = graph
        self.n = graph.n
        self.order, self.flags, self.pad = order, flags, pad
        self.fuse_masks = fuse_masks
        self.layers = []
        f = f_in
        ws_bytes = 0
        for p in params:
            h = p.w_self.shape[1]
            assert p.w_self.shape == (f, h) == p.w_neigh.shape
            L = {"f_in": f, "h": h}
            L["W_self"] = torch.from_numpy(np.ascontiguousarray(p.w_self)).to(device)
            L["W_neigh"] = torch.from_numpy(np.ascontiguousarray(p.w_neigh)).to(device)
            L["b_self"] = None if p.b_self is None else \
                torch.from_numpy(np.ascontiguousarray(p.b_self)).to(device)
            L["b_neigh"] = None if p.b_neigh is None else \
                torch.from_numpy(np.ascontiguousarray(p.b_neigh)).to(device)
            ld_y = _round_up(2 * h, pad)
            L["Y"] = torch.empty((max(self.n, 1), ld_y), device=device)[: self.n, : 2 * h]
            L["dW_self"] = torch.empty((f, h), device=device)
            L["dW_neigh"] = torch.empty((f, h), device=device)
            L["db_self"] = torch.empty(h, device=device) if p.b_self is not None else None
            L["db_neigh"] = torch.empty(h, device=device) if p.b_neigh is not None else None
            ld_x = _round_up(f, pad)
            L["dX"] = torch.empty((max(self.n, 1), ld_x), device=device)[: self.n, :f]
            self.layers.append(L)
            f = 2 * h
        self.f_in = f_in
        # layer structs need the input stride: filled at forward time
        for i, L in enumerate(self.layers):
            lay = self._layer(i, _round_up(L["f_in"], pad))
            sb = G.gnn_prop_saved_bytes(graph.struct(), lay)
            L["saved"] = torch.empty(max(sb, 256), dtype=torch.uint8, device=device)
            ws_bytes = max(ws_bytes, G.gnn_prop_workspace_bytes(graph.struct(), lay))
        self.workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=device)
        self.inputs: List[Optional[torch.Tensor]] = [None] * len(self.layers)

    def _layer(self, i: int, ld_x: int, extra_flags: int = 0) -> G.gnn_layer:
        L = self.layers[i]
        return G.make_layer(L["f_in"], L["h"], ld_x, L["Y"].stride(0) if self.n else 2 * L["h"],
                            L["dX"].stride(0) if self.n else L["f_in"], self.order,
                            self.flags | extra_flags)

    def forward(self, X: torch.Tensor, stream=None) -> torch.Tensor:
        csr = self.g.struct()
        x = X
        for i, L in enumerate(self.layers):
            self.inputs[i] = x
            ld_x = x.stride(0) if self.n else L["f_in"]
            G.gnn_prop_fwd(csr, self._layer(i, ld_x), x, L["W_self"], L["W_neigh"],
                           L["b_self"], L["b_neigh"], L["Y"], L["saved"],
                           self.workspace, stream)
            x = L["Y"]
        return x

    def backward(self, dY: torch.Tensor, want_dx_first: bool = True, stream=None):
        csr = self.g.struct()
        d = dY
        for i in reversed(range(len(self.layers))):
            L = self.layers[i]
            x = self.inputs[i]
            ld_x = x.stride(0) if self.n else L["f_in"]
            extra = 0
            if self.fuse_masks:
                if i < len(self.layers) - 1:
                    extra |= G.GNN_FLAG_DY_MASKED
                if i > 0:
                    extra |= G.GNN_FLAG_DX_MASKED
            lay = self._layer(i, ld_x, extra)
            # the upstream gradient must share Y's row stride
            if self.n and d.stride(0) != L["Y"].stride(0):
                d = padded(d.contiguous(), L["Y"].stride(0))
            dx = L["dX"] if (i > 0 or want_dx_first) else None
            G.gnn_prop_bwd(csr, lay, x, L["W_self"], L["W_neigh"], L["Y"], d,
                           L["saved"], dx, L["dW_self"], L["dW_neigh"],
                           L["db_self"], L["db_neigh"], self.workspace, stream)
            d = dx
        return self.layers[0]["dX"] if want_dx_first else None


class Trainer:
    """One training iteration of Algorithm 1 on a prepared subgraph: the
    stack's forward pass, the classifier and loss (Section 3.1), the backward
    pass from the classifier's input gradient down (Section 5.1), then SGD or
    Adam on every weight.  All arithmetic runs in libgnnprop; the loss stays
    on the device (read it with `loss.item()` when needed)."""

    def __init__(self, graph: DeviceGraph, params: Sequence, f_in: int, w_mlp,
                 multilabel: bool, optimizer: str = "adam", lr: float = 0.01,
                 betas=(0.9, 0.999), eps: float = 1e-8, order: int = 0,
                 flags: int = 0, pad: int = 16, fuse_masks: bool = False,
                 want_probs: bool = False, keep_xm: bool = False,
                 device: str = "cuda"):
        """want_probs / keep_xm: keep the class probabilities Y / the MLP
        output X_MLP = ReLU(X^(L) W_MLP) of the last iteration in `probs` /
        `xm` (n x C views)."""
        if optimizer not in ("sgd", "adam"):
            raise ValueError("optimizer must be 'sgd' or 'adam'")
        self.stack = SageStack(graph, params, f_in, order, flags, pad, fuse_masks, device)
        self.n = graph.n
        self.kind = G.GNN_LOSS_SIGMOID if multilabel else G.GNN_LOSS_SOFTMAX
        self.flags = flags & G.GNN_FLAG_BF16
        self.optimizer, self.lr, self.betas, self.eps = optimizer, lr, betas, eps
        top = self.stack.layers[-1]
        self.f_top = 2 * top["h"]
        self.C = int(w_mlp.shape[1])
        assert w_mlp.shape == (self.f_top, self.C)
        self.W_mlp = torch.from_numpy(np.ascontiguousarray(w_mlp, np.float32)).to(device)
        self.dW_mlp = torch.empty_like(self.W_mlp)
        # the classifier writes dX^(L) at the top layer's Y stride, which is
        # the stride the stack's backward pass expects
        self.dX_top = torch.empty((max(self.n, 1), top["Y"].stride(0)),
                                  device=device)[: self.n, : self.f_top]
        ld_p = _round_up(self.C, 4)
        self.probs = torch.empty((max(self.n, 1), ld_p), device=device)[: self.n, : self.C] \
            if want_probs else None
        self.xm = torch.empty((max(self.n, 1), ld_p), device=device)[: self.n, : self.C] \
            if keep_xm else None
        self.loss = torch.zeros(1, device=device)
        self.cls_ws = torch.empty(max(G.gnn_classifier_workspace_bytes(self.n, self.f_top,
                                                                      self.C), 256),
                                  dtype=torch.uint8, device=device)
        # (weight, gradient) pairs in a fixed order: W_MLP, then per layer
        # W_self, W_neigh (, b_self, b_neigh)
        self.pairs = [(self.W_mlp, self.dW_mlp)]
        for L in self.stack.layers:
            self.pairs += [(L["W_self"], L["dW_self"]), (L["W_neigh"], L["dW_neigh"])]
            if L["b_self"] is not None:
                self.pairs += [(L["b_self"], L["db_self"]), (L["b_neigh"], L["db_neigh"])]
        self.state = [(torch.zeros_like(w), torch.zeros_like(w)) for w, _ in self.pairs] \
            if optimizer == "adam" else None
        self.t = 0

    def step(self, X: torch.Tensor, targets: torch.Tensor, stream=None) -> torch.Tensor:
        """X: n x f_in (any row stride); targets: n x C 0/1 floats."""
        top = self.stack.forward(X, stream)
        ld_top = top.stride(0) if self.n else self.f_top
        ld_t = targets.stride(0) if self.n else self.C
        G.gnn_classifier(self.n, self.f_top, self.C, self.kind, self.flags, top, ld_top,
                         self.W_mlp, targets, ld_t, self.xm,
                         self.xm.stride(0) if self.xm is not None else self.C, self.probs,
                         self.probs.stride(0) if self.probs is not None else self.C,
                         self.loss, self.dW_mlp, self.dX_top,
                         self.dX_top.stride(0) if self.n else self.f_top, self.cls_ws,
                         stream)
        self.stack.backward(self.dX_top, want_dx_first=False, stream=stream)
        self.t += 1
        for i, (w, gr) in enumerate(self.pairs):
            if self.optimizer == "sgd":
                G.gnn_sgd_step(w.numel(), w, gr, self.lr, stream)
            else:
                m, v = self.state[i]
                G.gnn_adam_step(w.numel(), w, gr, m, v, self.lr, self.betas[0],
                                self.betas[1], self.eps, self.t, stream)
        return self.loss
