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


class _Rows:
    """A (rows, ld) float32 device buffer that grows on demand; view(n) is
    the first n rows, `cols` wide, at row stride ld."""

    def __init__(self, cols: int, ld: int, device):
        self.cols, self.ld, self.device = cols, ld, device
        self.buf = torch.empty((1, ld), device=device)

    def view(self, n: int) -> torch.Tensor:
        if n > self.buf.shape[0]:
            self.buf = torch.empty((n, self.ld), device=self.device)
        return self.buf[:n, : self.cols]


def _grown(buf: Optional[torch.Tensor], nbytes: int, device) -> torch.Tensor:
    """buf if it holds nbytes, else a new byte buffer of that size (>= 256)."""
    if buf is not None and buf.numel() >= nbytes:
        return buf
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


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
                  values: torch.Tensor, nnz: Optional[int] = None,
                  values_t: Optional[torch.Tensor] = None,
                  plan: Optional[torch.Tensor] = None) -> "DeviceGraph":
        """Wraps a CSR already in device memory (int32 indptr of n + 1,
        int32 indices and float32 values holding at least nnz entries);
        values_t / plan buffers are allocated unless given (large enough)."""
        g = cls.__new__(cls)
        g.n = int(n)
        g.nnz = int(indices.numel()) if nnz is None else int(nnz)
        g.device = indptr.device
        g.indptr, g.indices, g.values = indptr, indices, values
        g.values_t = values_t if values_t is not None else \
            torch.empty(max(g.nnz, 1), dtype=torch.float32, device=g.device)
        need = G.gnn_plan_bytes(g.n, g.nnz)
        g.plan = plan if plan is not None and plan.numel() >= need else \
            torch.empty(max(need, 256), dtype=torch.uint8, device=g.device)
        return g

    def struct(self) -> G.gnn_csr:
        return G.make_csr(self.n, self.nnz, self.indptr, self.indices, self.values,
                          self.values_t, self.plan)

    def prepare(self, stream=None):
        """Per-subgraph preparation: the work plan and (A_s)^T values, one
        launch."""
        G.gnn_csr_prepare(self.struct(), self.plan, self.values_t, stream)

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


class _Slot:
    """Buffers of one subgraph in flight through the pipeline."""

    def __init__(self, max_nodes: int, cap: int, f: int, C: int, pad: int, device):
        self.host_nodes = torch.empty(max_nodes, dtype=torch.int32).pin_memory()
        self.host_meta = torch.zeros(2, dtype=torch.int64).pin_memory()
        self.nodes = torch.empty(max(max_nodes, 1), dtype=torch.int32, device=device)
        self.indptr = torch.empty(max_nodes + 1, dtype=torch.int32, device=device)
        self.indices = torch.empty(max(cap, 1), dtype=torch.int32, device=device)
        self.values = torch.empty(max(cap, 1), dtype=torch.float32, device=device)
        self.values_t = torch.empty(max(cap, 1), dtype=torch.float32, device=device)
        self.plan = torch.empty(max(G.gnn_plan_bytes(max_nodes, cap), 256),
                                dtype=torch.uint8, device=device)
        self.meta = torch.zeros(2, dtype=torch.int64, device=device)  # nnz, status
        self.ws = torch.empty(max(G.gnn_induce_workspace_bytes(max_nodes), 256),
                              dtype=torch.uint8, device=device)
        self.X = torch.empty((max(max_nodes, 1), _round_up(f, pad)), device=device)
        self.T = torch.empty((max(max_nodes, 1), max(C, 1)), device=device)
        self.induced = torch.cuda.Event()
        self.consumed = torch.cuda.Event()
        self.n = 0
        self.sid = -1


class SubgraphPipeline:
    """Algorithm 8 on one GPU.  A pool of host sampler threads keeps node
    lists ready (gnn_sampler_pool); each subgraph is induced and its rows
    gathered on a preparation stream while the previous subgraph trains on
    the caller's stream, with `depth` sets of buffers in rotation.

        sub = pipe.next()       # (DeviceGraph prepared, X_s, T_s, id)
        ...launch the iteration on sub...
        pipe.release()          # after launching: frees the slot for reuse
                                # and starts preparing the following subgraph
    """

    def __init__(self, full_dev: FullGraphDevice, pool, max_nodes: int, depth: int = 2,
                 pad: int = 16):
        assert depth >= 2
        self.full, self.pool = full_dev, pool
        self.max_nodes = int(max_nodes)
        deg = np.sort(full_dev.deg)[::-1]
        cap = int(deg[: self.max_nodes].sum()) + self.max_nodes  # any max_nodes nodes fit
        f = full_dev.X.shape[1] if full_dev.X is not None else 1
        C = full_dev.labels.shape[1] if full_dev.labels is not None else 1
        dev = full_dev.device
        self.cap = cap
        self.slots = [_Slot(self.max_nodes, cap, f, C, pad, dev) for _ in range(depth)]
        self.prep = torch.cuda.Stream(device=dev)
        self.k = 0
        self._issue(self.slots[0])

    def _issue(self, s: _Slot):
        sid, nodes = self.pool.next()
        n = len(nodes)
        if n > self.max_nodes:
            raise ValueError("subgraph of %d nodes exceeds max_nodes %d" % (n, self.max_nodes))
        s.n, s.sid = n, sid
        s.host_nodes[:n].copy_(torch.from_numpy(nodes))
        full = self.full
        with torch.cuda.stream(self.prep):
            self.prep.wait_event(s.consumed)  # the iteration that last used s is done
            s.nodes[:n].copy_(s.host_nodes[:n], non_blocking=True)
            G.gnn_induce_subgraph(full.n, full.nnz, full.indptr, full.indices, n, s.nodes,
                                  full.norm, full.map, self.cap, s.indptr, s.indices,
                                  s.values, s.meta[0:1], s.meta[1:2].view(torch.int32), s.ws,
                                  self.prep.cuda_stream)
            if full.X is not None:
                G.gnn_gather_rows(n, s.nodes, full.X.shape[1], full.X, full.X.stride(0),
                                  full.n, s.X, s.X.stride(0), self.prep.cuda_stream)
            if full.labels is not None:
                G.gnn_gather_rows(n, s.nodes, full.labels.shape[1], full.labels,
                                  full.labels.stride(0), full.n, s.T, s.T.stride(0),
                                  self.prep.cuda_stream)
            s.host_meta.copy_(s.meta, non_blocking=True)
            s.induced.record(self.prep)

    def next(self):
        s = self.slots[self.k % len(self.slots)]
        s.induced.synchronize()
        nnz, status = int(s.host_meta[0]), int(s.host_meta[1])
        if status:
            raise ValueError("gnn_induce_subgraph status %d" % status)
        cur = torch.cuda.current_stream()
        cur.wait_event(s.induced)
        dg = DeviceGraph.on_device(s.n, s.indptr[: s.n + 1], s.indices, s.values, nnz=nnz,
                                   values_t=s.values_t, plan=s.plan)
        dg.prepare(cur.cuda_stream)
        f = self.full.X.shape[1] if self.full.X is not None else 0
        C = self.full.labels.shape[1] if self.full.labels is not None else 0
        return dg, s.X[: s.n, :f], s.T[: s.n, :C], s.sid

    def release(self):
        s = self.slots[self.k % len(self.slots)]
        s.consumed.record(torch.cuda.current_stream())
        self.k += 1
        self._issue(self.slots[self.k % len(self.slots)])


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
        self.order, self.flags, self.pad = order, flags, pad
        self.fuse_masks = fuse_masks
        self.device = device
        self.layers = []
        f = f_in
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
            L["dW_self"] = torch.empty((f, h), device=device)
            L["dW_neigh"] = torch.empty((f, h), device=device)
            L["db_self"] = torch.empty(h, device=device) if p.b_self is not None else None
            L["db_neigh"] = torch.empty(h, device=device) if p.b_neigh is not None else None
            L["_Y"] = _Rows(2 * h, _round_up(2 * h, pad), device)
            L["_dX"] = _Rows(f, _round_up(f, pad), device)
            L["saved"] = None
            self.layers.append(L)
            f = 2 * h
        self.f_in = f_in
        self.workspace = None
        self.inputs: List[Optional[torch.Tensor]] = [None] * len(self.layers)
        self.bind(graph)

    def bind(self, graph: DeviceGraph):
        """Moves the stack to another (prepared) subgraph: activation and
        gradient views of its size, saved state and workspace grown as
        needed.  Weights and their gradients are kept."""
        self.g = graph
        self.n = graph.n
        ws_bytes = 0
        for i, L in enumerate(self.layers):
            L["Y"] = L["_Y"].view(self.n)
            L["dX"] = L["_dX"].view(self.n)
            lay = self._layer(i, _round_up(L["f_in"], self.pad))
            L["saved"] = _grown(L["saved"], G.gnn_prop_saved_bytes(graph.struct(), lay),
                                self.device)
            ws_bytes = max(ws_bytes, G.gnn_prop_workspace_bytes(graph.struct(), lay))
        self.workspace = _grown(self.workspace, ws_bytes, self.device)
        self.inputs = [None] * len(self.layers)

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
        self.kind = G.GNN_LOSS_SIGMOID if multilabel else G.GNN_LOSS_SOFTMAX
        self.flags = flags & (G.GNN_FLAG_BF16 | G.GNN_FLAG_F32_MFMA)
        self.optimizer, self.lr, self.betas, self.eps = optimizer, lr, betas, eps
        self.device = device
        top = self.stack.layers[-1]
        self.f_top = 2 * top["h"]
        self.C = int(w_mlp.shape[1])
        assert w_mlp.shape == (self.f_top, self.C)
        self.W_mlp = torch.from_numpy(np.ascontiguousarray(w_mlp, np.float32)).to(device)
        self.dW_mlp = torch.empty_like(self.W_mlp)
        # the classifier writes dX^(L) at the top layer's Y stride, which is
        # the stride the stack's backward pass expects
        self._dX_top = _Rows(self.f_top, top["_Y"].ld, device)
        ld_p = _round_up(self.C, 4)
        self._probs = _Rows(self.C, ld_p, device) if want_probs else None
        self._xm = _Rows(self.C, ld_p, device) if keep_xm else None
        self.loss = torch.zeros(1, device=device)
        self.cls_ws = None
        self.bind(graph, rebind_stack=False)
        # Every weight, gradient and optimizer moment lives in one flat
        # buffer (tensors at 256-byte offsets, zero padding between them), so
        # that one update launch covers the whole model.  (weight, gradient)
        # pairs in a fixed order: W_MLP, then per layer W_self, W_neigh
        # (, b_self, b_neigh).
        names = [(None, "W_mlp", "dW_mlp")]
        for L in self.stack.layers:
            names += [(L, "W_self", "dW_self"), (L, "W_neigh", "dW_neigh")]
            if L["b_self"] is not None:
                names += [(L, "b_self", "db_self"), (L, "b_neigh", "db_neigh")]
        get = lambda L, k: getattr(self, k) if L is None else L[k]
        offs, total = [], 0
        for L, wk, _ in names:
            offs.append(total)
            total += _round_up(get(L, wk).numel(), 64)
        self.flat_w = torch.zeros(max(total, 64), device=device)
        self.flat_g = torch.zeros(max(total, 64), device=device)
        self.pairs = []
        for (L, wk, gk), o in zip(names, offs):
            w = get(L, wk)
            wv = self.flat_w[o: o + w.numel()].view(w.shape)
            wv.copy_(w)
            gv = self.flat_g[o: o + w.numel()].view(w.shape)
            if L is None:
                setattr(self, wk, wv)
                setattr(self, gk, gv)
            else:
                L[wk], L[gk] = wv, gv
            self.pairs.append((wv, gv))
        self.state = None
        if optimizer == "adam":
            self.flat_m = torch.zeros_like(self.flat_w)
            self.flat_v = torch.zeros_like(self.flat_w)
            self.state = [(self.flat_m[o: o + w.numel()].view(w.shape),
                           self.flat_v[o: o + w.numel()].view(w.shape))
                          for (w, _), o in zip(self.pairs, offs)]
        self.t = 0

    def bind(self, graph: DeviceGraph, rebind_stack: bool = True):
        """Moves the iteration to another prepared subgraph (weights and
        optimizer state are kept)."""
        if rebind_stack:
            self.stack.bind(graph)
        self.n = graph.n
        self.dX_top = self._dX_top.view(self.n)
        self.probs = self._probs.view(self.n) if self._probs is not None else None
        self.xm = self._xm.view(self.n) if self._xm is not None else None
        self.cls_ws = _grown(self.cls_ws, G.gnn_classifier_workspace_bytes(
            self.n, self.f_top, self.C), self.device)

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
        if self.optimizer == "sgd":
            G.gnn_sgd_step(self.flat_w.numel(), self.flat_w, self.flat_g, self.lr, stream)
        else:
            G.gnn_adam_step(self.flat_w.numel(), self.flat_w, self.flat_g, self.flat_m,
                            self.flat_v, self.lr, self.betas[0], self.betas[1], self.eps,
                            self.t, stream)
        return self.loss
