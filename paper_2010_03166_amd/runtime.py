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
