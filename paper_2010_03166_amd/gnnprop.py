"""Python binding of libgnnprop (ctypes).

Argument marshalling only: every function here has the name of the C entry
point it calls, takes torch tensors on the current HIP device (or plain
integers), passes their data pointers and the current stream, and raises
GnnError when the library returns an error status.  All computation happens
in the HIP kernels of libgnnprop.so; if that library is missing this module
raises instead of computing anything itself.
"""
from __future__ import annotations

import ctypes

import numpy as np
import os
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libgnnprop.so")

GNN_OK = 0
GNN_FLAG_BF16 = 0x1
GNN_FLAG_DY_MASKED = 0x2
GNN_FLAG_DX_MASKED = 0x4
GNN_FLAG_F32_MFMA = 0x8
GNN_FLAG_ROW_NORMALIZED = 0x10
GNN_LOSS_SOFTMAX = 0
GNN_LOSS_SIGMOID = 1
KERNELS = {"spmm": 0, "spmm_reduce": 1, "gemm_nn": 2, "gemm_tn": 3,
           "gemm_nt": 4, "gemm_tt": 5, "gemm_reduce": 6, "mask": 7,
           "colsum": 8, "plan": 9, "transpose": 10, "loss": 11, "update": 12,
           "induce": 13, "gather": 14, "sddmm": 15, "wsplit": 16}
GNN_NORM_ROW = 0
GNN_NORM_SYM = 1
GNN_PROBE_MFMA_BF16 = 0
GNN_PROBE_MFMA_F32 = 1
GNN_PROBE_MAX_BLOCKS = 65536
GNN_PROBE_MAX_ITERS = 100000

_lib = None


class GnnError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (where, status_string(status), status))


class gnn_csr(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("nnz", ctypes.c_int64),
                ("indptr", ctypes.c_void_p), ("indices", ctypes.c_void_p),
                ("values", ctypes.c_void_p), ("values_t", ctypes.c_void_p),
                ("plan", ctypes.c_void_p)]


class gnn_layer(ctypes.Structure):
    _fields_ = [("f_in", ctypes.c_int32), ("h", ctypes.c_int32),
                ("ld_x", ctypes.c_int64), ("ld_y", ctypes.c_int64),
                ("ld_dx", ctypes.c_int64), ("order", ctypes.c_int32),
                ("flags", ctypes.c_uint32)]


EXPORTS = {
    # name: (restype, argtypes)
    "gnn_status_string": (ctypes.c_char_p, [ctypes.c_int32]),
    "gnn_choose_order": (ctypes.c_int32, [ctypes.c_int32, ctypes.c_int32]),
    "gnn_plan_bytes": (ctypes.c_size_t, [ctypes.c_int32, ctypes.c_int64]),
    "gnn_csr_transpose_values": (ctypes.c_int32, [ctypes.POINTER(gnn_csr),
                                                  ctypes.c_void_p, ctypes.c_void_p]),
    "gnn_csr_build_plan": (ctypes.c_int32, [ctypes.POINTER(gnn_csr), ctypes.c_void_p,
                                            ctypes.c_size_t, ctypes.c_void_p]),
    "gnn_csr_prepare": (ctypes.c_int32, [ctypes.POINTER(gnn_csr), ctypes.c_void_p,
                                         ctypes.c_size_t, ctypes.c_void_p,
                                         ctypes.c_void_p]),
    "gnn_csr_validate": (ctypes.c_int32, [ctypes.POINTER(gnn_csr), ctypes.c_int32,
                                          ctypes.c_void_p]),
    "gnn_csr_validate_noalloc": (ctypes.c_int32, [ctypes.POINTER(gnn_csr),
                                                  ctypes.c_int32, ctypes.c_void_p]),
    "gnn_prop_saved_bytes": (ctypes.c_size_t, [ctypes.POINTER(gnn_csr),
                                               ctypes.POINTER(gnn_layer)]),
    "gnn_prop_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(gnn_csr),
                                                   ctypes.POINTER(gnn_layer)]),
    "gnn_prop_fwd": (ctypes.c_int32, [ctypes.POINTER(gnn_csr), ctypes.POINTER(gnn_layer)]
                     + [ctypes.c_void_p] * 8 + [ctypes.c_size_t, ctypes.c_void_p]),
    "gnn_prop_bwd": (ctypes.c_int32, [ctypes.POINTER(gnn_csr), ctypes.POINTER(gnn_layer)]
                     + [ctypes.c_void_p] * 12 + [ctypes.c_size_t, ctypes.c_void_p]),
    "gnn_spmm_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(gnn_csr),
                                                   ctypes.c_int32]),
    "gnn_spmm": (ctypes.c_int32, [ctypes.POINTER(gnn_csr), ctypes.c_int32, ctypes.c_int32,
                                  ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                  ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t,
                                  ctypes.c_void_p]),
    "gnn_spmm_gather_floor": (ctypes.c_int32, [ctypes.POINTER(gnn_csr), ctypes.c_int32,
                                               ctypes.c_int32, ctypes.c_void_p,
                                               ctypes.c_int64, ctypes.c_void_p,
                                               ctypes.c_int64, ctypes.c_void_p]),
    "gnn_gemm_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int32] * 3),
    "gnn_mfma_rate_probe": (ctypes.c_int32, [ctypes.c_int32] * 3 + [ctypes.c_void_p] * 3),
    "gnn_gemm": (ctypes.c_int32, [ctypes.c_int32] * 5 + [
        ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
        ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint32, ctypes.c_void_p,
        ctypes.c_size_t, ctypes.c_void_p]),
    "gnn_gcn_saved_bytes": (ctypes.c_size_t, [ctypes.POINTER(gnn_csr),
                                              ctypes.POINTER(gnn_layer)]),
    "gnn_gcn_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(gnn_csr),
                                                  ctypes.POINTER(gnn_layer)]),
    "gnn_gcn_fwd": (ctypes.c_int32, [ctypes.POINTER(gnn_csr), ctypes.POINTER(gnn_layer)]
                    + [ctypes.c_void_p] * 6 + [ctypes.c_size_t, ctypes.c_void_p]),
    "gnn_gcn_bwd": (ctypes.c_int32, [ctypes.POINTER(gnn_csr), ctypes.POINTER(gnn_layer)]
                    + [ctypes.c_void_p] * 9 + [ctypes.c_size_t, ctypes.c_void_p]),
    "gnn_mixhop_saved_bytes": (ctypes.c_size_t, [ctypes.POINTER(gnn_csr),
                                                 ctypes.POINTER(gnn_layer), ctypes.c_int32]),
    "gnn_mixhop_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(gnn_csr),
                                                     ctypes.POINTER(gnn_layer),
                                                     ctypes.c_int32]),
    "gnn_mixhop_fwd": (ctypes.c_int32, [ctypes.POINTER(gnn_csr), ctypes.POINTER(gnn_layer),
                                        ctypes.c_int32] + [ctypes.c_void_p] * 6
                       + [ctypes.c_size_t, ctypes.c_void_p]),
    "gnn_mixhop_bwd": (ctypes.c_int32, [ctypes.POINTER(gnn_csr), ctypes.POINTER(gnn_layer),
                                        ctypes.c_int32] + [ctypes.c_void_p] * 9
                       + [ctypes.c_size_t, ctypes.c_void_p]),
    "gnn_classifier_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int32] * 3),
    "gnn_classifier": (ctypes.c_int32, [ctypes.c_int32] * 4 + [ctypes.c_uint32,
                       ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                       ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                       ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                       ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "gnn_sgd_step": (ctypes.c_int32, [ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_double, ctypes.c_void_p]),
    "gnn_adam_step": (ctypes.c_int32, [ctypes.c_int64] + [ctypes.c_void_p] * 4
                      + [ctypes.c_double] * 4 + [ctypes.c_int32, ctypes.c_void_p]),
    "gnn_induce_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int32]),
    "gnn_induce_subgraph": (ctypes.c_int32, [ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                            ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                            ctypes.c_void_p, ctypes.c_int64] + [ctypes.c_void_p] * 6
                           + [ctypes.c_size_t, ctypes.c_void_p]),
    "gnn_gather_rows": (ctypes.c_int32, [ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                         ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                         ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]),
    "gnn_frontier_sample": (ctypes.c_int32, [ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                             ctypes.c_int32, ctypes.c_int32, ctypes.c_double,
                                             ctypes.c_int32, ctypes.c_uint64, ctypes.c_int64,
                                             ctypes.c_void_p, ctypes.c_void_p]),
    "gnn_sampler_create": (ctypes.c_int32, [ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_int32, ctypes.c_int32, ctypes.c_double,
                                            ctypes.c_int32, ctypes.c_uint64, ctypes.c_int32,
                                            ctypes.c_int32, ctypes.c_void_p]),
    "gnn_sampler_next": (ctypes.c_int32, [ctypes.c_void_p] * 4),
    "gnn_sampler_destroy": (None, [ctypes.c_void_p]),
    "gnn_gat_saved_bytes": (ctypes.c_size_t, [ctypes.POINTER(gnn_csr),
                                              ctypes.POINTER(gnn_layer)]),
    "gnn_gat_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(gnn_csr),
                                                  ctypes.POINTER(gnn_layer)]),
    "gnn_gat_fwd": (ctypes.c_int32, [ctypes.POINTER(gnn_csr), ctypes.POINTER(gnn_layer)]
                    + [ctypes.c_void_p] * 3 + [ctypes.c_float]
                    + [ctypes.c_void_p] * 4 + [ctypes.c_size_t, ctypes.c_void_p]),
    "gnn_gat_bwd": (ctypes.c_int32, [ctypes.POINTER(gnn_csr), ctypes.POINTER(gnn_layer)]
                    + [ctypes.c_void_p] * 3 + [ctypes.c_float]
                    + [ctypes.c_void_p] * 7 + [ctypes.c_size_t, ctypes.c_void_p]),
    "gnn_timer_enable": (ctypes.c_int32, [ctypes.c_int32]),
    "gnn_timer_reset": (ctypes.c_int32, []),
    "gnn_timer_read": (ctypes.c_int32, [ctypes.c_int32, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_int64),
                                        ctypes.POINTER(ctypes.c_double)]),
}


def lib():
    """The loaded libgnnprop.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                "libgnnprop.so is not built (expected at %s); run "
                "`python -c 'import __graft_entry__ as g; g.build()'`" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in EXPORTS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def status_string(s: int) -> str:
    return lib().gnn_status_string(int(s)).decode()


def _check(st: int, where: str):
    if st != GNN_OK:
        raise GnnError(st, where)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _ld(t) -> int:
    return int(t.stride(0)) if t.dim() == 2 else int(t.shape[-1])


# ------------------------------------------------------------ structures

def make_csr(n: int, nnz: int, indptr, indices, values, values_t=None,
             plan=None) -> gnn_csr:
    return gnn_csr(int(n), int(nnz), _ptr(indptr), _ptr(indices), _ptr(values),
                   _ptr(values_t), _ptr(plan))


def make_layer(f_in: int, h: int, ld_x: int, ld_y: int, ld_dx: int = 0,
               order: int = 0, flags: int = 0) -> gnn_layer:
    return gnn_layer(int(f_in), int(h), int(ld_x), int(ld_y),
                     int(ld_dx or ld_x), int(order), int(flags))


# ------------------------------------------------------------ entry points

def gnn_choose_order(f_in: int, h: int) -> int:
    return int(lib().gnn_choose_order(int(f_in), int(h)))


def gnn_plan_bytes(n: int, nnz: int) -> int:
    return int(lib().gnn_plan_bytes(int(n), int(nnz)))


def gnn_csr_transpose_values(csr: gnn_csr, values_t, stream=None):
    _check(lib().gnn_csr_transpose_values(ctypes.byref(csr), _ptr(values_t),
                                          _stream(stream)),
           "gnn_csr_transpose_values")


def gnn_csr_build_plan(csr: gnn_csr, plan, stream=None):
    nbytes = plan.numel() * plan.element_size()
    _check(lib().gnn_csr_build_plan(ctypes.byref(csr), _ptr(plan), nbytes,
                                    _stream(stream)), "gnn_csr_build_plan")


def gnn_csr_prepare(csr: gnn_csr, plan, values_t, stream=None):
    nbytes = plan.numel() * plan.element_size()
    _check(lib().gnn_csr_prepare(ctypes.byref(csr), _ptr(plan), nbytes, _ptr(values_t),
                                 _stream(stream)), "gnn_csr_prepare")


def gnn_csr_validate(csr: gnn_csr, require_symmetric: bool = True,
                     stream=None) -> int:
    """Returns the status (GNN_OK or an error code) without raising."""
    return int(lib().gnn_csr_validate(ctypes.byref(csr), int(require_symmetric),
                                      _stream(stream)))


def gnn_csr_validate_noalloc(csr: Optional[gnn_csr], require_symmetric: bool = True,
                             stream=None) -> int:
    """gnn_csr_validate without device allocation; returns the status."""
    return int(lib().gnn_csr_validate_noalloc(
        ctypes.byref(csr) if csr is not None else None, int(require_symmetric),
        _stream(stream)))


def gnn_prop_saved_bytes(csr: gnn_csr, layer: gnn_layer) -> int:
    return int(lib().gnn_prop_saved_bytes(ctypes.byref(csr), ctypes.byref(layer)))


def gnn_prop_workspace_bytes(csr: gnn_csr, layer: gnn_layer) -> int:
    return int(lib().gnn_prop_workspace_bytes(ctypes.byref(csr), ctypes.byref(layer)))


def _nbytes(t) -> int:
    return 0 if t is None else t.numel() * t.element_size()


def gnn_prop_fwd(csr: gnn_csr, layer: gnn_layer, X, W_self, W_neigh, b_self,
                 b_neigh, Y, saved, workspace, stream=None):
    _check(lib().gnn_prop_fwd(ctypes.byref(csr), ctypes.byref(layer), _ptr(X),
                              _ptr(W_self), _ptr(W_neigh), _ptr(b_self),
                              _ptr(b_neigh), _ptr(Y), _ptr(saved),
                              _ptr(workspace), _nbytes(workspace),
                              _stream(stream)), "gnn_prop_fwd")


def gnn_prop_bwd(csr: gnn_csr, layer: gnn_layer, X, W_self, W_neigh, Y, dY,
                 saved, dX, dW_self, dW_neigh, db_self, db_neigh, workspace,
                 stream=None):
    _check(lib().gnn_prop_bwd(ctypes.byref(csr), ctypes.byref(layer), _ptr(X),
                              _ptr(W_self), _ptr(W_neigh), _ptr(Y), _ptr(dY),
                              _ptr(saved), _ptr(dX), _ptr(dW_self),
                              _ptr(dW_neigh), _ptr(db_self), _ptr(db_neigh),
                              _ptr(workspace), _nbytes(workspace),
                              _stream(stream)), "gnn_prop_bwd")


def gnn_gcn_saved_bytes(csr: gnn_csr, layer: gnn_layer) -> int:
    return int(lib().gnn_gcn_saved_bytes(ctypes.byref(csr), ctypes.byref(layer)))


def gnn_gcn_workspace_bytes(csr: gnn_csr, layer: gnn_layer) -> int:
    return int(lib().gnn_gcn_workspace_bytes(ctypes.byref(csr), ctypes.byref(layer)))


def gnn_gcn_fwd(csr: gnn_csr, layer: gnn_layer, X, W, b, Y, saved, workspace,
                stream=None):
    _check(lib().gnn_gcn_fwd(ctypes.byref(csr), ctypes.byref(layer), _ptr(X), _ptr(W),
                             _ptr(b), _ptr(Y), _ptr(saved), _ptr(workspace),
                             _nbytes(workspace), _stream(stream)), "gnn_gcn_fwd")


def gnn_gcn_bwd(csr: gnn_csr, layer: gnn_layer, X, W, Y, dY, saved, dX, dW, db,
                workspace, stream=None):
    _check(lib().gnn_gcn_bwd(ctypes.byref(csr), ctypes.byref(layer), _ptr(X), _ptr(W),
                             _ptr(Y), _ptr(dY), _ptr(saved), _ptr(dX), _ptr(dW),
                             _ptr(db), _ptr(workspace), _nbytes(workspace),
                             _stream(stream)), "gnn_gcn_bwd")


def gnn_mixhop_saved_bytes(csr: gnn_csr, layer: gnn_layer, K: int) -> int:
    return int(lib().gnn_mixhop_saved_bytes(ctypes.byref(csr), ctypes.byref(layer), int(K)))


def gnn_mixhop_workspace_bytes(csr: gnn_csr, layer: gnn_layer, K: int) -> int:
    return int(lib().gnn_mixhop_workspace_bytes(ctypes.byref(csr), ctypes.byref(layer),
                                                int(K)))


def gnn_mixhop_fwd(csr: gnn_csr, layer: gnn_layer, K: int, X, W, b, Y, saved,
                   workspace, stream=None):
    _check(lib().gnn_mixhop_fwd(ctypes.byref(csr), ctypes.byref(layer), int(K), _ptr(X),
                                _ptr(W), _ptr(b), _ptr(Y), _ptr(saved), _ptr(workspace),
                                _nbytes(workspace), _stream(stream)), "gnn_mixhop_fwd")


def gnn_mixhop_bwd(csr: gnn_csr, layer: gnn_layer, K: int, X, W, Y, dY, saved, dX, dW,
                   db, workspace, stream=None):
    _check(lib().gnn_mixhop_bwd(ctypes.byref(csr), ctypes.byref(layer), int(K), _ptr(X),
                                _ptr(W), _ptr(Y), _ptr(dY), _ptr(saved), _ptr(dX),
                                _ptr(dW), _ptr(db), _ptr(workspace), _nbytes(workspace),
                                _stream(stream)), "gnn_mixhop_bwd")


def gnn_gat_saved_bytes(csr: gnn_csr, layer: gnn_layer) -> int:
    return int(lib().gnn_gat_saved_bytes(ctypes.byref(csr), ctypes.byref(layer)))


def gnn_gat_workspace_bytes(csr: gnn_csr, layer: gnn_layer) -> int:
    return int(lib().gnn_gat_workspace_bytes(ctypes.byref(csr), ctypes.byref(layer)))


def gnn_gat_fwd(csr: gnn_csr, layer: gnn_layer, X, W, a, alpha: float, Y, att_out, saved,
                workspace, stream=None):
    _check(lib().gnn_gat_fwd(ctypes.byref(csr), ctypes.byref(layer), _ptr(X), _ptr(W),
                             _ptr(a), float(alpha), _ptr(Y), _ptr(att_out), _ptr(saved),
                             _ptr(workspace), _nbytes(workspace), _stream(stream)),
           "gnn_gat_fwd")


def gnn_gat_bwd(csr: gnn_csr, layer: gnn_layer, X, W, a, alpha: float, Y, dY, saved, dX,
                dW, da, workspace, stream=None):
    _check(lib().gnn_gat_bwd(ctypes.byref(csr), ctypes.byref(layer), _ptr(X), _ptr(W),
                             _ptr(a), float(alpha), _ptr(Y), _ptr(dY), _ptr(saved),
                             _ptr(dX), _ptr(dW), _ptr(da), _ptr(workspace),
                             _nbytes(workspace), _stream(stream)), "gnn_gat_bwd")


def gnn_classifier_workspace_bytes(n: int, f: int, C: int) -> int:
    return int(lib().gnn_classifier_workspace_bytes(int(n), int(f), int(C)))


def gnn_classifier(n: int, f: int, C: int, kind: int, flags: int, X, ld_x: int, W, T,
                   ld_t: int, xm, ld_xm: int, probs, ld_p: int, loss, dW, dX, ld_dx: int,
                   workspace, stream=None):
    _check(lib().gnn_classifier(int(n), int(f), int(C), int(kind), int(flags), _ptr(X),
                                int(ld_x), _ptr(W), _ptr(T), int(ld_t), _ptr(xm),
                                int(ld_xm), _ptr(probs), int(ld_p), _ptr(loss), _ptr(dW),
                                _ptr(dX), int(ld_dx), _ptr(workspace), _nbytes(workspace),
                                _stream(stream)), "gnn_classifier")


def gnn_sgd_step(count: int, W, G_, lr: float, stream=None):
    _check(lib().gnn_sgd_step(int(count), _ptr(W), _ptr(G_), float(lr), _stream(stream)),
           "gnn_sgd_step")


def gnn_adam_step(count: int, W, G_, m, v, lr: float, beta1: float, beta2: float,
                  eps: float, t: int, stream=None):
    _check(lib().gnn_adam_step(int(count), _ptr(W), _ptr(G_), _ptr(m), _ptr(v), float(lr),
                               float(beta1), float(beta2), float(eps), int(t),
                               _stream(stream)), "gnn_adam_step")


def gnn_induce_workspace_bytes(n_s: int) -> int:
    return int(lib().gnn_induce_workspace_bytes(int(n_s)))


def gnn_induce_subgraph(n_full: int, nnz_full: int, indptr, indices, n_s: int, nodes,
                        norm: int, map_, capacity: int, sub_indptr, sub_indices, sub_values,
                        nnz_out, status_out, workspace, stream=None):
    _check(lib().gnn_induce_subgraph(int(n_full), int(nnz_full), _ptr(indptr), _ptr(indices),
                                     int(n_s), _ptr(nodes), int(norm), _ptr(map_),
                                     int(capacity), _ptr(sub_indptr), _ptr(sub_indices),
                                     _ptr(sub_values), _ptr(nnz_out), _ptr(status_out),
                                     _ptr(workspace), _nbytes(workspace), _stream(stream)),
           "gnn_induce_subgraph")


def gnn_gather_rows(rows: int, index, width: int, src, ld_src: int, src_rows: int, dst,
                    ld_dst: int, stream=None):
    _check(lib().gnn_gather_rows(int(rows), _ptr(index), int(width), _ptr(src), int(ld_src),
                                 int(src_rows), _ptr(dst), int(ld_dst), _stream(stream)),
           "gnn_gather_rows")


def _host_graph(full):
    ip = np.ascontiguousarray(full.indptr, np.int64)
    ix = np.ascontiguousarray(full.indices, np.int32)
    return ip, ix


def gnn_frontier_sample(full, m: int, budget: int, eta: float, clip: int, seed: int,
                        sub_id: int) -> np.ndarray:
    """Node list of subgraph sub_id (host arrays in, sorted int32 out)."""
    ip, ix = _host_graph(full)
    out = np.empty(max(int(budget), 1), np.int32)
    cnt = ctypes.c_int32(0)
    _check(lib().gnn_frontier_sample(int(full.n), ip.ctypes.data, ix.ctypes.data, int(m),
                                     int(budget), float(eta), int(clip),
                                     int(seed) & ((1 << 64) - 1), int(sub_id),
                                     out.ctypes.data, ctypes.addressof(cnt)),
           "gnn_frontier_sample")
    return out[: cnt.value].copy()


def gnn_sampler_create(n_full: int, indptr: np.ndarray, indices: np.ndarray, m: int,
                       budget: int, eta: float, clip: int, seed: int, threads: int,
                       depth: int) -> ctypes.c_void_p:
    """Handle of a new pool; indptr / indices are host numpy arrays that
    must outlive it."""
    h = ctypes.c_void_p()
    _check(lib().gnn_sampler_create(int(n_full), indptr.ctypes.data, indices.ctypes.data,
                                    int(m), int(budget), float(eta), int(clip),
                                    int(seed) & ((1 << 64) - 1), int(threads), int(depth),
                                    ctypes.addressof(h)), "gnn_sampler_create")
    return h


def gnn_sampler_next(h, room: int):
    """(subgraph id, sorted node list) of the pool's next subgraph."""
    out = np.empty(max(int(room), 1), np.int32)
    cnt, sid = ctypes.c_int32(0), ctypes.c_int64(0)
    _check(lib().gnn_sampler_next(h, out.ctypes.data, ctypes.addressof(cnt),
                                  ctypes.addressof(sid)), "gnn_sampler_next")
    return int(sid.value), out[: cnt.value].copy()


def gnn_sampler_destroy(h):
    lib().gnn_sampler_destroy(h)


class gnn_sampler_pool:
    """Owns a gnn_sampler and the host graph arrays it reads."""

    def __init__(self, full, m: int, budget: int, eta: float, clip: int, seed: int,
                 threads: int, depth: int):
        self._ip, self._ix = _host_graph(full)
        self.budget = int(budget)
        self._h = gnn_sampler_create(full.n, self._ip, self._ix, m, budget, eta, clip, seed,
                                     threads, depth)

    def next(self):
        """(subgraph id, sorted node list)."""
        return gnn_sampler_next(self._h, self.budget)

    def close(self):
        if getattr(self, "_h", None):
            gnn_sampler_destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()


def gnn_spmm_workspace_bytes(csr: gnn_csr, w: int) -> int:
    return int(lib().gnn_spmm_workspace_bytes(ctypes.byref(csr), int(w)))


def gnn_spmm(csr: gnn_csr, transpose: bool, w: int, inp, ld_in: int, out,
             ld_out: int, workspace, stream=None):
    _check(lib().gnn_spmm(ctypes.byref(csr), int(transpose), int(w), _ptr(inp),
                          int(ld_in), _ptr(out), int(ld_out), _ptr(workspace),
                          _nbytes(workspace), _stream(stream)), "gnn_spmm")


def gnn_spmm_gather_floor(csr: gnn_csr, transpose: bool, w: int, inp, ld_in: int,
                          out, ld_out: int, stream=None):
    _check(lib().gnn_spmm_gather_floor(ctypes.byref(csr), int(transpose), int(w),
                                       _ptr(inp), int(ld_in), _ptr(out), int(ld_out),
                                       _stream(stream)), "gnn_spmm_gather_floor")


def gnn_gemm_workspace_bytes(M: int, N: int, K: int) -> int:
    return int(lib().gnn_gemm_workspace_bytes(int(M), int(N), int(K)))


def gnn_gemm(trans_a: bool, trans_b: bool, M: int, N: int, K: int, A, lda: int,
             B, ldb: int, C, ldc: int, flags: int = 0, workspace=None,
             stream=None):
    _check(lib().gnn_gemm(int(trans_a), int(trans_b), int(M), int(N), int(K),
                          _ptr(A), int(lda), _ptr(B), int(ldb), _ptr(C), int(ldc),
                          int(flags), _ptr(workspace), _nbytes(workspace),
                          _stream(stream)), "gnn_gemm")


def gnn_mfma_rate_probe(kind: int, blocks: int, iters: int, sink, clocks, stream=None):
    _check(lib().gnn_mfma_rate_probe(int(kind), int(blocks), int(iters), _ptr(sink),
                                     _ptr(clocks), _stream(stream)), "gnn_mfma_rate_probe")


def gnn_timer_enable(enable: bool = True):
    _check(lib().gnn_timer_enable(int(enable)), "gnn_timer_enable")


def gnn_timer_reset():
    _check(lib().gnn_timer_reset(), "gnn_timer_reset")


def gnn_timer_read(kernel) -> tuple:
    """(milliseconds, launches, algorithmic work) of one kernel."""
    k = KERNELS[kernel] if isinstance(kernel, str) else int(kernel)
    ms, n, w = ctypes.c_double(), ctypes.c_int64(), ctypes.c_double()
    _check(lib().gnn_timer_read(k, ctypes.byref(ms), ctypes.byref(n),
                                ctypes.byref(w)), "gnn_timer_read")
    return ms.value, n.value, w.value
