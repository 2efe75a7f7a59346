"""Python face of the CPU oracle (test infrastructure only).

The oracle is plain C in double precision (gnn_oracle.c); this module
compiles it with gcc on first use, loads it with ctypes and converts numpy
arrays.  Only the tests, the smoke check and the benchmark's CPU-baseline
leg use it; the GPU library never does.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gnn_oracle.c")
_LIB = os.path.join(_HERE, "libgnn_oracle.so")
_lock = threading.Lock()
_lib = None

_I32P = ctypes.POINTER(ctypes.c_int32)
_F64P = ctypes.POINTER(ctypes.c_double)
_U8P = ctypes.POINTER(ctypes.c_uint8)
_I64P = ctypes.POINTER(ctypes.c_int64)


def build(force: bool = True) -> str:
    """Compile the oracle into oracle/libgnn_oracle.so (gcc, OpenMP)."""
    if not force and os.path.exists(_LIB):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O3", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-shared", "-fPIC", "-std=c99", "-Wall", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB) or \
                    os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build()
            L = ctypes.CDLL(_LIB)
            i32, i64 = ctypes.c_int32, ctypes.c_int64
            sigs = {
                "oracle_spmm": [i32, _I32P, _I32P, _F64P, i32, _F64P, _F64P],
                "oracle_spmm_transpose": [i32, _I32P, _I32P, _F64P, i32, _F64P,
                                          _F64P],
                "oracle_transpose_values": [i32, _I32P, _I32P, _F64P, _F64P],
                "oracle_choose_order": [i64, i64],
                "oracle_mm_nn": [i32, i32, i32, _F64P, _F64P, _F64P],
                "oracle_mm_tn": [i32, i32, i32, _F64P, _F64P, _F64P],
                "oracle_mm_nt": [i32, i32, i32, _F64P, _F64P, _F64P],
                "oracle_sage_fwd": [i32, _I32P, _I32P, _F64P, i32, i32, _F64P,
                                    _F64P, _F64P, _F64P, _F64P, _F64P, _F64P],
                "oracle_sage_bwd": [i32, _I32P, _I32P, _F64P, i32, i32, _F64P,
                                    _F64P, _F64P, _F64P, _F64P, _F64P, _F64P,
                                    _F64P, _F64P, _F64P],
                "oracle_sage_fwd_rows": [i32, _I32P, _I32P, _F64P, i32, i32,
                                         _F64P, _F64P, _F64P, _F64P, _F64P,
                                         i32, _I32P, _F64P],
                "oracle_sage_bwd_dx_rows": [i32, _I32P, _I32P, _F64P, i32, i32,
                                            _F64P, _F64P, _F64P, _F64P, i32,
                                            _I32P, _F64P],
                "oracle_sage_bwd_dw_entries": [i32, _I32P, _I32P, _F64P, i32,
                                               i32, _F64P, _F64P, _F64P, i32,
                                               _I32P, _I32P, _F64P, _F64P],
                "oracle_round_bf16": [i64, _F64P, _F64P],
                "oracle_gcn_fwd": [i32, _I32P, _I32P, _F64P, i32, i32, _F64P,
                                   _F64P, _F64P, _F64P, _F64P],
                "oracle_gcn_bwd": [i32, _I32P, _I32P, _F64P, i32, i32, _F64P,
                                   _F64P, _F64P, _F64P, _F64P, _F64P, _F64P],
                "oracle_classifier": [i32, i32, i32, _F64P, _F64P, _F64P, i32,
                                      _F64P, _F64P, _F64P, _U8P],
                "oracle_sgd": [i64, _F64P, _F64P, ctypes.c_double],
                "oracle_induce": [i64, _I64P, _I32P, i32, _I32P, i32, _I32P, _I32P,
                                  _F64P],
                "oracle_gat_fwd": [i32, _I32P, _I32P, i32, i32, _F64P, _F64P, _F64P,
                                   ctypes.c_double, _F64P, _F64P],
                "oracle_gat_bwd": [i32, _I32P, _I32P, i32, i32, _F64P, _F64P, _F64P,
                                   ctypes.c_double, _F64P, _F64P, _F64P, _F64P, _F64P,
                                   _U8P],
                "oracle_adam": [i64, _F64P, _F64P, _F64P, _F64P, ctypes.c_double,
                                ctypes.c_double, ctypes.c_double, ctypes.c_double, i32],
                "oracle_mixhop_fwd": [i32, _I32P, _I32P, _F64P, i32, i32, i32,
                                      _F64P, _F64P, _F64P, _F64P],
                "oracle_mixhop_bwd": [i32, _I32P, _I32P, _F64P, i32, i32, i32,
                                      _F64P, _F64P, _F64P, _F64P, _F64P, _F64P,
                                      _F64P],
                "oracle_num_threads": [],
                "oracle_set_num_threads": [i32],
            }
            for name, args in sigs.items():
                fn = getattr(L, name)
                fn.argtypes = args
                fn.restype = ctypes.c_int32 if name in (
                    "oracle_transpose_values", "oracle_choose_order",
                    "oracle_num_threads") else None
                if name == "oracle_classifier":
                    fn.restype = ctypes.c_double
                if name == "oracle_induce":
                    fn.restype = ctypes.c_int64
            _lib = L
        return _lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _p(a: Optional[np.ndarray], t):
    if a is None:
        return None
    return a.ctypes.data_as(t)


def _csr(g) -> Tuple[int, np.ndarray, np.ndarray, np.ndarray]:
    return g.n, _i32(g.indptr), _i32(g.indices), _f64(g.values)


def round_bf16(a) -> np.ndarray:
    """float -> nearest bfloat16 (ties to even), returned as double."""
    a = np.asarray(a)
    x = _f64(a).reshape(-1)
    out = np.empty_like(x)
    lib().oracle_round_bf16(x.size, _p(x, _F64P), _p(out, _F64P))
    return out.reshape(a.shape)


def num_threads() -> int:
    return int(lib().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """OpenMP threads of the oracle's later calls (results are identical for
    any count)."""
    lib().oracle_set_num_threads(int(n))


def spmm(g, x: np.ndarray) -> np.ndarray:
    n, ip, ix, v = _csr(g)
    x = _f64(x)
    w = x.shape[1]
    out = np.empty((n, w), np.float64)
    lib().oracle_spmm(n, _p(ip, _I32P), _p(ix, _I32P), _p(v, _F64P), w,
                      _p(x, _F64P), _p(out, _F64P))
    return out


def spmm_transpose(g, u: np.ndarray) -> np.ndarray:
    n, ip, ix, v = _csr(g)
    u = _f64(u)
    w = u.shape[1]
    out = np.empty((n, w), np.float64)
    lib().oracle_spmm_transpose(n, _p(ip, _I32P), _p(ix, _I32P), _p(v, _F64P),
                                w, _p(u, _F64P), _p(out, _F64P))
    return out


def transpose_values(g) -> np.ndarray:
    n, ip, ix, v = _csr(g)
    vt = np.full(v.shape, np.nan, np.float64)
    rc = lib().oracle_transpose_values(n, _p(ip, _I32P), _p(ix, _I32P),
                                       _p(v, _F64P), _p(vt, _F64P))
    if rc != 0:
        raise ValueError("pattern is not symmetric")
    return vt


def choose_order(f1: int, f2: int) -> int:
    return int(lib().oracle_choose_order(int(f1), int(f2)))


def _mm(name, M, N, K, a, b):
    a, b = _f64(a), _f64(b)
    c = np.empty((M, N), np.float64)
    getattr(lib(), name)(M, N, K, _p(a, _F64P), _p(b, _F64P), _p(c, _F64P))
    return c


def mm_nn(a, b):
    return _mm("oracle_mm_nn", a.shape[0], b.shape[1], a.shape[1], a, b)


def mm_tn(a, b):
    return _mm("oracle_mm_tn", a.shape[1], b.shape[1], a.shape[0], a, b)


def mm_nt(a, b):
    return _mm("oracle_mm_nt", a.shape[0], b.shape[0], a.shape[1], a, b)


def sage_fwd(g, x, w_self, w_neigh, b_self=None, b_neigh=None,
             want_s: bool = False):
    """Returns Y (n x 2h) [and S = A_s X]."""
    n, ip, ix, v = _csr(g)
    x, ws, wn = _f64(x), _f64(w_self), _f64(w_neigh)
    f_in, h = ws.shape
    assert x.shape == (n, f_in) and wn.shape == (f_in, h)
    bs = None if b_self is None else _f64(b_self)
    bn = None if b_neigh is None else _f64(b_neigh)
    y = np.empty((n, 2 * h), np.float64)
    s = np.empty((n, f_in), np.float64) if want_s else None
    lib().oracle_sage_fwd(n, _p(ip, _I32P), _p(ix, _I32P), _p(v, _F64P), f_in,
                          h, _p(x, _F64P), _p(ws, _F64P), _p(wn, _F64P),
                          _p(bs, _F64P), _p(bn, _F64P), _p(y, _F64P),
                          _p(s, _F64P))
    return (y, s) if want_s else y


def sage_bwd(g, x, w_self, w_neigh, y, dy, want_dx: bool = True,
             want_db: bool = False) -> dict:
    n, ip, ix, v = _csr(g)
    x, ws, wn, y, dy = _f64(x), _f64(w_self), _f64(w_neigh), _f64(y), _f64(dy)
    f_in, h = ws.shape
    assert x.shape == (n, f_in) and y.shape == (n, 2 * h) == dy.shape
    out = {"dW_self": np.empty((f_in, h)), "dW_neigh": np.empty((f_in, h))}
    out["dX"] = np.empty((n, f_in)) if want_dx else None
    out["db_self"] = np.empty(h) if want_db else None
    out["db_neigh"] = np.empty(h) if want_db else None
    lib().oracle_sage_bwd(n, _p(ip, _I32P), _p(ix, _I32P), _p(v, _F64P), f_in,
                          h, _p(x, _F64P), _p(ws, _F64P), _p(wn, _F64P),
                          _p(y, _F64P), _p(dy, _F64P), _p(out["dX"], _F64P),
                          _p(out["dW_self"], _F64P), _p(out["dW_neigh"], _F64P),
                          _p(out["db_self"], _F64P), _p(out["db_neigh"], _F64P))
    return out


def sage_fwd_rows(g, x, w_self, w_neigh, rows, b_self=None, b_neigh=None):
    n, ip, ix, v = _csr(g)
    x, ws, wn = _f64(x), _f64(w_self), _f64(w_neigh)
    f_in, h = ws.shape
    rows = _i32(rows)
    bs = None if b_self is None else _f64(b_self)
    bn = None if b_neigh is None else _f64(b_neigh)
    y = np.empty((rows.size, 2 * h), np.float64)
    lib().oracle_sage_fwd_rows(n, _p(ip, _I32P), _p(ix, _I32P), _p(v, _F64P),
                               f_in, h, _p(x, _F64P), _p(ws, _F64P),
                               _p(wn, _F64P), _p(bs, _F64P), _p(bn, _F64P),
                               rows.size, _p(rows, _I32P), _p(y, _F64P))
    return y


def sage_bwd_dx_rows(g, w_self, w_neigh, y, dy, rows):
    n, ip, ix, v = _csr(g)
    ws, wn, y, dy = _f64(w_self), _f64(w_neigh), _f64(y), _f64(dy)
    f_in, h = ws.shape
    rows = _i32(rows)
    out = np.empty((rows.size, f_in), np.float64)
    lib().oracle_sage_bwd_dx_rows(n, _p(ip, _I32P), _p(ix, _I32P),
                                  _p(v, _F64P), f_in, h, _p(ws, _F64P),
                                  _p(wn, _F64P), _p(y, _F64P), _p(dy, _F64P),
                                  rows.size, _p(rows, _I32P), _p(out, _F64P))
    return out


def sage_bwd_dw_entries(g, x, y, dy, h, ei, ej):
    n, ip, ix, v = _csr(g)
    x, y, dy = _f64(x), _f64(y), _f64(dy)
    f_in = x.shape[1]
    ei, ej = _i32(ei), _i32(ej)
    ws = np.empty(ei.size, np.float64)
    wn = np.empty(ei.size, np.float64)
    lib().oracle_sage_bwd_dw_entries(n, _p(ip, _I32P), _p(ix, _I32P),
                                     _p(v, _F64P), f_in, h, _p(x, _F64P),
                                     _p(y, _F64P), _p(dy, _F64P), ei.size,
                                     _p(ei, _I32P), _p(ej, _I32P),
                                     _p(ws, _F64P), _p(wn, _F64P))
    return ws, wn


def gcn_fwd(g, x, w, b=None, want_s: bool = False):
    """Y = ReLU(A_hat X W + b); g.values must hold A_hat."""
    n, ip, ix, v = _csr(g)
    x, w = _f64(x), _f64(w)
    f_in, h = w.shape
    assert x.shape == (n, f_in)
    bb = None if b is None else _f64(b)
    y = np.empty((n, h), np.float64)
    s = np.empty((n, f_in), np.float64) if want_s else None
    lib().oracle_gcn_fwd(n, _p(ip, _I32P), _p(ix, _I32P), _p(v, _F64P), f_in, h,
                         _p(x, _F64P), _p(w, _F64P), _p(bb, _F64P), _p(y, _F64P),
                         _p(s, _F64P))
    return (y, s) if want_s else y


def gcn_bwd(g, x, w, y, dy, want_dx: bool = True, want_db: bool = False) -> dict:
    n, ip, ix, v = _csr(g)
    x, w, y, dy = _f64(x), _f64(w), _f64(y), _f64(dy)
    f_in, h = w.shape
    assert y.shape == (n, h) == dy.shape
    out = {"dW": np.empty((f_in, h)),
           "dX": np.empty((n, f_in)) if want_dx else None,
           "db": np.empty(h) if want_db else None}
    lib().oracle_gcn_bwd(n, _p(ip, _I32P), _p(ix, _I32P), _p(v, _F64P), f_in, h,
                         _p(x, _F64P), _p(w, _F64P), _p(y, _F64P), _p(dy, _F64P),
                         _p(out["dX"], _F64P), _p(out["dW"], _F64P),
                         _p(out["db"], _F64P))
    return out


def mixhop_fwd(g, x, w, K: int, b=None):
    """Y = ReLU(||_k A_hat^k X W_k + b); w is f_in x (K+1)h."""
    n, ip, ix, v = _csr(g)
    x, w = _f64(x), _f64(w)
    f_in, wy = w.shape
    assert wy % (K + 1) == 0 and x.shape == (n, f_in)
    h = wy // (K + 1)
    bb = None if b is None else _f64(b)
    y = np.empty((n, wy), np.float64)
    lib().oracle_mixhop_fwd(n, _p(ip, _I32P), _p(ix, _I32P), _p(v, _F64P), K, f_in,
                            h, _p(x, _F64P), _p(w, _F64P), _p(bb, _F64P),
                            _p(y, _F64P))
    return y


def mixhop_bwd(g, x, w, K: int, y, dy, want_dx: bool = True,
               want_db: bool = False) -> dict:
    n, ip, ix, v = _csr(g)
    x, w, y, dy = _f64(x), _f64(w), _f64(y), _f64(dy)
    f_in, wy = w.shape
    h = wy // (K + 1)
    assert y.shape == (n, wy) == dy.shape
    out = {"dW": np.empty((f_in, wy)),
           "dX": np.empty((n, f_in)) if want_dx else None,
           "db": np.empty(wy) if want_db else None}
    lib().oracle_mixhop_bwd(n, _p(ip, _I32P), _p(ix, _I32P), _p(v, _F64P), K, f_in,
                            h, _p(x, _F64P), _p(w, _F64P), _p(y, _F64P),
                            _p(dy, _F64P), _p(out["dX"], _F64P), _p(out["dW"], _F64P),
                            _p(out["db"], _F64P))
    return out


SOFTMAX, SIGMOID = 0, 1


GAT_ALPHA = 0.2  # LeakyReLU slope of the attention scores


def gat_fwd(g, x, w, a, alpha: float = GAT_ALPHA, want_att: bool = False):
    """Y = ReLU(A_att X W) with att_uv = LeakyReLU(a1 . P_u + a2 . P_v)."""
    n, ip, ix, _ = _csr(g)
    x, w, a = _f64(x), _f64(w), _f64(a)
    f_in, h = w.shape
    assert x.shape == (n, f_in) and a.shape == (2 * h,)
    y = np.empty((n, h))
    att = np.empty(int(ip[-1])) if want_att else None
    lib().oracle_gat_fwd(n, _p(ip, _I32P), _p(ix, _I32P), f_in, h, _p(x, _F64P),
                         _p(w, _F64P), _p(a, _F64P), float(alpha), _p(y, _F64P),
                         _p(att, _F64P))
    return (y, att) if want_att else y


def gat_bwd(g, x, w, a, y, dy, alpha: float = GAT_ALPHA, want_dx: bool = True,
            z_pos=None) -> dict:
    """z_pos: optional per-entry booleans, the LeakyReLU's decisions."""
    n, ip, ix, _ = _csr(g)
    zp = None if z_pos is None else np.ascontiguousarray(z_pos, np.uint8)
    x, w, a, y, dy = _f64(x), _f64(w), _f64(a), _f64(y), _f64(dy)
    f_in, h = w.shape
    assert y.shape == (n, h) == dy.shape
    out = {"dW": np.empty((f_in, h)), "da": np.empty(2 * h),
           "dX": np.empty((n, f_in)) if want_dx else None}
    lib().oracle_gat_bwd(n, _p(ip, _I32P), _p(ix, _I32P), f_in, h, _p(x, _F64P),
                         _p(w, _F64P), _p(a, _F64P), float(alpha), _p(y, _F64P),
                         _p(dy, _F64P), _p(out["dX"], _F64P), _p(out["dW"], _F64P),
                         _p(out["da"], _F64P), _p(zp, _U8P))
    return out


def classifier(x, w, t, kind: int, want_dx: bool = True, relu_on=None) -> dict:
    """Head + loss: returns loss, probs, dW, dX (see oracle_classifier).
    relu_on: optional n x C booleans, the MLP ReLU's decision."""
    x, w, t = _f64(x), _f64(w), _f64(t)
    n, f = x.shape
    C = w.shape[1]
    assert w.shape == (f, C) and t.shape == (n, C)
    on = None
    if relu_on is not None:
        on = np.ascontiguousarray(relu_on, np.uint8)
        assert on.shape == (n, C)
    probs = np.empty((n, C))
    dw = np.empty((f, C))
    dx = np.empty((n, f)) if want_dx else None
    loss = lib().oracle_classifier(n, f, C, _p(x, _F64P), _p(w, _F64P), _p(t, _F64P),
                                   int(kind), _p(probs, _F64P), _p(dw, _F64P),
                                   _p(dx, _F64P), _p(on, _U8P))
    return {"loss": float(loss), "probs": probs, "dW": dw, "dX": dx}


def sgd(w, g, lr: float) -> np.ndarray:
    w = _f64(w).copy()
    g = _f64(g)
    lib().oracle_sgd(w.size, _p(w, _F64P), _p(g, _F64P), float(lr))
    return w


def adam(w, g, m, v, lr, b1, b2, eps, t: int):
    """Returns updated (w, m, v) as new arrays."""
    w, m, v = _f64(w).copy(), _f64(m).copy(), _f64(v).copy()
    g = _f64(g)
    lib().oracle_adam(w.size, _p(w, _F64P), _p(g, _F64P), _p(m, _F64P), _p(v, _F64P),
                      float(lr), float(b1), float(b2), float(eps), int(t))
    return w, m, v


def sage_stack(g, x, params, dy_top, want_dx_first: bool = True):
    """L layers forward then backward (Algorithm 1's layer loop with a given
    top gradient in place of the classifier and loss).  Every layer's input
    is the previous layer's double-precision output."""
    acts, ys = [_f64(x)], []
    for p in params:
        y = sage_fwd(g, acts[-1], p.w_self, p.w_neigh, p.b_self, p.b_neigh)
        ys.append(y)
        acts.append(y)
    grads = [None] * len(params)
    dy = _f64(dy_top)
    for l in reversed(range(len(params))):
        p = params[l]
        need_dx = l > 0 or want_dx_first
        r = sage_bwd(g, acts[l], p.w_self, p.w_neigh, ys[l], dy,
                     want_dx=need_dx, want_db=p.b_self is not None)
        grads[l] = r
        dy = r["dX"]
    return {"acts": acts, "ys": ys, "grads": grads}


def train_step(g, x, params, w_mlp, targets, kind: int, opt: str = "sgd",
               lr: float = 0.01, state=None, t: int = 1, b1: float = 0.9,
               b2: float = 0.999, eps: float = 1e-8, forced=None):
    """One iteration of Algorithm 1 on a given subgraph: the L layers forward,
    classifier and loss (Section 3.1), the backward pass of Section 5.1 from
    the classifier's input gradient down, then every weight updated by SGD or
    Adam.  state: per-parameter (m, v) pairs for Adam, in the order
    [W_MLP, then W_self, W_neigh (, b_self, b_neigh) of each layer].
    forced: optional {"ys": [Y of layer 1..L], "relu_on": n x C booleans}
    taken in place of the forward pass's own layer outputs (the inputs of
    the layers above, the ReLU masks of the backward pass) and of the MLP
    ReLU's decision, so that every ReLU decision is another implementation's.
    Returns the loss, the gradients, the updated weights and the new state."""
    acts, ys = [_f64(x)], []
    for l, p in enumerate(params):
        if forced is not None:
            y = _f64(forced["ys"][l])
        else:
            y = sage_fwd(g, acts[-1], p.w_self, p.w_neigh, p.b_self, p.b_neigh)
        ys.append(y)
        acts.append(y)
    head = classifier(acts[-1], w_mlp, targets, kind, want_dx=True,
                      relu_on=None if forced is None else forced.get("relu_on"))
    grads = [None] * len(params)
    dy = head["dX"]
    for l in reversed(range(len(params))):
        p = params[l]
        r = sage_bwd(g, acts[l], p.w_self, p.w_neigh, ys[l], dy, want_dx=l > 0,
                     want_db=p.b_self is not None)
        grads[l] = r
        dy = r["dX"]
    weights = [_f64(w_mlp)]
    gs = [head["dW"]]
    for p, r in zip(params, grads):
        weights += [_f64(p.w_self), _f64(p.w_neigh)]
        gs += [r["dW_self"], r["dW_neigh"]]
        if p.b_self is not None:
            weights += [_f64(p.b_self), _f64(p.b_neigh)]
            gs += [r["db_self"], r["db_neigh"]]
    if state is None:
        state = [(np.zeros_like(w), np.zeros_like(w)) for w in weights]
    new_w, new_state = [], []
    for w, gr, (m, v) in zip(weights, gs, state):
        if opt == "sgd":
            new_w.append(sgd(w, gr, lr))
            new_state.append((m, v))
        else:
            w2, m2, v2 = adam(w, gr, m, v, lr, b1, b2, eps, t)
            new_w.append(w2)
            new_state.append((m2, v2))
    return {"loss": head["loss"], "probs": head["probs"], "acts": acts,
            "head": head, "grads": grads, "flat_grads": gs, "weights": new_w,
            "state": new_state}


class SubgraphCsr:
    """CSR of an induced subgraph (the oracle's own result type)."""

    def __init__(self, n, indptr, indices, values):
        self.n, self.indptr, self.indices, self.values = n, indptr, indices, values

    @property
    def nnz(self) -> int:
        return int(self.indptr[-1])


def induce(full, nodes, norm: int = 0) -> SubgraphCsr:
    """Subgraph of `full` (n, indptr, indices) induced by the sorted,
    distinct node list `nodes`, self loops added, normalised by rows
    (norm 0) or symmetrically (norm 1); see oracle_induce."""
    ip = np.ascontiguousarray(full.indptr, np.int64)
    ix = _i32(full.indices)
    nd = _i32(nodes)
    assert nd.ndim == 1 and (nd.size < 2 or np.all(nd[1:] > nd[:-1]))
    assert nd.size == 0 or (nd[0] >= 0 and nd[-1] < full.n)
    cap = int((ip[nd + 1] - ip[nd]).sum()) + nd.size
    out_ip = np.zeros(nd.size + 1, np.int32)
    out_ix = np.empty(max(cap, 1), np.int32)
    out_v = np.empty(max(cap, 1), np.float64)
    nnz = lib().oracle_induce(int(full.n), _p(ip, _I64P), _p(ix, _I32P), nd.size,
                              _p(nd, _I32P), int(norm), _p(out_ip, _I32P),
                              _p(out_ix, _I32P), _p(out_v, _F64P))
    return SubgraphCsr(nd.size, out_ip, out_ix[:nnz].copy(), out_v[:nnz].copy())
