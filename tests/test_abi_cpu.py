"""Host-side checks of the C-ABI library; no GPU needed.

The library must load, export every function include/gnnprop.h declares,
and reject bad arguments synchronously, before anything is enqueued.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import oracle as O
from paper_2010_03166_amd import gnnprop as G

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gnnprop.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"\b(gnn_[a-z_0-9]+)\s*\(", src)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(G.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return G.lib()


def test_header_declares_the_boundary():
    names = declared_functions()
    for must in ("gnn_prop_fwd", "gnn_prop_bwd", "gnn_csr_transpose_values",
                 "gnn_csr_build_plan", "gnn_csr_validate", "gnn_spmm", "gnn_gemm",
                 "gnn_choose_order", "gnn_status_string"):
        assert must in names


def test_library_exports_every_declared_symbol(lib):
    names = declared_functions()
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing
    # and the binding wraps every one of them by the same name
    assert set(names) <= set(G.EXPORTS), set(names) - set(G.EXPORTS)


def test_binding_has_same_names(lib):
    for n in declared_functions():
        if n == "gnn_status_string":
            continue
        assert callable(getattr(G, n)), n


def test_status_strings(lib):
    for s in range(0, -8, -1):
        assert G.status_string(s)
    assert G.status_string(-99) == "unknown status"


@pytest.mark.parametrize("f_in,h", [(50, 128), (602, 512), (300, 512), (512, 512),
                                    (1024, 512), (200, 512), (256, 1024),
                                    (2048, 1024), (1, 1), (7, 3)])
def test_order_rule_agrees_with_oracle(lib, f_in, h):
    assert G.gnn_choose_order(f_in, h) == O.choose_order(f_in, h)


def test_plan_bytes_monotone(lib):
    a = G.gnn_plan_bytes(1000, 10000)
    assert a >= 4 * 10000  # the row of every entry
    assert G.gnn_plan_bytes(2000, 10000) >= a
    assert G.gnn_plan_bytes(1000, 100000) > a
    assert G.gnn_plan_bytes(0, 0) > 0
    assert G.gnn_plan_bytes(-1, 0) == 0


def _fake_csr(n=10, nnz=30):
    # host addresses stand in for device pointers: these calls must fail
    # before dereferencing or launching anything
    return G.make_csr(n, nnz, 0x1000, 0x2000, 0x3000, 0x4000, 0x5000)


def test_size_queries(lib):
    c = _fake_csr(8000, 128000)
    l1 = G.make_layer(602, 512, 604, 1024, 604, order=1)
    l2 = G.make_layer(602, 512, 604, 1024, 604, order=2)
    # split products: the forward also saves the input gradient's bf16
    # pieces of W_self^T and W_neigh^T (three planes of ceil(h / 16) groups
    # x f_in columns x 16 bf16 each)
    pieces = 2 * (3 * 32 * 602 * 16 * 2)
    assert G.gnn_prop_saved_bytes(c, l1) >= 8000 * 604 * 4 + pieces
    assert G.gnn_prop_saved_bytes(c, l2) == pieces
    for flag in (G.GNN_FLAG_BF16, G.GNN_FLAG_F32_MFMA):  # no pieces
        l2f = G.make_layer(602, 512, 604, 1024, 604, order=2, flags=flag)
        assert G.gnn_prop_saved_bytes(c, l2f) == 0
        l1f = G.make_layer(602, 512, 604, 1024, 604, order=1, flags=flag)
        assert 8000 * 604 * 4 <= G.gnn_prop_saved_bytes(c, l1f) < 8000 * 604 * 4 + 256
    for l in (l1, l2):
        assert G.gnn_prop_workspace_bytes(c, l) > 8000 * 512 * 4
    auto = G.make_layer(602, 512, 604, 1024, 604, order=0)
    assert G.gnn_prop_saved_bytes(c, auto) == pieces  # 602 > 512: order 2
    # one block per tile (no partial tiles); the split products' B pieces:
    # three planes of ceil(K / 16) groups x N columns x 16 bf16
    assert G.gnn_gemm_workspace_bytes(8000, 1024, 602) == 3 * 38 * 1024 * 16 * 2
    assert G.gnn_gemm_workspace_bytes(602, 512, 8000) > 0  # split along K
    assert G.gnn_spmm_workspace_bytes(c, 512) == 0  # one kernel, no partials


def _st(fn, *args):
    return getattr(G.lib(), fn)(*args)


def test_argument_errors_are_synchronous(lib):
    L = G.lib()
    c = _fake_csr()
    lay = G.make_layer(8, 4, 8, 8, 8)
    P = ctypes.c_void_p
    ws = 1 << 30
    # NULL structs
    assert L.gnn_prop_fwd(None, ctypes.byref(lay), *([P(0x10)] * 8), ws, None) == -1
    assert L.gnn_prop_fwd(ctypes.byref(c), None, *([P(0x10)] * 8), ws, None) == -1
    # bad shapes
    bad = G.make_layer(8, 4, 7, 8, 8)  # ld_x < f_in
    assert L.gnn_prop_fwd(ctypes.byref(c), ctypes.byref(bad), *([P(0x10)] * 8), ws, None) == -2
    bad = G.make_layer(8, 4, 8, 7, 8)  # ld_y < 2h
    assert L.gnn_prop_fwd(ctypes.byref(c), ctypes.byref(bad), *([P(0x10)] * 8), ws, None) == -2
    bad = G.make_layer(0, 4, 8, 8, 8)
    assert L.gnn_prop_fwd(ctypes.byref(c), ctypes.byref(bad), *([P(0x10)] * 8), ws, None) == -2
    bad = G.make_layer(8, 4, 8, 8, 8, order=3)
    assert L.gnn_prop_fwd(ctypes.byref(c), ctypes.byref(bad), *([P(0x10)] * 8), ws, None) == -2
    bad = G.make_layer(8, 4, 8, 8, 8, flags=0x80)
    assert L.gnn_prop_fwd(ctypes.byref(c), ctypes.byref(bad), *([P(0x10)] * 8), ws, None) == -4
    # negative sizes
    neg = G.make_csr(-1, 0, 0x1000, 0x2000, 0x3000, 0x4000, 0x5000)
    assert L.gnn_prop_fwd(ctypes.byref(neg), ctypes.byref(lay), *([P(0x10)] * 8), ws, None) == -2
    # workspace too small
    assert L.gnn_prop_fwd(ctypes.byref(c), ctypes.byref(lay), *([P(0x10)] * 8), 16, None) == -5
    # missing values_t for the backward pass
    c2 = G.make_csr(10, 30, 0x1000, 0x2000, 0x3000, None, 0x5000)
    assert L.gnn_prop_bwd(ctypes.byref(c2), ctypes.byref(lay), *([P(0x10)] * 12), ws, None) == -1
    # output overlapping an input
    xs = 0x100000
    assert L.gnn_prop_fwd(ctypes.byref(c), ctypes.byref(lay), P(xs), P(0x10), P(0x20),
                          None, None, P(xs + 8), P(0x40), P(0x50), ws, None) == -7
    # spmm / gemm
    assert L.gnn_spmm(ctypes.byref(c), 0, 8, P(0x10), 4, P(0x20), 8, None, 0, None) == -2
    # gather floor: the same checks, plus 16-byte aligned rows
    assert L.gnn_spmm_gather_floor(ctypes.byref(c), 0, 8, P(0x10), 4, P(0x20), 8, None) == -2
    assert L.gnn_spmm_gather_floor(None, 0, 8, P(0x10), 8, P(0x20), 8, None) == -1
    assert L.gnn_spmm_gather_floor(ctypes.byref(c), 0, 8, P(0x14), 8, P(0x20), 8, None) == -4
    assert L.gnn_spmm_gather_floor(ctypes.byref(c), 0, 8, P(0x10), 9, P(0x20), 8, None) == -4
    assert L.gnn_spmm_gather_floor(ctypes.byref(c), 0, 8, P(0x1000), 8, P(0x1010), 8,
                                   None) == -7
    assert L.gnn_gemm(0, 0, 4, 4, 4, P(0x10), 3, P(0x20), 4, P(0x30), 4, 0, None, 0, None) == -2
    assert L.gnn_gemm(0, 0, 4, 4, 4, P(0x10), 4, P(0x20), 4, P(0x30), 4, 0x80, None, 0, None) == -4
    assert L.gnn_gemm(0, 0, -1, 4, 4, P(0x10), 4, P(0x20), 4, P(0x30), 4, 0, None, 0, None) == -2
    # bf16 and fp32-instruction products at once: not a mode
    both = G.GNN_FLAG_BF16 | G.GNN_FLAG_F32_MFMA
    assert L.gnn_gemm(0, 0, 4, 4, 4, P(0x10), 4, P(0x20), 4, P(0x30), 4, both, None, 0, None) == -4
    bad = G.make_layer(8, 4, 8, 8, 8, flags=both)
    assert L.gnn_prop_fwd(ctypes.byref(c), ctypes.byref(bad), *([P(0x10)] * 8), ws, None) == -4
    # plan buffer too small
    assert L.gnn_csr_build_plan(ctypes.byref(c), P(0x10), 8, None) == -5


def test_misaligned_buffers_rejected(lib):
    """Workspace, saved and plan buffers must start 16-byte aligned (the
    kernels access them 16 bytes at a time): any other address is refused
    before anything is enqueued."""
    L = G.lib()
    P = ctypes.c_void_p
    ws = 1 << 30
    c = _fake_csr()
    odd_plan = G.make_csr(10, 30, 0x1000, 0x2000, 0x3000, 0x4000, 0x5004)
    lay = G.make_layer(8, 4, 8, 8, 8)
    args = [P(0x10)] * 8
    assert L.gnn_prop_fwd(ctypes.byref(odd_plan), ctypes.byref(lay), *args, ws, None) == -4
    assert L.gnn_prop_fwd(ctypes.byref(c), ctypes.byref(lay), *args[:6], P(0x18), P(0x10),
                          ws, None) == -4  # saved
    assert L.gnn_prop_fwd(ctypes.byref(c), ctypes.byref(lay), *args[:7], P(0x14), ws,
                          None) == -4  # workspace
    assert L.gnn_prop_bwd(ctypes.byref(c), ctypes.byref(lay), *([P(0x10)] * 11), P(0x14), ws,
                          None) == -4
    assert L.gnn_csr_build_plan(ctypes.byref(c), P(0x14), 1 << 20, None) == -4
    need = int(L.gnn_plan_bytes(c.n, c.nnz))
    assert L.gnn_csr_prepare(ctypes.byref(c), P(0x800004), need, P(0x900000), None) == -4
    assert L.gnn_spmm(ctypes.byref(odd_plan), 0, 8, P(0x10), 8, P(0x20), 8, None, 0,
                      None) == -4
    assert L.gnn_gemm(0, 0, 4, 4, 4, P(0x10), 4, P(0x20), 4, P(0x30), 4, 0, P(0x44), ws,
                      None) == -4
    assert L.gnn_gcn_fwd(ctypes.byref(c), ctypes.byref(lay), P(0x10), P(0x20), None,
                         P(0x30), P(0x40), P(0x54), ws, None) == -4
    ml = G.make_layer(8, 4, 8, 12, 8)
    assert L.gnn_mixhop_fwd(ctypes.byref(c), ctypes.byref(ml), 2, P(0x10), P(0x20), None,
                            P(0x30), P(0x48), P(0x50), ws, None) == -4
    gl = G.make_layer(8, 4, 8, 4, 8)
    assert L.gnn_gat_fwd(ctypes.byref(c), ctypes.byref(gl), P(0x10), P(0x20), P(0x30),
                         ctypes.c_float(0.2), P(0x40), None, P(0x50), P(0x64), ws, None) == -4
    assert L.gnn_classifier(16, 8, 4, G.GNN_LOSS_SOFTMAX, 0, P(0x10), 8, P(0x20), P(0x30), 4,
                            None, 4, None, 4, P(0x40), P(0x50), None, 8, P(0x6c), ws,
                            None) == -4


def test_saved_buffer_required_where_it_holds_something(lib):
    """Order 2 saves the input gradient's weight pieces with split products,
    so forward and backward then need `saved`; with GNN_FLAG_BF16 or
    GNN_FLAG_F32_MFMA order 2 saves nothing and NULL is accepted (the calls
    below stop at the workspace size instead)."""
    L = G.lib()
    P = ctypes.c_void_p
    c = _fake_csr()
    split = G.make_layer(8, 4, 8, 8, 8, order=2)
    assert G.gnn_prop_saved_bytes(c, split) > 0
    fwd = [P(0x10)] * 6 + [None, P(0x20)]   # X .. Y, saved = NULL, workspace
    bwd = [P(0x10)] * 5 + [None] + [P(0x30)] * 5 + [P(0x20)]
    assert L.gnn_prop_fwd(ctypes.byref(c), ctypes.byref(split), *fwd, 1 << 30, None) == -1
    assert L.gnn_prop_bwd(ctypes.byref(c), ctypes.byref(split), *bwd, 1 << 30, None) == -1
    for flag in (G.GNN_FLAG_BF16, G.GNN_FLAG_F32_MFMA):
        lay = G.make_layer(8, 4, 8, 8, 8, order=2, flags=flag)
        assert G.gnn_prop_saved_bytes(c, lay) == 0
        assert L.gnn_prop_fwd(ctypes.byref(c), ctypes.byref(lay), *fwd, 16, None) == -5
        assert L.gnn_prop_bwd(ctypes.byref(c), ctypes.byref(lay), *bwd, 16, None) == -5


def test_prepare_and_gat_argument_errors(lib):
    L = G.lib()
    P = ctypes.c_void_p
    c = _fake_csr()
    need = int(L.gnn_plan_bytes(c.n, c.nnz))
    # fused preparation: plan too small, no plan, transposed values over the values
    assert L.gnn_csr_prepare(ctypes.byref(c), P(0x10), need - 1, P(0x900000), None) == -5
    assert L.gnn_csr_prepare(ctypes.byref(c), None, need, P(0x900000), None) == -1
    assert L.gnn_csr_prepare(ctypes.byref(c), P(0x800000), need, P(c.values), None) == -7
    assert L.gnn_csr_prepare(ctypes.byref(c), P(0x800000), need, None, None) == -1
    # GAT: slope outside [0, 1] (and NaN), bad widths, workspace too small
    lay = G.make_layer(8, 4, 8, 4, 8)
    ws = 1 << 30
    for alpha in (-0.1, 1.5, float("nan")):
        assert L.gnn_gat_fwd(ctypes.byref(c), ctypes.byref(lay), P(0x10), P(0x20), P(0x30),
                             ctypes.c_float(alpha), P(0x40), None, P(0x50), P(0x60), ws,
                             None) == -2
    bad = G.make_layer(8, 4, 8, 3, 8)  # ld_y < h
    assert L.gnn_gat_fwd(ctypes.byref(c), ctypes.byref(bad), P(0x10), P(0x20), P(0x30),
                         ctypes.c_float(0.2), P(0x40), None, P(0x50), P(0x60), ws, None) == -2
    assert L.gnn_gat_fwd(ctypes.byref(c), ctypes.byref(lay), P(0x10), P(0x20), P(0x30),
                         ctypes.c_float(0.2), P(0x40), None, P(0x50), P(0x60), 16, None) == -5
    assert int(L.gnn_gat_workspace_bytes(ctypes.byref(c), ctypes.byref(bad))) == 0


def test_both_product_flags_rejected_everywhere(lib):
    """GNN_FLAG_BF16 | GNN_FLAG_F32_MFMA is not a mode: every entry point with
    GEMM products refuses it before touching its (fake) pointers."""
    L = G.lib()
    P = ctypes.c_void_p
    c = _fake_csr()
    both = G.GNN_FLAG_BF16 | G.GNN_FLAG_F32_MFMA
    lay = G.make_layer(8, 4, 8, 8, 8, flags=both)
    ws = 1 << 30
    assert L.gnn_gcn_fwd(ctypes.byref(c), ctypes.byref(lay), P(0x10), P(0x20), None,
                         P(0x30), P(0x40), P(0x50), ws, None) == -4
    ml = G.make_layer(8, 4, 8, 12, 8, flags=both)  # (K + 1) h = 12 columns
    assert L.gnn_mixhop_fwd(ctypes.byref(c), ctypes.byref(ml), 2, P(0x10), P(0x20), None,
                            P(0x30), P(0x40), P(0x50), ws, None) == -4
    gl = G.make_layer(8, 4, 8, 4, 8, flags=both)
    assert L.gnn_gat_fwd(ctypes.byref(c), ctypes.byref(gl), P(0x10), P(0x20), P(0x30),
                         ctypes.c_float(0.2), P(0x40), None, P(0x50), P(0x60), ws, None) == -4
    assert L.gnn_classifier(16, 8, 4, G.GNN_LOSS_SOFTMAX, both, P(0x10), 8, P(0x20), P(0x30), 4,
                            None, 4, None, 4, P(0x40), P(0x50), None, 8, P(0x60), ws, None) == -4


def test_row_normalized_flag_arguments(lib):
    """GNN_FLAG_ROW_NORMALIZED: the GraphSAGE layer needs no value arrays
    (the checks pass NULL values / values_t and stop at the workspace size
    instead); the other layers refuse the flag."""
    L = G.lib()
    P = ctypes.c_void_p
    rn = G.GNN_FLAG_ROW_NORMALIZED
    nov = G.make_csr(10, 30, 0x1000, 0x2000, None, None, 0x5000)
    lay = G.make_layer(8, 4, 8, 8, 8, flags=rn)
    plain = G.make_layer(8, 4, 8, 8, 8)
    assert L.gnn_prop_fwd(ctypes.byref(nov), ctypes.byref(lay), *([P(0x10)] * 8), 16,
                          None) == -5
    assert L.gnn_prop_bwd(ctypes.byref(nov), ctypes.byref(lay), *([P(0x10)] * 12), 16,
                          None) == -5
    assert L.gnn_prop_fwd(ctypes.byref(nov), ctypes.byref(plain), *([P(0x10)] * 8), 16,
                          None) == -1
    assert L.gnn_prop_bwd(ctypes.byref(nov), ctypes.byref(plain), *([P(0x10)] * 12), 16,
                          None) == -1
    c = _fake_csr()
    ws = 1 << 30
    assert L.gnn_gcn_fwd(ctypes.byref(c), ctypes.byref(lay), P(0x10), P(0x20), None,
                         P(0x30), P(0x40), P(0x50), ws, None) == -4
    ml = G.make_layer(8, 4, 8, 12, 8, flags=rn)
    assert L.gnn_mixhop_fwd(ctypes.byref(c), ctypes.byref(ml), 2, P(0x10), P(0x20), None,
                            P(0x30), P(0x40), P(0x50), ws, None) == -4
    gl = G.make_layer(8, 4, 8, 4, 8, flags=rn)
    assert L.gnn_gat_fwd(ctypes.byref(c), ctypes.byref(gl), P(0x10), P(0x20), P(0x30),
                         ctypes.c_float(0.2), P(0x40), None, P(0x50), P(0x60), ws, None) == -4
    assert L.gnn_classifier(16, 8, 4, G.GNN_LOSS_SOFTMAX, rn, P(0x10), 8, P(0x20), P(0x30), 4,
                            None, 4, None, 4, P(0x40), P(0x50), None, 8, P(0x60), ws, None) == -4


def test_empty_problems_need_no_launch(lib):
    L = G.lib()
    P = ctypes.c_void_p
    # M = 0 or N = 0: nothing to do, nothing dereferenced
    assert L.gnn_gemm(0, 0, 0, 4, 4, None, 4, None, 4, None, 4, 0, None, 0, None) == 0
    c = G.make_csr(0, 0, 0x1000, None, None, None, None)
    assert L.gnn_spmm(ctypes.byref(c), 0, 8, P(0x10), 8, P(0x20), 8, None, 0, None) == 0
    assert L.gnn_spmm_gather_floor(ctypes.byref(c), 0, 8, P(0x10), 8, P(0x20), 8, None) == 0


def test_mfma_rate_probe_argument_errors(lib):
    L = G.lib()
    P = ctypes.c_void_p
    bf, f32 = G.GNN_PROBE_MFMA_BF16, G.GNN_PROBE_MFMA_F32
    assert L.gnn_mfma_rate_probe(2, 512, 100, P(0x1000), P(0x8000), None) == -4
    assert L.gnn_mfma_rate_probe(-1, 512, 100, P(0x1000), P(0x8000), None) == -4
    for blocks, iters in ((0, 100), (G.GNN_PROBE_MAX_BLOCKS + 1, 100), (512, 0),
                          (512, G.GNN_PROBE_MAX_ITERS + 1), (-3, 100)):
        assert L.gnn_mfma_rate_probe(bf, blocks, iters, P(0x1000), P(0x8000), None) == -2
    assert L.gnn_mfma_rate_probe(f32, 512, 100, None, P(0x8000), None) == -1
    assert L.gnn_mfma_rate_probe(f32, 512, 100, P(0x1000), None, None) == -1
    assert L.gnn_mfma_rate_probe(bf, 512, 100, P(0x1002), P(0x100000), None) == -4
    assert L.gnn_mfma_rate_probe(bf, 512, 100, P(0x1000), P(0x100004), None) == -4
    # clocks inside sink (512 x 512 floats from 0x1000)
    assert L.gnn_mfma_rate_probe(bf, 512, 100, P(0x1000), P(0x2000), None) == -7
    assert G.GNN_PROBE_MAX_BLOCKS == 65536 and G.GNN_PROBE_MAX_ITERS == 100000
