"""GCN and MixHop layers on the GPU against the CPU oracle (through the C ABI).

Forward outputs are compared with the oracle's; the backward pass is
teacher-forced from the oracle's side: the GPU backward receives the
oracle's forward output Y (rounded to fp32) in place of its own, and the
oracle's backward the same fp32 Y, so both take the oracle's ReLU mask.  The
ReLU decisions of the GPU's own forward that differ from the oracle's must
lie at the kink (gpu_helpers.decision_flips).  Tolerance: per-tensor
max |gpu - oracle| / max |oracle| of 1e-4 in fp32, 2e-2 with bf16 GEMM
operands.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2010_03166_amd import gnnprop as G
from paper_2010_03166_amd import runtime, synth

from gpu_helpers import decision_flips, maxrel, prepared, to_dev

pytestmark = pytest.mark.gpu

TOL = 1e-4


def graphs():
    return {
        "random": synth.random_graph(300, 6.0, 1, values="sym-normalized"),
        "powerlaw": synth.sym_normalized(synth.power_law_graph(3000, 2.1, 12.0, seed=2)),
        "star700": synth.sym_normalized(synth.star_graph(700)),
        "identity": synth.sym_normalized(synth.identity_graph(64)),
    }


GRAPHS = graphs()


def _buf(nbytes):
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device="cuda")


def _out(n, w, ld):
    return torch.full((max(n, 1), ld), float("nan"), device="cuda")[:n, :w]


def _params(f_in, wy, bias, seed):
    rng = np.random.default_rng(seed)
    w = synth.glorot(f_in, wy, rng)
    b = rng.standard_normal(wy).astype(np.float32) if bias else None
    return w, b


def run_gcn(g, f_in, h, order, bias, flags=0, seed=0, pad=8):
    dg = prepared(g)
    c = dg.struct()
    w, b = _params(f_in, h, bias, seed)
    x = synth.features(g.n, f_in, seed + 1)
    dy = np.random.default_rng(seed + 2).standard_normal((g.n, h)).astype(np.float32)
    ld_x, ld_y = f_in + pad, h + pad
    lay = G.make_layer(f_in, h, ld_x, ld_y, ld_x, order, flags)
    X, Y = to_dev(x, ld_x), _out(g.n, h, ld_y)
    W = to_dev(w)
    B = to_dev(b) if bias else None
    saved = _buf(G.gnn_gcn_saved_bytes(c, lay))
    ws = _buf(G.gnn_gcn_workspace_bytes(c, lay))
    G.gnn_gcn_fwd(c, lay, X, W, B, Y, saved, ws)
    torch.cuda.synchronize()
    y_gpu = Y.cpu().numpy()
    y_ref = O.gcn_fwd(g, x, w, b)
    y32 = y_ref.astype(np.float32)
    Y.copy_(torch.from_numpy(y32).cuda())  # the oracle's mask for the backward
    dX, dW = _out(g.n, f_in, ld_x), torch.empty((f_in, h), device="cuda")
    db = torch.empty(h, device="cuda") if bias else None
    G.gnn_gcn_bwd(c, lay, X, W, Y, to_dev(dy, ld_y), saved, dX, dW, db, ws)
    torch.cuda.synchronize()
    return dict(x=x, w=w, b=b, dy=dy, Y=y_gpu, Y_ref=y_ref, Y32=y32, dX=dX.cpu().numpy(),
                dW=dW.cpu().numpy(), db=None if db is None else db.cpu().numpy())


@pytest.mark.parametrize("name", list(GRAPHS))
@pytest.mark.parametrize("order", [1, 2])
@pytest.mark.parametrize("bias", [False, True])
def test_gcn_layer_parity(name, order, bias):
    g = GRAPHS[name]
    f_in, h = (24, 40) if order == 1 else (40, 24)
    r = run_gcn(g, f_in, h, order, bias)
    assert maxrel(r["Y"], r["Y_ref"]) <= TOL
    decision_flips(r["Y"], r["Y_ref"], TOL)
    ref = O.gcn_bwd(g, r["x"], r["w"], r["Y32"], r["dy"], want_db=bias)
    for k in ("dX", "dW") + (("db",) if bias else ()):
        assert maxrel(r[k], ref[k]) <= TOL, k


def test_gcn_full_size_bench_graph():
    wl = synth.WORKLOADS["cl2.1-n8000-f602-h512-L2"]
    g = synth.sym_normalized(synth.workload_graph(wl))
    r = run_gcn(g, 602, 512, 0, True, pad=6)  # order chosen by the rule: 2
    assert maxrel(r["Y"], r["Y_ref"]) <= TOL
    decision_flips(r["Y"], r["Y_ref"], TOL)
    ref = O.gcn_bwd(g, r["x"], r["w"], r["Y32"], r["dy"], want_db=True)
    for k in ("dX", "dW", "db"):
        assert maxrel(r[k], ref[k]) <= TOL, k


def test_gcn_bf16_mode():
    g = GRAPHS["powerlaw"]
    r = run_gcn(g, 64, 48, 2, False, flags=G.GNN_FLAG_BF16)
    assert maxrel(r["Y"], r["Y_ref"]) <= 2e-2
    decision_flips(r["Y"], r["Y_ref"], 2e-2)
    ref = O.gcn_bwd(g, r["x"], r["w"], r["Y32"], r["dy"])
    for k in ("dX", "dW"):
        assert maxrel(r[k], ref[k]) <= 2e-2, k


def test_gcn_f32_mfma_mode():
    """GNN_FLAG_F32_MFMA: the fp32 matrix-core products, fp32 tolerance."""
    g = GRAPHS["powerlaw"]
    r = run_gcn(g, 64, 48, 2, True, flags=G.GNN_FLAG_F32_MFMA)
    assert maxrel(r["Y"], r["Y_ref"]) <= TOL
    decision_flips(r["Y"], r["Y_ref"], TOL)
    ref = O.gcn_bwd(g, r["x"], r["w"], r["Y32"], r["dy"], want_db=True)
    for k in ("dX", "dW", "db"):
        assert maxrel(r[k], ref[k]) <= TOL, k


def run_mixhop(g, K, f_in, h, bias, seed=0, pad=8, want_dx=True, flags=0):
    dg = prepared(g)
    c = dg.struct()
    wy = (K + 1) * h
    w, b = _params(f_in, wy, bias, seed)
    x = synth.features(g.n, f_in, seed + 1)
    dy = np.random.default_rng(seed + 2).standard_normal((g.n, wy)).astype(np.float32)
    ld_x, ld_y = f_in + pad, wy + pad
    lay = G.make_layer(f_in, h, ld_x, ld_y, ld_x, 0, flags)
    X, Y = to_dev(x, ld_x), _out(g.n, wy, ld_y)
    W = to_dev(w)
    B = to_dev(b) if bias else None
    saved = _buf(G.gnn_mixhop_saved_bytes(c, lay, K))
    ws = _buf(G.gnn_mixhop_workspace_bytes(c, lay, K))
    G.gnn_mixhop_fwd(c, lay, K, X, W, B, Y, saved, ws)
    torch.cuda.synchronize()
    y_gpu = Y.cpu().numpy()
    y_ref = O.mixhop_fwd(g, x, w, K, b)
    y32 = y_ref.astype(np.float32)
    Y.copy_(torch.from_numpy(y32).cuda())  # the oracle's mask for the backward
    dX = _out(g.n, f_in, ld_x) if want_dx else None
    dW = torch.empty((f_in, wy), device="cuda")
    db = torch.empty(wy, device="cuda") if bias else None
    G.gnn_mixhop_bwd(c, lay, K, X, W, Y, to_dev(dy, ld_y), saved, dX, dW, db, ws)
    torch.cuda.synchronize()
    return dict(x=x, w=w, b=b, dy=dy, Y=y_gpu, Y_ref=y_ref, Y32=y32,
                dX=None if dX is None else dX.cpu().numpy(), dW=dW.cpu().numpy(),
                db=None if db is None else db.cpu().numpy())


@pytest.mark.parametrize("name", list(GRAPHS))
@pytest.mark.parametrize("K", [0, 1, 2, 3, 4])
def test_mixhop_layer_parity(name, K):
    g = GRAPHS[name]
    bias = K % 2 == 1
    r = run_mixhop(g, K, 36, 20, bias, seed=K)
    assert maxrel(r["Y"], r["Y_ref"]) <= TOL
    decision_flips(r["Y"], r["Y_ref"], TOL)
    ref = O.mixhop_bwd(g, r["x"], r["w"], K, r["Y32"], r["dy"], want_db=bias)
    for k in ("dX", "dW") + (("db",) if bias else ()):
        assert maxrel(r[k], ref[k]) <= TOL, (k, K)


def test_mixhop_f32_mfma_mode():
    g = GRAPHS["powerlaw"]
    r = run_mixhop(g, 2, 36, 20, True, seed=4, flags=G.GNN_FLAG_F32_MFMA)
    assert maxrel(r["Y"], r["Y_ref"]) <= TOL
    decision_flips(r["Y"], r["Y_ref"], TOL)
    ref = O.mixhop_bwd(g, r["x"], r["w"], 2, r["Y32"], r["dy"], want_db=True)
    for k in ("dX", "dW", "db"):
        assert maxrel(r[k], ref[k]) <= TOL, k


@pytest.mark.parametrize("K", [2, 4])
def test_mixhop_without_dx_and_unaligned_widths(K):
    """Without dX the last weight-gradient launch's reduction runs on its
    own (K = 4: three launches, each summing its predecessor's tiles)."""
    g = GRAPHS["random"]
    r = run_mixhop(g, K, 13, 7, True, pad=1, want_dx=False)
    assert maxrel(r["Y"], r["Y_ref"]) <= TOL
    decision_flips(r["Y"], r["Y_ref"], TOL)
    ref = O.mixhop_bwd(g, r["x"], r["w"], K, r["Y32"], r["dy"], want_dx=False, want_db=True)
    assert maxrel(r["dW"], ref["dW"]) <= TOL and maxrel(r["db"], ref["db"]) <= TOL


def test_mixhop_full_size_bench_graph():
    wl = synth.WORKLOADS["cl2.1-n8000-f602-h512-L2"]
    g = synth.sym_normalized(synth.workload_graph(wl))
    r = run_mixhop(g, 2, 602, 256, True, pad=6)
    assert maxrel(r["Y"], r["Y_ref"]) <= TOL
    decision_flips(r["Y"], r["Y_ref"], TOL)
    ref = O.mixhop_bwd(g, r["x"], r["w"], 2, r["Y32"], r["dy"], want_db=True)
    for k in ("dX", "dW", "db"):
        assert maxrel(r[k], ref[k]) <= TOL, k


def _random_variant_cases(count=30, seed=808):
    """Seeded random GCN / MixHop layers: graph size and density (uniform or
    power-law), widths, order (GCN) or hop count (MixHop), bias, product
    mode, row-stride padding and, for MixHop, whether dX is wanted."""
    rng = np.random.default_rng(seed)
    modes = [0, G.GNN_FLAG_F32_MFMA, G.GNN_FLAG_BF16]
    cases = []
    for i in range(count):
        cases.append((i, int(rng.integers(1, 1500)), float(rng.uniform(0.5, 20.0)),
                      bool(rng.integers(0, 2)), int(rng.integers(1, 200)),
                      int(rng.integers(1, 160)), int(rng.integers(0, 3)),
                      int(rng.integers(0, 5)), bool(rng.integers(0, 2)), modes[i % 3],
                      int(rng.integers(0, 9)), bool(rng.integers(0, 2))))
    return cases


def _random_graph(i, n, mean, powerlaw):
    if powerlaw and n > 2:
        return synth.sym_normalized(synth.power_law_graph(n, 2.1, min(mean, n - 1.0),
                                                          seed=400 + i))
    return synth.random_graph(n, min(mean, max(n - 1.0, 0.0)), 500 + i,
                              values="sym-normalized")


@pytest.mark.parametrize("case", _random_variant_cases(), ids=lambda c: "case%d" % c[0])
def test_gcn_random_shapes(case):
    i, n, mean, powerlaw, f_in, h, order, _, bias, flags, pad, _ = case
    g = _random_graph(i, n, mean, powerlaw)
    tol = 2e-2 if flags == G.GNN_FLAG_BF16 else TOL
    r = run_gcn(g, f_in, h, order, bias, flags=flags, seed=i, pad=pad)
    assert maxrel(r["Y"], r["Y_ref"]) <= tol
    decision_flips(r["Y"], r["Y_ref"], tol)
    ref = O.gcn_bwd(g, r["x"], r["w"], r["Y32"], r["dy"], want_db=bias)
    for k in ("dX", "dW") + (("db",) if bias else ()):
        assert maxrel(r[k], ref[k]) <= tol, k


@pytest.mark.parametrize("case", _random_variant_cases(seed=909), ids=lambda c: "case%d" % c[0])
def test_mixhop_random_shapes(case):
    i, n, mean, powerlaw, f_in, h, _, K, bias, flags, pad, want_dx = case
    g = _random_graph(i + 1000, n, mean, powerlaw)
    tol = 2e-2 if flags == G.GNN_FLAG_BF16 else TOL
    r = run_mixhop(g, K, f_in, h, bias, seed=i, pad=pad, want_dx=want_dx, flags=flags)
    assert maxrel(r["Y"], r["Y_ref"]) <= tol
    decision_flips(r["Y"], r["Y_ref"], tol)
    ref = O.mixhop_bwd(g, r["x"], r["w"], K, r["Y32"], r["dy"], want_dx=want_dx,
                       want_db=bias)
    for k in (("dX",) if want_dx else ()) + ("dW",) + (("db",) if bias else ()):
        assert maxrel(r[k], ref[k]) <= tol, (k, K)


def test_variant_argument_errors():
    g = GRAPHS["random"]
    dg = prepared(g)
    c = dg.struct()
    lay = G.make_layer(8, 4, 8, 12, 8, 2, 0)
    with pytest.raises(G.GnnError):  # MixHop propagates features first only
        G.gnn_mixhop_fwd(c, lay, 2, None, None, None, None, None, None)
    lay = G.make_layer(8, 4, 8, 4, 8, 0, G.GNN_FLAG_DY_MASKED)
    assert G.gnn_gcn_workspace_bytes(c, lay) == 0  # flag not supported here
