"""Classifier head, loss, weight updates and the full training iteration on
the GPU against the CPU oracle (through the C ABI).

Tolerances: max |gpu - oracle| / max |oracle| per tensor of 1e-4 in fp32
(2e-2 with bf16 products); the loss, a mean of n positive terms, to 1e-5
relative.  ReLU decisions are the GPU's: a logit or activation that rounding
puts on the other side of 0 flips a whole gradient entry (for a sigmoid head
by (1/2 - t)/n), so the oracle takes the GPU's X_MLP sign and layer outputs
as its decisions (teacher forcing), and the forward values themselves are
compared separately.  Every such decision that differs from the one the
oracle takes on its own must lie at the kink: both values within the
tolerance times the tensor's maximum of 0 (gpu_helpers.decision_flips).  Adam divides by sqrt(v), so its update is likewise
checked on the GPU's own gradients.
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
TOL_LOSS = 1e-5


def _buf(nbytes):
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device="cuda")


def _head_case(n, f, C, multilabel, seed):
    rng = np.random.default_rng(seed)
    x = np.maximum(rng.standard_normal((n, f)), 0).astype(np.float32)  # post-ReLU
    w = synth.glorot(f, C, rng) * 4.0  # logits of order 1
    t = synth.labels(n, C, multilabel, rng)
    return x, w, t


def run_head(x, w, t, kind, flags=0, pad=3, want_probs=True, want_dx=True):
    n, f = x.shape
    C = w.shape[1]
    X, W, T = to_dev(x, f + pad), to_dev(w), to_dev(t, C + pad)
    XM = torch.full((max(n, 1), C + 2), float("nan"), device="cuda")[:n, :C]
    P = torch.full((max(n, 1), C + 1), float("nan"), device="cuda")[:n, :C] \
        if want_probs else None
    dX = torch.full((max(n, 1), f + 5), float("nan"), device="cuda")[:n, :f] \
        if want_dx else None
    loss = torch.full((1,), float("nan"), device="cuda")
    dW = torch.full((f, C), float("nan"), device="cuda")
    ws = _buf(G.gnn_classifier_workspace_bytes(n, f, C))
    G.gnn_classifier(n, f, C, kind, flags, X, X.stride(0) if n else f, W, T,
                     T.stride(0) if n else C, XM, XM.stride(0) if n else C,
                     P, P.stride(0) if P is not None else C,
                     loss, dW, dX, dX.stride(0) if dX is not None else f, ws)
    torch.cuda.synchronize()
    return dict(loss=float(loss.item()), probs=None if P is None else P.cpu().numpy(),
                dW=dW.cpu().numpy(), dX=None if dX is None else dX.cpu().numpy(),
                xm=XM.cpu().numpy())


HEAD_CASES = [  # n, f, C, multilabel
    (1000, 256, 41, False),   # one lane stride of columns
    (777, 100, 121, True),    # two strides, ragged
    (300, 1024, 130, False),  # three strides
    (5, 3, 1, False),         # one class: Y = 1, loss 0
    (1, 7, 64, True),
]


@pytest.mark.parametrize("case", HEAD_CASES, ids=lambda c: "n%d-f%d-C%d-%s" % (
    c[0], c[1], c[2], "sig" if c[3] else "soft"))
def test_classifier_parity(case):
    n, f, C, multi = case
    kind = G.GNN_LOSS_SIGMOID if multi else G.GNN_LOSS_SOFTMAX
    x, w, t = _head_case(n, f, C, multi, seed=n + C)
    r = run_head(x, w, t, kind)
    xm_ref = np.maximum(O.mm_nn(x, w), 0)
    assert maxrel(r["xm"], xm_ref) <= TOL
    decision_flips(r["xm"], xm_ref, TOL)
    ref = O.classifier(x, w, t, kind, relu_on=r["xm"] > 0)
    assert abs(r["loss"] - ref["loss"]) <= TOL_LOSS * max(abs(ref["loss"]), 1e-30) or \
        abs(r["loss"] - ref["loss"]) < 1e-7
    for k in ("probs", "dW", "dX"):
        assert maxrel(r[k], ref[k]) <= TOL, k


def test_classifier_bf16_mode():
    x, w, t = _head_case(2000, 512, 41, False, seed=9)
    r = run_head(x, w, t, G.GNN_LOSS_SOFTMAX, flags=G.GNN_FLAG_BF16)
    xm_ref = np.maximum(O.mm_nn(x, w), 0)
    assert maxrel(r["xm"], xm_ref) <= 2e-2
    decision_flips(r["xm"], xm_ref, 2e-2)
    ref = O.classifier(x, w, t, G.GNN_LOSS_SOFTMAX, relu_on=r["xm"] > 0)
    assert abs(r["loss"] - ref["loss"]) <= 2e-2 * ref["loss"]
    for k in ("probs", "dW", "dX"):
        assert maxrel(r[k], ref[k]) <= 2e-2, k


def test_classifier_f32_mfma_mode():
    x, w, t = _head_case(2000, 512, 41, False, seed=10)
    r = run_head(x, w, t, G.GNN_LOSS_SOFTMAX, flags=G.GNN_FLAG_F32_MFMA)
    xm_ref = np.maximum(O.mm_nn(x, w), 0)
    assert maxrel(r["xm"], xm_ref) <= TOL
    decision_flips(r["xm"], xm_ref, TOL)
    ref = O.classifier(x, w, t, G.GNN_LOSS_SOFTMAX, relu_on=r["xm"] > 0)
    assert abs(r["loss"] - ref["loss"]) <= TOL * ref["loss"]
    for k in ("probs", "dW", "dX"):
        assert maxrel(r[k], ref[k]) <= TOL, k


def test_classifier_optional_outputs_and_empty():
    x, w, t = _head_case(200, 40, 17, True, seed=2)
    r = run_head(x, w, t, G.GNN_LOSS_SIGMOID, want_probs=False, want_dx=False)
    decision_flips(r["xm"], np.maximum(O.mm_nn(x, w), 0), TOL)
    ref = O.classifier(x, w, t, G.GNN_LOSS_SIGMOID, want_dx=False, relu_on=r["xm"] > 0)
    assert maxrel(r["dW"], ref["dW"]) <= TOL
    assert abs(r["loss"] - ref["loss"]) <= TOL_LOSS * ref["loss"]
    # no rows: loss 0, zero weight gradient
    e = run_head(np.zeros((0, 40), np.float32), w, np.zeros((0, 17), np.float32),
                 G.GNN_LOSS_SOFTMAX)
    assert e["loss"] == 0.0 and np.all(e["dW"] == 0)


def _random_head_cases(count=30, seed=3131):
    """Seeded random classifier heads: rows, features, classes, softmax or
    sigmoid, product mode, row-stride padding, optional outputs."""
    rng = np.random.default_rng(seed)
    modes = [0, G.GNN_FLAG_F32_MFMA, G.GNN_FLAG_BF16]
    return [(i, int(rng.integers(1, 2500)), int(rng.integers(1, 600)),
             int(rng.integers(1, 200)), bool(rng.integers(0, 2)), modes[i % 3],
             int(rng.integers(0, 6)), bool(rng.integers(0, 2)), bool(rng.integers(0, 2)))
            for i in range(count)]


@pytest.mark.parametrize("case", _random_head_cases(), ids=lambda c: "case%d" % c[0])
def test_classifier_random_shapes(case):
    i, n, f, C, multi, flags, pad, want_probs, want_dx = case
    kind = G.GNN_LOSS_SIGMOID if multi else G.GNN_LOSS_SOFTMAX
    tol = 2e-2 if flags == G.GNN_FLAG_BF16 else TOL
    x, w, t = _head_case(n, f, C, multi, seed=900 + i)
    r = run_head(x, w, t, kind, flags=flags, pad=pad, want_probs=want_probs,
                 want_dx=want_dx)
    xm_ref = np.maximum(O.mm_nn(x, w), 0)
    assert maxrel(r["xm"], xm_ref) <= tol
    decision_flips(r["xm"], xm_ref, tol)
    ref = O.classifier(x, w, t, kind, want_dx=want_dx, relu_on=r["xm"] > 0)
    loss_tol = 2e-2 if flags == G.GNN_FLAG_BF16 else TOL_LOSS
    assert abs(r["loss"] - ref["loss"]) <= loss_tol * abs(ref["loss"]) or \
        abs(r["loss"] - ref["loss"]) < 1e-7
    keys = ("dW",) + (("probs",) if want_probs else ()) + (("dX",) if want_dx else ())
    for k in keys:
        assert maxrel(r[k], ref[k]) <= tol, k


def test_classifier_deterministic():
    x, w, t = _head_case(5000, 128, 41, False, seed=4)
    a = run_head(x, w, t, G.GNN_LOSS_SOFTMAX)
    b = run_head(x, w, t, G.GNN_LOSS_SOFTMAX)
    assert a["loss"] == b["loss"]
    for k in ("probs", "dW", "dX"):
        assert np.array_equal(a[k], b[k]), k


def test_classifier_argument_errors():
    n, f, C = 8, 4, 3
    X, W = torch.zeros((n, f), device="cuda"), torch.zeros((f, C), device="cuda")
    T, loss = torch.zeros((n, C), device="cuda"), torch.zeros(1, device="cuda")
    dW = torch.zeros((f, C), device="cuda")
    ws = _buf(G.gnn_classifier_workspace_bytes(n, f, C))
    with pytest.raises(G.GnnError):  # unknown loss
        G.gnn_classifier(n, f, C, 7, 0, X, f, W, T, C, None, C, None, C, loss, dW, None, f,
                         ws)
    with pytest.raises(G.GnnError):  # row stride below the width
        G.gnn_classifier(n, f, C, 0, 0, X, f - 1, W, T, C, None, C, None, C, loss, dW, None,
                         f, ws)
    with pytest.raises(G.GnnError):  # workspace too small
        G.gnn_classifier(n, f, C, 0, 0, X, f, W, T, C, None, C, None, C, loss, dW, None, f,
                         _buf(0)[:8])
    with pytest.raises(G.GnnError):  # output aliases an input
        G.gnn_classifier(n, f, C, 0, 0, X, f, W, T, C, None, C, None, C, loss, W, None, f, ws)
    with pytest.raises(G.GnnError):  # two outputs overlap
        G.gnn_classifier(n, f, C, 0, 0, X, f, W, T, C, dW, C, None, C, loss, dW, None, f, ws)
    with pytest.raises(G.GnnError):  # Adam step counts from 1
        G.gnn_adam_step(4, dW, W, T, X, 0.1, 0.9, 0.999, 1e-8, 0)


@pytest.mark.parametrize("count", [1, 1000, 3_000_001])
def test_sgd_adam_parity(count):
    rng = np.random.default_rng(count)
    w0 = rng.standard_normal(count).astype(np.float32)
    W, Wa = to_dev(w0), to_dev(w0)
    m, v = torch.zeros(count, device="cuda"), torch.zeros(count, device="cuda")
    wr, wa = w0.astype(np.float64), w0.astype(np.float64)
    mr, vr = np.zeros(count), np.zeros(count)
    for step in range(1, 4):
        gr = (rng.standard_normal(count) * 10.0 ** -step).astype(np.float32)
        Gd = to_dev(gr)
        G.gnn_sgd_step(count, W, Gd, 0.05)
        G.gnn_adam_step(count, Wa, Gd, m, v, 1e-3, 0.9, 0.999, 1e-8, step)
        wr = O.sgd(wr, gr, 0.05)
        wa, mr, vr = O.adam(wa, gr, mr, vr, 1e-3, 0.9, 0.999, 1e-8, step)
    torch.cuda.synchronize()
    assert maxrel(W, wr) <= 1e-6
    assert maxrel(Wa, wa) <= 1e-6
    assert maxrel(m, mr) <= 1e-6 and maxrel(v, vr) <= 1e-5


# ---------------------------------------------------------- full iteration

def _trainer_inputs(wl, bias):
    d = synth.workload_inputs(wl, bias=bias)
    c = synth.classifier_inputs(wl)
    return d["graph"], d["x"], d["params"], c["w_mlp"], c["targets"]


def _gpu_grads(tr):
    return [gr.cpu().numpy() for _, gr in tr.pairs]


def _gpu_weights(tr):
    return [w.cpu().numpy() for w, _ in tr.pairs]


def _params_from(flat, nlayers, bias):
    """Per-layer parameters from the flat [W_MLP, W_self, W_neigh (, b...)]."""
    per = 4 if bias else 2
    return flat[0], [synth.LayerParams(*flat[1 + per * l: 1 + per * (l + 1)])
                     for l in range(nlayers)]


def check_iteration(tr, g, x, t, kind, tol, before=None, rows=None):
    """After tr.step(): the forward layer by layer against the oracle on the
    GPU's own layer inputs, then loss, probabilities and every gradient
    against the oracle's iteration with the GPU's ReLU decisions.  Returns
    the oracle's result.  before: the flat weights the step started from
    (default: the trainer's construction weights must be passed)."""
    nl = len(tr.stack.layers)
    bias = tr.stack.layers[0]["b_self"] is not None
    w_mlp, params = _params_from(before, nl, bias)
    ys = [L["Y"].cpu().numpy() for L in tr.stack.layers]
    inp = [x] + ys[:-1]
    for l, p in enumerate(params):
        if rows is None:
            ref = O.sage_fwd(g, inp[l], p.w_self, p.w_neigh, p.b_self, p.b_neigh)
            assert maxrel(ys[l], ref) <= tol, ("Y", l)
            decision_flips(ys[l], ref, tol)
        else:
            ref = O.sage_fwd_rows(g, inp[l], p.w_self, p.w_neigh, rows, p.b_self, p.b_neigh)
            assert maxrel(ys[l][rows], ref) <= tol, ("Y", l)
            decision_flips(ys[l][rows], ref, tol)
    xm = tr.xm.cpu().numpy()
    xm_ref = np.maximum(O.mm_nn(ys[-1], w_mlp), 0)
    assert maxrel(xm, xm_ref) <= tol
    decision_flips(xm, xm_ref, tol)
    ref = O.train_step(g, x, params, w_mlp, t, kind, "sgd", lr=0.0,
                       forced={"ys": ys, "relu_on": xm > 0})
    loss = float(tr.loss.item())
    assert abs(loss - ref["loss"]) <= max(TOL_LOSS, tol / 10) * ref["loss"]
    if tr.probs is not None:
        assert maxrel(tr.probs, ref["probs"]) <= tol
    for k, (a, b) in enumerate(zip(_gpu_grads(tr), ref["flat_grads"])):
        assert maxrel(a, b) <= tol, ("grad", k)
    return ref


@pytest.mark.parametrize("multilabel", [False, True])
@pytest.mark.parametrize("bias", [False, True])
def test_train_iteration_sgd_tiny(multilabel, bias):
    """Two SGD iterations of the 1,000-node workload (softmax or sigmoid
    head); each checked on its own inputs, the update exactly as SGD
    defines it on the GPU's gradients."""
    wl = synth.WORKLOADS[synth.TINY_WORKLOAD]
    g, x, params, w_mlp, t = _trainer_inputs(wl, bias)
    kind = G.GNN_LOSS_SIGMOID if multilabel else G.GNN_LOSS_SOFTMAX
    if multilabel != wl.multilabel:
        t = synth.labels(g.n, wl.classes, multilabel, np.random.default_rng(3))
    tr = runtime.Trainer(prepared(g), params, wl.f_in, w_mlp, multilabel, "sgd", lr=0.05,
                         want_probs=True, keep_xm=True)
    X, T = to_dev(x, wl.f_in + 14), to_dev(t)
    for it in range(2):
        before = _gpu_weights(tr)
        tr.step(X, T)
        check_iteration(tr, g, x, t, kind, TOL, before)
        for k, (w0, gr, w1) in enumerate(zip(before, _gpu_grads(tr), _gpu_weights(tr))):
            assert maxrel(w1, O.sgd(w0, gr, 0.05)) <= 1e-6, (it, k)


def test_train_iteration_adam_tiny():
    """Three Adam iterations: each iteration's gradients against the oracle,
    the update against the oracle's Adam on the GPU's gradients."""
    wl = synth.WORKLOADS[synth.TINY_WORKLOAD]
    g, x, params, w_mlp, t = _trainer_inputs(wl, True)
    tr = runtime.Trainer(prepared(g), params, wl.f_in, w_mlp, wl.multilabel, "adam",
                         lr=1e-3, keep_xm=True)
    X, T = to_dev(x), to_dev(t)
    state = [(np.zeros(w.shape), np.zeros(w.shape)) for w, _ in tr.pairs]
    for it in range(1, 4):
        before = _gpu_weights(tr)
        tr.step(X, T)
        check_iteration(tr, g, x, t, G.GNN_LOSS_SIGMOID, TOL, before)
        grads = _gpu_grads(tr)
        for k, (w0, gr, w1) in enumerate(zip(before, grads, _gpu_weights(tr))):
            m, v = state[k]
            wr, m, v = O.adam(w0, gr, m, v, 1e-3, 0.9, 0.999, 1e-8, it)
            state[k] = (m, v)
            assert maxrel(w1, wr) <= 1e-6, (it, k)
        for k, (m, v) in enumerate(tr.state):
            assert maxrel(m, state[k][0]) <= 1e-6 and maxrel(v, state[k][1]) <= 1e-6, (it, k)


def test_train_iteration_full_size_bench_workload():
    """One Adam iteration of the 8,000-node, 602-feature workload with its
    41-class softmax head (the benchmark's iteration), every gradient
    against the oracle's; the forward on sampled rows."""
    wl = synth.WORKLOADS[synth.BENCH_WORKLOAD]
    g, x, params, w_mlp, t = _trainer_inputs(wl, False)
    tr = runtime.Trainer(prepared(g), params, wl.f_in, w_mlp, wl.multilabel, "adam",
                         lr=1e-3, keep_xm=True)
    before = _gpu_weights(tr)
    tr.step(to_dev(x, 608), to_dev(t))
    rows = np.unique(np.r_[0, g.n - 1, int(np.argmax(g.degrees())),
                           np.random.default_rng(0).choice(g.n, 40, replace=False)])
    check_iteration(tr, g, x, t, G.GNN_LOSS_SOFTMAX, TOL, before, rows=rows)


def test_train_iteration_bf16_mode():
    wl = synth.WORKLOADS[synth.TINY_WORKLOAD]
    g, x, params, w_mlp, t = _trainer_inputs(wl, False)
    tr = runtime.Trainer(prepared(g), params, wl.f_in, w_mlp, wl.multilabel, "sgd", lr=0.05,
                         flags=G.GNN_FLAG_BF16, keep_xm=True)
    before = _gpu_weights(tr)
    tr.step(to_dev(x), to_dev(t))
    check_iteration(tr, g, x, t, G.GNN_LOSS_SIGMOID, 2e-2, before)
def test_trainer_graph_replay():
    """The iteration captured in a HIP graph and replayed matches the same
    iterations run eagerly (every replay checked)."""
    wl = synth.WORKLOADS[synth.TINY_WORKLOAD]
    g, x, params, w_mlp, t = _trainer_inputs(wl, False)
    dg = prepared(g)
    X, T = to_dev(x), to_dev(t)
    # the Adam step count is a host argument of its launch, so a captured
    # iteration replays one fixed t; the captured trainer here uses SGD
    cap = runtime.Trainer(dg, params, wl.f_in, w_mlp, wl.multilabel, "sgd", lr=1e-3)
    eager = runtime.Trainer(dg, params, wl.f_in, w_mlp, wl.multilabel, "sgd", lr=1e-3)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        cap.step(X, T, stream=s.cuda_stream)  # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    eager.step(X, T)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        cap.step(X, T, stream=s.cuda_stream)
    for it in range(3):
        graph.replay()
        torch.cuda.synchronize()
        eager.step(X, T)
        torch.cuda.synchronize()
        assert float(cap.loss.item()) == float(eager.loss.item()), it
        for a, b in zip(_gpu_weights(cap), _gpu_weights(eager)):
            assert np.array_equal(a, b), it
