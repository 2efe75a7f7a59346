"""Whole-tensor parity of chained GraphSAGE stacks at full size.

The 8,000-node workloads (2 layers of 602 -> 2 x 512, 3 layers of 300 ->
2 x 512) and the 20,000-node deep one (5 layers of 200 -> 2 x 512) run
through the C ABI exactly as the benchmark chains them (Algorithm 1's layer
loop: forward l = 1..L, backward l = L..1 with each layer's dX as the dY of
the layer below, the first layer's dX included), and every element of every
layer's Y, dX, dW_self and dW_neigh (and db with biases) is compared with
the double-precision oracle:

  - forward: the GPU chain runs free (each layer takes the GPU's own output
    of the layer below); the oracle chain carries fp32 activations between
    layers.  Y must match to max |gpu - oracle| / max |oracle| <= 1e-4 per
    tensor (2e-2 with bf16 products), and every ReLU decision the GPU takes
    differently from the oracle must lie at the kink (both values within the
    tolerance times max |Y| of 0); the number of such flips is reported;
  - backward: teacher-forced per layer (Section 5.1's gradient equations
    read the forward's Y through the mask): the oracle's fp32 layer outputs
    are written into the GPU stack's Y buffers, which are also the inputs of
    the layers above, so both sides take the same masks; the gradient chain
    runs on the GPU.  dX, dW_self, dW_neigh (and db) to the same tolerance.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2010_03166_amd import gnnprop as G
from paper_2010_03166_amd import runtime, synth

from gpu_helpers import decision_flips, maxrel, prepared, to_dev

pytestmark = pytest.mark.gpu

STACKS = ["cl2.1-n8000-f602-h512-L2", "cl2.3-n8000-f300-h512-L3",
          "cl2.1-n20000-f200-h512-L5"]
MODES = {"split": (0, 1e-4), "f32_mfma": (G.GNN_FLAG_F32_MFMA, 1e-4),
         "bf16": (G.GNN_FLAG_BF16, 2e-2)}

_CACHE = {}


def oracle_chain(name, bias):
    """Inputs of the workload and the oracle's chained stack: fp32 layer
    inputs xs[0..L] (xs[l+1] = fp32 of layer l+1's double output ys[l]),
    and the backward from the workload's top dY with those fp32 inputs and
    outputs, the gradients chained in double."""
    key = (name, bias)
    if key in _CACHE:
        return _CACHE[key]
    _CACHE.clear()  # one workload's arrays at a time (the deep stack's are large)
    wl = synth.WORKLOADS[name]
    inp = synth.workload_inputs(wl, bias=bias)
    g, x, params, dy = inp["graph"], inp["x"], inp["params"], inp["dy"]
    xs, ys = [x], []
    for p in params:
        y = O.sage_fwd(g, xs[-1], p.w_self, p.w_neigh, p.b_self, p.b_neigh)
        ys.append(y)
        xs.append(y.astype(np.float32))
    grads = [None] * len(params)
    d = dy.astype(np.float64)
    for l in reversed(range(len(params))):
        p = params[l]
        r = O.sage_bwd(g, xs[l], p.w_self, p.w_neigh, xs[l + 1], d, want_dx=True,
                       want_db=bias)
        grads[l] = r
        d = r["dX"]
    out = {"wl": wl, "graph": g, "x": x, "params": params, "dy": dy, "xs": xs,
           "ys": ys, "grads": grads}
    _CACHE[key] = out
    return out


def run_and_check(name, mode, bias=False):
    ref = oracle_chain(name, bias)
    wl, g, params = ref["wl"], ref["graph"], ref["params"]
    flags, tol = MODES[mode]
    dg = prepared(g)
    st = runtime.SageStack(dg, params, wl.f_in, flags=flags)
    ld_x = (wl.f_in + 15) // 16 * 16
    st.forward(runtime.padded(torch.from_numpy(ref["x"]).cuda(), ld_x))
    torch.cuda.synchronize()
    flips = []
    for l, L in enumerate(st.layers):
        y = L["Y"].cpu().numpy()
        assert maxrel(y, ref["ys"][l]) <= tol, (name, mode, "Y", l, maxrel(y, ref["ys"][l]))
        flips.append(decision_flips(y, ref["ys"][l], bound=tol))
    print("%s %s: ReLU decisions flipped per layer %s of %d each"
          % (name, mode, flips, g.n * 2 * wl.hidden))
    # teacher forcing: the oracle's fp32 outputs become the masks and the
    # inputs of the layers above
    for l, L in enumerate(st.layers):
        L["Y"].copy_(torch.from_numpy(ref["xs"][l + 1]).cuda())
    st.backward(to_dev(ref["dy"]), want_dx_first=True)
    torch.cuda.synchronize()
    keys = ("dX", "dW_self", "dW_neigh") + (("db_self", "db_neigh") if bias else ())
    worst = {}
    for l, L in enumerate(st.layers):
        R = ref["grads"][l]
        for k in keys:
            e = maxrel(L[k].cpu().numpy(), R[k])
            worst[k] = max(worst.get(k, 0.0), e)
            assert e <= tol, (name, mode, k, l, e)
    print("%s %s: worst max-normalised error over the layers %s"
          % (name, mode, {k: "%.2e" % v for k, v in worst.items()}))
    del st
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("name", STACKS)
def test_stack_whole_tensors(name, mode):
    run_and_check(name, mode)


@pytest.mark.parametrize("mode", ["split", "f32_mfma"])
def test_stack_whole_tensors_with_bias(mode):
    """The 3-layer 8,000-node stack with per-half biases: db_self and
    db_neigh of every layer as well."""
    run_and_check("cl2.3-n8000-f300-h512-L3", mode, bias=True)


def _random_stack_cases(count=16, seed=6060):
    """Seeded random small stacks: 2 to 5 layers with random widths per
    layer, product mode, bias, and the cross-layer mask fusion on or off."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(count):
        L = int(rng.integers(2, 6))
        cases.append((i, int(rng.integers(2, 1500)), int(rng.integers(1, 200)),
                      [int(rng.integers(1, 128)) for _ in range(L)], list(MODES)[i % 3],
                      bool(rng.integers(0, 2)), bool(rng.integers(0, 2))))
    return cases


@pytest.mark.parametrize("case", _random_stack_cases(), ids=lambda c: "case%d" % c[0])
def test_stack_random_shapes(case):
    """Chained stacks of random shapes, checked the same way as the full-size
    ones (forward free, backward teacher-forced from the oracle's fp32 layer
    outputs, every element of every layer); with the mask fusion, dX of the
    layers above the first comes back masked by the sign of their input."""
    i, n, f_in, hs, mode, bias, fuse = case
    flags, tol = MODES[mode]
    rng = np.random.default_rng(7000 + i)
    g = synth.power_law_graph(n, 2.1, min(10.0, n - 1.0), seed=7100 + i)
    x = rng.standard_normal((n, f_in)).astype(np.float32)
    params, f = [], f_in
    for h in hs:
        p = synth.LayerParams(synth.glorot(f, h, rng), synth.glorot(f, h, rng))
        if bias:
            p.b_self = (0.1 * rng.standard_normal(h)).astype(np.float32)
            p.b_neigh = (0.1 * rng.standard_normal(h)).astype(np.float32)
        params.append(p)
        f = 2 * h
    dy = rng.standard_normal((n, f)).astype(np.float32)
    xs, ys = [x], []
    for p in params:
        y = O.sage_fwd(g, xs[-1], p.w_self, p.w_neigh, p.b_self, p.b_neigh)
        ys.append(y)
        xs.append(y.astype(np.float32))
    grads = [None] * len(params)
    d = dy.astype(np.float64)
    for l in reversed(range(len(params))):
        p = params[l]
        grads[l] = O.sage_bwd(g, xs[l], p.w_self, p.w_neigh, xs[l + 1], d, want_dx=True,
                              want_db=bias)
        d = grads[l]["dX"]
    st = runtime.SageStack(prepared(g), params, f_in, flags=flags, fuse_masks=fuse)
    st.forward(to_dev(x, (f_in + 15) // 16 * 16))
    torch.cuda.synchronize()
    for l, L in enumerate(st.layers):
        y = L["Y"].cpu().numpy()
        assert maxrel(y, ys[l]) <= tol, ("Y", l)
        decision_flips(y, ys[l], bound=tol)
    for l, L in enumerate(st.layers):
        L["Y"].copy_(torch.from_numpy(xs[l + 1]).cuda())
    st.backward(to_dev(dy), want_dx_first=True)
    torch.cuda.synchronize()
    keys = ("dX", "dW_self", "dW_neigh") + (("db_self", "db_neigh") if bias else ())
    for l, L in enumerate(st.layers):
        for k in keys:
            ref = grads[l][k]
            if k == "dX" and fuse and l > 0:
                ref = ref * (xs[l] > 0)
            assert maxrel(L[k].cpu().numpy(), ref) <= tol, (k, l)
