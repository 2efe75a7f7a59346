"""Subgraph preparation on the GPU (induced subgraph of a device-resident
full graph, feature / label gather) against the CPU oracle, through the C
ABI.  Structure (row pointers, column indices) bit-exact; values are the
correctly rounded fp32 of the oracle's double values up to one rounding of
the square root: max relative error 1e-7.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2010_03166_amd import gnnprop as G
from paper_2010_03166_amd import runtime, synth

from gpu_helpers import decision_flips, maxrel, to_dev

pytestmark = pytest.mark.gpu

FULL = {
    "kron12": synth.kronecker_graph(12, 16.0, 1),
    "kron15": synth.kronecker_graph(15, 16.0, 2),
}


def _buf(nbytes):
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device="cuda")


def run_induce(full, nodes, norm, capacity=None, dev=None):
    dev = dev or runtime.FullGraphDevice(full, norm=norm)
    n_s = len(nodes)
    cap = dev.capacity(nodes) if capacity is None else capacity
    nd = torch.from_numpy(np.ascontiguousarray(nodes, np.int32)).cuda() if n_s else \
        torch.empty(1, dtype=torch.int32, device="cuda")
    guard = 64
    ip = torch.full((n_s + 1,), -7, dtype=torch.int32, device="cuda")
    ix = torch.full((cap + guard,), -7, dtype=torch.int32, device="cuda")
    vals = torch.full((cap + guard,), float("nan"), device="cuda")
    nnz = torch.full((1,), -1, dtype=torch.int64, device="cuda")
    st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    ws = _buf(G.gnn_induce_workspace_bytes(n_s))
    G.gnn_induce_subgraph(full.n, full.nnz, dev.indptr, dev.indices, n_s, nd, norm, dev.map,
                          cap, ip, ix, vals, nnz, st, ws)
    torch.cuda.synchronize()
    return dict(indptr=ip.cpu().numpy(), indices=ix.cpu().numpy(), values=vals.cpu().numpy(),
                nnz=int(nnz.item()), status=int(st.item()), cap=cap, guard=guard,
                map=dev.map.cpu().numpy())


def check_parity(full, nodes, norm, r):
    ref = O.induce(full, nodes, norm)
    assert r["status"] == 0
    assert r["nnz"] == ref.nnz
    assert np.array_equal(r["indptr"], ref.indptr)
    assert np.array_equal(r["indices"][: ref.nnz], ref.indices)
    assert maxrel(r["values"][: ref.nnz], ref.values) <= 1e-7
    # nothing written past the entries, the map restored
    assert np.all(r["indices"][ref.nnz:] == -7)
    assert np.all(r["map"] == -1)


def _sets(full, seed):
    rng = np.random.default_rng(seed)
    deg = full.degrees()
    hub = int(np.argmax(deg))
    iso = np.flatnonzero(deg == 0)
    out = {
        "one": np.array([hub], np.int32),
        "two_adjacent": np.sort(np.array([hub, full.indices[full.indptr[hub]]], np.int32)),
        "uniform100": synth.uniform_node_sample(full, 100, rng),
        "uniform3000": synth.uniform_node_sample(full, 3000, rng),
        "hubs_and_isolated": np.unique(np.r_[np.argsort(deg)[-50:],
                                            iso[:20]]).astype(np.int32),
        "all": np.arange(full.n, dtype=np.int32),
    }
    return out


@pytest.mark.parametrize("name", list(FULL))
@pytest.mark.parametrize("norm", [G.GNN_NORM_ROW, G.GNN_NORM_SYM])
def test_induce_parity(name, norm):
    full = FULL[name]
    dev = runtime.FullGraphDevice(full, norm=norm)
    for k, nodes in _sets(full, 3).items():
        if k == "all" and full.n > 5000:
            continue
        r = run_induce(full, nodes, norm, dev=dev)
        check_parity(full, nodes, norm, r)


def _random_induce_cases(count=24, seed=4545):
    """Seeded random inductions: Kronecker full graphs of random scale and
    density, node sets of random size drawn uniformly or in proportion to
    degree, both normalisations."""
    rng = np.random.default_rng(seed)
    return [(i, int(rng.integers(8, 14)), float(rng.uniform(2.0, 24.0)),
             float(rng.uniform(0.0, 1.0)), bool(rng.integers(0, 2)),
             [G.GNN_NORM_ROW, G.GNN_NORM_SYM][int(rng.integers(0, 2))])
            for i in range(count)]


@pytest.mark.parametrize("case", _random_induce_cases(), ids=lambda c: "case%d" % c[0])
def test_induce_random_sets(case):
    i, scale, deg, frac, biased, norm = case
    full = synth.kronecker_graph(scale, deg, 50 + i)
    rng = np.random.default_rng(60 + i)
    size = max(1, int(frac * min(full.n, 5000)))
    if biased and full.nnz > 0:
        p = full.degrees() + 1.0
        nodes = np.unique(rng.choice(full.n, size=size, p=p / p.sum())).astype(np.int32)
    else:
        nodes = np.sort(rng.choice(full.n, size=size, replace=False)).astype(np.int32)
    check_parity(full, nodes, norm, run_induce(full, nodes, norm))


def test_induce_frontier_like_large_set():
    """8,000 nodes drawn with probability proportional to degree (the bias
    of the frontier sampler) from a 2^15-node graph: hub rows spread over
    many workgroups."""
    full = FULL["kron15"]
    rng = np.random.default_rng(5)
    p = full.degrees() / full.degrees().sum()
    nodes = np.unique(rng.choice(full.n, size=9000, p=p)).astype(np.int32)
    r = run_induce(full, nodes, G.GNN_NORM_ROW)
    check_parity(full, nodes, G.GNN_NORM_ROW, r)


def test_induce_empty_and_loop_in_full_graph():
    full = FULL["kron12"]
    r = run_induce(full, np.zeros(0, np.int32), G.GNN_NORM_ROW)
    assert r["status"] == 0 and r["nnz"] == 0 and r["indptr"].tolist() == [0]
    loop = synth.FullGraph(3, np.array([0, 2, 3, 4], np.int64),
                           np.array([0, 1, 0, 2], np.int32))
    nodes = np.array([0, 1, 2], np.int32)
    check_parity(loop, nodes, G.GNN_NORM_ROW, run_induce(loop, nodes, G.GNN_NORM_ROW))


def test_induce_status_flags():
    """Invalid node lists are reported, never read out of bounds: an id past
    the end keeps only its self loop; a capacity below the entry count
    writes nothing past the capacity."""
    full = FULL["kron12"]
    dev = runtime.FullGraphDevice(full)
    nodes = np.array([3, 10, full.n + 5], np.int32)
    cap = int(full.degrees()[[3, 10]].sum()) + 3
    r = run_induce(full, nodes, G.GNN_NORM_ROW, capacity=cap, dev=dev)
    assert r["status"] & 1
    row = r["indices"][r["indptr"][2]: r["indptr"][3]]
    assert row.tolist() == [2]
    assert np.all(r["map"] == -1)
    nodes = synth.uniform_node_sample(full, 500, 1)
    ref = O.induce(full, nodes, 0)
    r = run_induce(full, nodes, G.GNN_NORM_ROW, capacity=ref.nnz - 10, dev=dev)
    assert r["status"] & 4 and r["nnz"] == ref.nnz
    assert np.all(r["indices"][ref.nnz - 10:] == -7)
    assert np.all(r["map"] == -1)
    r = run_induce(full, nodes[::-1].copy(), G.GNN_NORM_ROW, dev=dev)
    assert r["status"] & 2
    assert np.all(r["map"] == -1)


@pytest.mark.parametrize("width,pad", [(602, 6), (41, 0), (50, 3), (1, 0)])
def test_gather_rows_exact(width, pad):
    rng = np.random.default_rng(width)
    src = rng.standard_normal((700, width)).astype(np.float32)
    idx = rng.integers(0, 700, size=333).astype(np.int32)
    idx[5] = 700  # out of range: a row of zeros
    S = to_dev(src, width + pad)
    D = torch.full((333, width + pad), float("nan"), device="cuda")[:, :width]
    G.gnn_gather_rows(333, torch.from_numpy(idx).cuda(), width, S, S.stride(0), 700, D,
                      D.stride(0))
    torch.cuda.synchronize()
    ref = src[np.minimum(idx, 699)]
    ref[5] = 0
    assert np.array_equal(D.cpu().numpy(), ref)


def test_prepared_subgraph_trains_like_oracle():
    """Subgraph built on the GPU from a sampled node list, then one SGD
    iteration of a 2-layer stack with a 7-class head, against the oracle
    on the oracle's own induced subgraph and gathered rows."""
    full = FULL["kron12"]
    rng = np.random.default_rng(11)
    f, C, h = 40, 7, 24
    X = rng.standard_normal((full.n, f)).astype(np.float32)
    Y = synth.labels(full.n, C, False, rng)
    dev = runtime.FullGraphDevice(full, X, Y)
    p = full.degrees() / full.degrees().sum()
    nodes = np.unique(rng.choice(full.n, size=900, p=p)).astype(np.int32)
    dg, Xs, Ts = dev.induce(nodes)
    sub = O.induce(full, nodes, 0)
    assert dg.nnz == sub.nnz
    assert np.array_equal(Xs.cpu().numpy(), X[nodes])
    assert np.array_equal(Ts.cpu().numpy(), Y[nodes])
    params = [synth.LayerParams(synth.glorot(f, h, rng), synth.glorot(f, h, rng)),
              synth.LayerParams(synth.glorot(2 * h, h, rng), synth.glorot(2 * h, h, rng))]
    w_mlp = synth.glorot(2 * h, C, rng)
    tr = runtime.Trainer(dg, params, f, w_mlp, False, "sgd", lr=0.1, keep_xm=True)
    tr.step(Xs, Ts)
    ys = [L["Y"].cpu().numpy() for L in tr.stack.layers]
    xm = tr.xm.cpu().numpy()
    sub.values = sub.values.astype(np.float32).astype(np.float64)
    # the forward layer by layer on the GPU's own layer inputs, and every
    # ReLU decision the oracle is then handed bounded to the kink
    inp = [X[nodes]] + ys[:-1]
    for l, p in enumerate(params):
        y_ref = O.sage_fwd(sub, inp[l], p.w_self, p.w_neigh)
        assert maxrel(ys[l], y_ref) <= 1e-4, l
        decision_flips(ys[l], y_ref, 1e-4)
    xm_ref = np.maximum(O.mm_nn(ys[-1], w_mlp), 0)
    assert maxrel(xm, xm_ref) <= 1e-4
    decision_flips(xm, xm_ref, 1e-4)
    ref = O.train_step(sub, X[nodes], params, w_mlp, Y[nodes], G.GNN_LOSS_SOFTMAX, "sgd",
                       lr=0.0, forced={"ys": ys, "relu_on": xm > 0})
    assert abs(float(tr.loss.item()) - ref["loss"]) <= 1e-5 * ref["loss"]
    for k, (_, gr) in enumerate(tr.pairs):
        assert maxrel(gr, ref["flat_grads"][k]) <= 1e-4, k


def _train_loop(full, X, Y, params, w_mlp, pipelined, iters, m=60, budget=700, seed=9):
    dev = runtime.FullGraphDevice(full, X, Y)
    f, C = X.shape[1], Y.shape[1]
    losses, ids = [], []
    if pipelined:
        pool = G.gnn_sampler_pool(full, m, budget, 2.0, 16, seed, 3, 4)
        pipe = runtime.SubgraphPipeline(dev, pool, max_nodes=budget)
        tr = None
        for _ in range(iters):
            dg, Xs, Ts, sid = pipe.next()
            if tr is None:
                tr = runtime.Trainer(dg, params, f, w_mlp, False, "adam", lr=1e-2)
            else:
                tr.bind(dg)
            tr.step(Xs, Ts)
            losses.append(tr.loss.clone())
            ids.append(sid)
            pipe.release()
        pool.close()
    else:
        tr = None
        for k in range(iters):
            nodes = G.gnn_frontier_sample(full, m, budget, 2.0, 16, seed, k)
            dg, Xs, Ts = dev.induce(nodes)
            if tr is None:
                tr = runtime.Trainer(dg, params, f, w_mlp, False, "adam", lr=1e-2)
            else:
                tr.bind(dg)
            tr.step(Xs, Ts)
            losses.append(tr.loss.clone())
            ids.append(k)
    torch.cuda.synchronize()
    return ids, [float(l.item()) for l in losses], [w.cpu().numpy() for w, _ in tr.pairs]


def test_pipeline_matches_serial_iterations():
    """Six Adam iterations on frontier-sampled subgraphs: the overlapped
    pipeline (host sampler threads, induction on its own stream one subgraph
    ahead) gives bit-for-bit the losses and weights of the serial loop."""
    full = FULL["kron12"]
    rng = np.random.default_rng(21)
    f, C, h = 32, 5, 16
    X = rng.standard_normal((full.n, f)).astype(np.float32)
    Y = synth.labels(full.n, C, False, rng)
    params = [synth.LayerParams(synth.glorot(f, h, rng), synth.glorot(f, h, rng)),
              synth.LayerParams(synth.glorot(2 * h, h, rng), synth.glorot(2 * h, h, rng))]
    w_mlp = synth.glorot(2 * h, C, rng)
    a = _train_loop(full, X, Y, params, w_mlp, True, 6)
    b = _train_loop(full, X, Y, params, w_mlp, False, 6)
    assert a[0] == b[0] == list(range(6))
    assert a[1] == b[1]
    for wa, wb in zip(a[2], b[2]):
        assert np.array_equal(wa, wb)
    # the subgraphs differ in size from one iteration to the next
    sizes = {len(G.gnn_frontier_sample(full, 60, 700, 2.0, 16, 9, k)) for k in range(6)}
    assert len(sizes) > 1
