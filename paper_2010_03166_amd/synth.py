"""Seeded synthetic inputs for the GraphSAGE feature-propagation path.

This module builds the *inputs* of one sampled-subgraph training step and
nothing else: a CSR adjacency with a symmetric, row-sorted pattern and self
loops, the row-normalised values D^-1 A of that pattern (the subgraph
adjacency the paper feeds to each layer, Section 2.1, Eq. "graphsage
forward"), node features, Glorot weights and a random upstream gradient.
It holds none of the layer arithmetic (aggregation, transforms, activation,
gradients) and is shared, as plain numpy arrays, by the CPU oracle tests and
the GPU path alike.

Workload shapes stand in for frontier-sampled subgraphs of the paper's
datasets (Table 2 feature widths 50/602/300/200; subgraph budget n = 8000,
Section 7.5; sampled-graph degree d ~ 15, Section 5.3).  Degrees follow a
Chung-Lu power law; the tiny case is an Erdos-Renyi graph.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np

# Random streams (SeedSequence([case, stream])).
STREAM_GRAPH = 0
STREAM_X = 1
STREAM_DY = 99
STREAM_LABELS = 98
STREAM_W_MLP = 97
STREAM_W0 = 10  # + layer index


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic subgraph-training workload."""
    name: str
    case: int             # seed namespace
    n: int                # subgraph nodes
    graph: str            # "er" or "chung-lu"
    mean_deg: float       # mean degree without the self loop
    gamma: float = 0.0    # power-law tail exponent (chung-lu)
    kmax: Optional[float] = None  # cap on expected degree (None: n-1)
    f_in: int = 50        # input feature width
    layers: int = 2
    hidden: int = 128     # width of each concat half
    classes: int = 2      # C: columns of the classifier output
    multilabel: bool = False  # sigmoid + per-class CE, else softmax + CE


WORKLOADS: Dict[str, Workload] = {w.name: w for w in [
    Workload("er-n1000-f50-h128-L2", 0, 1000, "er", 10.0,
             f_in=50, layers=2, hidden=128, classes=121, multilabel=True),
    Workload("cl2.1-n8000-f602-h512-L2", 1, 8000, "chung-lu", 15.0,
             gamma=2.1, kmax=1000.0, f_in=602, layers=2, hidden=512, classes=41),
    Workload("cl2.3-n8000-f300-h512-L3", 2, 8000, "chung-lu", 20.0,
             gamma=2.3, f_in=300, layers=3, hidden=512, classes=100, multilabel=True),
    Workload("cl2.1-n20000-f200-h512-L5", 3, 20000, "chung-lu", 30.0,
             gamma=2.1, f_in=200, layers=5, hidden=512, classes=107, multilabel=True),
    Workload("cl1.9-n50000-f256-h1024-L3", 4, 50000, "chung-lu", 40.0,
             gamma=1.9, kmax=5000.0, f_in=256, layers=3, hidden=1024, classes=107,
             multilabel=True),
]}
# Classes follow the paper's dataset table for the feature width each
# workload copies (50: 121 labels, 602: 41 classes, 300: 100 labels, 200: 107
# labels); the 256-wide one takes 107 labels.

# The workload the benchmark times and the small one the oracle finishes fast.
BENCH_WORKLOAD = "cl2.1-n8000-f602-h512-L2"
TINY_WORKLOAD = "er-n1000-f50-h128-L2"


def rng_for(case: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([case, stream]))


# ---------------------------------------------------------------- CSR build

@dataclasses.dataclass
class Csr:
    n: int
    indptr: np.ndarray    # int32 [n+1]
    indices: np.ndarray   # int32 [nnz], ascending within each row
    values: np.ndarray    # float32 [nnz]

    @property
    def nnz(self) -> int:
        return int(self.indices.shape[0])

    def degrees(self) -> np.ndarray:
        return np.diff(self.indptr.astype(np.int64))

    def stats(self) -> dict:
        d = self.degrees()
        return {"n": self.n, "nnz": self.nnz,
                "mean_deg": float(d.mean()) if self.n else 0.0,
                "max_deg": int(d.max()) if self.n else 0,
                "rows_deg_le4": int((d <= 4).sum()),
                "rows_deg_ge256": int((d >= 256).sum())}


def csr_from_pairs(n: int, rows: np.ndarray, cols: np.ndarray,
                   values: Optional[np.ndarray] = None) -> Csr:
    """Sort (row, col[, value]) triples into CSR with ascending columns.

    Duplicate (row, col) pairs are not merged; callers pass unique pairs.
    If `values` is None the binary pattern is row-normalised (1/deg).
    """
    rows = np.asarray(rows, dtype=np.int64)
    cols = np.asarray(cols, dtype=np.int64)
    key = rows * max(n, 1) + cols
    order = np.argsort(key, kind="stable")
    rows, cols = rows[order], cols[order]
    counts = np.bincount(rows, minlength=n) if n else np.zeros(0, np.int64)
    indptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(counts, out=indptr[1:])
    if values is None:
        deg = counts.astype(np.float64)
        vals = (1.0 / deg[rows]).astype(np.float32) if rows.size else \
            np.zeros(0, np.float32)
    else:
        vals = np.asarray(values, dtype=np.float32)[order]
    return Csr(n, indptr.astype(np.int32), cols.astype(np.int32), vals)


def symmetric_csr(n: int, edges: np.ndarray, self_loops: bool = True,
                  values: str = "row-normalized",
                  rng: Optional[np.random.Generator] = None) -> Csr:
    """Undirected graph from unique edges (u != v) -> symmetric CSR.

    values: "row-normalized" (1/deg, deg counting the self loop),
            "sym-normalized" (1/sqrt(deg_u deg_v), the symmetric
            normalisation a GCN or MixHop layer aggregates with; with the
            self loops this is (I + D)^-1/2 (I + A) (I + D)^-1/2),
            "ones", or "random" (independent N(0,1) per stored entry, a
            pattern-symmetric but value-asymmetric matrix for tests).
    """
    edges = np.asarray(edges, dtype=np.int64).reshape(-1, 2)
    r = [edges[:, 0], edges[:, 1]]
    c = [edges[:, 1], edges[:, 0]]
    if self_loops:
        ar = np.arange(n, dtype=np.int64)
        r.append(ar)
        c.append(ar)
    rows = np.concatenate(r) if r else np.zeros(0, np.int64)
    cols = np.concatenate(c) if c else np.zeros(0, np.int64)
    if values == "row-normalized":
        return csr_from_pairs(n, rows, cols, None)
    if values == "sym-normalized":
        return sym_normalized(csr_from_pairs(n, rows, cols, None))
    if values == "ones":
        return csr_from_pairs(n, rows, cols, np.ones(rows.size, np.float32))
    if values == "random":
        rng = rng or np.random.default_rng(0)
        return csr_from_pairs(n, rows, cols,
                              rng.standard_normal(rows.size).astype(np.float32))
    raise ValueError(values)


def sym_normalized(g: Csr) -> Csr:
    """The same pattern with values 1/sqrt(deg_u deg_v) (deg = stored
    entries of the row, self loop included)."""
    deg = g.degrees().astype(np.float64)
    rows = np.repeat(np.arange(g.n), g.degrees())
    cols = g.indices.astype(np.int64)
    vals = (1.0 / np.sqrt(deg[rows] * deg[cols])).astype(np.float32) if g.nnz else \
        np.zeros(0, np.float32)
    return Csr(g.n, g.indptr.copy(), g.indices.copy(), vals)


# ------------------------------------------------------------- graph models

def er_edges(n: int, mean_deg: float, rng: np.random.Generator) -> np.ndarray:
    """G(n, p) with p = mean_deg/(n-1) over the upper triangle."""
    if n < 2:
        return np.zeros((0, 2), np.int64)
    p = mean_deg / (n - 1)
    iu, ju = np.triu_indices(n, 1)
    keep = rng.random(iu.size) < p
    return np.stack([iu[keep], ju[keep]], axis=1).astype(np.int64)


def chung_lu_weights(n: int, gamma: float, mean_deg: float,
                     kmax: Optional[float]) -> np.ndarray:
    """Expected degrees w_i = c (i+1)^(-1/(gamma-1)), capped at kmax, with c
    chosen by bisection so that mean(w) = mean_deg."""
    kmax = float(n - 1) if kmax is None else float(kmax)
    base = np.arange(1, n + 1, dtype=np.float64) ** (-1.0 / (gamma - 1.0))
    lo, hi = 0.0, kmax / base[-1] + 1.0
    for _ in range(200):
        c = 0.5 * (lo + hi)
        m = np.minimum(c * base, kmax).mean()
        if m < mean_deg:
            lo = c
        else:
            hi = c
    return np.minimum(0.5 * (lo + hi) * base, kmax)


def chung_lu_edges(n: int, gamma: float, mean_deg: float,
                   kmax: Optional[float], rng: np.random.Generator) -> np.ndarray:
    """round(n*mean/2) distinct undirected non-loop edges (at most all
    n(n-1)/2 of them, for tiny n), both endpoints drawn independently with
    probability proportional to the weights; the first distinct pairs in
    draw order are kept."""
    target = min(int(round(n * mean_deg / 2.0)), n * (n - 1) // 2)
    w = chung_lu_weights(n, gamma, mean_deg, kmax)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    kept = np.zeros(0, np.int64)
    while kept.size < target:
        m = int((target - kept.size) * 1.3) + 4096
        u = rng.random(2 * m)
        idx = np.minimum(np.searchsorted(cdf, u, side="right"), n - 1)
        a, b = idx[:m], idx[m:]
        ok = a != b
        key = np.minimum(a, b)[ok] * n + np.maximum(a, b)[ok]
        allk = np.concatenate([kept, key])
        _, first = np.unique(allk, return_index=True)
        first.sort()
        kept = allk[first]
    kept = kept[:target]
    return np.stack([kept // n, kept % n], axis=1)


def workload_graph(wl: Workload) -> Csr:
    rng = rng_for(wl.case, STREAM_GRAPH)
    if wl.graph == "er":
        e = er_edges(wl.n, wl.mean_deg, rng)
    elif wl.graph == "chung-lu":
        e = chung_lu_edges(wl.n, wl.gamma, wl.mean_deg, wl.kmax, rng)
    else:
        raise ValueError(wl.graph)
    return symmetric_csr(wl.n, e, self_loops=True)


# ------------------------------------------------------- small test graphs

def star_graph(k: int, self_loops: bool = True) -> Csr:
    """Centre 0 joined to leaves 1..k."""
    e = np.stack([np.zeros(k, np.int64), np.arange(1, k + 1)], axis=1)
    return symmetric_csr(k + 1, e, self_loops)


def complete_graph(n: int, self_loops: bool = True) -> Csr:
    iu, ju = np.triu_indices(n, 1)
    return symmetric_csr(n, np.stack([iu, ju], axis=1), self_loops)


def identity_graph(n: int) -> Csr:
    return symmetric_csr(n, np.zeros((0, 2), np.int64), self_loops=True)


def path_graph(n: int, self_loops: bool = True) -> Csr:
    e = np.stack([np.arange(n - 1), np.arange(1, n)], axis=1)
    return symmetric_csr(n, e, self_loops)


def random_graph(n: int, mean_deg: float, seed: int, self_loops: bool = True,
                 values: str = "row-normalized") -> Csr:
    rng = np.random.default_rng(seed)
    e = er_edges(n, mean_deg, rng)
    return symmetric_csr(n, e, self_loops, values, rng)


def power_law_graph(n: int, gamma: float, mean_deg: float, seed: int,
                    kmax: Optional[float] = None) -> Csr:
    rng = np.random.default_rng(seed)
    return symmetric_csr(n, chung_lu_edges(n, gamma, mean_deg, kmax, rng))


# ------------------------------------------------------- dense layer inputs

def features(n: int, f: int, seed_or_rng, ld: Optional[int] = None) -> np.ndarray:
    """N(0,1) float32 features, shape (n, f); with ld > f the array is an
    (n, ld) buffer whose trailing columns are NaN padding (never read)."""
    rng = seed_or_rng if isinstance(seed_or_rng, np.random.Generator) else \
        np.random.default_rng(seed_or_rng)
    x = rng.standard_normal((n, f)).astype(np.float32)
    if ld is None or ld == f:
        return x
    buf = np.full((n, ld), np.nan, np.float32)
    buf[:, :f] = x
    return buf


def glorot(f_in: int, h: int, rng: np.random.Generator) -> np.ndarray:
    a = math.sqrt(6.0 / (f_in + h))
    return rng.uniform(-a, a, size=(f_in, h)).astype(np.float32)


@dataclasses.dataclass
class LayerParams:
    w_self: np.ndarray   # (f_in, h)
    w_neigh: np.ndarray  # (f_in, h)
    b_self: Optional[np.ndarray] = None
    b_neigh: Optional[np.ndarray] = None


def layer_dims(wl: Workload) -> List[tuple]:
    """(f_in, h) per layer; each layer's output width is 2h."""
    dims, f = [], wl.f_in
    for _ in range(wl.layers):
        dims.append((f, wl.hidden))
        f = 2 * wl.hidden
    return dims


def workload_inputs(wl: Workload, bias: bool = False) -> dict:
    """Graph, X, per-layer Glorot weights and the top-layer dY."""
    g = workload_graph(wl)
    x = features(wl.n, wl.f_in, rng_for(wl.case, STREAM_X))
    params = []
    for l, (f_in, h) in enumerate(layer_dims(wl)):
        r = rng_for(wl.case, STREAM_W0 + l)
        p = LayerParams(glorot(f_in, h, r), glorot(f_in, h, r))
        if bias:
            p.b_self = (0.1 * r.standard_normal(h)).astype(np.float32)
            p.b_neigh = (0.1 * r.standard_normal(h)).astype(np.float32)
        params.append(p)
    dy = rng_for(wl.case, STREAM_DY).standard_normal(
        (wl.n, 2 * wl.hidden)).astype(np.float32)
    return {"graph": g, "x": x, "params": params, "dy": dy}


# ------------------------------------------------------ classifier inputs

LABEL_DENSITY = 0.25  # probability that a label is on (multi-label targets)


def labels(n: int, C: int, multilabel: bool, seed_or_rng) -> np.ndarray:
    """0/1 float32 targets (n, C): one uniform class per row (single label),
    or each label on independently with probability LABEL_DENSITY."""
    rng = seed_or_rng if isinstance(seed_or_rng, np.random.Generator) else \
        np.random.default_rng(seed_or_rng)
    if multilabel:
        return (rng.random((n, C)) < LABEL_DENSITY).astype(np.float32)
    t = np.zeros((n, C), np.float32)
    t[np.arange(n), rng.integers(0, C, size=n)] = 1.0
    return t


def classifier_inputs(wl: Workload) -> dict:
    """Glorot W_MLP (2 * hidden x C) and the synthetic targets."""
    w = glorot(2 * wl.hidden, wl.classes, rng_for(wl.case, STREAM_W_MLP))
    t = labels(wl.n, wl.classes, wl.multilabel, rng_for(wl.case, STREAM_LABELS))
    return {"w_mlp": w, "targets": t}


# ------------------------------------------------- full graphs (for prep)

@dataclasses.dataclass
class FullGraph:
    """Unweighted, undirected training graph: CSR with int64 row pointers,
    rows sorted, every edge stored both ways, no self loops."""
    n: int
    indptr: np.ndarray   # int64, n + 1
    indices: np.ndarray  # int32

    @property
    def nnz(self) -> int:
        return int(self.indptr[-1])

    def degrees(self) -> np.ndarray:
        return np.diff(self.indptr)


# Kronecker initiator of the paper's synthetic graphs (proportional to it)
KRONECKER_INITIATOR = ((0.9, 0.5), (0.5, 0.1))


def full_from_pairs(n: int, rows: np.ndarray, cols: np.ndarray) -> FullGraph:
    """Symmetric CSR from undirected pairs (loops and duplicates dropped)."""
    keep = rows != cols
    r = np.concatenate([rows[keep], cols[keep]]).astype(np.int64)
    c = np.concatenate([cols[keep], rows[keep]]).astype(np.int64)
    key = np.unique(r * n + c)
    r, c = key // n, key % n
    indptr = np.zeros(n + 1, np.int64)
    np.cumsum(np.bincount(r, minlength=n), out=indptr[1:])
    return FullGraph(n, indptr, c.astype(np.int32))


def kronecker_graph(scale: int, mean_deg: float, seed: int,
                    initiator=KRONECKER_INITIATOR) -> FullGraph:
    """Stochastic Kronecker graph on 2^scale nodes: each edge descends
    `scale` levels, choosing a quadrant with probability proportional to the
    initiator entry; pairs are drawn until round(n * mean_deg / 2) distinct
    undirected non-loop pairs exist (the first ones drawn are kept)."""
    n = 1 << scale
    p = np.asarray(initiator, np.float64).ravel()
    p = p / p.sum()
    target = int(round(n * mean_deg / 2))
    rng = np.random.default_rng(np.random.SeedSequence([7, seed, scale]))
    keys = np.empty(0, np.int64)
    while keys.size < target:
        m = int((target - keys.size) * 1.3) + 16
        r = np.zeros(m, np.int64)
        c = np.zeros(m, np.int64)
        for _ in range(scale):
            q = rng.choice(4, size=m, p=p)
            r = (r << 1) | (q >> 1)
            c = (c << 1) | (q & 1)
        lo, hi = np.minimum(r, c), np.maximum(r, c)
        k = (lo * n + hi)[lo != hi]
        allk = np.concatenate([keys, k])
        _, first = np.unique(allk, return_index=True)
        keys = allk[np.sort(first)]
    keys = keys[:target]
    return full_from_pairs(n, keys // n, keys % n)


def uniform_node_sample(full: FullGraph, k: int, seed_or_rng) -> np.ndarray:
    """k distinct nodes chosen uniformly, sorted (int32)."""
    rng = seed_or_rng if isinstance(seed_or_rng, np.random.Generator) else \
        np.random.default_rng(seed_or_rng)
    return np.sort(rng.choice(full.n, size=min(k, full.n), replace=False)).astype(np.int32)
