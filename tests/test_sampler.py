"""Frontier sampler: the oracle pinned to what Algorithm 2 fixes, then the
library's host implementation (Dashboard, Algorithms 3 and 4) and its pool
(Algorithm 8) against the oracle, node list for node list.  Host code only:
no GPU involved."""
import collections

import numpy as np
import pytest

from oracle import frontier as F
from paper_2010_03166_amd import gnnprop as G
from paper_2010_03166_amd import synth


def cycle(n):
    nb = np.stack([(np.arange(n) - 1) % n, (np.arange(n) + 1) % n], 1)
    nb.sort(axis=1)
    return synth.FullGraph(n, np.arange(0, 2 * n + 1, 2, dtype=np.int64),
                           nb.ravel().astype(np.int32))


def path3():
    # a - b - c: degrees 1, 2, 1
    return synth.FullGraph(3, np.array([0, 1, 3, 4], np.int64),
                           np.array([1, 0, 2, 1], np.int32))


KRON = {10: synth.kronecker_graph(10, 8.0, 4), 12: synth.kronecker_graph(12, 16.0, 5)}


# ------------------------------------------------------------ oracle pins

def test_splitmix_uniform():
    # integers below K are uniform: chi-square over 20 buckets
    s = F.Stream(12345, 0, 1)
    counts = np.bincount([s.below(20) for _ in range(40000)], minlength=20)
    chi2 = float(((counts - 2000.0) ** 2 / 2000.0).sum())
    assert chi2 < 50.0  # 19 degrees of freedom; P(chi2 > 50) < 1e-4
    # streams of different ids or purposes differ
    a = [F.Stream(7, 0, 1).next() for _ in range(1)]
    assert a != [F.Stream(7, 1, 1).next()] and a != [F.Stream(7, 0, 2).next()]


def test_single_frontier_node_is_a_random_walk():
    # m = 1: the only frontier node is always popped and replaced by a
    # uniform neighbour, so V_s is the start node plus a random walk
    g = cycle(40)
    trace = []
    vs = F.frontier_sample(g, 1, 12, 2.0, seed=3, sub_id=0, trace=trace)
    start = trace[0][1][0]
    walk = [start]
    nbr = F.Stream(3, 0, 2)
    for _ in range(11):
        v = walk[-1]
        walk.append(int(g.indices[g.indptr[v] + nbr.below(2)]))
    assert [p for p, _ in trace[1:]] == walk[:-1]
    assert [q for _, q in trace[1:]] == walk[1:]
    assert vs.tolist() == sorted(set(walk))


def test_pop_probability_proportional_to_degree():
    # frontier = the whole path a-b-c (degrees 1, 2, 1): the first pop is b
    # with probability 1/2, a and c with 1/4 each
    g = path3()
    first = collections.Counter()
    runs = 4000
    for s in range(runs):
        trace = []
        F.frontier_sample(g, 3, 4, 2.0, seed=s, sub_id=0, trace=trace)
        first[trace[1][0]] += 1
    sd = np.sqrt(0.25 / runs)
    assert abs(first[1] / runs - 0.5) < 4 * sd
    assert abs(first[0] / runs - 0.25) < 4 * np.sqrt(0.1875 / runs)


@pytest.mark.parametrize("eta", [1.0, 1.2, 4.0])
def test_frontier_invariants(eta):
    # every pop takes a node of the current frontier (a multiset of m
    # nodes), every new node is a neighbour of the popped one, V_s is the
    # initial frontier plus the new nodes; with eta = 1 cleanups happen
    # often and hubs get truncated pin ranges
    g = KRON[10]
    for sid in range(3):
        trace = []
        vs = F.frontier_sample(g, 20, 300, eta, seed=11, sub_id=sid, trace=trace)
        fs = collections.Counter(trace[0][1])
        assert len(trace[0][1]) == 20 == len(set(trace[0][1]))
        seen = set(trace[0][1])
        for v_pop, v_new in trace[1:]:
            assert fs[v_pop] > 0
            fs[v_pop] -= 1
            fs[v_new] += 1
            assert v_new in g.indices[g.indptr[v_pop]:g.indptr[v_pop + 1]]
            seen.add(v_new)
        assert sum(fs.values()) == 20
        assert vs.tolist() == sorted(seen) and len(vs) <= 300


def test_clipping_and_degenerate_cases():
    g = KRON[10]
    full = F.frontier_sample(g, 20, 300, 2.0, seed=1, sub_id=4)
    clipped = F.frontier_sample(g, 20, 300, 2.0, seed=1, sub_id=4, clip=16)
    assert len(clipped) % 16 == 0 and len(full) - len(clipped) == len(full) % 16
    assert set(clipped.tolist()) <= set(full.tolist())
    # budget = m: V_s is the initial frontier
    assert len(F.frontier_sample(g, 50, 50, 2.0, seed=2, sub_id=0)) == 50
    # an edgeless graph: nothing to pop, V_s = the initial frontier
    empty = synth.FullGraph(30, np.zeros(31, np.int64), np.zeros(0, np.int32))
    assert len(F.frontier_sample(empty, 5, 100, 2.0, seed=2, sub_id=0)) == 5


# ----------------------------------------------- library against the oracle

CASES = [  # scale, m, budget, eta, clip
    (10, 1, 40, 2.0, 0),
    (10, 20, 300, 1.0, 0),
    (10, 20, 300, 1.2, 16),
    (12, 100, 1000, 2.0, 0),
    (12, 50, 800, 1.0, 32),
    (12, 500, 500, 2.0, 0),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "s%d-m%d-n%d-eta%g-clip%d" % c)
def test_library_sampler_matches_oracle(case):
    scale, m, budget, eta, clip = case
    g = KRON[scale]
    for sid in (0, 1, 7):
        ref = F.frontier_sample(g, m, budget, eta, seed=99, sub_id=sid, clip=clip)
        got = G.gnn_frontier_sample(g, m, budget, eta, clip, 99, sid)
        assert np.array_equal(got, ref), sid


def test_library_sampler_large_seed_and_errors():
    g = KRON[10]
    seed = (1 << 64) - 5
    assert np.array_equal(G.gnn_frontier_sample(g, 10, 100, 1.5, 0, seed, 3),
                          F.frontier_sample(g, 10, 100, 1.5, seed=seed, sub_id=3))
    with pytest.raises(G.GnnError):
        G.gnn_frontier_sample(g, 10, 5, 2.0, 0, 0, 0)  # budget below m
    with pytest.raises(G.GnnError):
        G.gnn_frontier_sample(g, 10, 50, 0.5, 0, 0, 0)  # eta below 1


@pytest.mark.parametrize("threads,depth", [(1, 1), (3, 2), (8, 5)])
def test_pool_hands_out_subgraphs_in_order(threads, depth):
    g = KRON[12]
    pool = G.gnn_sampler_pool(g, 100, 1000, 2.0, 16, 42, threads, depth)
    try:
        for k in range(12):
            sid, nodes = pool.next()
            assert sid == k
            assert np.array_equal(nodes, G.gnn_frontier_sample(g, 100, 1000, 2.0, 16, 42, k))
    finally:
        pool.close()
