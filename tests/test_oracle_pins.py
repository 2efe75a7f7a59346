"""Pins of the CPU oracle to facts other than itself.

Each check ties the oracle to something the paper or plain mathematics fixes:
a hand-worked example (tests/golden), brute force against dense matrices,
closed forms on star / complete / identity graphs, invariants (row sums of a
row-normalised adjacency, the adjoint identity), the order rule's MAC counts,
and central finite differences of the backward pass.  No GPU is used.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O
from paper_2010_03166_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def dense(g, vals=None):
    """Dense matrix of a CSR (test-side brute force)."""
    vals = g.values if vals is None else vals
    a = np.zeros((g.n, g.n), np.float64)
    for v in range(g.n):
        for j in range(g.indptr[v], g.indptr[v + 1]):
            a[v, g.indices[j]] += float(vals[j])
    return a


def fr(a):
    return np.array([[float(Fraction(x)) for x in row] for row in a]) \
        if isinstance(a[0], list) else np.array([float(Fraction(x)) for x in a])


def rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    s = max(np.abs(b).max(), 1e-300) if b.size else 1.0
    return float(np.abs(a - b).max() / s) if b.size else 0.0


# ------------------------------------------------------------------ golden

@pytest.fixture(scope="module")
def path4():
    d = json.load(open(os.path.join(GOLDEN, "sage_path4.json")))
    g = synth.symmetric_csr(4, np.array(d["edges"]), self_loops=True)
    assert g.indptr.tolist() == d["csr"]["indptr"]
    assert g.indices.tolist() == d["csr"]["indices"]
    np.testing.assert_allclose(g.values, fr(d["csr"]["values"]), rtol=1e-7)
    # use the exact fractions as double values
    g.values = fr(d["csr"]["values"])
    return g, d


def test_golden_transpose_values(path4):
    g, d = path4
    np.testing.assert_array_equal(O.transpose_values(g), fr(d["values_t"]))


def test_golden_aggregation(path4):
    g, d = path4
    x = fr(d["X"])
    np.testing.assert_allclose(O.spmm(g, x), fr(d["AX"]), rtol=0, atol=1e-15)
    np.testing.assert_allclose(O.spmm_transpose(g, x), fr(d["ATX"]),
                               rtol=0, atol=1e-15)


def test_golden_layer(path4):
    g, d = path4
    x, ws, wn = fr(d["X"]), fr(d["W_self"]), fr(d["W_neigh"])
    y = O.sage_fwd(g, x, ws, wn)
    np.testing.assert_allclose(y, fr(d["Y"]), rtol=0, atol=1e-15)
    r = O.sage_bwd(g, x, ws, wn, fr(d["Y"]), fr(d["dY"]), want_db=True)
    for k in ("dW_self", "dW_neigh", "dX"):
        np.testing.assert_allclose(r[k], fr(d[k]), rtol=0, atol=1e-14, err_msg=k)
    np.testing.assert_allclose(r["db_self"], fr(d["db_self"]), atol=1e-15)
    np.testing.assert_allclose(r["db_neigh"], fr(d["db_neigh"]), atol=1e-15)


# --------------------------------------------------------------- aggregation

@pytest.mark.parametrize("seed,self_loops,values", [
    (0, True, "row-normalized"), (1, False, "row-normalized"),
    (2, True, "random"), (3, False, "random")])
def test_spmm_brute_force(seed, self_loops, values):
    g = synth.random_graph(40, 4.0, seed, self_loops=self_loops, values=values)
    x = np.random.default_rng(seed).standard_normal((g.n, 7))
    a = dense(g)
    assert rel(O.spmm(g, x), a @ x) < 1e-13
    assert rel(O.spmm_transpose(g, x), a.T @ x) < 1e-13


def test_spmm_empty_rows_give_zero():
    # isolated nodes without self loops have empty rows
    g = synth.symmetric_csr(5, np.array([[0, 1]]), self_loops=False)
    assert g.degrees().tolist() == [1, 1, 0, 0, 0]
    x = np.arange(15, dtype=np.float64).reshape(5, 3) + 1
    out = O.spmm(g, x)
    np.testing.assert_array_equal(out[2:], 0.0)
    np.testing.assert_array_equal(out[0], x[1])


def exact_row_norm(g):
    """The same graph with D^-1 values held in double (not rounded to f32)."""
    d = g.degrees()
    g.values = 1.0 / np.repeat(d, d).astype(np.float64)
    return g


def test_row_sum_invariant():
    g = exact_row_norm(synth.power_law_graph(300, 2.1, 8.0, seed=5))
    ones = np.ones((g.n, 3))
    np.testing.assert_allclose(O.spmm(g, ones), 1.0, rtol=0, atol=1e-13)
    c = np.tile(np.array([[2.5, -1.0, 7.0]]), (g.n, 1))
    np.testing.assert_allclose(O.spmm(g, c), c, rtol=0, atol=1e-12)


@pytest.mark.parametrize("k", [1, 3, 17])
def test_star_closed_form(k):
    g = exact_row_norm(synth.star_graph(k))
    x = np.random.default_rng(k).standard_normal((k + 1, 5))
    out = O.spmm(g, x)
    np.testing.assert_allclose(out[0], x.sum(0) / (k + 1), atol=1e-13)
    np.testing.assert_allclose(out[1:], (x[1:] + x[0]) / 2, atol=1e-13)
    t = O.spmm_transpose(g, x)
    np.testing.assert_allclose(t[0], x[0] / (k + 1) + x[1:].sum(0) / 2,
                               atol=1e-13)
    np.testing.assert_allclose(t[1:], x[0] / (k + 1) + x[1:] / 2, atol=1e-13)
    # column sums of A: centre 1/(k+1) + k/2, leaf 1/(k+1) + 1/2, total n
    cs = O.spmm_transpose(g, np.ones((k + 1, 1)))[:, 0]
    np.testing.assert_allclose(cs[0], 1 / (k + 1) + k / 2, atol=1e-14)
    np.testing.assert_allclose(cs[1:], 1 / (k + 1) + 0.5, atol=1e-14)
    np.testing.assert_allclose(cs.sum(), k + 1, atol=1e-12)


def test_complete_graph_closed_form():
    n = 9
    x = np.random.default_rng(1).standard_normal((n, 4))
    out = O.spmm(exact_row_norm(synth.complete_graph(n, True)), x)
    np.testing.assert_allclose(out, np.tile(x.mean(0), (n, 1)), atol=1e-13)
    out = O.spmm(exact_row_norm(synth.complete_graph(n, False)), x)
    np.testing.assert_allclose(out, (x.sum(0) - x) / (n - 1), atol=1e-13)


def test_identity_graph():
    x = np.random.default_rng(2).standard_normal((6, 3))
    g = synth.identity_graph(6)
    np.testing.assert_array_equal(O.spmm(g, x), x)
    np.testing.assert_array_equal(O.spmm_transpose(g, x), x)


def test_adjoint_identity():
    g = synth.random_graph(60, 5.0, 7, values="random")
    r = np.random.default_rng(7)
    x, u = r.standard_normal((60, 6)), r.standard_normal((60, 6))
    lhs = np.sum(O.spmm(g, x) * u)
    rhs = np.sum(x * O.spmm_transpose(g, u))
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))


# ------------------------------------------------------------- Algorithm 6

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_transpose_values_is_dense_transpose(seed):
    g = synth.random_graph(50, 6.0, seed, values="random")
    vt = O.transpose_values(g)
    # exact: a pure permutation of the stored values
    np.testing.assert_array_equal(dense(g, vt), dense(g).T)
    np.testing.assert_array_equal(np.sort(vt), np.sort(g.values.astype(float)))


def test_transpose_values_regular_graph_unchanged():
    n = 12  # cycle + self loops: every degree is 3, so A is symmetric
    e = np.stack([np.arange(n), (np.arange(n) + 1) % n], 1)
    g = synth.symmetric_csr(n, e)
    np.testing.assert_array_equal(O.transpose_values(g),
                                  g.values.astype(np.float64))


def test_transpose_values_rejects_asymmetric_pattern():
    g = synth.csr_from_pairs(3, np.array([0, 0, 1, 2]), np.array([0, 1, 1, 2]))
    with pytest.raises(ValueError):
        O.transpose_values(g)


# ------------------------------------------------------------ order choice

@pytest.mark.parametrize("f1,f2", [(50, 128), (602, 512), (300, 512),
                                   (512, 512), (1024, 512), (256, 1024),
                                   (2048, 1024), (1, 1000)])
def test_order_rule_matches_mac_counts(f1, f2):
    n, delta = 8000, 16 / 8000
    mac1 = delta * n * n * f1 + n * f1 * f2   # (A W1) W2
    mac2 = delta * n * n * f2 + n * f1 * f2   # A (W1 W2)
    assert O.choose_order(f1, f2) == (1 if mac1 <= mac2 else 2)


def test_orders_agree():
    g = synth.power_law_graph(200, 2.1, 6.0, seed=3)
    r = np.random.default_rng(3)
    x, w = r.standard_normal((200, 9)), r.standard_normal((9, 5))
    o1 = O.mm_nn(O.spmm(g, x), w)
    o2 = O.spmm(g, O.mm_nn(x, w))
    assert rel(o1, o2) < 1e-13


# ----------------------------------------------------------- dense products

def test_dense_products_vs_numpy():
    r = np.random.default_rng(4)
    a, b = r.standard_normal((13, 7)), r.standard_normal((7, 11))
    assert rel(O.mm_nn(a, b), a @ b) < 1e-14
    assert rel(O.mm_tn(a.T.copy(), b), a @ b) < 1e-14
    assert rel(O.mm_nt(a, b.T.copy()), a @ b) < 1e-14


# -------------------------------------------------------------- whole layer

def layer_case(seed, n=30, f_in=6, h=4, bias=False, graph="random"):
    r = np.random.default_rng(seed)
    if graph == "random":
        g = synth.random_graph(n, 4.0, seed)
    elif graph == "identity":
        g = synth.identity_graph(n)
    else:
        g = exact_row_norm(synth.complete_graph(n))
    x = r.standard_normal((n, f_in))
    ws, wn = r.standard_normal((f_in, h)), r.standard_normal((f_in, h))
    bs = r.standard_normal(h) if bias else None
    bn = r.standard_normal(h) if bias else None
    return g, x, ws, wn, bs, bn


def test_layer_identity_graph_is_two_path_mlp():
    g, x, ws, wn, _, _ = layer_case(0, graph="identity")
    y = O.sage_fwd(g, x, ws, wn)
    np.testing.assert_allclose(y, np.maximum(np.hstack([x @ ws, x @ wn]), 0),
                               atol=1e-13)


def test_layer_dense_brute_force_with_bias():
    g, x, ws, wn, bs, bn = layer_case(1, bias=True)
    a = dense(g)
    z = np.hstack([x @ ws + bs, (a @ x) @ wn + bn])
    y, s = O.sage_fwd(g, x, ws, wn, bs, bn, want_s=True)
    assert rel(y, np.maximum(z, 0)) < 1e-13
    assert rel(s, a @ x) < 1e-13


def test_layer_zero_weights():
    g, x, ws, wn, _, _ = layer_case(2)
    y = O.sage_fwd(g, x, ws, np.zeros_like(wn))
    np.testing.assert_array_equal(y[:, 4:], 0.0)
    y = O.sage_fwd(g, x, np.zeros_like(ws), wn)
    np.testing.assert_array_equal(y[:, :4], 0.0)


def test_layer_complete_graph_neighbour_half_rows_equal():
    g, x, ws, wn, _, _ = layer_case(3, n=12, graph="complete")
    y = O.sage_fwd(g, x, ws, wn)
    np.testing.assert_allclose(y[:, 4:], np.tile(y[0, 4:], (12, 1)), atol=1e-13)
    dy = np.random.default_rng(3).standard_normal(y.shape)
    r = O.sage_bwd(g, x, ws, wn, y, dy)
    # dW_neigh = mu^T (1^T G_n): rank one, mu = column mean of X
    gn = dy[:, 4:] * (y[:, 4:] > 0)
    np.testing.assert_allclose(r["dW_neigh"], np.outer(x.mean(0), gn.sum(0)),
                               atol=1e-12)


def _loss(g, x, ws, wn, bs, bn, dy):
    return float(np.sum(dy * O.sage_fwd(g, x, ws, wn, bs, bn)))


def _preact(g, x, ws, wn, bs, bn):
    a = dense(g)
    z = np.hstack([x @ ws, (a @ x) @ wn])
    if bs is not None:
        z = z + np.concatenate([bs, bn])
    return z


@pytest.mark.parametrize("seed,bias", [(10, False), (11, True), (12, False)])
def test_backward_finite_differences(seed, bias):
    # central differences of L = <dY, Y> in double; the layer is piecewise
    # linear, so away from ReLU kinks the difference quotient is exact up to
    # rounding.  Cases whose pre-activations come near 0 are re-drawn.
    for s in range(seed, seed + 50):
        g, x, ws, wn, bs, bn = layer_case(s, n=10, f_in=4, h=3, bias=bias)
        if np.abs(_preact(g, x, ws, wn, bs, bn)).min() > 1e-3:
            break
    dy = np.random.default_rng(seed + 100).standard_normal((10, 6))
    y = O.sage_fwd(g, x, ws, wn, bs, bn)
    r = O.sage_bwd(g, x, ws, wn, y, dy, want_db=bias)
    eps = 1e-6

    def fd(arr):
        out = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + eps
            lp = _loss(g, x, ws, wn, bs, bn, dy)
            arr[idx] = old - eps
            lm = _loss(g, x, ws, wn, bs, bn, dy)
            arr[idx] = old
            out[idx] = (lp - lm) / (2 * eps)
        return out

    assert rel(r["dX"], fd(x)) < 1e-6
    assert rel(r["dW_self"], fd(ws)) < 1e-6
    assert rel(r["dW_neigh"], fd(wn)) < 1e-6
    if bias:
        assert rel(r["db_self"], fd(bs)) < 1e-6
        assert rel(r["db_neigh"], fd(bn)) < 1e-6


def test_two_layer_stack_finite_differences():
    for s in range(50):
        r = np.random.default_rng(s)
        g = synth.random_graph(8, 3.0, s)
        x = r.standard_normal((8, 3))
        p1 = synth.LayerParams(r.standard_normal((3, 2)), r.standard_normal((3, 2)))
        p2 = synth.LayerParams(r.standard_normal((4, 2)), r.standard_normal((4, 2)))
        y1 = O.sage_fwd(g, x, p1.w_self, p1.w_neigh)
        z1 = _preact(g, x, p1.w_self, p1.w_neigh, None, None)
        z2 = _preact(g, y1, p2.w_self, p2.w_neigh, None, None)
        if min(np.abs(z1).min(), np.abs(z2).min()) > 1e-3:
            break
    dy = np.random.default_rng(99).standard_normal((8, 4))
    res = O.sage_stack(g, x, [p1, p2], dy)

    def loss():
        y1 = O.sage_fwd(g, x, p1.w_self, p1.w_neigh)
        return float(np.sum(dy * O.sage_fwd(g, y1, p2.w_self, p2.w_neigh)))

    eps = 1e-6
    for arr, got in [(x, res["grads"][0]["dX"]),
                     (p1.w_neigh, res["grads"][0]["dW_neigh"]),
                     (p2.w_self, res["grads"][1]["dW_self"])]:
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + eps
            lp = loss()
            arr[idx] = old - eps
            lm = loss()
            arr[idx] = old
            num[idx] = (lp - lm) / (2 * eps)
        assert rel(got, num) < 1e-6


# ------------------------------------------------------ per-output spot evals

def test_spot_evaluations_match_full_layer():
    g = synth.power_law_graph(120, 2.1, 6.0, seed=9)
    r = np.random.default_rng(9)
    f_in, h = 7, 5
    x = r.standard_normal((120, f_in))
    ws, wn = r.standard_normal((f_in, h)), r.standard_normal((f_in, h))
    bs, bn = r.standard_normal(h), r.standard_normal(h)
    y = O.sage_fwd(g, x, ws, wn, bs, bn)
    rows = np.array([0, 5, 119, 64, 5])
    assert rel(O.sage_fwd_rows(g, x, ws, wn, rows, bs, bn), y[rows]) < 1e-14
    ysyn = r.standard_normal((120, 2 * h))  # any sign pattern is a valid mask
    dy = r.standard_normal((120, 2 * h))
    full = O.sage_bwd(g, x, ws, wn, ysyn, dy)
    assert rel(O.sage_bwd_dx_rows(g, ws, wn, ysyn, dy, rows), full["dX"][rows]) \
        < 1e-13
    ei, ej = np.array([0, 6, 3, 2]), np.array([4, 0, 2, 2])
    a, b = O.sage_bwd_dw_entries(g, x, ysyn, dy, h, ei, ej)
    assert rel(a, full["dW_self"][ei, ej]) < 1e-13
    assert rel(b, full["dW_neigh"][ei, ej]) < 1e-13


def test_result_independent_of_thread_count(monkeypatch):
    # fixed summation order: the same bits with any OpenMP thread count
    import subprocess
    import sys
    code = ("import numpy as np,sys;sys.path.insert(0,%r);"
            "from oracle import oracle as O;from paper_2010_03166_amd import synth;"
            "g=synth.power_law_graph(500,2.1,8.0,seed=1);"
            "x=np.random.default_rng(0).standard_normal((500,33));"
            "w=np.random.default_rng(1).standard_normal((33,8));"
            "y=O.sage_fwd(g,x,w,w);r=O.sage_bwd(g,x,w,w,y,y);"
            "sys.stdout.write(str(hash(y.tobytes()+r['dX'].tobytes()+r['dW_neigh'].tobytes()"
            "+O.spmm_transpose(g,x).tobytes())))") % os.path.dirname(GOLDEN + "/..")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = code.replace(repr(os.path.dirname(GOLDEN + "/..")), repr(root))
    outs = []
    for t in ("1", "3", "8"):
        env = dict(os.environ, OMP_NUM_THREADS=t, PYTHONHASHSEED="0")
        outs.append(subprocess.run([sys.executable, "-c", code], env=env,
                                   capture_output=True, text=True,
                                   check=True).stdout)
    assert outs[0] == outs[1] == outs[2]


# ------------------------------------------------------- bfloat16 rounding

def test_round_bf16_closed_forms():
    # bfloat16 has 8 significant bits: representable neighbours of 1 are
    # 1 - 2^-8 and 1 + 2^-7
    vals = np.array([1.0, 1 + 2.0**-8, 1 + 3 * 2.0**-9, 1 + 2.0**-7 + 2.0**-8,
                     -(1 + 2.0**-8 + 2.0**-20), 0.0, -0.0, 2.0**-130,
                     3.0e38, 1.0 + 2.0**-9])
    exp = np.array([1.0, 1.0,                # tie -> even (1.0)
                    1 + 2.0**-7,             # above the tie -> up
                    1 + 2.0**-6,             # tie between 1+2^-7 (odd) and 1+2^-6
                    -(1 + 2.0**-7),          # above the tie (negative) -> away
                    0.0, -0.0, 2.0**-130,    # float subnormal 2^-130 is exact
                    np.float32(3.0e38).astype(np.float64),
                    1.0])
    exp[8] = np.inf if False else exp[8]
    got = O.round_bf16(vals)
    assert got[:8].tolist() == exp[:8].tolist()
    assert np.signbit(got[6])
    # 3e38 rounds to a value with 8 significant bits, within half an ulp
    b = got[8]
    assert abs(b - 3.0e38) <= 2.0**(127 - 8) and b == O.round_bf16([b])[0]
    assert got[9] == 1.0


def test_round_bf16_is_idempotent_and_monotone():
    r = np.random.default_rng(0)
    x = np.sort(r.standard_normal(5000) * 10.0 ** r.uniform(-5, 5, 5000))
    y = O.round_bf16(x)
    assert np.all(np.diff(y) >= 0)
    assert np.array_equal(O.round_bf16(y), y)
    # at most half a bfloat16 ulp (relative 2^-8) from the float value
    f = x.astype(np.float32).astype(np.float64)
    assert np.all(np.abs(y - f) <= np.abs(f) * 2.0**-8 * (1 + 1e-12))


# --------------------------------------------------- GCN and MixHop layers

def gcn_graph(seed, n=14, deg=3.0):
    return synth.sym_normalized(synth.random_graph(n, deg, seed))


def test_sym_normalization_matches_definition():
    # A_hat = (I + D)^-1/2 (I + A) (I + D)^-1/2 with A the binary adjacency
    # without self loops and D its degree matrix, written out densely.
    g0 = synth.random_graph(25, 4.0, 3, self_loops=False, values="ones")
    a = dense(g0)
    d = a.sum(axis=1)
    ref = np.diag((1 + d) ** -0.5) @ (np.eye(25) + a) @ np.diag((1 + d) ** -0.5)
    g = synth.sym_normalized(synth.random_graph(25, 4.0, 3))
    assert np.allclose(dense(g), ref, rtol=1e-6, atol=0)
    assert np.allclose(dense(g), dense(g).T)


def test_gcn_forward_dense_brute_force():
    rng = np.random.default_rng(4)
    g = gcn_graph(5)
    x, w, b = rng.standard_normal((14, 5)), rng.standard_normal((5, 3)), rng.standard_normal(3)
    ref = np.maximum(dense(g) @ x @ w + b, 0)
    assert rel(O.gcn_fwd(g, x, w, b), ref) < 1e-14


def test_gcn_regular_graph_preserves_constant_rows():
    # On a cycle (2-regular, 3 stored entries per row) every A_hat entry is
    # 1/3, so A_hat maps constant columns to themselves: Y = ReLU(X W), up
    # to the float32 storage of 1/3 (relative 3e-8).
    n = 9
    e = np.array([[i, (i + 1) % n] for i in range(n)])
    g = synth.sym_normalized(synth.symmetric_csr(n, e))
    assert np.all(g.values == np.float32(1 / 3))
    x = np.tile(np.random.default_rng(1).standard_normal(4), (n, 1))
    w = np.random.default_rng(2).standard_normal((4, 3))
    assert rel(O.gcn_fwd(g, x, w), np.maximum(x @ w, 0)) < 1e-7


def test_mixhop_forward_dense_matrix_powers():
    rng = np.random.default_rng(6)
    g = gcn_graph(7)
    K, f_in, h = 3, 4, 2
    x = rng.standard_normal((14, f_in))
    w = rng.standard_normal((f_in, (K + 1) * h))
    b = rng.standard_normal((K + 1) * h)
    a = dense(g)
    ref = np.hstack([np.linalg.matrix_power(a, k) @ x @ w[:, k * h:(k + 1) * h]
                     for k in range(K + 1)]) + b
    assert rel(O.mixhop_fwd(g, x, w, K, b), np.maximum(ref, 0)) < 1e-13


def test_mixhop_special_cases():
    rng = np.random.default_rng(8)
    g = gcn_graph(9)
    x = rng.standard_normal((14, 5))
    w0, w1 = rng.standard_normal((5, 3)), rng.standard_normal((5, 3))
    # K = 0: a dense layer
    assert rel(O.mixhop_fwd(g, x, w0, 0), np.maximum(x @ w0, 0)) < 1e-14
    # K = 1: the two-path GraphSAGE layer aggregating with A_hat
    assert rel(O.mixhop_fwd(g, x, np.hstack([w0, w1]), 1),
               O.sage_fwd(g, x, w0, w1)) < 1e-14
    # K = 1 with W_0 = 0: hop 0 is zero, hop 1 is the GCN layer
    y = O.mixhop_fwd(g, x, np.hstack([np.zeros_like(w0), w1]), 1)
    assert np.all(y[:, :3] == 0) and rel(y[:, 3:], O.gcn_fwd(g, x, w1)) < 1e-14


def _fd_grads(loss, arrays, eps=1e-6):
    out = []
    for arr in arrays:
        d = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + eps
            lp = loss()
            arr[idx] = old - eps
            lm = loss()
            arr[idx] = old
            d[idx] = (lp - lm) / (2 * eps)
        out.append(d)
    return out


@pytest.mark.parametrize("bias", [False, True])
def test_gcn_backward_finite_differences(bias):
    # L = <dY, Y>; cases with a pre-activation near the ReLU kink re-drawn
    for s in range(20, 80):
        rng = np.random.default_rng(s)
        g = synth.sym_normalized(synth.random_graph(10, 3.0, s))
        x, w = rng.standard_normal((10, 4)), rng.standard_normal((4, 3))
        b = rng.standard_normal(3) if bias else None
        z = dense(g) @ x @ w + (b if bias else 0)
        if np.abs(z).min() > 1e-3:
            break
    dy = np.random.default_rng(5).standard_normal((10, 3))
    r = O.gcn_bwd(g, x, w, O.gcn_fwd(g, x, w, b), dy, want_db=bias)
    arrs = [x, w] + ([b] if bias else [])
    fds = _fd_grads(lambda: float(np.sum(dy * O.gcn_fwd(g, x, w, b))), arrs)
    assert rel(r["dX"], fds[0]) < 1e-6 and rel(r["dW"], fds[1]) < 1e-6
    if bias:
        assert rel(r["db"], fds[2]) < 1e-6


@pytest.mark.parametrize("K", [1, 2, 3])
def test_mixhop_backward_finite_differences(K):
    h = 2
    for s in range(40, 120):
        rng = np.random.default_rng(s)
        g = synth.sym_normalized(synth.random_graph(9, 3.0, s))
        x = rng.standard_normal((9, 3))
        w = rng.standard_normal((3, (K + 1) * h))
        b = rng.standard_normal((K + 1) * h)
        a = dense(g)
        z = np.hstack([np.linalg.matrix_power(a, k) @ x @ w[:, k * h:(k + 1) * h]
                       for k in range(K + 1)]) + b
        if np.abs(z).min() > 1e-3:
            break
    dy = np.random.default_rng(6).standard_normal((9, (K + 1) * h))
    y = O.mixhop_fwd(g, x, w, K, b)
    r = O.mixhop_bwd(g, x, w, K, y, dy, want_db=True)
    fds = _fd_grads(lambda: float(np.sum(dy * O.mixhop_fwd(g, x, w, K, b))), [x, w, b])
    assert rel(r["dX"], fds[0]) < 1e-6
    assert rel(r["dW"], fds[1]) < 1e-6
    assert rel(r["db"], fds[2]) < 1e-6


def test_mixhop_backward_on_asymmetric_values():
    # the backward uses A_hat^T, not A_hat: random (value-asymmetric)
    # entries on a symmetric pattern check the transposes against dense
    # matrix powers of the transpose
    rng = np.random.default_rng(12)
    g = synth.random_graph(12, 3.0, 4, values="random")
    K, h = 2, 2
    x, w = rng.standard_normal((12, 3)), rng.standard_normal((3, (K + 1) * h))
    y = O.mixhop_fwd(g, x, w, K)
    dy = rng.standard_normal(y.shape)
    r = O.mixhop_bwd(g, x, w, K, y, dy)
    at = dense(g).T
    gm = np.where(y > 0, dy, 0)
    ref = sum(np.linalg.matrix_power(at, k) @ gm[:, k * h:(k + 1) * h] @ w[:, k * h:(k + 1) * h].T
              for k in range(K + 1))
    assert rel(r["dX"], ref) < 1e-13


# ------------------------------------ classifier head, loss, weight update

def _cls_case(seed, n=12, f=5, C=4, kind=0):
    for s in range(seed, seed + 60):
        rng = np.random.default_rng(s)
        x, w = rng.standard_normal((n, f)), rng.standard_normal((f, C))
        if np.abs(x @ w).min() > 1e-3:  # away from the MLP ReLU kink
            break
    if kind == O.SOFTMAX:
        t = np.eye(C)[rng.integers(0, C, n)]
    else:
        t = (rng.random((n, C)) < 0.4).astype(np.float64)
    return x, w, t


@pytest.mark.parametrize("kind", [0, 1])
def test_classifier_gradients_finite_differences(kind):
    x, w, t = _cls_case(30 + kind, kind=kind)
    r = O.classifier(x, w, t, kind)
    fd = _fd_grads(lambda: O.classifier(x, w, t, kind, want_dx=False)["loss"], [x, w])
    assert rel(r["dX"], fd[0]) < 1e-6 and rel(r["dW"], fd[1]) < 1e-6


def test_classifier_zero_weights_closed_forms():
    x, _, t = _cls_case(5, C=7)
    w = np.zeros((5, 7))
    r = O.classifier(x, w, t, O.SOFTMAX)
    assert abs(r["loss"] - np.log(7)) < 1e-15 and np.allclose(r["probs"], 1 / 7)
    ts = (np.random.default_rng(1).random((12, 7)) < 0.5).astype(float)
    r = O.classifier(x, w, ts, O.SIGMOID)
    assert abs(r["loss"] - 7 * np.log(2)) < 1e-14 and np.allclose(r["probs"], 0.5)
    # all logits at the ReLU floor: no gradient reaches W or X
    assert np.all(r["dW"] == 0) and np.all(r["dX"] == 0)


def test_classifier_probabilities():
    x, w, t = _cls_case(8, kind=0)
    p = O.classifier(x, w, t, O.SOFTMAX)["probs"]
    assert np.allclose(p.sum(axis=1), 1, rtol=0, atol=1e-15) and np.all(p > 0)
    z = np.maximum(x @ w, 0)
    ps = O.classifier(x, w, t, O.SIGMOID)["probs"]
    assert np.allclose(ps, 1 / (1 + np.exp(-z)), rtol=1e-14, atol=0)


def test_classifier_confident_loss_closed_form():
    # logit 20 on the true class, 0 on the other two: every row's softmax
    # cross-entropy is log(1 + 2 e^-20) = 4.12e-9, here reached through
    # log(sum of exponentials), i.e. to within the rounding of log near 1
    n, C = 6, 3
    x = np.eye(C)[np.arange(n) % C]
    w = np.eye(C) * 20.0
    r = O.classifier(x, w, x.copy(), O.SOFTMAX)
    assert abs(r["loss"] - np.log1p(2 * np.exp(-20.0))) < 5e-16


def test_adam_constant_gradient_closed_form():
    # with a constant gradient the bias-corrected moments are g and g^2, so
    # every step moves W by lr * g / (|g| + eps)
    rng = np.random.default_rng(3)
    w0, g = rng.standard_normal(50), rng.standard_normal(50)
    w, m, v = w0.copy(), np.zeros(50), np.zeros(50)
    lr, eps = 1e-3, 1e-8
    for step in range(1, 6):
        w, m, v = O.adam(w, g, m, v, lr, 0.9, 0.999, eps, step)
    assert np.allclose(w, w0 - 5 * lr * g / (np.abs(g) + eps), rtol=0, atol=1e-12)
    assert np.array_equal(O.sgd(w0, g, 0.5), w0 - 0.5 * g)


# ------------------------------------------------- full training iteration

def _train_case(kind, bias, seed=4):
    g = synth.random_graph(10, 3.0, seed)
    g.values = g.values.astype(np.float64)
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((10, 4))
    params = []
    for f, h in ((4, 3), (6, 3)):
        p = synth.LayerParams(rng.standard_normal((f, h)), rng.standard_normal((f, h)))
        if bias:
            p.b_self, p.b_neigh = rng.standard_normal(h), rng.standard_normal(h)
        params.append(p)
    w_mlp = rng.standard_normal((6, 3))
    t = np.eye(3)[rng.integers(0, 3, 10)] if kind == O.SOFTMAX else \
        (rng.random((10, 3)) < 0.4).astype(np.float64)
    return g, x, params, w_mlp, t


def _loss_only(g, x, params, w_mlp, t, kind):
    a = x
    for p in params:
        a = O.sage_fwd(g, a, p.w_self, p.w_neigh, p.b_self, p.b_neigh)
    return O.classifier(a, w_mlp, t, kind, want_dx=False)["loss"]


@pytest.mark.parametrize("kind", [0, 1])
@pytest.mark.parametrize("bias", [False, True])
def test_train_step_gradients_finite_differences(kind, bias):
    # the composed backward pass (classifier gradient fed into the top layer
    # as its dY, the top layer's ReLU mask applied there) against central
    # differences of the end-to-end loss in every weight
    g, x, params, w_mlp, t = _train_case(kind, bias)
    r = O.train_step(g, x, params, w_mlp, t, kind, "sgd", lr=0.0)
    arrays = [w_mlp]
    for p in params:
        arrays += [p.w_self, p.w_neigh] + ([p.b_self, p.b_neigh] if bias else [])
    fd = _fd_grads(lambda: _loss_only(g, x, params, w_mlp, t, kind), arrays)
    assert len(fd) == len(r["flat_grads"])
    for a, b in zip(r["flat_grads"], fd):
        assert rel(a, b) < 1e-6
    assert abs(r["loss"] - _loss_only(g, x, params, w_mlp, t, kind)) < 1e-14
    # lr = 0 leaves every weight as it was
    for a, b in zip(r["weights"], arrays):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("kind", [0, 1])
def test_train_step_descends(kind):
    # a small SGD step along the gradient lowers the loss by about
    # lr * |grad|^2 (first-order Taylor term)
    g, x, params, w_mlp, t = _train_case(kind, True, seed=7)
    lr = 1e-5
    r = O.train_step(g, x, params, w_mlp, t, kind, "sgd", lr=lr)
    ws = r["weights"]
    newp, k = [], 1
    for p in params:
        newp.append(synth.LayerParams(ws[k], ws[k + 1], ws[k + 2], ws[k + 3]))
        k += 4
    drop = r["loss"] - _loss_only(g, x, newp, ws[0], t, kind)
    sq = sum(float((gr ** 2).sum()) for gr in r["flat_grads"])
    assert drop > 0 and abs(drop - lr * sq) < 1e-3 * lr * sq


def test_train_step_adam_first_step():
    # at t = 1 the bias-corrected moments are g and g^2: each weight moves by
    # lr * g / (|g| + eps)
    g, x, params, w_mlp, t = _train_case(O.SOFTMAX, False)
    r = O.train_step(g, x, params, w_mlp, t, O.SOFTMAX, "adam", lr=1e-2, t=1)
    arrays = [w_mlp] + [a for p in params for a in (p.w_self, p.w_neigh)]
    for w0, w1, gr in zip(arrays, r["weights"], r["flat_grads"]):
        assert np.allclose(w1, w0 - 1e-2 * gr / (np.abs(gr) + 1e-8), rtol=0, atol=1e-15)


def test_classifier_supplied_relu_decision():
    # the natural decision given explicitly reproduces the default exactly;
    # with every unit on, the head is linear and its loss smooth, so central
    # differences of that loss pin the gradient under a supplied decision
    for kind in (O.SOFTMAX, O.SIGMOID):
        x, w, t = _cls_case(40 + kind, kind=kind)
        a = O.classifier(x, w, t, kind)
        b = O.classifier(x, w, t, kind, relu_on=(x @ w) > 0)
        assert a["loss"] == b["loss"]
        for k in ("probs", "dW", "dX"):
            assert np.array_equal(a[k], b[k]), k
        on = np.ones((x.shape[0], w.shape[1]), bool)
        r = O.classifier(x, w, t, kind, relu_on=on)
        fd = _fd_grads(lambda: O.classifier(x, w, t, kind, want_dx=False, relu_on=on)["loss"],
                       [x, w])
        assert rel(r["dX"], fd[0]) < 1e-6 and rel(r["dW"], fd[1]) < 1e-6
        # and it differs from the ReLU head (some logits are negative)
        assert not np.allclose(r["dW"], a["dW"])


def test_train_step_forced_decisions_reproduce_default():
    # supplying the oracle's own layer outputs and MLP decision changes nothing
    g, x, params, w_mlp, t = _train_case(O.SIGMOID, True)
    r = O.train_step(g, x, params, w_mlp, t, O.SIGMOID, "sgd", lr=0.1)
    z = r["acts"][-1] @ w_mlp
    f = O.train_step(g, x, params, w_mlp, t, O.SIGMOID, "sgd", lr=0.1,
                     forced={"ys": r["acts"][1:], "relu_on": z > 0})
    assert f["loss"] == r["loss"]
    for a, b in zip(f["flat_grads"] + f["weights"], r["flat_grads"] + r["weights"]):
        assert np.array_equal(a, b)


# ------------------------------------------------- induced subgraph (prep)

def _dense_full(full):
    A = np.zeros((full.n, full.n))
    for u in range(full.n):
        A[u, full.indices[full.indptr[u]:full.indptr[u + 1]]] = 1.0
    return A


def _dense_of(s):
    D = np.zeros((s.n, s.n))
    for u in range(s.n):
        for j in range(s.indptr[u], s.indptr[u + 1]):
            D[u, s.indices[j]] += s.values[j]
    return D


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_induce_dense_brute_force(seed):
    # A_s = A[V_s, V_s] + I, then D^-1 A_s (row norm) or D^-1/2 A_s D^-1/2
    full = synth.kronecker_graph(6, 6.0, seed)
    A = _dense_full(full)
    rng = np.random.default_rng(seed)
    nodes = np.sort(rng.choice(full.n, size=23, replace=False)).astype(np.int32)
    sub = A[np.ix_(nodes, nodes)] + np.eye(len(nodes))
    d = sub.sum(axis=1)
    r = O.induce(full, nodes, 0)
    assert np.array_equal(_dense_of(r), sub / d[:, None])
    s = O.induce(full, nodes, 1)
    assert np.allclose(_dense_of(s), sub / np.sqrt(np.outer(d, d)), rtol=1e-15, atol=0)
    # rows sorted, pattern symmetric, row sums 1
    for u in range(r.n):
        row = r.indices[r.indptr[u]:r.indptr[u + 1]]
        assert np.all(np.diff(row) > 0) and u in row
    assert np.array_equal(_dense_of(r) > 0, (_dense_of(r) > 0).T)
    assert np.allclose(_dense_of(r).sum(axis=1), 1.0, rtol=0, atol=1e-15)


def test_induce_special_cases():
    full = synth.kronecker_graph(7, 8.0, 3)
    # all nodes: the full graph with self loops, values 1/deg
    allv = np.arange(full.n, dtype=np.int32)
    r = O.induce(full, allv, 0)
    assert np.array_equal(r.indptr, full.indptr + np.arange(full.n + 1))
    pairs = np.stack([np.repeat(np.arange(full.n), full.degrees()), full.indices], 1)
    ref = synth.symmetric_csr(full.n, pairs[pairs[:, 0] < pairs[:, 1]], self_loops=True)
    assert np.array_equal(r.indices, ref.indices)
    assert np.allclose(r.values, np.repeat(1.0 / (full.degrees() + 1), full.degrees() + 1),
                       rtol=1e-15, atol=0)
    # one node: a single self loop of value 1
    one = O.induce(full, np.array([5], np.int32), 1)
    assert one.indptr.tolist() == [0, 1] and one.indices.tolist() == [0] and one.values[0] == 1
    # isolated nodes keep only their loop; an independent set gives I
    deg = full.degrees()
    iso = np.flatnonzero(deg == 0)[:4].astype(np.int32)
    if iso.size:
        r = O.induce(full, iso, 0)
        assert np.array_equal(r.indices, np.arange(iso.size)) and np.all(r.values == 1)
    # a stored loop in the full graph is not counted twice
    loop = synth.FullGraph(3, np.array([0, 2, 3, 4], np.int64), np.array([0, 1, 0, 2], np.int32))
    r = O.induce(loop, np.array([0, 1, 2], np.int32), 0)
    assert r.indptr.tolist() == [0, 2, 4, 5] and r.indices.tolist() == [0, 1, 0, 1, 2]


def test_kronecker_graph_properties():
    g = synth.kronecker_graph(10, 16.0, 0)
    assert g.n == 1024 and g.nnz == 2 * round(1024 * 16 / 2)
    A = _dense_full(g)
    assert np.array_equal(A, A.T) and np.all(np.diag(A) == 0)
    for u in range(g.n):
        row = g.indices[g.indptr[u]:g.indptr[u + 1]]
        assert np.all(np.diff(row) > 0)
    # the initiator's heavy corner: node 0 has the largest expected degree
    assert g.degrees()[0] == g.degrees().max()


# ------------------------------------------------------------- GAT layer

def _gat_case(seed, n=9, f=4, h=3):
    g = synth.random_graph(n, 2.5, seed)
    for s in range(seed, seed + 200):
        rng = np.random.default_rng(s)
        x, w = rng.standard_normal((n, f)), rng.standard_normal((f, h))
        a = rng.standard_normal(2 * h)
        P = x @ w
        z = np.array([a[:h] @ P[u] + a[h:] @ P[v] for u in range(n)
                      for v in g.indices[g.indptr[u]:g.indptr[u + 1]]])
        y = O.gat_fwd(g, x, w, a)
        pre = _gat_dense(g, x, w, a) @ P
        # away from both kinks, so that central differences are smooth
        if np.abs(z).min() > 1e-3 and np.abs(pre).min() > 1e-3:
            return g, x, w, a
    raise AssertionError("no smooth case")


def _gat_dense(g, x, w, a, alpha=O.GAT_ALPHA):
    h = w.shape[1]
    P = x @ w
    A = np.zeros((g.n, g.n))
    for u in range(g.n):
        for v in g.indices[g.indptr[u]:g.indptr[u + 1]]:
            z = a[:h] @ P[u] + a[h:] @ P[v]
            A[u, v] = z if z > 0 else alpha * z
    return A


def test_gat_forward_dense_brute_force():
    g, x, w, a = _gat_case(3)
    y, att = O.gat_fwd(g, x, w, a, want_att=True)
    A = _gat_dense(g, x, w, a)
    assert rel(y, np.maximum(A @ (x @ w), 0)) < 1e-14
    got = np.zeros((g.n, g.n))
    for u in range(g.n):
        got[u, g.indices[g.indptr[u]:g.indptr[u + 1]]] = att[g.indptr[u]:g.indptr[u + 1]]
    assert rel(got, A) < 1e-14


def test_gat_linear_attention_closed_form():
    # slope 1: the attention is linear, A_att = diag(s) B + B diag(t) on the
    # pattern B, with s = P a1 and t = P a2
    g, x, w, a = _gat_case(5)
    h = w.shape[1]
    P = x @ w
    B = np.zeros((g.n, g.n))
    for u in range(g.n):
        B[u, g.indices[g.indptr[u]:g.indptr[u + 1]]] = 1.0
    s, t = P @ a[:h], P @ a[h:]
    Z = np.diag(s) @ B @ P + B @ np.diag(t) @ P
    assert rel(O.gat_fwd(g, x, w, a, alpha=1.0), np.maximum(Z, 0)) < 1e-13


def test_gat_zero_attention_vector():
    g, x, w, a = _gat_case(7)
    a0 = np.zeros_like(a)
    assert np.all(O.gat_fwd(g, x, w, a0) == 0)
    dy = np.random.default_rng(1).standard_normal((g.n, w.shape[1]))
    r = O.gat_bwd(g, x, w, a0, O.gat_fwd(g, x, w, a0), dy)
    assert np.all(r["dW"] == 0) and np.all(r["dX"] == 0) and np.all(r["da"] == 0)


@pytest.mark.parametrize("seed", [11, 12])
def test_gat_gradients_finite_differences(seed):
    g, x, w, a = _gat_case(seed)
    dy = np.random.default_rng(seed).standard_normal((g.n, w.shape[1]))
    y = O.gat_fwd(g, x, w, a)
    r = O.gat_bwd(g, x, w, a, y, dy)
    fd = _fd_grads(lambda: float((dy * O.gat_fwd(g, x, w, a)).sum()), [x, w, a])
    assert rel(r["dX"], fd[0]) < 1e-6
    assert rel(r["dW"], fd[1]) < 1e-6
    assert rel(r["da"], fd[2]) < 1e-6


def test_gat_supplied_decisions():
    # the natural decisions given explicitly change nothing; all-positive
    # decisions equal slope 1 (the attention taken as linear)
    g, x, w, a = _gat_case(13)
    dy = np.random.default_rng(2).standard_normal((g.n, w.shape[1]))
    y, att = O.gat_fwd(g, x, w, a, want_att=True)
    r0 = O.gat_bwd(g, x, w, a, y, dy)
    r1 = O.gat_bwd(g, x, w, a, y, dy, z_pos=att > 0)
    for k in ("dX", "dW", "da"):
        assert np.array_equal(r0[k], r1[k])
    y1 = O.gat_fwd(g, x, w, a, alpha=1.0)
    ra = O.gat_bwd(g, x, w, a, y1, dy, z_pos=np.ones(att.size, bool))
    rb = O.gat_bwd(g, x, w, a, y1, dy, alpha=1.0)
    for k in ("dX", "dW", "da"):
        assert rel(ra[k], rb[k]) < 1e-14
