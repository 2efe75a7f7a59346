"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Every comparison uses the same seeded inputs on both sides.  Floating-point
results must agree to max |gpu - oracle| / max |oracle| <= 1e-4 per tensor
(fp32 arithmetic against the double-precision oracle); the aggregation alone
is held to 1e-5; the transposed value array and the work plan are checked
bit for bit.
"""

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2010_03166_amd import gnnprop as G
from paper_2010_03166_amd import runtime, synth

from gpu_helpers import (empty_out, maxrel, prepared, read_plan, sample_rows,
                         to_dev, unaligned)

pytestmark = pytest.mark.gpu

TOL = 1e-4
TOL_SPMM = 1e-5


def boundary_graph():
    """Rows of every kind the aggregation plan distinguishes, side by side:
    empty rows, rows of exactly 64 and 65 entries (the long-row threshold),
    long rows next to short ones, and short rows straddling 64-entry
    windows; random values (asymmetric), no self loops."""
    rng = np.random.default_rng(11)
    e = [(3, v) for v in range(100, 164)]            # row 3: 64 entries
    e += [(4, v) for v in range(200, 265)]           # row 4: 65 entries
    e += [(10, v) for v in range(100, 400) if v != 10]  # a long row
    e += [(11, v) for v in range(300, 380)]          # adjacent long row
    for u in range(20, 60):                          # short rows
        for v in rng.choice(np.arange(20, 60), size=3, replace=False):
            if u < v:
                e.append((u, int(v)))
    # rows 70..89 stay empty
    e = np.unique(np.array([(min(a, b), max(a, b)) for a, b in e]), axis=0)
    return synth.symmetric_csr(400, e, self_loops=False, values="random",
                               rng=np.random.default_rng(12))


def graphs():
    return {
        "boundary": boundary_graph(),
        "path4": synth.path_graph(4),
        "random": synth.random_graph(300, 6.0, 1, values="random"),
        "powerlaw": synth.power_law_graph(3000, 2.1, 12.0, seed=2),
        "star700": synth.star_graph(700),
        "no_self_loops": synth.random_graph(200, 1.5, 3, self_loops=False),
        "identity": synth.identity_graph(64),
        "single": synth.identity_graph(1),
    }


GRAPHS = graphs()


# ------------------------------------------------- per-subgraph preparation

@pytest.mark.parametrize("name", list(GRAPHS))
def test_transpose_values_bit_exact(name):
    g = GRAPHS[name]
    dg = prepared(g)
    torch.cuda.synchronize()
    got = dg.values_t[: g.nnz].cpu().numpy()
    ref = O.transpose_values(g).astype(np.float32)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("name", ["powerlaw", "star700", "random"])
def test_transpose_values_without_plan(name):
    # with plan == NULL the transpose runs one wavefront per row
    g = GRAPHS[name]
    dg = runtime.DeviceGraph(g)
    c = dg.struct()
    c.plan = None
    G.gnn_csr_transpose_values(c, dg.values_t)
    torch.cuda.synchronize()
    got = dg.values_t[: g.nnz].cpu().numpy()
    ref = O.transpose_values(g).astype(np.float32)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


EDGELESS = synth.symmetric_csr(5, np.zeros((0, 2), np.int64), self_loops=False)


@pytest.mark.parametrize("name", list(GRAPHS) + ["edgeless"])
def test_prepare_fused_equals_separate(name):
    """gnn_csr_prepare (one launch) writes bit for bit the plan and the
    transposed values of gnn_csr_build_plan + gnn_csr_transpose_values."""
    g = EDGELESS if name == "edgeless" else GRAPHS[name]
    a, b = runtime.DeviceGraph(g), runtime.DeviceGraph(g)
    for dg in (a, b):  # stale bytes must not survive either path
        dg.plan.fill_(0xA5)
        dg.values_t.fill_(float("nan"))
    G.gnn_csr_prepare(a.struct(), a.plan, a.values_t)
    cb = b.struct()
    G.gnn_csr_build_plan(cb, b.plan)
    G.gnn_csr_transpose_values(cb, b.values_t)
    torch.cuda.synchronize()
    nb = G.gnn_plan_bytes(g.n, g.nnz)
    assert np.array_equal(a.plan[:nb].cpu().numpy(), b.plan[:nb].cpu().numpy())
    va = a.values_t[: g.nnz].cpu().numpy().view(np.uint32)
    vb = b.values_t[: g.nnz].cpu().numpy().view(np.uint32)
    assert np.array_equal(va, vb)


def test_prepare_argument_errors():
    g = GRAPHS["random"]
    dg = runtime.DeviceGraph(g)
    with pytest.raises(G.GnnError):  # plan too small
        G.gnn_csr_prepare(dg.struct(), dg.plan[:16], dg.values_t)
    with pytest.raises(G.GnnError):  # transposed values over the values
        G.gnn_csr_prepare(dg.struct(), dg.plan, dg.values)


def _ru(x, m=256):
    return (x + m - 1) // m * m


@pytest.mark.parametrize("name", ["powerlaw", "star700", "no_self_loops", "single",
                                  "random", "boundary"])
def test_plan_exact(name):
    g = GRAPHS[name]
    dg = prepared(g)
    torch.cuda.synchronize()
    hdr, raw = read_plan(dg)
    nblk, be, n, nnz = [int(v) for v in hdr[:4]]
    assert (n, nnz) == (g.n, g.nnz)
    assert be >= 64 and be & (be - 1) == 0
    assert nblk == max(1, -(-g.nnz // be))
    # window table right after the 256-byte header, then the entry rows
    binfo = raw[64: 64 + 4 * nblk].reshape(-1, 4).astype(np.int64)
    off_erow = _ru(256 + 16 * nblk)
    erow = raw[off_erow // 4: off_erow // 4 + g.nnz]
    ip = g.indptr.astype(np.int64)
    deg = np.diff(ip)
    # workgroup k owns the rows whose first entry is in window k (the last
    # one also the trailing empty rows): derived from the row pointers alone
    lo = [int(np.searchsorted(ip, k * be, side="left")) for k in range(nblk)] + [g.n]
    exp = np.array([(lo[k], lo[k + 1], ip[lo[k]], ip[lo[k + 1]]) for k in range(nblk)],
                   np.int64)
    assert np.array_equal(binfo, exp)
    # the windows partition rows and entries
    assert binfo[0, 0] == 0 and binfo[-1, 1] == g.n and binfo[-1, 3] == g.nnz
    assert (binfo[1:, 0] == binfo[:-1, 1]).all() and (binfo[1:, 2] == binfo[:-1, 3]).all()
    assert np.array_equal(erow, np.repeat(np.arange(g.n), deg))


# ---------------------------------------------------------------- aggregation

WIDTHS = [1, 3, 16, 50, 64, 128, 200, 300, 512, 602, 1024, 1030]


@pytest.mark.parametrize("name", ["powerlaw", "star700", "no_self_loops",
                                  "identity", "random", "boundary"])
@pytest.mark.parametrize("w", WIDTHS)
@pytest.mark.parametrize("transpose", [0, 1])
@pytest.mark.parametrize("layout", ["aligned", "unaligned"])
def test_spmm_parity(name, w, transpose, layout):
    g = GRAPHS[name]
    if g.n * w > 3_000_000:
        w = max(1, 3_000_000 // g.n)
    dg = prepared(g)
    x = np.random.default_rng(w).standard_normal((g.n, w)).astype(np.float32)
    if layout == "aligned":
        ld = (w + 3) // 4 * 4
        xin, out = to_dev(x, ld), empty_out(g.n, w, ld)
    else:
        ld = w + 1
        xin, out = unaligned(x, ld), empty_out(g.n, w, ld, shift=True)
    ws = torch.empty(max(G.gnn_spmm_workspace_bytes(dg.struct(), w), 256),
                     dtype=torch.uint8, device="cuda")
    G.gnn_spmm(dg.struct(), transpose, w, xin, xin.stride(0), out, out.stride(0), ws)
    torch.cuda.synchronize()
    ref = O.spmm_transpose(g, x) if transpose else O.spmm(g, x)
    assert maxrel(out, ref) <= TOL_SPMM


def _random_spmm_cases(count=48, seed=555):
    """Seeded random aggregations: uniform or power-law degrees (hub rows
    over several windows), with or without self loops, random values;
    widths from 1 to 1100 (narrow slices, the 10-lane groups, ragged
    ends), padded or odd row strides, both directions."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(count):
        n = int(rng.integers(1, 4000))
        w = int(rng.choice([int(rng.integers(1, 1100)), int(rng.integers(1, 128)) * 8]))
        w = max(1, min(w, 3_000_000 // n))
        cases.append((i, n, w, float(rng.uniform(0.3, 40.0)), bool(rng.integers(0, 2)),
                      bool(rng.integers(0, 2)), int(rng.integers(0, 2)),
                      int(rng.integers(0, 8)), bool(rng.integers(0, 2))))
    return cases


@pytest.mark.parametrize("case", _random_spmm_cases(), ids=lambda c: "case%d" % c[0])
def test_spmm_random_graphs(case):
    i, n, w, mean, powerlaw, loops, transpose, pad, shift = case
    if powerlaw and n > 2:
        g = synth.power_law_graph(n, 2.1, min(mean, n - 1.0), seed=100 + i)
    else:
        g = synth.random_graph(n, min(mean, max(n - 1.0, 0.0)), 200 + i,
                               self_loops=loops, values="random")
    dg = prepared(g)
    x = np.random.default_rng(300 + i).standard_normal((g.n, w)).astype(np.float32)
    ld = w + pad
    if shift:
        xin, out = unaligned(x, ld), empty_out(g.n, w, ld, shift=True)
    else:
        ld = (ld + 3) // 4 * 4
        xin, out = to_dev(x, ld), empty_out(g.n, w, ld)
    G.gnn_spmm(dg.struct(), transpose, w, xin, xin.stride(0), out, out.stride(0), None)
    torch.cuda.synchronize()
    ref = O.spmm_transpose(g, x) if transpose else O.spmm(g, x)
    assert maxrel(out, ref) <= TOL_SPMM


@pytest.mark.parametrize("w", [40, 200, 256])
@pytest.mark.parametrize("transpose", [0, 1])
def test_spmm_two_windows_per_workgroup(w, transpose):
    """Launches of more than 16,384 workgroups give each workgroup two
    consecutive plan windows: the 20,000-node workload graph (about 620 k
    entries, 2,400 windows, 8 column slices), hubs spanning several windows,
    checked against the oracle."""
    g = synth.workload_graph(synth.WORKLOADS["cl2.1-n20000-f200-h512-L5"])
    dg = prepared(g)
    assert -(-g.nnz // 256) * 8 > 16384
    x = np.random.default_rng(w + transpose).standard_normal((g.n, w)).astype(np.float32)
    xin, out = to_dev(x, w), empty_out(g.n, w, w)
    G.gnn_spmm(dg.struct(), transpose, w, xin, w, out, w, None)
    torch.cuda.synchronize()
    ref = O.spmm_transpose(g, x) if transpose else O.spmm(g, x)
    assert maxrel(out, ref) <= TOL_SPMM


FLOOR_CASES = [("powerlaw", 16), ("powerlaw", 300), ("star700", 512), ("boundary", 602),
               ("random", 64), ("identity", 1030)]


@pytest.mark.parametrize("name,w", FLOOR_CASES + [("workload", 512), ("workload", 602)])
@pytest.mark.parametrize("transpose", [0, 1])
def test_spmm_gather_floor_column_sums(name, w, transpose):
    """The gather floor (a measurement aid) writes every output row once and
    keeps the column sums of the aggregation: sum_v out[v, :] equals
    1^T (A_s X) (resp. 1^T (A_s^T X)), up to fp32 summation error measured
    against the column sums of |A_s| |X|."""
    g = (synth.workload_graph(synth.WORKLOADS["cl2.1-n8000-f602-h512-L2"])
         if name == "workload" else GRAPHS[name])
    if g.n * w > 3_000_000 and name != "workload":
        w = max(4, 3_000_000 // g.n // 4 * 4)
    dg = prepared(g)
    x = np.random.default_rng(w + 7).standard_normal((g.n, w)).astype(np.float32)
    ld = (w + 3) // 4 * 4
    xin, out = to_dev(x, ld), empty_out(g.n, w, ld)
    G.gnn_spmm_gather_floor(dg.struct(), transpose, w, xin, ld, out, ld)
    torch.cuda.synchronize()
    o = out.cpu().numpy().astype(np.float64)
    assert np.isfinite(o).all()
    ref = (O.spmm_transpose(g, x) if transpose else O.spmm(g, x)).sum(axis=0)
    # |A| |X| column sums (the transpose has the same entries, moved)
    rows = np.repeat(np.arange(g.n), np.diff(g.indptr.astype(np.int64)))
    src = rows if transpose else g.indices
    absx = np.abs(x.astype(np.float64))
    scale = (np.abs(g.values.astype(np.float64))[:, None] * absx[src]).sum(axis=0)
    assert np.all(np.abs(o.sum(axis=0) - ref) <= 1e-5 * scale + 1e-30)


def test_spmm_empty_graph_and_empty_rows():
    g = synth.symmetric_csr(6, np.array([[0, 1]]), self_loops=False)
    dg = prepared(g)
    x = np.arange(24, dtype=np.float32).reshape(6, 4)
    out = empty_out(6, 4)
    G.gnn_spmm(dg.struct(), 0, 4, to_dev(x), 4, out, 4, None)
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    assert np.array_equal(o[2:], np.zeros((4, 4), np.float32))
    assert np.array_equal(o[0], x[1]) and np.array_equal(o[1], x[0])


# ------------------------------------------------------------------- GEMM

# one block per tile; split-K (few tiles, long K); stream-K (tiles that do
# not fill the chip, e.g. 2000 x 1300); ragged and empty shapes
GEMM_SHAPES = [(1, 1, 1), (37, 45, 29), (128, 128, 32), (130, 257, 70),
               (1000, 128, 50), (602, 512, 8000), (300, 96, 4099), (64, 64, 0),
               (2001, 1300, 100), (8000, 602, 1024)]


# the two fp32 product paths: three-piece bf16 split (default) and the
# fp32 matrix-core instruction
MODES = {"split": 0, "f32_mfma": G.GNN_FLAG_F32_MFMA}


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
@pytest.mark.parametrize("ta", [0, 1])
@pytest.mark.parametrize("tb", [0, 1])
@pytest.mark.parametrize("layout", ["aligned", "unaligned"])
@pytest.mark.parametrize("mode", list(MODES))
def test_gemm_parity(M, N, K, ta, tb, layout, mode):
    rng = np.random.default_rng(M * 7 + N * 3 + K)
    a = rng.standard_normal((K, M) if ta else (M, K)).astype(np.float32)
    b = rng.standard_normal((N, K) if tb else (K, N)).astype(np.float32)
    if layout == "aligned":
        A = to_dev(a, (a.shape[1] + 3) // 4 * 4)
        B = to_dev(b, (b.shape[1] + 3) // 4 * 4)
        C = empty_out(M, N, (N + 3) // 4 * 4)
    else:
        A = unaligned(a, a.shape[1] + 1)
        B = unaligned(b, b.shape[1] + 3)
        C = empty_out(M, N, N + 1, shift=True)
    ws = torch.empty(max(G.gnn_gemm_workspace_bytes(M, N, K), 256),
                     dtype=torch.uint8, device="cuda")
    G.gnn_gemm(ta, tb, M, N, K, A, A.stride(0), B, B.stride(0), C, C.stride(0),
               MODES[mode], ws)
    torch.cuda.synchronize()
    aa = a.T if ta else a
    bb = b.T if tb else b
    ref = O.mm_nn(aa, bb) if K > 0 else np.zeros((M, N))
    assert maxrel(C, ref) <= TOL


def _random_gemm_cases(count=90, seed=77):
    """Seeded random shapes over the work-split regimes (one block per tile,
    split-K for few tiles over a long K, stream-K in between), all four
    transposes, aligned or shifted layouts and the three product modes."""
    rng = np.random.default_rng(seed)
    modes = [0, G.GNN_FLAG_F32_MFMA, G.GNN_FLAG_BF16]
    cases = []
    for i in range(count):
        kind = i % 3
        if kind == 0:    # many tiles
            M, N, K = int(rng.integers(1500, 6000)), int(rng.integers(200, 1100)), \
                int(rng.integers(1, 700))
        elif kind == 1:  # few tiles, long K
            M, N, K = int(rng.integers(1, 700)), int(rng.integers(1, 600)), \
                int(rng.integers(1000, 9000))
        else:            # in between
            M, N, K = int(rng.integers(300, 3000)), int(rng.integers(100, 1400)), \
                int(rng.integers(20, 3000))
        cases.append((i, M, N, K, int(rng.integers(0, 2)), int(rng.integers(0, 2)),
                      bool(rng.integers(0, 2)), modes[int(rng.integers(0, 3))]))
    return cases


@pytest.mark.parametrize("case", _random_gemm_cases(), ids=lambda c: "case%d" % c[0])
def test_gemm_random_shapes(case):
    _, M, N, K, ta, tb, aligned, flags = case
    rng = np.random.default_rng(M + 5 * N + 11 * K)
    a = rng.standard_normal((K, M) if ta else (M, K)).astype(np.float32)
    b = rng.standard_normal((N, K) if tb else (K, N)).astype(np.float32)
    if aligned:
        A = to_dev(a, (a.shape[1] + 3) // 4 * 4)
        B = to_dev(b, (b.shape[1] + 3) // 4 * 4)
        C = empty_out(M, N, (N + 3) // 4 * 4)
    else:
        A = unaligned(a, a.shape[1] + 1)
        B = unaligned(b, b.shape[1] + 3)
        C = empty_out(M, N, N + 1, shift=True)
    ws = torch.empty(max(G.gnn_gemm_workspace_bytes(M, N, K), 256),
                     dtype=torch.uint8, device="cuda")
    G.gnn_gemm(ta, tb, M, N, K, A, A.stride(0), B, B.stride(0), C, C.stride(0), flags, ws)
    torch.cuda.synchronize()
    if flags == G.GNN_FLAG_BF16:   # exact products of the rounded operands
        a, b = O.round_bf16(a), O.round_bf16(b)
    ref = O.mm_nn(a.T if ta else a, b.T if tb else b)
    assert maxrel(C, ref) <= (TOL_BF16_KERNEL if flags == G.GNN_FLAG_BF16 else TOL)


def _gemm(a, b, flags):
    M, K = a.shape
    N = b.shape[1]
    A, B = to_dev(a), to_dev(b)
    C = empty_out(M, N, N)
    ws = torch.empty(max(G.gnn_gemm_workspace_bytes(M, N, K), 256),
                     dtype=torch.uint8, device="cuda")
    G.gnn_gemm(0, 0, M, N, K, A, K, B, N, C, N, flags, ws)
    torch.cuda.synchronize()
    return C.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("ta_tb", [(0, 0), (1, 0), (0, 1), (1, 1)])
@pytest.mark.parametrize("full", ["a", "b"])
def test_gemm_split_keeps_every_operand_bit(ta_tb, full):
    """One operand has all 24 significand bits in use (1 + 2^-9 + 2^-18 +
    2^-23, scaled by powers of two: hi, mid and lo pieces all nonzero), the
    other selects one entry per output with a power-of-two weight, so every
    exact result is an fp32 number.  The split path and the fp32 path must
    return it bit for bit; the bf16 path, which keeps 8 bits, cannot."""
    ta, tb = ta_tb
    M, N, K = 96, 80, 64
    rng = np.random.default_rng(5)
    sig = 1.0 + 2.0 ** -9 + 2.0 ** -18 + 2.0 ** -23

    def dense(r, c):
        return (sig * rng.choice([1.0, -1.0], size=(r, c))
                * np.ldexp(1.0, rng.integers(-3, 4, size=(r, c))))

    def select(r, c, axis):
        m = np.zeros((r, c))
        if axis == 0:   # one nonzero per column
            m[rng.integers(0, r, size=c), np.arange(c)] = np.ldexp(1.0, -rng.integers(0, 3, size=c))
        else:           # one nonzero per row
            m[np.arange(r), rng.integers(0, c, size=r)] = np.ldexp(1.0, -rng.integers(0, 3, size=r))
        return m

    if full == "a":
        a, b = dense(M, K), select(K, N, 0)
    else:
        a, b = select(M, K, 1), dense(K, N)
    a, b = a.astype(np.float32), b.astype(np.float32)
    ref = a.astype(np.float64) @ b.astype(np.float64)
    assert np.array_equal(ref.astype(np.float32).astype(np.float64), ref)
    A = to_dev(np.ascontiguousarray(a.T) if ta else a)
    B = to_dev(np.ascontiguousarray(b.T) if tb else b)
    out = {}
    for name, fl in (("split", 0), ("f32_mfma", G.GNN_FLAG_F32_MFMA),
                     ("bf16", G.GNN_FLAG_BF16)):
        C = empty_out(M, N, N)
        ws = torch.empty(max(G.gnn_gemm_workspace_bytes(M, N, K), 256),
                         dtype=torch.uint8, device="cuda")
        G.gnn_gemm(ta, tb, M, N, K, A, A.stride(0), B, B.stride(0), C, C.stride(0),
                   fl, ws)
        torch.cuda.synchronize()
        out[name] = C.cpu().numpy().astype(np.float64)
    assert np.array_equal(out["split"], ref)
    assert np.array_equal(out["f32_mfma"], ref)
    assert not np.array_equal(out["bf16"], ref)


@pytest.mark.parametrize("M,N,K", [(2001, 1300, 100), (1000, 512, 64), (256, 384, 700)])
@pytest.mark.parametrize("flags", [0, G.GNN_FLAG_F32_MFMA, G.GNN_FLAG_BF16])
def test_gemm_epilogue_paths_bit_identical(M, N, K, flags):
    """Whole interior tiles of a float4-aligned C are written through LDS as
    float4 rows; the same product into a C 4 bytes off alignment takes the
    per-element path.  Both must hold the same bits everywhere."""
    rng = np.random.default_rng(M + N + K + flags)
    a = rng.standard_normal((M, K)).astype(np.float32)
    b = rng.standard_normal((K, N)).astype(np.float32)
    A, B = to_dev(a), to_dev(b)
    ws = torch.empty(max(G.gnn_gemm_workspace_bytes(M, N, K), 256),
                     dtype=torch.uint8, device="cuda")
    outs = []
    for shift in (False, True):
        C = empty_out(M, N, N + 4, shift=shift)
        G.gnn_gemm(0, 0, M, N, K, A, K, B, N, C, C.stride(0), flags, ws)
        torch.cuda.synchronize()
        outs.append(C.cpu().numpy().copy())
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
    assert maxrel(outs[0], O.mm_nn(a, b)) <= (TOL if flags != G.GNN_FLAG_BF16 else 2e-2)


@pytest.mark.parametrize("M,N,K", [(2000, 1024, 1024), (602, 512, 8000)])
def test_gemm_split_accuracy_matches_f32_mfma(M, N, K):
    """Against the double-precision product, the split path's error is of
    the fp32 path's size (measured: 1.1e-6 against 1.5e-6 at 8000 x 1024 x
    1024): no more than twice it, and far inside the layer tolerance."""
    rng = np.random.default_rng(M + N + K)
    a = rng.standard_normal((M, K)).astype(np.float32)
    b = (rng.standard_normal((K, N)) * 0.05).astype(np.float32)
    ref = O.mm_nn(a, b)
    scale = np.abs(ref).max()
    e_split = np.abs(_gemm(a, b, 0) - ref).max() / scale
    e_f32 = np.abs(_gemm(a, b, G.GNN_FLAG_F32_MFMA) - ref).max() / scale
    assert e_split <= 2 * e_f32 + 1e-7, (e_split, e_f32)
    assert e_split <= 1e-5


# --------------------------------------------------------------- one layer

def layer_inputs(n, f_in, h, seed, bias):
    rng = np.random.default_rng(seed)
    g = synth.power_law_graph(n, 2.1, 8.0, seed=seed) if n > 1 else synth.identity_graph(n)
    x = rng.standard_normal((n, f_in)).astype(np.float32)
    p = synth.LayerParams(synth.glorot(f_in, h, rng), synth.glorot(f_in, h, rng))
    if bias:
        p.b_self = rng.standard_normal(h).astype(np.float32) * 0.1
        p.b_neigh = rng.standard_normal(h).astype(np.float32) * 0.1
    dy = rng.standard_normal((n, 2 * h)).astype(np.float32)
    return g, x, p, dy


def run_layer(g, x, p, y_for_bwd, dy, order, pad=16, want_dx=True, flags=0):
    f_in, h = p.w_self.shape
    dg = prepared(g)
    st = runtime.SageStack(dg, [p], f_in, order=order, pad=pad, flags=flags)
    xd = to_dev(x, (f_in + pad - 1) // pad * pad)
    st.forward(xd)
    torch.cuda.synchronize()
    y = st.layers[0]["Y"].cpu().numpy().copy()
    # the backward pass gets the oracle's forward output as Y (teacher forcing)
    st.layers[0]["Y"].copy_(torch.from_numpy(y_for_bwd.astype(np.float32)).cuda())
    st.backward(to_dev(dy), want_dx_first=want_dx)
    torch.cuda.synchronize()
    L = st.layers[0]
    out = {"Y": y, "dW_self": L["dW_self"].cpu().numpy(),
           "dW_neigh": L["dW_neigh"].cpu().numpy(),
           "dX": L["dX"].cpu().numpy() if want_dx else None}
    if p.b_self is not None:
        out["db_self"] = L["db_self"].cpu().numpy()
        out["db_neigh"] = L["db_neigh"].cpu().numpy()
    return out


LAYER_CASES = [(1, 7, 5), (37, 7, 5), (500, 50, 128), (400, 130, 64),
               (300, 64, 64), (257, 33, 100)]


@pytest.mark.parametrize("n,f_in,h", LAYER_CASES)
@pytest.mark.parametrize("order", [1, 2])
@pytest.mark.parametrize("bias", [False, True])
@pytest.mark.parametrize("mode", list(MODES))
def test_layer_parity(n, f_in, h, order, bias, mode):
    g, x, p, dy = layer_inputs(n, f_in, h, n + f_in + h, bias)
    y_ref = O.sage_fwd(g, x, p.w_self, p.w_neigh, p.b_self, p.b_neigh)
    y32 = y_ref.astype(np.float32)
    got = run_layer(g, x, p, y32, dy, order, flags=MODES[mode])
    assert maxrel(got["Y"], y_ref) <= TOL
    r = O.sage_bwd(g, x, p.w_self, p.w_neigh, y32, dy, want_db=bias)
    for k in ("dX", "dW_self", "dW_neigh") + (("db_self", "db_neigh") if bias else ()):
        assert maxrel(got[k], r[k]) <= TOL, k


def _random_layer_cases(count=96, seed=2024):
    """Seeded random layer shapes and options: odd and aligned widths,
    padded strides, with or without bias and dX, all three product modes
    (the split-K and stream-K launches, held reductions and bf16 operand
    storage all come up across them)."""
    rng = np.random.default_rng(seed)
    modes = [0, G.GNN_FLAG_F32_MFMA, G.GNN_FLAG_BF16]
    cases = []
    for i in range(count):
        n = int(rng.integers(2, 900))
        f_in = int(rng.choice([int(rng.integers(1, 160)), int(rng.integers(1, 40)) * 8]))
        h = int(rng.choice([int(rng.integers(1, 140)), int(rng.integers(1, 32)) * 8]))
        cases.append((i, n, f_in, h, int(rng.integers(1, 3)), bool(rng.integers(0, 2)),
                      bool(rng.integers(0, 2)), modes[i % 3], int(rng.choice([1, 4, 16]))))
    return cases


@pytest.mark.parametrize("case", _random_layer_cases(), ids=lambda c: "case%d" % c[0])
def test_layer_random_shapes(case):
    _, n, f_in, h, order, bias, want_dx, flags, pad = case
    g, x, p, dy = layer_inputs(n, f_in, h, 1000 + n + f_in + h, bias)
    y_ref = O.sage_fwd(g, x, p.w_self, p.w_neigh, p.b_self, p.b_neigh)
    y32 = y_ref.astype(np.float32)
    got = run_layer(g, x, p, y32, dy, order, pad=pad, want_dx=want_dx, flags=flags)
    tol = 2e-2 if flags == G.GNN_FLAG_BF16 else TOL
    assert maxrel(got["Y"], y_ref) <= tol
    r = O.sage_bwd(g, x, p.w_self, p.w_neigh, y32, dy, want_dx=want_dx, want_db=bias)
    keys = ("dW_self", "dW_neigh") + (("dX",) if want_dx else ()) + \
        (("db_self", "db_neigh") if bias else ())
    for k in keys:
        assert maxrel(got[k], r[k]) <= tol, k


@pytest.mark.parametrize("case", _random_layer_cases(count=24, seed=3033),
                         ids=lambda c: "case%d" % c[0])
def test_layer_random_shapes_row_normalized(case):
    """The random layer cases with GNN_FLAG_ROW_NORMALIZED added to the
    product mode: A_s = D^-1 A taken from the pattern (the graphs store
    1/deg, so the oracle's value-based layer is the same operator)."""
    _random_row_normalized_layer(case[:7] + (case[7] | G.GNN_FLAG_ROW_NORMALIZED, case[8]))


def _random_row_normalized_layer(case):
    _, n, f_in, h, order, bias, want_dx, flags, pad = case
    g, x, p, dy = layer_inputs(n, f_in, h, 4000 + n + f_in + h, bias)
    y_ref = O.sage_fwd(g, x, p.w_self, p.w_neigh, p.b_self, p.b_neigh)
    y32 = y_ref.astype(np.float32)
    got = run_layer(g, x, p, y32, dy, order, pad=pad, want_dx=want_dx, flags=flags)
    tol = 2e-2 if flags & G.GNN_FLAG_BF16 else TOL
    assert maxrel(got["Y"], y_ref) <= tol
    r = O.sage_bwd(g, x, p.w_self, p.w_neigh, y32, dy, want_dx=want_dx, want_db=bias)
    keys = ("dW_self", "dW_neigh") + (("dX",) if want_dx else ()) + \
        (("db_self", "db_neigh") if bias else ())
    for k in keys:
        assert maxrel(got[k], r[k]) <= tol, k


@pytest.mark.parametrize("flags", [0, G.GNN_FLAG_F32_MFMA, G.GNN_FLAG_BF16])
@pytest.mark.parametrize("order", [1, 2])
def test_layer_zero_nodes(flags, order):
    """An empty subgraph: the forward writes nothing and the backward gives
    zero weight and bias gradients, in every product mode (the weight
    gradients are products over K = 0)."""
    g = synth.identity_graph(0)
    dg = prepared(g)
    f_in, h = 6, 5
    rng = np.random.default_rng(3)
    p = synth.LayerParams(synth.glorot(f_in, h, rng), synth.glorot(f_in, h, rng),
                          rng.standard_normal(h).astype(np.float32),
                          rng.standard_normal(h).astype(np.float32))
    st = runtime.SageStack(dg, [p], f_in, order=order, flags=flags)
    st.forward(torch.empty((0, f_in), device="cuda"))
    L = st.layers[0]
    keys = ("dW_self", "dW_neigh", "db_self", "db_neigh")
    for k in keys:
        L[k].fill_(float("nan"))
    st.backward(torch.empty((0, 2 * h), device="cuda"))
    torch.cuda.synchronize()
    for k in keys:
        assert np.array_equal(L[k].cpu().numpy(), np.zeros(L[k].shape, np.float32)), k


@pytest.mark.parametrize("flags", [0, G.GNN_FLAG_F32_MFMA, G.GNN_FLAG_BF16])
@pytest.mark.parametrize("order", [1, 2])
def test_layer_edgeless_subgraph(flags, order):
    """A subgraph whose nodes hold no stored entries at all (no self loops:
    every row empty, one window owning all of them).  Section 2.1's
    aggregation of an empty row is zero, so Y's neighbour half is
    ReLU(b_neigh), the weight gradient dW_neigh is exactly zero and the
    transposed aggregation adds nothing to dX; forward and backward against
    the oracle in every product mode and both orders."""
    n, f_in, h = 37, 12, 10
    g = synth.symmetric_csr(n, np.zeros((0, 2), np.int64), self_loops=False)
    assert g.nnz == 0
    rng = np.random.default_rng(11)
    x = rng.standard_normal((n, f_in)).astype(np.float32)
    p = synth.LayerParams(synth.glorot(f_in, h, rng), synth.glorot(f_in, h, rng),
                          rng.standard_normal(h).astype(np.float32) * 0.1,
                          rng.standard_normal(h).astype(np.float32) * 0.1)
    dy = rng.standard_normal((n, 2 * h)).astype(np.float32)
    y_ref = O.sage_fwd(g, x, p.w_self, p.w_neigh, p.b_self, p.b_neigh)
    y32 = y_ref.astype(np.float32)
    got = run_layer(g, x, p, y32, dy, order, flags=flags)
    tol = TOL_BF16_LAYER if flags == G.GNN_FLAG_BF16 else TOL
    assert maxrel(got["Y"], y_ref) <= tol
    nb = np.broadcast_to(np.maximum(p.b_neigh, 0), (n, h))
    assert np.array_equal(got["Y"][:, h:], nb.astype(np.float32))
    r = O.sage_bwd(g, x, p.w_self, p.w_neigh, y32, dy, want_db=True)
    assert not np.any(r["dW_neigh"])
    for k in ("dX", "dW_self", "dW_neigh", "db_self", "db_neigh"):
        assert maxrel(got[k], r[k]) <= tol, k


@pytest.mark.parametrize("order", [1, 2])
def test_layer_without_input_gradient(order):
    g, x, p, dy = layer_inputs(200, 40, 24, 5, False)
    y32 = O.sage_fwd(g, x, p.w_self, p.w_neigh).astype(np.float32)
    got = run_layer(g, x, p, y32, dy, order, want_dx=False)
    r = O.sage_bwd(g, x, p.w_self, p.w_neigh, y32, dy, want_dx=False)
    assert maxrel(got["dW_self"], r["dW_self"]) <= TOL
    assert maxrel(got["dW_neigh"], r["dW_neigh"]) <= TOL


@pytest.mark.parametrize("order", [1, 2])
def test_layer_unpadded_rows(order):
    # row strides equal to the widths (602 floats is not a multiple of 4)
    g, x, p, dy = layer_inputs(300, 602, 40, 11, False)
    y_ref = O.sage_fwd(g, x, p.w_self, p.w_neigh)
    y32 = y_ref.astype(np.float32)
    got = run_layer(g, x, p, y32, dy, order, pad=1)
    r = O.sage_bwd(g, x, p.w_self, p.w_neigh, y32, dy)
    assert maxrel(got["Y"], y_ref) <= TOL
    for k in ("dX", "dW_self", "dW_neigh"):
        assert maxrel(got[k], r[k]) <= TOL, k


# ------------------------------------------- GNN_FLAG_ROW_NORMALIZED

RN = G.GNN_FLAG_ROW_NORMALIZED


def run_rn_pair(g, x, p, y32, dy, order, pad=16):
    """The same layer through the general path (values = fp32(1/deg), the
    transposed values from the preparation) and with GNN_FLAG_ROW_NORMALIZED,
    for which the value arrays are overwritten with NaN first (a read of
    them would show); both backward passes take y32 as Y."""
    f_in, h = p.w_self.shape
    outs = {}
    for rn in (False, True):
        dg = prepared(g)
        if rn:
            torch.cuda.synchronize()
            dg.values.fill_(float("nan"))
            dg.values_t.fill_(float("nan"))
        st = runtime.SageStack(dg, [p], f_in, order=order, pad=pad,
                               flags=RN if rn else 0)
        st.forward(to_dev(x, (f_in + pad - 1) // pad * pad))
        torch.cuda.synchronize()
        o = {"Y": st.layers[0]["Y"].cpu().numpy().copy()}
        st.layers[0]["Y"].copy_(torch.from_numpy(y32).cuda())
        st.backward(to_dev(dy))
        torch.cuda.synchronize()
        for k in ("dX", "dW_self", "dW_neigh"):
            o[k] = st.layers[0][k].cpu().numpy().copy()
        outs[rn] = o
        del st
    return outs


RN_GRAPHS = {k: GRAPHS[k] for k in ("powerlaw", "star700", "no_self_loops", "identity",
                                    "path4", "single")}
RN_GRAPHS["random_rownorm"] = synth.random_graph(300, 6.0, 1)  # values 1/deg


@pytest.mark.parametrize("name", list(RN_GRAPHS))
@pytest.mark.parametrize("order", [1, 2])
def test_row_normalized_flag(name, order):
    """Section 2.1's A_s = D^-1 A taken from the pattern alone: within 1e-5
    of the general path on every output (forward and backward, both
    orders; empty rows in no_self_loops), and within 1e-4 of the oracle."""
    g = RN_GRAPHS[name]
    assert np.array_equal(g.values, (1.0 / np.repeat(g.degrees(), g.degrees())
                                     ).astype(np.float32))
    f_in, h = (24, 40) if order == 1 else (40, 24)
    rng = np.random.default_rng(order + g.n)
    x = rng.standard_normal((g.n, f_in)).astype(np.float32)
    p = synth.LayerParams(synth.glorot(f_in, h, rng), synth.glorot(f_in, h, rng))
    dy = rng.standard_normal((g.n, 2 * h)).astype(np.float32)
    y_ref = O.sage_fwd(g, x, p.w_self, p.w_neigh)
    y32 = y_ref.astype(np.float32)
    outs = run_rn_pair(g, x, p, y32, dy, order)
    r = O.sage_bwd(g, x, p.w_self, p.w_neigh, y32, dy)
    for k in ("Y", "dX", "dW_self", "dW_neigh"):
        assert maxrel(outs[True][k], outs[False][k]) <= TOL_SPMM, k
        assert maxrel(outs[True][k], y_ref if k == "Y" else r[k]) <= TOL, k


@pytest.mark.parametrize("name,layer", [("cl2.1-n8000-f602-h512-L2", 0),
                                        ("cl2.1-n8000-f602-h512-L2", 1),
                                        ("cl2.1-n20000-f200-h512-L5", 0)])
def test_row_normalized_flag_full_size(name, layer):
    """The benchmark's layer shapes at full size (8,000 nodes: 602 -> 2 x 512
    and 1024 -> 2 x 512, order 2; 20,000 nodes: 200 -> 2 x 512, order 1 with
    two plan windows per workgroup): every element within 1e-5 of the
    general path."""
    wl = synth.WORKLOADS[name]
    g = synth.workload_graph(wl)
    f_in, h = synth.layer_dims(wl)[layer]
    rng = np.random.default_rng(77 + layer)
    x = rng.standard_normal((g.n, f_in)).astype(np.float32)
    if layer:
        x = np.maximum(x, 0)
    p = synth.LayerParams(synth.glorot(f_in, h, rng), synth.glorot(f_in, h, rng))
    ysyn = np.maximum(rng.standard_normal((g.n, 2 * h)), 0).astype(np.float32)
    dy = rng.standard_normal((g.n, 2 * h)).astype(np.float32)
    outs = run_rn_pair(g, x, p, ysyn, dy, 0)
    for k in ("Y", "dX", "dW_self", "dW_neigh"):
        assert maxrel(outs[True][k], outs[False][k]) <= TOL_SPMM, k


# ------------------------------------------------------ whole stacks, C ABI

@pytest.mark.parametrize("fuse", [True, False])
def test_tiny_workload_stack_end_to_end(fuse):
    wl = synth.WORKLOADS[synth.TINY_WORKLOAD]
    inp = synth.workload_inputs(wl)
    g, x, params, dy = inp["graph"], inp["x"], inp["params"], inp["dy"]
    ref = O.sage_stack(g, x, params, dy)
    dg = prepared(g)
    st = runtime.SageStack(dg, params, wl.f_in, fuse_masks=fuse)
    y = st.forward(to_dev(x, 64))
    st.backward(to_dev(dy))
    torch.cuda.synchronize()
    assert maxrel(y, ref["ys"][-1]) <= TOL
    for l in range(wl.layers):
        L, R = st.layers[l], ref["grads"][l]
        assert maxrel(L["Y"], ref["ys"][l]) <= TOL
        for k in ("dW_self", "dW_neigh"):
            assert maxrel(L[k], R[k]) <= TOL, (l, k)
        dx_ref = R["dX"]
        if fuse and l > 0:  # masked by the sign of this layer's input
            dx_ref = dx_ref * (st.layers[l - 1]["Y"].cpu().numpy() > 0)
        assert maxrel(L["dX"], dx_ref) <= TOL, (l, "dX")


def test_stack_step_graph_replay():
    """One propagation step (plan, transposed values, forward and backward of
    the whole stack) captured in a HIP graph: every replay, with eager steps
    and synchronisations between replays, gives bit for bit the eager step's
    outputs and gradients."""
    wl = synth.WORKLOADS[synth.TINY_WORKLOAD]
    inp = synth.workload_inputs(wl)
    g, x, params, dy = inp["graph"], inp["x"], inp["params"], inp["dy"]
    X, dY = to_dev(x, 64), to_dev(dy)
    dg_cap, dg_eag = runtime.DeviceGraph(g), runtime.DeviceGraph(g)
    cap = runtime.SageStack(dg_cap, params, wl.f_in)
    eag = runtime.SageStack(dg_eag, params, wl.f_in)

    def step(dg, st):
        dg.prepare()
        st.forward(X)
        st.backward(dY)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step(dg_cap, cap)  # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        step(dg_cap, cap)
    keys = ("Y", "dW_self", "dW_neigh", "dX")
    for it in range(3):
        for L in cap.layers:  # stale results must not survive a replay
            for k in keys:
                L[k].fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        step(dg_eag, eag)
        torch.cuda.synchronize()
        for l in range(wl.layers):
            for k in keys:
                a = cap.layers[l][k].cpu().numpy()
                b = eag.layers[l][k].cpu().numpy()
                assert np.array_equal(a, b), (it, l, k)


@pytest.mark.parametrize("order", [1, 2])
@pytest.mark.parametrize("bias", [False, True])
@pytest.mark.parametrize("mode,f_in,h", [("split", 40, 24), ("bf16", 40, 24),
                                         ("bf16", 37, 16)])
def test_layer_mask_flags_exact(order, bias, mode, f_in, h):
    """GNN_FLAG_DY_MASKED with a pre-masked dY, plus GNN_FLAG_DX_MASKED,
    gives bit for bit the plain backward's weight and bias gradients and its
    dX with the input's sign mask applied.  In bf16 mode (order 2) the plain
    backward keeps G_s and T as bf16 in its workspace and the GEMMs read
    them as bf16 operands, while the pre-masked path hands them over in
    fp32 and the GEMMs round them: the same values, so the same bits.  (h is
    a multiple of 4 so that the pre-masked dY's neighbour half, G_n = dY + h,
    is aggregated with the same lane groups and summation order as the
    masking pass's aligned G_n.)"""
    g = GRAPHS["powerlaw"]
    base = G.GNN_FLAG_BF16 if mode == "bf16" else 0
    rng = np.random.default_rng(7)
    p = synth.LayerParams(synth.glorot(f_in, h, rng), synth.glorot(f_in, h, rng),
                          rng.standard_normal(h) if bias else None,
                          rng.standard_normal(h) if bias else None)
    x = np.maximum(rng.standard_normal((g.n, f_in)), 0).astype(np.float32)  # post-ReLU input
    x[: g.n // 3] = rng.standard_normal((g.n // 3, f_in))   # and some signed rows
    dy = rng.standard_normal((g.n, 2 * h)).astype(np.float32)
    dg = prepared(g)
    outs = {}
    for how in ("plain", "fused"):
        st = runtime.SageStack(dg, [p], f_in, order=order, flags=base)
        xin = to_dev(x, 48)
        y = st.forward(xin)
        torch.cuda.synchronize()
        L = st.layers[0]
        d = to_dev(dy, L["Y"].stride(0))
        flags = 0
        if how == "fused":
            d = to_dev(np.where(y.cpu().numpy() > 0, dy, 0), L["Y"].stride(0))
            flags = G.GNN_FLAG_DY_MASKED | G.GNN_FLAG_DX_MASKED
        lay = st._layer(0, xin.stride(0), flags)
        G.gnn_prop_bwd(dg.struct(), lay, xin, L["W_self"], L["W_neigh"], L["Y"], d,
                       L["saved"], L["dX"], L["dW_self"], L["dW_neigh"],
                       L["db_self"], L["db_neigh"], st.workspace)
        torch.cuda.synchronize()
        outs[how] = {k: L[k].cpu().numpy().copy() for k in
                     ("dX", "dW_self", "dW_neigh") + (("db_self", "db_neigh") if bias else ())}
    a, b = outs["plain"], outs["fused"]
    for k in a:
        exp = a[k] if k != "dX" else np.where(x > 0, a[k], 0).astype(np.float32)
        assert np.array_equal(b[k].view(np.uint32), exp.view(np.uint32)), k


def test_bitwise_reproducible():
    wl = synth.WORKLOADS[synth.TINY_WORKLOAD]
    inp = synth.workload_inputs(wl)
    outs = []
    for _ in range(2):
        dg = prepared(inp["graph"])
        st = runtime.SageStack(dg, inp["params"], wl.f_in)
        st.forward(to_dev(inp["x"], 64))
        st.backward(to_dev(inp["dy"]))
        torch.cuda.synchronize()
        outs.append([t.cpu().numpy().copy() for L in st.layers
                     for t in (L["Y"], L["dX"], L["dW_self"], L["dW_neigh"])])
    for a, b in zip(*outs):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


# ---------------------------------------- full-size workloads, spot checked

@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_workload_layers_full_size(name):
    """Every layer shape of every workload at its real size, in the launch
    configuration the benchmark uses; outputs checked on sampled rows and
    weight-gradient entries against the oracle's per-output evaluation."""
    wl = synth.WORKLOADS[name]
    g = synth.workload_graph(wl)
    dg = prepared(g)
    deg = g.degrees()
    hub = int(np.argmax(deg))
    for l, (f_in, h) in enumerate(synth.layer_dims(wl)):
        rng = np.random.default_rng(1000 + l)
        x = rng.standard_normal((g.n, f_in)).astype(np.float32)
        if l > 0:  # post-ReLU activations
            x = np.maximum(x, 0)
        p = synth.LayerParams(synth.glorot(f_in, h, rng), synth.glorot(f_in, h, rng))
        ysyn = rng.standard_normal((g.n, 2 * h)).astype(np.float32)
        dy = rng.standard_normal((g.n, 2 * h)).astype(np.float32)
        st = runtime.SageStack(dg, [p], f_in)
        st.forward(to_dev(x, (f_in + 15) // 16 * 16))
        torch.cuda.synchronize()
        rows = sample_rows(g.n, 24, l, must=(0, g.n - 1, hub))
        y = st.layers[0]["Y"][torch.from_numpy(rows).cuda()].cpu().numpy()
        yr = O.sage_fwd_rows(g, x, p.w_self, p.w_neigh, rows)
        assert maxrel(y, yr) <= TOL, ("Y", l)
        st.layers[0]["Y"].copy_(torch.from_numpy(ysyn).cuda())
        st.backward(to_dev(dy))
        torch.cuda.synchronize()
        dx = st.layers[0]["dX"][torch.from_numpy(rows).cuda()].cpu().numpy()
        dxr = O.sage_bwd_dx_rows(g, p.w_self, p.w_neigh, ysyn, dy, rows)
        assert maxrel(dx, dxr) <= TOL, ("dX", l)
        ei = np.concatenate([[0, f_in - 1], rng.integers(0, f_in, 14)])
        ej = np.concatenate([[0, h - 1], rng.integers(0, h, 14)])
        ws, wn = O.sage_bwd_dw_entries(g, x, ysyn, dy, h, ei, ej)
        gs = st.layers[0]["dW_self"].cpu().numpy()[ei, ej]
        gn = st.layers[0]["dW_neigh"].cpu().numpy()[ei, ej]
        assert maxrel(gs, ws) <= TOL, ("dW_self", l)
        assert maxrel(gn, wn) <= TOL, ("dW_neigh", l)
        del st
        torch.cuda.empty_cache()


# -------------------------------------------------------------- validation

def test_validate_accepts_and_rejects():
    good = prepared(synth.power_law_graph(500, 2.1, 6.0, seed=4))
    assert good.validate(True) == G.GNN_OK
    # asymmetric pattern
    g = synth.csr_from_pairs(3, np.array([0, 0, 1, 2]), np.array([0, 1, 1, 2]))
    assert runtime.DeviceGraph(g).validate(True) == -3
    assert runtime.DeviceGraph(g).validate(False) == G.GNN_OK
    # unsorted row
    g = synth.path_graph(5)
    g.indices = g.indices.copy()
    g.indices[[0, 1]] = g.indices[[1, 0]]
    assert runtime.DeviceGraph(g).validate(False) == -3
    # index out of range
    g = synth.path_graph(5)
    g.indices = g.indices.copy()
    g.indices[-1] = 5
    assert runtime.DeviceGraph(g).validate(False) == -3
    # indptr not ending at nnz
    g = synth.path_graph(5)
    g.indptr = g.indptr.copy()
    g.indptr[-1] -= 1
    assert runtime.DeviceGraph(g).validate(False) == -3


# ----------------------------------------------------- bf16 matrix-core mode

TOL_BF16_KERNEL = 1e-5   # vs the oracle on bf16-rounded operands
TOL_BF16_LAYER = 2e-2    # vs the double-precision oracle on the fp32 inputs


@pytest.mark.parametrize("M,N,K", [(37, 45, 29), (128, 128, 64), (130, 257, 70),
                                   (602, 512, 8000), (2001, 1300, 100),
                                   (8000, 602, 1024), (64, 64, 0), (300, 96, 4099),
                                   (1000, 128, 50)])
@pytest.mark.parametrize("ta", [0, 1])
@pytest.mark.parametrize("tb", [0, 1])
def test_gemm_bf16_parity(M, N, K, ta, tb):
    # operands rounded to bf16 (nearest, ties to even) and multiplied exactly;
    # only the fp32 accumulation order differs from the oracle
    rng = np.random.default_rng(M + 3 * N + 7 * K)
    a = rng.standard_normal((K, M) if ta else (M, K)).astype(np.float32)
    b = rng.standard_normal((N, K) if tb else (K, N)).astype(np.float32)
    A = to_dev(a, (a.shape[1] + 3) // 4 * 4)
    B = to_dev(b, (b.shape[1] + 3) // 4 * 4)
    C = empty_out(M, N, (N + 3) // 4 * 4)
    ws = torch.empty(max(G.gnn_gemm_workspace_bytes(M, N, K), 256),
                     dtype=torch.uint8, device="cuda")
    G.gnn_gemm(ta, tb, M, N, K, A, A.stride(0), B, B.stride(0), C, C.stride(0),
               G.GNN_FLAG_BF16, ws)
    torch.cuda.synchronize()
    ra, rb = O.round_bf16(a), O.round_bf16(b)
    ref = O.mm_nn(ra.T if ta else ra, rb.T if tb else rb) if K > 0 else np.zeros((M, N))
    assert maxrel(C, ref) <= TOL_BF16_KERNEL


@pytest.mark.parametrize("n,f_in,h,bias", [(500, 50, 128, False), (400, 130, 64, True),
                                           (300, 602, 40, False), (300, 37, 13, True)])
@pytest.mark.parametrize("order", [1, 2])
def test_layer_bf16(n, f_in, h, bias, order):
    """bf16 products against the double-precision oracle at the bf16
    tolerance; h = 13 takes the per-element mask and the ragged bf16 stores
    of the transposed aggregation, the bias cases the bias gradients summed
    from Y and dY."""
    g, x, p, dy = layer_inputs(n, f_in, h, 77 + n, bias)
    y_ref = O.sage_fwd(g, x, p.w_self, p.w_neigh, p.b_self, p.b_neigh)
    y32 = y_ref.astype(np.float32)
    dg = prepared(g)
    st = runtime.SageStack(dg, [p], f_in, order=order, flags=G.GNN_FLAG_BF16)
    st.forward(to_dev(x, (f_in + 15) // 16 * 16))
    torch.cuda.synchronize()
    assert maxrel(st.layers[0]["Y"], y_ref) <= TOL_BF16_LAYER
    st.layers[0]["Y"].copy_(torch.from_numpy(y32).cuda())
    st.backward(to_dev(dy))
    torch.cuda.synchronize()
    r = O.sage_bwd(g, x, p.w_self, p.w_neigh, y32, dy, want_db=bias)
    for k in ("dX", "dW_self", "dW_neigh") + (("db_self", "db_neigh") if bias else ()):
        assert maxrel(st.layers[0][k], r[k]) <= TOL_BF16_LAYER, k


@pytest.mark.parametrize("name", ["cl2.1-n8000-f602-h512-L2", "cl2.3-n8000-f300-h512-L3"])
def test_workload_bf16_full_size(name):
    """The 8,000-node workloads at full size in bf16 mode, spot-checked
    against the double-precision oracle at the bf16 tolerance."""
    wl = synth.WORKLOADS[name]
    g = synth.workload_graph(wl)
    dg = prepared(g)
    hub = int(np.argmax(g.degrees()))
    for l, (f_in, h) in enumerate(synth.layer_dims(wl)):
        rng = np.random.default_rng(2000 + l)
        x = rng.standard_normal((g.n, f_in)).astype(np.float32)
        if l > 0:
            x = np.maximum(x, 0)
        p = synth.LayerParams(synth.glorot(f_in, h, rng), synth.glorot(f_in, h, rng))
        ysyn = rng.standard_normal((g.n, 2 * h)).astype(np.float32)
        dy = rng.standard_normal((g.n, 2 * h)).astype(np.float32)
        st = runtime.SageStack(dg, [p], f_in, flags=G.GNN_FLAG_BF16)
        st.forward(to_dev(x, (f_in + 15) // 16 * 16))
        torch.cuda.synchronize()
        rows = sample_rows(g.n, 16, l, must=(0, hub))
        y = st.layers[0]["Y"][torch.from_numpy(rows).cuda()].cpu().numpy()
        assert maxrel(y, O.sage_fwd_rows(g, x, p.w_self, p.w_neigh, rows)) <= TOL_BF16_LAYER
        st.layers[0]["Y"].copy_(torch.from_numpy(ysyn).cuda())
        st.backward(to_dev(dy))
        torch.cuda.synchronize()
        dx = st.layers[0]["dX"][torch.from_numpy(rows).cuda()].cpu().numpy()
        dxr = O.sage_bwd_dx_rows(g, p.w_self, p.w_neigh, ysyn, dy, rows)
        assert maxrel(dx, dxr) <= TOL_BF16_LAYER
        ei, ej = rng.integers(0, f_in, 12), rng.integers(0, h, 12)
        ws_, wn_ = O.sage_bwd_dw_entries(g, x, ysyn, dy, h, ei, ej)
        assert maxrel(st.layers[0]["dW_self"].cpu().numpy()[ei, ej], ws_) <= TOL_BF16_LAYER
        assert maxrel(st.layers[0]["dW_neigh"].cpu().numpy()[ei, ej], wn_) <= TOL_BF16_LAYER
        del st
