"""Shared helpers of the GPU parity tests (upload, compare, sampling)."""
import numpy as np
import torch

from paper_2010_03166_amd import gnnprop as G
from paper_2010_03166_amd import runtime


def maxrel(got, ref) -> float:
    """max |got - ref| / max |ref| over one tensor (0 for empty tensors)."""
    if isinstance(got, torch.Tensor):
        got = got.detach().cpu().numpy()
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    den = np.abs(ref).max()
    if den == 0:
        return float(np.abs(got).max())
    return float(np.abs(got - ref).max() / den)


def to_dev(a, ld=None) -> torch.Tensor:
    """float32 upload; with ld the rows are placed at that stride (the pad
    columns hold NaN so that a kernel reading them would show up)."""
    t = torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    if ld is None or t.dim() != 2 or ld == t.shape[1]:
        return t
    buf = torch.full((t.shape[0], ld), float("nan"), device="cuda")
    buf[:, : t.shape[1]] = t
    return buf[:, : t.shape[1]]


def unaligned(a, ld) -> torch.Tensor:
    """float32 matrix whose base address is 4 bytes past a 16-byte boundary
    and whose row stride is ld (forces the scalar paths)."""
    a = np.ascontiguousarray(a, np.float32)
    rows, cols = a.shape
    buf = torch.full((rows * ld + 8,), float("nan"), device="cuda")
    view = buf[1: 1 + rows * ld].view(rows, ld)[:, :cols] if rows else \
        buf[1:1].view(0, cols)
    view.copy_(torch.from_numpy(a).cuda())
    return view


def empty_out(rows, cols, ld=None, shift=False) -> torch.Tensor:
    ld = ld or cols
    if shift:
        buf = torch.full((rows * ld + 8,), float("nan"), device="cuda")
        return buf[1: 1 + rows * ld].view(rows, ld)[:, :cols]
    return torch.full((rows, ld), float("nan"), device="cuda")[:, :cols]


def prepared(csr) -> runtime.DeviceGraph:
    g = runtime.DeviceGraph(csr)
    g.prepare()
    return g


def read_plan(g: runtime.DeviceGraph):
    raw = g.plan.cpu().numpy().view(np.int32)
    hdr = raw[:8]
    # the header's first four words: items, long rows, chunk, n
    return hdr, raw


def sample_rows(n, k, seed, must=()):
    rng = np.random.default_rng(seed)
    rows = list(must) + list(rng.choice(n, size=min(k, n), replace=False))
    return np.array(sorted(set(int(r) for r in rows if 0 <= r < n)), np.int64)


def decision_flips(gpu_act, ref_act, bound=1e-4) -> int:
    """Activation decisions (value > 0: a ReLU or LeakyReLU passes its input
    unscaled) that the GPU took differently from the oracle's own forward
    pass.  Asserts that every such decision lies at the kink, i.e. that both
    activation values there are within bound * max|ref| of 0 (so rounding
    alone decided it), and returns how many there were."""
    if isinstance(gpu_act, torch.Tensor):
        gpu_act = gpu_act.detach().cpu().numpy()
    g = np.asarray(gpu_act, np.float64)
    r = np.asarray(ref_act, np.float64)
    assert g.shape == r.shape, (g.shape, r.shape)
    flip = (g > 0) != (r > 0)
    count = int(flip.sum())
    if count:
        lim = bound * max(float(np.abs(r).max()), 1e-300)
        worst = float(np.maximum(np.abs(g[flip]), np.abs(r[flip])).max())
        assert worst <= lim, ("decision far from the kink", count, worst, lim)
    return count
