"""The matrix-core rate probe (gnn_mfma_rate_probe), a measurement aid.

Each wavefront adds the same register-operand product into its four
accumulators once per iteration, so doubling the iterations doubles every
thread's sum up to the rounding inside the matrix instruction's
accumulation (checked against the largest sum).  The clock pair gives a
shader clock in a plausible range.
"""
import pytest
import torch

from paper_2010_03166_amd import gnnprop as G

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("kind", [G.GNN_PROBE_MFMA_BF16, G.GNN_PROBE_MFMA_F32])
@pytest.mark.parametrize("blocks", [1, 7, 512])
def test_probe_sums_scale_with_iterations(kind, blocks):
    sink1 = torch.full((blocks * 512,), float("nan"), device="cuda")
    sink2 = torch.full((blocks * 512,), float("nan"), device="cuda")
    clocks = torch.zeros(2, dtype=torch.int64, device="cuda")
    G.gnn_mfma_rate_probe(kind, blocks, 1, sink1, clocks)
    G.gnn_mfma_rate_probe(kind, blocks, 2, sink2, clocks)
    torch.cuda.synchronize()
    a, b = sink1.cpu(), sink2.cpu()
    assert torch.isfinite(a).all() and torch.isfinite(b).all()
    scale = (2 * a).abs().max().item()
    assert scale > 0
    assert (b - 2 * a).abs().max().item() <= 1e-5 * scale


@pytest.mark.parametrize("kind", [G.GNN_PROBE_MFMA_BF16, G.GNN_PROBE_MFMA_F32])
def test_probe_clock_plausible(kind):
    sink = torch.empty(512 * 512, device="cuda")
    clocks = torch.zeros(2, dtype=torch.int64, device="cuda")
    G.gnn_mfma_rate_probe(kind, 512, 200, sink, clocks)
    torch.cuda.synchronize()
    cyc, ticks = (int(v) for v in clocks.cpu())
    assert cyc > 0 and ticks > 0
    assert 0.3 < 0.1 * cyc / ticks < 3.5


def test_probe_rejects_arguments_before_launch():
    sink = torch.empty(512, device="cuda")
    clocks = torch.zeros(2, dtype=torch.int64, device="cuda")
    with pytest.raises(G.GnnError):
        G.gnn_mfma_rate_probe(2, 1, 1, sink, clocks)
    with pytest.raises(G.GnnError):
        G.gnn_mfma_rate_probe(G.GNN_PROBE_MFMA_BF16, 1, 0, sink, clocks)
