"""The streaming probe behind bench.py's hbm_ceiling (GPU): each kind moves
the bytes it claims (the write fills, the copy copies, the read leaves its
buffer alone) and reports a positive time."""
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    from paper_2402_09633_amd import gnn
    return gnn


def test_probe_kinds_move_their_bytes(G):
    n = (1 << 22) + 4  # floats: a ragged tail past the last full grid pass
    a = torch.arange(n, dtype=torch.float32, device="cuda")
    b = torch.full((n,), -7.0, device="cuda")
    ms = G.gnn_hbm_probe(G.GNN_PROBE_READ, a, b, 4 * n, 64, 2)
    torch.cuda.synchronize()
    assert ms > 0.0
    assert torch.equal(a, torch.arange(n, dtype=torch.float32, device="cuda"))
    assert float(b[0]) == -7.0  # the sink is written only for an impossible sum
    ms = G.gnn_hbm_probe(G.GNN_PROBE_COPY, a, b, 4 * n, 0, 2)
    torch.cuda.synchronize()
    assert ms > 0.0 and torch.equal(a, b)
    ms = G.gnn_hbm_probe(G.GNN_PROBE_WRITE, b, a, 4 * n, 3, 1)
    torch.cuda.synchronize()
    want = torch.tensor([1.0, 2.0, 3.0, 4.0], device="cuda").repeat(n // 4)
    assert ms > 0.0 and torch.equal(b, want)
