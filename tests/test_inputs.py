"""Seeded generators: shapes, reproducibility and the geometric invariants."""
import math

import numpy as np
import pytest

from paper_2402_09633_amd import inputs as I


def test_tiny_graph_shape_and_no_self_loops():
    g = I.make_graph(I.CONFIGS["tiny"])
    assert g.x.shape == (2000, 3) and g.x.dtype == np.float32
    assert g.edge_index.shape == (2, 8000) and g.edge_index.dtype == np.int32
    assert (g.edge_index[0] != g.edge_index[1]).all()
    assert g.edge_index.min() >= 0 and g.edge_index.max() < 2000
    # features (r/1000, phi/pi, z/1000) inside their ranges
    assert (g.x[:, 0] >= 0.03 - 1e-7).all() and (g.x[:, 0] <= 1.0 + 1e-7).all()
    assert (np.abs(g.x[:, 1]) <= 1.0 + 1e-7).all() and (np.abs(g.x[:, 2]) <= 1.0 + 1e-7).all()


def test_generators_are_reproducible():
    a = I.make_graph(I.CONFIGS["tiny"])
    b = I.make_graph(I.CONFIGS["tiny"])
    assert a.digest() == b.digest()
    w1 = I.make_weights(3, 64, 1, 2000)
    w2 = I.make_weights(3, 64, 1, 2000)
    assert np.array_equal(w1, w2)


@pytest.mark.parametrize("n_nodes,scale", [(20_000, 1.0), (30_000, I.FULL_WINDOW_SCALE)])
def test_layered_graph_invariants(n_nodes, scale):
    dphi, dz = I.DPHI_MID * scale, I.DZ_MID * scale
    g = I.layered_graph(n_nodes, 7, dphi, dz)
    src, dst = g.edge_index.astype(np.int64)
    per = n_nodes // 10
    layer = np.minimum(np.arange(n_nodes) // per, 9)
    assert (layer[dst] == layer[src] + 1).all()          # adjacent layers only
    phi = g.x[:, 1].astype(np.float64) * math.pi
    z = g.x[:, 2].astype(np.float64) * 1000.0
    dp = np.abs((phi[dst] - phi[src] + math.pi) % (2 * math.pi) - math.pi)
    assert (dp < dphi + 1e-5).all() and (np.abs(z[dst] - z[src]) < dz + 1e-3).all()
    assert np.bincount(src, minlength=n_nodes).max() <= I.MAX_OUT_DEGREE
    assert (np.diff(src) >= 0).all()                     # emitted grouped by source
    r = g.x[:, 0] * 1000.0
    assert np.allclose(np.unique(np.round(r, 3)).size, 10)


def test_full_config_edge_count_near_one_million():
    g = I.make_graph(I.CONFIGS["full"])
    assert g.n_nodes == 300_000
    assert 0.98e6 < g.n_edges < 1.02e6


def test_weight_blob_layout():
    for F, H, S in [(3, 64, 1), (3, 128, 1), (3, 128, 8), (5, 64, 2)]:
        w = I.make_weights(F, H, S, 1)
        assert w.size == I.weight_count(F, H, S)
        v = I.blob_views(w, F, H, S)
        assert v["node_enc.0.W"].shape == (H, F)
        assert v["edge_cls.1.W"].shape == (1, H)
        a = math.sqrt(6.0 / (3 * H + H))
        assert np.abs(v["edge_cls.0.W"]).max() <= a
        assert (v["edge_mlp0.0.g"] == 1).all() and (v["edge_mlp0.0.beta"] == 0).all()
    assert I.weight_count(3, 128, 1) == 249_729


def test_batch_sizes_in_range():
    sizes = I.batch_sizes(I.CONFIGS["batch"])
    assert len(sizes) == 8 and all(240_000 <= n <= 360_000 for n in sizes)
