"""The library's per-stage profiler, through the C ABI: every stage of every
call (mode 1) or one iteration's three per-iteration stages per call
(GNN_PROFILE_SAMPLE); stage times come from events bound to the stages'
kernel dispatches, so each lies inside the call's total."""
import numpy as np
import pytest
import torch

from paper_2402_09633_amd import inputs as I
from tests.gpu_util import dev

pytestmark = pytest.mark.gpu
PER_ITER = ("edge_update", "aggregate", "node_update")
ONCE = ("csr", "node_enc", "edge_enc", "classifier")


@pytest.fixture(scope="module")
def G():
    from paper_2402_09633_amd import gnn
    return gnn


def _event():
    rng = np.random.default_rng(31)
    n, e = 20000, 70000
    x = rng.normal(size=(n, 3)).astype(np.float32)
    ei = rng.integers(0, n, size=(2, e)).astype(np.int32)
    return dev(x), dev(ei)


@pytest.mark.parametrize("dtype,flags", [(0, 0), (1, 0), (1, 8), (0, 4)])
def test_profile_modes_count_and_time_stages(G, dtype, flags):
    T, calls = 4, 3
    w = I.make_weights(3, 64, 1, 33)
    m = G.Model(w, G.make_dims(3, 64, T, dtype=dtype, flags=flags))
    x, ei = _event()
    out = torch.empty(ei.shape[1], device="cuda")
    try:
        m(x, ei, out)  # warm-up, not profiled
        torch.cuda.synchronize()
        G.gnn_profile_enable(m.handle, True)
        for _ in range(calls):
            m(x, ei, out)
        p = G.gnn_profile_read(m.handle)
        print(f"dtype={dtype} flags={flags} full: " +
              ", ".join(f"{k} {p[k]['launches']}/{p[k]['ms']:.3f}" for k in PER_ITER + ONCE + ("total",)),
              flush=True)
        assert p["n_calls"] == calls
        # fp16 weights: the edge encoder runs inside the first edge update
        inside = dtype == G.GNN_BF16 and flags & G.GNN_F16_WEIGHTS
        for k in ONCE + ("total",):
            if k == "edge_enc" and inside:
                assert p[k]["launches"] == 0 and p[k]["ms"] == 0.0, k
            else:
                assert p[k]["launches"] == calls and p[k]["ms"] > 0, k
        for k in PER_ITER:
            assert p[k]["launches"] == calls * T and p[k]["ms"] > 0, k
        # stage times are kernel run times inside the call's span
        parts = sum(p[k]["ms"] for k in PER_ITER + ONCE)
        assert parts <= p["total"]["ms"] * 1.001, (parts, p["total"]["ms"])

        G.gnn_profile_enable(m.handle, G.GNN_PROFILE_SAMPLE)
        for _ in range(calls):
            m(x, ei, out)
        q = G.gnn_profile_read(m.handle)
        assert q["n_calls"] == calls
        for k in PER_ITER:
            assert q[k]["launches"] == calls and q[k]["ms"] > 0, k
        for k in ONCE + ("total",):
            assert q[k]["launches"] == 0 and q[k]["ms"] == 0.0, k
        # a sampled launch takes about what an average full-mode launch takes
        for k in PER_ITER:
            full = p[k]["ms"] / p[k]["launches"]
            samp = q[k]["ms"] / q[k]["launches"]
            assert 0.5 * full < samp < 2.0 * full, (k, full, samp)

        G.gnn_profile_enable(m.handle, False)
        m(x, ei, out)
        r = G.gnn_profile_read(m.handle)
        assert r["n_calls"] == 0 and all(r[k]["launches"] == 0 for k in PER_ITER + ONCE)
        with pytest.raises(G.GnnError) as e:
            G.gnn_profile_enable(m.handle, 3)
        assert e.value.code == G.GNN_E_INVALID_ARG
    finally:
        m.close()


@pytest.mark.parametrize("T", [0, 1])
def test_profile_sampled_mode_few_iterations(G, T):
    """T = 0 has no iteration to sample (no stage timed, calls still
    counted); T = 1 samples its only iteration."""
    w = I.make_weights(3, 64, 1, 34)
    m = G.Model(w, G.make_dims(3, 64, T))
    x, ei = _event()
    out = torch.empty(ei.shape[1], device="cuda")
    try:
        G.gnn_profile_enable(m.handle, G.GNN_PROFILE_SAMPLE)
        for _ in range(2):
            m(x, ei, out)
        q = G.gnn_profile_read(m.handle)
        assert q["n_calls"] == 2
        for k in PER_ITER:
            assert q[k]["launches"] == (2 if T == 1 else 0), k
        for k in ONCE + ("total",):
            assert q[k]["launches"] == 0, k
        G.gnn_profile_enable(m.handle, True)
        m(x, ei, out)
        p = G.gnn_profile_read(m.handle)
        assert p["total"]["launches"] == 1 and p["classifier"]["launches"] == 1
        for k in PER_ITER:
            assert p[k]["launches"] == T, k
    finally:
        m.close()
