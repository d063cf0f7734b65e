"""End-to-end parity of the HIP path with the CPU oracle, through the C ABI.

fp32: per-edge logits within 1e-4 * max(1, |z|) of the fp64 oracle.
bf16: per-edge scores within 2e-2 of the fp64 oracle of the same fp32 model.
Full-size events are compared on the stored oracle sample (tests/golden/),
after checking that the regenerated graph has the stored digest.
"""
import json
import os

import numpy as np
import pytest
import torch

from paper_2402_09633_amd import inputs as I
from tests.gpu_util import BF16_SCORE_ATOL, assert_logits_close, dev, run_model

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.fixture(scope="module")
def G():
    from paper_2402_09633_amd import gnn
    return gnn


def _tiny_random(seed, n, e, loops=False):
    rng = np.random.default_rng(seed)
    x = rng.normal(size=(n, 3)).astype(np.float32)
    ei = rng.integers(0, n, size=(2, e)).astype(np.int32)
    if not loops and n > 1:
        ei[1] = np.where(ei[0] == ei[1], (ei[1] + 1) % n, ei[1])
    return x, ei


# fp32 runs three kernel sets: the default regrouping of the edge MLPs'
# first layer at node level with split-precision products on the fp16/bf16
# matrix cores (flags 0), the same regrouping on the fp32 matrix cores
# (GNN_FP32_MFMA = 4), and the per-edge gather (GNN_LITERAL_GATHER = 2).
PATHS = [0, 4, 2]
# bf16 runs the regrouped kernels (flags 0) and the per-edge gather (2).
BF16_PATHS = [0, 2, 8]  # default, per-edge first layer, fp16 weights


@pytest.mark.parametrize("flags", PATHS)
@pytest.mark.parametrize("H,T,S,noise", [(64, 2, 1, 0.0), (64, 2, 1, 0.3), (128, 2, 1, 0.3),
                                         (64, 3, 3, 0.3), (128, 0, 1, 0.3), (64, 1, 1, 0.3),
                                         (128, 4, 4, 0.3)])
def test_tiny_fp32_logits(G, oracle_mod, H, T, S, noise, flags):
    c = I.CONFIGS["tiny"]
    g = I.make_graph(c)
    w = I.make_weights(3, H, S, c.weight_seed, affine_noise=noise)
    print(f"tiny H={H} T={T} S={S} noise={noise} flags={flags}", flush=True)
    ref = oracle_mod.forward(w, g.x, g.edge_index, H, T, S)
    got = run_model(G, w, G.make_dims(3, H, T, S, flags=flags), g.x, g.edge_index)
    assert_logits_close(got, ref["logits"])
    sc = run_model(G, w, G.make_dims(3, H, T, S, flags=flags), g.x, g.edge_index, logits=False)
    np.testing.assert_allclose(sc, ref["scores"], rtol=0, atol=1e-5)


@pytest.mark.parametrize("flags", PATHS)
@pytest.mark.parametrize("n,e,seed", [(50, 1, 0), (50, 31, 1), (50, 33, 2), (3000, 8001, 3),
                                      (1, 7, 4), (700, 129, 5)])
def test_ragged_and_small_graphs(G, oracle_mod, n, e, seed, flags):
    x, ei = _tiny_random(seed, n, e, loops=(n == 1))
    w = I.make_weights(3, 64, 1, seed, affine_noise=0.3)
    print(f"ragged n={n} e={e} flags={flags}", flush=True)
    ref = oracle_mod.forward(w, x, ei, 64, 2)
    got = run_model(G, w, G.make_dims(3, 64, 2, flags=flags), x, ei)
    assert_logits_close(got, ref["logits"])


@pytest.mark.parametrize("flags", PATHS)
def test_stage_parity_tiny(G, oracle_mod, flags):
    c = I.CONFIGS["tiny"]
    g = I.make_graph(c)
    H, T = c.hidden, 3
    w = I.make_weights(3, H, 1, c.weight_seed, affine_noise=0.3)
    h = G.gnn_create(w, G.make_dims(3, H, T, flags=flags))
    try:
        xd, eid = dev(g.x), dev(g.edge_index)
        N, E = g.n_nodes, g.n_edges
        for t in range(T + 1):
            ref = oracle_mod.forward(w, g.x, g.edge_index, H, T, dump_iter=t)
            outs = {k: torch.zeros(n, H, device="cuda") for k, n in
                    (("h", N), ("e", E), ("agg_in", N), ("agg_out", N))}
            G.gnn_debug_stages(h, xd, eid, N, E, t, outs["h"], outs["e"], outs["agg_in"],
                               outs["agg_out"])
            torch.cuda.synchronize()
            for k in (("h", "e") if t == 0 else ("h", "e", "agg_in", "agg_out")):
                assert_logits_close(outs[k].cpu().numpy(), ref[k], what=f"{k} after {t}")
    finally:
        G.gnn_destroy(h)


@pytest.mark.slow
def test_mid_fp32_full_compare(G, oracle_mod):
    c = I.CONFIGS["mid"]
    g = I.make_graph(c)
    w = I.make_weights(3, c.hidden, 1, c.weight_seed, affine_noise=0.1)
    print(f"mid N={g.n_nodes} E={g.n_edges}", flush=True)
    ref = oracle_mod.forward(w, g.x, g.edge_index, c.hidden, c.n_iters)
    for flags in PATHS:
        got = run_model(G, w, G.make_dims(3, c.hidden, c.n_iters, flags=flags), g.x,
                        g.edge_index)
        err = assert_logits_close(got, ref["logits"])
        print(f"mid flags={flags} max scaled logit error {err:.2e}", flush=True)
    for flags in BF16_PATHS:
        sc = run_model(G, w, G.make_dims(3, c.hidden, c.n_iters, dtype=G.GNN_BF16, flags=flags),
                       g.x, g.edge_index, logits=False)
        err = np.abs(sc - ref["scores"])
        print(f"mid bf16 flags={flags} max score error {err.max():.3e}", flush=True)
        assert err.max() <= BF16_SCORE_ATOL


def _golden(name):
    with open(os.path.join(GOLDEN, f"{name}_oracle_sample.json")) as f:
        return json.load(f)


@pytest.mark.parametrize("flags", PATHS)
def test_full_fp32_vs_stored_oracle(G, flags):
    gold = _golden("full")
    c = I.CONFIGS["full"]
    g = I.make_graph(c)
    assert g.digest() == gold["graph_digest"]
    w = I.make_weights(3, c.hidden, 1, c.weight_seed)
    ids = np.array(gold["edge_ids"])
    dims = G.make_dims(3, c.hidden, c.n_iters, flags=flags)
    got = run_model(G, w, dims, g.x, g.edge_index)
    err = assert_logits_close(got[ids], gold["logits"])
    print(f"full fp32 flags={flags} max scaled logit error {err:.2e}", flush=True)
    sc = run_model(G, w, dims, g.x, g.edge_index, logits=False)
    np.testing.assert_allclose(sc[ids], gold["scores"], rtol=0, atol=2e-5)


@pytest.mark.parametrize("flags", BF16_PATHS)
def test_full_bf16_scores_vs_stored_oracle(G, flags):
    gold = _golden("full")
    c = I.CONFIGS["full_bf16"]
    g = I.make_graph(c)
    assert g.digest() == gold["graph_digest"] and c.weight_seed == gold["weight_seed"]
    w = I.make_weights(3, c.hidden, 1, c.weight_seed)
    ids = np.array(gold["edge_ids"])
    sc = run_model(G, w, G.make_dims(3, c.hidden, c.n_iters, dtype=G.GNN_BF16, flags=flags),
                   g.x, g.edge_index, logits=False)
    err = np.abs(sc[ids] - np.array(gold["scores"]))
    print(f"full bf16 flags={flags} max score error {err.max():.3e} "
          f"p99 {np.percentile(err, 99):.3e}", flush=True)
    assert err.max() <= BF16_SCORE_ATOL


@pytest.mark.parametrize("flags", BF16_PATHS)
@pytest.mark.parametrize("H,T,S,noise", [(64, 2, 1, 0.0), (64, 2, 1, 0.3), (128, 3, 1, 0.3),
                                         (64, 3, 3, 0.3), (128, 0, 1, 0.3), (128, 1, 1, 0.3)])
def test_tiny_bf16_scores(G, oracle_mod, H, T, S, noise, flags):
    c = I.CONFIGS["tiny"]
    g = I.make_graph(c)
    w = I.make_weights(3, H, S, c.weight_seed, affine_noise=noise)
    ref = oracle_mod.forward(w, g.x, g.edge_index, H, T, S)
    sc = run_model(G, w, G.make_dims(3, H, T, S, dtype=G.GNN_BF16, flags=flags), g.x,
                   g.edge_index, logits=False)
    err = np.abs(sc - ref["scores"]).max()
    print(f"tiny bf16 H={H} T={T} S={S} flags={flags} max score error {err:.3e}", flush=True)
    assert err <= BF16_SCORE_ATOL


@pytest.mark.parametrize("dtype,flags", [(0, f) for f in PATHS] + [(1, f) for f in BF16_PATHS])
@pytest.mark.parametrize("F,H", [(1, 64), (5, 128), (16, 64), (16, 128)])
def test_feature_counts_other_than_three(G, oracle_mod, F, H, dtype, flags):
    # The node encoder's first layer takes 1..16 input features (the hit
    # features of other detectors); every other test uses 3.
    rng = np.random.default_rng(100 + F)
    n, e = 900, 3000
    x = rng.normal(size=(n, F)).astype(np.float32)
    ei = rng.integers(0, n, size=(2, e)).astype(np.int32)
    w = I.make_weights(F, H, 1, 300 + F, affine_noise=0.3)
    print(f"F={F} H={H} dtype={dtype} flags={flags}", flush=True)
    ref = oracle_mod.forward(w, x, ei, H, 2)
    dims = G.make_dims(F, H, 2, dtype=dtype, flags=flags)
    if dtype == 0:
        assert_logits_close(run_model(G, w, dims, x, ei), ref["logits"])
    else:
        sc = run_model(G, w, dims, x, ei, logits=False)
        assert np.abs(sc - ref["scores"]).max() <= BF16_SCORE_ATOL


@pytest.mark.parametrize("dtype,flags", [(0, f) for f in PATHS] + [(1, f) for f in BF16_PATHS])
@pytest.mark.parametrize("eps", [0.5, 3.0e-3])
def test_layernorm_eps(G, oracle_mod, eps, dtype, flags):
    # A LayerNorm eps far from the default: the split kernels carry it as
    # eps * s^2 next to accumulators scaled by a power of two s.
    c = I.CONFIGS["tiny"]
    g = I.make_graph(c)
    w = I.make_weights(3, 128, 1, c.weight_seed, affine_noise=0.3)
    print(f"eps={eps} dtype={dtype} flags={flags}", flush=True)
    ref = oracle_mod.forward(w, g.x, g.edge_index, 128, 3, eps=eps)
    dims = G.make_dims(3, 128, 3, dtype=dtype, ln_eps=eps, flags=flags)
    if dtype == 0:
        assert_logits_close(run_model(G, w, dims, g.x, g.edge_index), ref["logits"])
    else:
        sc = run_model(G, w, dims, g.x, g.edge_index, logits=False)
        assert np.abs(sc - ref["scores"]).max() <= BF16_SCORE_ATOL


@pytest.mark.parametrize("dtype", [0, 1])
@pytest.mark.parametrize("bias", [0.0, 3.25, -80.0])
def test_zero_weights_closed_form(G, dtype, bias):
    g = I.make_graph(I.CONFIGS["tiny"])
    w = np.zeros(I.weight_count(3, 64, 1), np.float32)
    v = I.blob_views(w, 3, 64, 1)
    for k in v:
        if k.endswith(".g"):
            v[k][:] = 1.0
    v["edge_cls.1.b"][:] = bias
    d = G.make_dims(3, 64, 2, dtype=dtype)
    z = run_model(G, w, d, g.x, g.edge_index)
    assert (z == np.float32(bias)).all()
    s = run_model(G, w, d, g.x, g.edge_index, logits=False)
    if bias == 0.0:
        assert (s == 0.5).all()
    else:
        np.testing.assert_allclose(s, 1 / (1 + np.exp(-np.float64(bias))), rtol=1e-6, atol=0)


@pytest.mark.parametrize("dtype", [0, 1])
def test_constant_messages_aggregate_to_degrees_full_scale(G, dtype):
    c = I.CONFIGS["full"]
    g = I.make_graph(c)
    H = c.hidden
    w = I.make_weights(3, H, 1, c.weight_seed)
    v = I.blob_views(w, 3, H, 1)
    v["edge_mlp0.1.W"][:] = 0.0
    v["edge_mlp0.1.beta"][:] = 1.0
    h = G.gnn_create(w, G.make_dims(3, H, c.n_iters, dtype=dtype))
    try:
        N, E = g.n_nodes, g.n_edges
        ain = torch.zeros(N, H, device="cuda")
        aout = torch.zeros(N, H, device="cuda")
        e = torch.zeros(E, H, device="cuda")
        G.gnn_debug_stages(h, dev(g.x), dev(g.edge_index), N, E, 2, None, e, ain, aout)
        torch.cuda.synchronize()
        assert (e == 1).all()
        indeg = np.bincount(g.edge_index[1], minlength=N).astype(np.float32)
        outdeg = np.bincount(g.edge_index[0], minlength=N).astype(np.float32)
        np.testing.assert_array_equal(ain.cpu().numpy(), np.repeat(indeg[:, None], H, 1))
        np.testing.assert_array_equal(aout.cpu().numpy(), np.repeat(outdeg[:, None], H, 1))
    finally:
        G.gnn_destroy(h)


@pytest.mark.parametrize("dtype", [0, 1])
def test_large_event_edge_rows_beyond_4gib(G, dtype):
    # 2M nodes, 10M uniform edges: the fp32 edge-row buffer is 5.1 GB, so
    # every per-edge row offset must be 64-bit (a 32-bit byte offset wraps
    # after 8.4M fp32 rows).  Constant messages (edge MLP layer 2 W = 0,
    # beta = 1) make every message exactly 1 and the aggregates exact
    # degrees; the unmodified model is then run twice for bitwise
    # determinism and scores in [0, 1].
    N, E, H = 2_000_000, 10_000_000, 128
    rng = np.random.default_rng(4242)
    ei = rng.integers(0, N, size=(2, E), dtype=np.int32)
    x = rng.normal(size=(N, 3)).astype(np.float32)
    xd, eid = dev(x), dev(ei)
    print(f"large event N={N} E={E} dtype={dtype}", flush=True)
    w = I.make_weights(3, H, 1, 4242)
    wc = w.copy()
    v = I.blob_views(wc, 3, H, 1)
    v["edge_mlp0.1.W"][:] = 0.0
    v["edge_mlp0.1.beta"][:] = 1.0
    h = G.gnn_create(wc, G.make_dims(3, H, 2, dtype=dtype))
    try:
        e = torch.zeros(E, H, device="cuda")
        ain = torch.zeros(N, H, device="cuda")
        aout = torch.zeros(N, H, device="cuda")
        G.gnn_debug_stages(h, xd, eid, N, E, 1, None, e, ain, aout)
        torch.cuda.synchronize()
        assert bool((e == 1).all())
        del e
        indeg = torch.bincount(eid[1].long(), minlength=N).float()
        outdeg = torch.bincount(eid[0].long(), minlength=N).float()
        assert torch.equal(ain, indeg[:, None].expand(N, H))
        assert torch.equal(aout, outdeg[:, None].expand(N, H))
    finally:
        G.gnn_destroy(h)
    m = G.Model(w, G.make_dims(3, H, 2, dtype=dtype))
    try:
        s1 = m(xd, eid, logits=False).clone()
        s2 = m(xd, eid, logits=False)
        torch.cuda.synchronize()
        assert torch.equal(s1, s2)
        assert bool(((s1 >= 0) & (s1 <= 1)).all())
    finally:
        m.close()


@pytest.mark.parametrize("dtype,flags", [(0, f) for f in PATHS] + [(1, f) for f in BF16_PATHS])
@pytest.mark.parametrize("H", [64, 128])
def test_out_sums_every_run_offset_exact(G, dtype, flags, H):
    # Out-degrees 0..129 and random ones, with nodes without out-edges in
    # between and the edge list in a random order: in source order the runs
    # of one node start and end at every offset of a 32-row unit and span up
    # to five units.  With constant messages the sums are exact degrees
    # (in bf16 too: every degree here is below 256).
    rng = np.random.default_rng(77)
    degs = np.concatenate([np.arange(130), rng.integers(0, 40, 400), np.zeros(50, np.int64)])
    rng.shuffle(degs)
    N = len(degs)
    src = np.repeat(np.arange(N), degs)
    E = len(src)
    dst = rng.integers(0, N, E)
    p = rng.permutation(E)
    ei = np.stack([src[p], dst[p]]).astype(np.int32)
    x = rng.normal(size=(N, 3)).astype(np.float32)
    w = I.make_weights(3, H, 1, 77)
    v = I.blob_views(w, 3, H, 1)
    v["edge_mlp0.1.W"][:] = 0.0
    v["edge_mlp0.1.beta"][:] = 1.0
    h = G.gnn_create(w, G.make_dims(3, H, 2, dtype=dtype, flags=flags))
    try:
        ain = torch.zeros(N, H, device="cuda")
        aout = torch.zeros(N, H, device="cuda")
        e = torch.zeros(E, H, device="cuda")
        G.gnn_debug_stages(h, dev(x), dev(ei), N, E, 1, None, e, ain, aout)
        torch.cuda.synchronize()
        assert (e == 1).all()
        indeg = np.bincount(ei[1], minlength=N).astype(np.float32)
        np.testing.assert_array_equal(aout.cpu().numpy(), np.repeat(degs[:, None], H, 1).astype(np.float32))
        np.testing.assert_array_equal(ain.cpu().numpy(), np.repeat(indeg[:, None], H, 1))
    finally:
        G.gnn_destroy(h)


@pytest.mark.parametrize("flags", PATHS)
@pytest.mark.parametrize("H", [64, 128])
def test_in_sums_every_degree_stage_parity(G, oracle_mod, flags, H):
    # In-degrees 0..70 (each once) and random small ones, edges in a random
    # order, distinct messages: the in-direction sums take one, two and three
    # loads of row ids (16 or 32 per load), every ragged tail of a batch of
    # four row loads, and both sides of the compensated-summation threshold.
    rng = np.random.default_rng(91)
    indeg = np.concatenate([np.arange(71), rng.integers(0, 12, 300)])
    rng.shuffle(indeg)
    N = len(indeg)
    dst = np.repeat(np.arange(N), indeg)
    E = len(dst)
    src = rng.integers(0, N, E)
    p = rng.permutation(E)
    ei = np.stack([src[p], dst[p]]).astype(np.int32)
    x = rng.normal(size=(N, 3)).astype(np.float32)
    w = I.make_weights(3, H, 1, 91, affine_noise=0.3)
    print(f"in-degree sweep H={H} flags={flags} N={N} E={E}", flush=True)
    ref = oracle_mod.forward(w, x, ei, H, 2, dump_iter=1)
    h = G.gnn_create(w, G.make_dims(3, H, 2, flags=flags))
    try:
        outs = {k: torch.zeros(n, H, device="cuda") for k, n in
                (("h", N), ("e", E), ("agg_in", N), ("agg_out", N))}
        G.gnn_debug_stages(h, dev(x), dev(ei), N, E, 1, outs["h"], outs["e"], outs["agg_in"],
                           outs["agg_out"])
        torch.cuda.synchronize()
        for k in ("agg_in", "agg_out", "h", "e"):
            assert_logits_close(outs[k].cpu().numpy(), ref[k], what=f"{k} after 1")
    finally:
        G.gnn_destroy(h)


def test_full_deterministic_and_permutation_equivariant(G):
    c = I.CONFIGS["full"]
    g = I.make_graph(c)
    w = I.make_weights(3, c.hidden, 1, c.weight_seed)
    m = G.Model(w, G.make_dims(3, c.hidden, c.n_iters))
    try:
        xd, eid = dev(g.x), dev(g.edge_index)
        a = m(xd, eid, logits=True).cpu().numpy()
        b = m(xd, eid, logits=True).cpu().numpy()
        assert np.array_equal(a, b)  # bitwise run-to-run
        gs, p = I.shuffled(g, 21)
        s = m(xd, dev(gs.edge_index), logits=True).cpu().numpy()
        assert_logits_close(s, a[p].astype(np.float64), rtol=2e-4, what="shuffled")
    finally:
        m.close()


def test_batch_event0_vs_stored_oracle(G):
    # Event 0 of the ragged batch regenerates to the stored digest and
    # matches the stored oracle sample (all 8 events on 8 streams and every
    # edge against a live oracle run: test_gpu_full_parity.py).
    c = I.CONFIGS["batch"]
    gold = _golden("batch_event0")
    n0 = I.batch_sizes(c)[0]
    g = I.layered_graph(n0, c.graph_seed + 1, I.DPHI_MID * c.window_scale,
                        I.DZ_MID * c.window_scale)
    assert g.digest() == gold["graph_digest"]
    w = I.make_weights(3, c.hidden, 1, c.weight_seed)
    z = run_model(G, w, G.make_dims(3, c.hidden, c.n_iters), g.x, g.edge_index)
    ids = np.array(gold["edge_ids"])
    assert_logits_close(z[ids], gold["logits"], what="batch event 0")


def test_empty_edge_list_writes_nothing(G):
    w = I.make_weights(3, 64, 1, 0)
    m = G.Model(w, G.make_dims(3, 64, 2))
    try:
        out = torch.full((4,), 7.0, device="cuda")
        x = dev(np.zeros((5, 3), np.float32))
        ei = torch.zeros(2, 0, dtype=torch.int32, device="cuda")
        G.gnn_infer(m.handle, x, ei, 5, 0, out)
        torch.cuda.synchronize()
        assert (out == 7.0).all()
    finally:
        m.close()


def test_validate_indices_reports_bad_index(G):
    w = I.make_weights(3, 64, 1, 0)
    m = G.Model(w, G.make_dims(3, 64, 2, flags=G.GNN_VALIDATE_INDICES))
    try:
        x, ei = _tiny_random(1, 100, 300)
        ei[1, 17] = 100
        with pytest.raises(G.GnnError) as e:
            m(dev(x), dev(ei))
        assert e.value.code == G.GNN_E_INDEX
        ei[1, 17] = 5
        m(dev(x), dev(ei))  # the same handle still works
        torch.cuda.synchronize()
    finally:
        m.close()


@pytest.mark.parametrize("flags", PATHS)
def test_hub_graph_long_segments(G, oracle_mod, flags):
    # one node receives half of all edges and another sends a fifth of them:
    # aggregation rows of ~150k and ~60k messages
    rng = np.random.default_rng(31)
    n, e = 5000, 300_000
    x = rng.normal(size=(n, 3)).astype(np.float32)
    ei = rng.integers(0, n, size=(2, e)).astype(np.int32)
    ei[1, rng.random(e) < 0.5] = 17
    ei[0, rng.random(e) < 0.2] = 4999
    w = I.make_weights(3, 64, 1, 31, affine_noise=0.2)
    ref = oracle_mod.forward(w, x, ei, 64, 2)
    got = run_model(G, w, G.make_dims(3, 64, 2, flags=flags), x, ei)
    assert_logits_close(got, ref["logits"])


@pytest.mark.parametrize("flags", BF16_PATHS)
@pytest.mark.parametrize("H,n,e,seed", [(64, 50, 1, 0), (128, 50, 33, 2), (64, 1, 7, 4),
                                        (128, 700, 129, 5)])
def test_ragged_and_small_graphs_bf16(G, oracle_mod, H, n, e, seed, flags):
    # the bf16 model's kernels (with fp16 weights the edge encoder runs inside
    # the first edge update) on one edge, ragged last units and a self-loop
    # graph of one node
    x, ei = _tiny_random(seed, n, e, loops=(n == 1))
    w = I.make_weights(3, H, 1, seed, affine_noise=0.3)
    print(f"ragged bf16 H={H} n={n} e={e} flags={flags}", flush=True)
    ref = oracle_mod.forward(w, x, ei, H, 2)
    sc = run_model(G, w, G.make_dims(3, H, 2, dtype=G.GNN_BF16, flags=flags), x, ei, logits=False)
    assert np.abs(sc - ref["scores"]).max() <= BF16_SCORE_ATOL


@pytest.mark.parametrize("flags", BF16_PATHS)
def test_hub_graph_long_segments_bf16(G, oracle_mod, flags):
    # the hub graph of test_hub_graph_long_segments, H = 128, bf16 model
    rng = np.random.default_rng(31)
    n, e = 5000, 300_000
    x = rng.normal(size=(n, 3)).astype(np.float32)
    ei = rng.integers(0, n, size=(2, e)).astype(np.int32)
    ei[1, rng.random(e) < 0.5] = 17
    ei[0, rng.random(e) < 0.2] = 4999
    w = I.make_weights(3, 128, 1, 31, affine_noise=0.2)
    ref = oracle_mod.forward(w, x, ei, 128, 2)
    sc = run_model(G, w, G.make_dims(3, 128, 2, dtype=G.GNN_BF16, flags=flags), x, ei,
                   logits=False)
    err = np.abs(sc - ref["scores"]).max()
    print(f"hub bf16 flags={flags} max score error {err:.3e}", flush=True)
    assert err <= BF16_SCORE_ATOL


@pytest.mark.parametrize("flags", PATHS)
def test_hidden64_many_tiles_per_workgroup(G, oracle_mod, flags):
    # 300k nodes: every persistent node workgroup walks several 256-node
    # tiles; with H=64 the encoder's weight stream has an odd number of LDS
    # chunks per tile (regression: the buffer parity must carry across tiles)
    rng = np.random.default_rng(41)
    n, e = 300_000, 150_000
    x = rng.normal(size=(n, 3)).astype(np.float32)
    ei = rng.integers(0, n, size=(2, e)).astype(np.int32)
    w = I.make_weights(3, 64, 1, 41, affine_noise=0.2)
    ref = oracle_mod.forward(w, x, ei, 64, 2)
    got = run_model(G, w, G.make_dims(3, 64, 2, flags=flags), x, ei)
    assert_logits_close(got, ref["logits"])


def _hub_free_graph(seed, n=3000, e=12000):
    rng = np.random.default_rng(seed)
    x = rng.normal(size=(n, 3)).astype(np.float32)
    ei = rng.integers(0, n, size=(2, e)).astype(np.int32)
    return x, ei


def test_split_products_take_fp32_mfma_path_outside_fp16_range(G, oracle_mod):
    # gamma = 5000 on one LayerNorm: its outputs can reach 5000 sqrt(63) > 2^15,
    # beyond what the fp16 parts of a split product can hold, so the handle
    # must use the fp32 matrix-core kernels: bitwise the GNN_FP32_MFMA result.
    x, ei = _hub_free_graph(51)
    w = I.make_weights(3, 64, 1, 51, affine_noise=0.2)
    V = I.blob_views(w, 3, 64, 1)
    V["edge_mlp0.0.g"][:] = 5000.0
    ref = oracle_mod.forward(w, x, ei, 64, 2)
    dflt = run_model(G, w, G.make_dims(3, 64, 2), x, ei)
    f32 = run_model(G, w, G.make_dims(3, 64, 2, flags=G.GNN_FP32_MFMA), x, ei)
    assert np.array_equal(dflt, f32)
    assert_logits_close(dflt, ref["logits"])


def test_split_products_large_but_in_range_activations(G, oracle_mod):
    # every gamma and beta times 1000 (gamma ~ 1000, |beta| <= 200): LayerNorm
    # outputs up to ~1e4, inside the fp16 range of the split parts (the split
    # path runs).  Logits of O(1) are then differences of O(1e4) terms, so
    # fp32 itself is off by more than 1e-4 here: the split products must stay
    # within twice the fp32 matrix-core path's error.
    x, ei = _hub_free_graph(52)
    w = I.make_weights(3, 64, 1, 52, affine_noise=0.2)
    V = I.blob_views(w, 3, 64, 1)
    for k in V:
        if k.endswith(".g") or k.endswith(".beta"):
            V[k][:] *= 1000.0
    ref = oracle_mod.forward(w, x, ei, 64, 2)["logits"]
    dflt = run_model(G, w, G.make_dims(3, 64, 2), x, ei)
    f32 = run_model(G, w, G.make_dims(3, 64, 2, flags=G.GNN_FP32_MFMA), x, ei)
    assert not np.array_equal(dflt, f32)  # the split kernels ran
    scale = np.maximum(1.0, np.abs(ref))
    e_split = float(np.max(np.abs(dflt - ref) / scale))
    e_f32 = float(np.max(np.abs(f32 - ref) / scale))
    print(f"large activations: split {e_split:.2e} fp32 mfma {e_f32:.2e}", flush=True)
    assert e_split <= 2 * e_f32 + 1e-6


@pytest.mark.parametrize("H", [64, 128])
def test_split_products_error_matches_fp32_mfma(G, oracle_mod, H):
    # The split products are meant to be as accurate as fp32 ones: on the
    # tiny event their worst logit error stays within twice that of the
    # fp32 matrix-core path (plus a floor of 1e-6).
    c = I.CONFIGS["tiny"]
    g = I.make_graph(c)
    w = I.make_weights(3, H, 1, c.weight_seed, affine_noise=0.3)
    ref = oracle_mod.forward(w, g.x, g.edge_index, H, 4)["logits"]
    def err(flags):
        z = run_model(G, w, G.make_dims(3, H, 4, flags=flags), g.x, g.edge_index)
        return float(np.max(np.abs(z - ref) / np.maximum(1.0, np.abs(ref))))
    e_split, e_f32 = err(0), err(G.GNN_FP32_MFMA)
    print(f"H={H} split {e_split:.2e} fp32 mfma {e_f32:.2e}", flush=True)
    assert e_split <= 2 * e_f32 + 1e-6


def test_split_products_hub_rows_match_fp32_mfma(G, oracle_mod):
    # A node with ~60k incoming messages: its aggregate (up to ~60k times the
    # message bound) is far outside the fp16 range, so the node MLP's first
    # layer scales that node's input row by a power of two before splitting
    # it.  The result must stay as accurate as the fp32 matrix-core path.
    rng = np.random.default_rng(61)
    n, e = 4000, 120_000
    x = rng.normal(size=(n, 3)).astype(np.float32)
    ei = rng.integers(0, n, size=(2, e)).astype(np.int32)
    ei[1, rng.random(e) < 0.5] = 123
    w = I.make_weights(3, 64, 1, 61, affine_noise=0.2)
    ref = oracle_mod.forward(w, x, ei, 64, 2)["logits"]
    scale = np.maximum(1.0, np.abs(ref))
    errs = {}
    for flags in (0, G.GNN_FP32_MFMA):
        z = run_model(G, w, G.make_dims(3, 64, 2, flags=flags), x, ei)
        errs[flags] = float(np.max(np.abs(z - ref) / scale))
    print(f"hub rows: split {errs[0]:.2e} fp32 mfma {errs[G.GNN_FP32_MFMA]:.2e}", flush=True)
    assert errs[0] <= 2 * errs[G.GNN_FP32_MFMA] + 1e-6
