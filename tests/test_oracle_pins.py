"""Pins of the CPU oracle against things other than itself.

* one hidden layer vs torch-CPU F.linear / F.layer_norm / relu (library);
* the CSR vs numpy's stable argsort and bincount (library);
* the whole model vs the incidence-matrix brute force on tiny graphs,
  including every intermediate stage;
* closed forms: all-zero weights give z = b_cls exactly; constant messages
  give aggregates equal to the node degrees exactly; node-determined
  messages aggregate to a dense adjacency matmul;
* invariances: edge order, node labels, duplicated edges, isolated nodes,
  an empty edge list.
"""
import numpy as np
import pytest
import scipy.special
import torch
import torch.nn.functional as Fn

from paper_2402_09633_amd import inputs as I
from tests import brute_force as B


def _tiny(seed, n=40, e=160, loops=False):
    rng = np.random.default_rng(seed)
    x = rng.normal(size=(n, 3)).astype(np.float32)
    ei = rng.integers(0, n, size=(2, e)).astype(np.int32)
    if not loops:
        ei[1] = np.where(ei[0] == ei[1], (ei[1] + 1) % n, ei[1])
    return x, ei


def test_hidden_layer_matches_torch(oracle_mod):
    rng = np.random.default_rng(0)
    for fin, fout in [(3, 8), (24, 16), (384, 128)]:
        W = rng.normal(size=(fout, fin)).astype(np.float32)
        b = rng.normal(size=fout).astype(np.float32)
        g = rng.uniform(0.5, 1.5, fout).astype(np.float32)
        be = rng.normal(size=fout).astype(np.float32)
        x = rng.normal(size=(50, fin))
        got = oracle_mod.hidden_layer(W, b, g, be, x, eps=1e-5)
        t = lambda a: torch.as_tensor(np.asarray(a, np.float64))
        ref = torch.relu(Fn.layer_norm(Fn.linear(t(x), t(W), t(b)), (fout,), t(g), t(be), 1e-5))
        np.testing.assert_allclose(got, ref.numpy(), rtol=0, atol=1e-12)


def test_hidden_layer_zero_variance_row_gives_relu_beta(oracle_mod):
    fout = 8
    W = np.zeros((fout, 4), np.float32)
    b = np.full(fout, 0.7, np.float32)
    g = np.full(fout, 3.0, np.float32)
    be = np.linspace(-1, 1, fout).astype(np.float32)
    out = oracle_mod.hidden_layer(W, b, g, be, np.ones((2, 4)))
    np.testing.assert_array_equal(out, np.maximum(be.astype(np.float64), 0)[None].repeat(2, 0))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_csr_matches_stable_argsort(oracle_mod, seed):
    rng = np.random.default_rng(seed)
    n = 37
    keys = rng.integers(0, n, 500).astype(np.int32)
    keys[:40] = 5  # a long segment
    rp, perm = oracle_mod.csr(keys, n)
    np.testing.assert_array_equal(perm, np.argsort(keys, kind="stable"))
    np.testing.assert_array_equal(rp, np.concatenate([[0], np.cumsum(np.bincount(keys, minlength=n))]))


def test_csr_rejects_out_of_range(oracle_mod):
    with pytest.raises(ValueError):
        oracle_mod.csr(np.array([0, 3], np.int32), 3)


@pytest.mark.parametrize("H,T,S,seed", [(4, 0, 1, 0), (8, 1, 1, 1), (8, 2, 1, 2),
                                        (4, 3, 3, 3), (8, 3, 1, 4)])
def test_forward_matches_brute_force(oracle_mod, H, T, S, seed):
    x, ei = _tiny(seed)
    w = I.make_weights(3, H, S, 100 + seed, affine_noise=0.3)
    ref = B.forward(w, x, ei, 3, H, T, S)
    got = oracle_mod.forward(w, x, ei, H, T, S)
    np.testing.assert_allclose(got["logits"], ref["logits"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(got["scores"], ref["scores"], rtol=0, atol=1e-13)
    for t in range(T + 1):
        d = oracle_mod.forward(w, x, ei, H, T, S, dump_iter=t)
        for k, v in ref["dumps"][t].items():
            np.testing.assert_allclose(d[k], v, rtol=0, atol=1e-11, err_msg=f"{k} after {t}")


def test_forward_with_self_loops_and_duplicates(oracle_mod):
    x, ei = _tiny(9, n=12, e=90, loops=True)
    ei[:, 10] = ei[:, 11]  # an explicit duplicate
    assert (ei[0] == ei[1]).any()
    w = I.make_weights(3, 8, 1, 9, affine_noise=0.3)
    ref = B.forward(w, x, ei, 3, 8, 2)
    got = oracle_mod.forward(w, x, ei, 8, 2)
    np.testing.assert_allclose(got["logits"], ref["logits"], rtol=0, atol=1e-12)


@pytest.mark.parametrize("bias", [0.0, 2.5, -40.0, 700.0, -750.0])
def test_zero_weights_closed_form(oracle_mod, bias):
    x, ei = _tiny(5)
    w = np.zeros(I.weight_count(3, 8, 1), np.float32)
    v = I.blob_views(w, 3, 8, 1)
    for k in v:
        if k.endswith(".g"):
            v[k][:] = 1.0
    v["edge_cls.1.b"][:] = bias
    got = oracle_mod.forward(w, x, ei, 8, 2)
    assert (got["logits"] == np.float64(np.float32(bias))).all()
    np.testing.assert_allclose(got["scores"], scipy.special.expit(np.float64(np.float32(bias))),
                               rtol=1e-15, atol=0)
    if bias == 0.0:
        assert (got["scores"] == 0.5).all()


def test_constant_messages_give_degrees(oracle_mod):
    n, e = 60, 400
    x, ei = _tiny(11, n, e)
    ei[1, :50] = 7  # a hub
    w = I.make_weights(3, 8, 1, 11, affine_noise=0.3)
    v = I.blob_views(w, 3, 8, 1)
    v["edge_mlp0.1.W"][:] = 0.0
    v["edge_mlp0.1.b"][:] = 0.0
    v["edge_mlp0.1.beta"][:] = 1.0
    for t in (1, 2):
        d = oracle_mod.forward(w, x, ei, 8, 2, dump_iter=t)
        assert (d["e"] == 1.0).all()
        indeg = np.bincount(ei[1], minlength=n).astype(np.float64)
        outdeg = np.bincount(ei[0], minlength=n).astype(np.float64)
        np.testing.assert_array_equal(d["agg_in"], indeg[:, None].repeat(8, 1))
        np.testing.assert_array_equal(d["agg_out"], outdeg[:, None].repeat(8, 1))


def test_node_determined_messages_equal_adjacency_matmul(oracle_mod):
    n, e, H = 30, 200, 8
    x, ei = _tiny(12, n, e)
    w = I.make_weights(3, H, 1, 12, affine_noise=0.3)
    v = I.blob_views(w, 3, H, 1)
    v["edge_mlp0.0.W"][:, H:] = 0.0  # the message depends on h_src only
    h0 = oracle_mod.forward(w, x, ei, H, 1, dump_iter=0)["h"]
    d1 = oracle_mod.forward(w, x, ei, H, 1, dump_iter=1)
    a0 = np.concatenate([h0, np.zeros((n, 2 * H))], 1)
    g = oracle_mod.hidden_layer(v["edge_mlp0.0.W"], v["edge_mlp0.0.b"], v["edge_mlp0.0.g"],
                                v["edge_mlp0.0.beta"], a0)
    g = oracle_mod.hidden_layer(v["edge_mlp0.1.W"], v["edge_mlp0.1.b"], v["edge_mlp0.1.g"],
                                v["edge_mlp0.1.beta"], g)
    A = np.zeros((n, n))
    np.add.at(A, (ei[0], ei[1]), 1.0)  # A[u, v] = multiplicity of u -> v
    np.testing.assert_allclose(d1["agg_in"], A.T @ g, rtol=0, atol=1e-12)
    # every edge out of u carries g[u], so agg_out[u] = outdeg(u) * g[u]
    outdeg = A.sum(1)
    np.testing.assert_allclose(d1["agg_out"], outdeg[:, None] * g, rtol=0, atol=1e-12)


def test_edge_permutation_permutes_outputs(oracle_mod):
    c = I.CONFIGS["tiny"]
    g = I.make_graph(c)
    w = I.make_weights(3, c.hidden, 1, c.weight_seed, affine_noise=0.2)
    a = oracle_mod.forward(w, g.x, g.edge_index, c.hidden, c.n_iters)
    gs, p = I.shuffled(g, 77)
    b = oracle_mod.forward(w, gs.x, gs.edge_index, c.hidden, c.n_iters)
    np.testing.assert_allclose(b["logits"], a["logits"][p], rtol=1e-12, atol=1e-13)


def test_node_relabel_leaves_scores_unchanged(oracle_mod):
    x, ei = _tiny(13, 50, 300)
    w = I.make_weights(3, 8, 1, 13, affine_noise=0.2)
    a = oracle_mod.forward(w, x, ei, 8, 3)
    q = np.random.default_rng(1).permutation(50)  # old id i -> new id q[i]
    x2 = np.empty_like(x)
    x2[q] = x
    b = oracle_mod.forward(w, x2, q[ei].astype(np.int32), 8, 3)
    np.testing.assert_allclose(b["logits"], a["logits"], rtol=1e-12, atol=1e-13)


def test_duplicate_edge_doubles_its_contribution(oracle_mod):
    x, ei = _tiny(14, 20, 60)
    w = I.make_weights(3, 8, 1, 14, affine_noise=0.2)
    ei2 = np.concatenate([ei, ei[:, :1]], 1)
    a = oracle_mod.forward(w, x, ei, 8, 1, dump_iter=1)
    b = oracle_mod.forward(w, x, ei2, 8, 1, dump_iter=1)
    u, v = ei[0, 0], ei[1, 0]
    np.testing.assert_allclose(b["agg_in"][v] - a["agg_in"][v], a["e"][0], rtol=0, atol=1e-12)
    np.testing.assert_allclose(b["agg_out"][u] - a["agg_out"][u], a["e"][0], rtol=0, atol=1e-12)
    np.testing.assert_allclose(b["logits"][-1], b["logits"][0], rtol=0, atol=1e-13)


def test_isolated_nodes_have_zero_aggregates(oracle_mod):
    x, ei = _tiny(15, 30, 80)
    ei = np.where(ei >= 25, ei % 25, ei).astype(np.int32)  # nodes 25..29 isolated
    w = I.make_weights(3, 8, 1, 15, affine_noise=0.2)
    d = oracle_mod.forward(w, x, ei, 8, 2, dump_iter=2)
    assert (d["agg_in"][25:] == 0).all() and (d["agg_out"][25:] == 0).all()


def test_empty_edge_list(oracle_mod):
    x, _ = _tiny(16, 10, 1)
    w = I.make_weights(3, 8, 1, 16)
    out = oracle_mod.forward(w, x, np.zeros((2, 0), np.int32), 8, 2)
    assert out["logits"].size == 0 and out["scores"].size == 0


def test_forward_rejects_bad_indices(oracle_mod):
    x, ei = _tiny(17, 10, 20)
    ei[0, 3] = 10
    w = I.make_weights(3, 8, 1, 17)
    with pytest.raises(ValueError):
        oracle_mod.forward(w, x, ei, 8, 1)


def _canonical(labels):
    """Map any component labelling to 'smallest node id of the component'."""
    labels = np.asarray(labels)
    first = {}
    for v, c in enumerate(labels):
        first.setdefault(c, v)
    return np.array([first[c] for c in labels], np.int32)


@pytest.mark.parametrize("seed,n,e,thr", [(0, 50, 40, 0.5), (1, 300, 400, 0.3), (2, 1000, 900, 0.7),
                                          (3, 20, 0, 0.5), (4, 1, 3, 0.5)])
def test_wcc_matches_scipy(oracle_mod, seed, n, e, thr):
    from scipy.sparse import coo_matrix
    from scipy.sparse.csgraph import connected_components
    rng = np.random.default_rng(seed)
    ei = rng.integers(0, n, size=(2, e)).astype(np.int32)
    sc = rng.random(e).astype(np.float32)
    got = oracle_mod.wcc(ei, n, sc, thr)
    keep = sc > thr
    A = coo_matrix((np.ones(keep.sum()), (ei[0, keep], ei[1, keep])), shape=(n, n))
    _, lab = connected_components(A, directed=True, connection="weak")
    np.testing.assert_array_equal(got, _canonical(lab))
    assert (got <= np.arange(n)).all() and (got[got] == got).all()


def test_wcc_threshold_and_order_invariance(oracle_mod):
    rng = np.random.default_rng(5)
    n, e = 500, 700
    ei = rng.integers(0, n, size=(2, e)).astype(np.int32)
    sc = rng.random(e).astype(np.float32)
    a = oracle_mod.wcc(ei, n, sc, 0.4)
    keep = sc > 0.4
    np.testing.assert_array_equal(a, oracle_mod.wcc(ei[:, keep], n))        # pre-filtered
    p = rng.permutation(e)
    np.testing.assert_array_equal(a, oracle_mod.wcc(ei[:, p], n, sc[p], 0.4))  # edge order
    np.testing.assert_array_equal(a, oracle_mod.wcc(ei[::-1].copy(), n, sc, 0.4))  # direction
    assert (oracle_mod.wcc(ei, n, np.zeros(e, np.float32), 0.5) == np.arange(n)).all()


def _filter_brute(w, x, ei, F, H, eps=1e-5):
    V = {k: torch.as_tensor(np.asarray(v, np.float64)) for k, v in
         I.filter_blob_views(np.asarray(w, np.float32), F, H).items()}
    xx = torch.as_tensor(np.asarray(x, np.float64))
    a = torch.cat([xx[torch.as_tensor(ei[0], dtype=torch.long)],
                   xx[torch.as_tensor(ei[1], dtype=torch.long)]], 1)
    for name in ("filter.0", "filter.1"):
        y = Fn.linear(a, V[name + ".W"], V[name + ".b"])
        a = torch.relu(Fn.layer_norm(y, (H,), V[name + ".g"], V[name + ".beta"], eps))
    return torch.sigmoid(Fn.linear(a, V["filter.2.W"], V["filter.2.b"])[:, 0]).numpy()


@pytest.mark.parametrize("H,seed", [(8, 0), (16, 1)])
def test_filter_matches_brute_force(oracle_mod, H, seed):
    x, ei = _tiny(seed, 40, 300)
    w = I.make_filter_weights(3, H, seed, affine_noise=0.3)
    sc, kept = oracle_mod.filter_edges(w, x, ei, H, 0.5)
    ref = _filter_brute(w, x, ei, 3, H)
    np.testing.assert_allclose(sc, ref, rtol=0, atol=1e-13)
    np.testing.assert_array_equal(kept, np.nonzero(ref > 0.5)[0])


def test_filter_closed_forms(oracle_mod):
    x, ei = _tiny(3, 30, 100)
    w = np.zeros(I.filter_weight_count(3, 8), np.float32)
    v = I.filter_blob_views(w, 3, 8)
    v["filter.0.g"][:] = 1.0
    v["filter.1.g"][:] = 1.0
    v["filter.2.b"][:] = 1.5
    sc, kept = oracle_mod.filter_edges(w, x, ei, 8, 0.5)
    assert (sc == scipy.special.expit(1.5)).all() and (kept == np.arange(100)).all()
    sc, kept = oracle_mod.filter_edges(w, x, ei, 8, 0.9)  # sigmoid(1.5) = 0.818 < 0.9
    assert kept.size == 0
    assert oracle_mod.filter_edges(w, x, np.zeros((2, 0), np.int32), 8)[1].size == 0


# ---- graph construction: embedding MLP and fixed-radius neighbours ----

def _embed_torch(w, x, F, H, D, eps=1e-5):
    V = {k: torch.as_tensor(np.array(v, np.float64))
         for k, v in I.embed_blob_views(w, F, H, D).items()}
    a = torch.as_tensor(x.astype(np.float64))
    for name in ("embed.0", "embed.1"):
        y = Fn.linear(a, V[name + ".W"], V[name + ".b"])
        a = torch.relu(Fn.layer_norm(y, (H,), V[name + ".g"], V[name + ".beta"], eps))
    return Fn.linear(a, V["embed.2.W"], V["embed.2.b"]).numpy()


@pytest.mark.parametrize("H,D,seed", [(8, 4, 0), (16, 8, 1), (32, 3, 2)])
def test_embed_matches_torch(oracle_mod, H, D, seed):
    x = np.random.default_rng(seed).normal(size=(50, 3)).astype(np.float32)
    w = I.make_embed_weights(3, H, D, seed, affine_noise=0.3)
    np.testing.assert_allclose(oracle_mod.embed(w, x, H, D), _embed_torch(w, x, 3, H, D),
                               rtol=0, atol=1e-13)


def test_embed_closed_form(oracle_mod):
    # zero weights except the output bias: every point maps to that bias
    w = np.zeros(I.embed_weight_count(3, 8, 5), np.float32)
    v = I.embed_blob_views(w, 3, 8, 5)
    v["embed.2.b"][:] = np.arange(5, dtype=np.float32) - 1.5
    z = oracle_mod.embed(w, np.random.default_rng(0).normal(size=(7, 3)).astype(np.float32), 8, 5)
    assert (z == np.arange(5) - 1.5).all()


def _pair_set(p):
    return set(map(tuple, np.asarray(p).reshape(-1, 2).tolist()))


@pytest.mark.parametrize("seed,n,D,r", [(0, 300, 8, 0.05), (1, 800, 3, 0.03), (2, 500, 5, 0.1)])
def test_frnn_matches_kdtree(oracle_mod, seed, n, D, r):
    # scipy's k-d tree in float64 brackets the fp32 decision: every pair
    # closer than r(1 - 1e-5) must be found, none farther than r(1 + 1e-5)
    from scipy.spatial import cKDTree
    z = I.clustered_points(n, D, seed)
    got = _pair_set(oracle_mod.frnn(z, np.float32(r * r)))
    t = cKDTree(z.astype(np.float64))
    inner = t.query_pairs(r * (1 - 1e-5))
    outer = t.query_pairs(r * (1 + 1e-5))
    assert inner <= got <= outer
    assert len(got) > 0


def test_frnn_exact_on_integer_lattice(oracle_mod):
    # integer coordinates: every fp32 squared distance is exact, so the pairs
    # are exactly those a float64 k-d tree finds for r2 = 2.5 (distances^2 of
    # 1 and 2 pass, 3 fails)
    from scipy.spatial import cKDTree
    g = np.stack(np.meshgrid(np.arange(6), np.arange(5), np.arange(4), indexing="ij"), -1)
    z = g.reshape(-1, 3).astype(np.float32)
    got = oracle_mod.frnn(z, 2.5)
    assert _pair_set(got) == cKDTree(z.astype(np.float64)).query_pairs(np.sqrt(2.5))
    assert (np.diff(got[:, 0]) >= 0).all() and (got[:, 0] < got[:, 1]).all()


def test_frnn_permutation_and_edge_cases(oracle_mod):
    z = I.clustered_points(400, 6, 9)
    p = np.random.default_rng(3).permutation(400)
    a = _pair_set(oracle_mod.frnn(z, 0.003))
    # row k of z[p] is row p[k] of z
    b = {tuple(sorted((int(p[i]), int(p[j])))) for i, j in _pair_set(oracle_mod.frnn(z[p], 0.003))}
    assert a == b and len(a) > 0
    assert oracle_mod.frnn(z, 0.0).shape == (0, 2)
    assert oracle_mod.frnn(z[:1], 1e9).shape == (0, 2)
    assert len(oracle_mod.frnn(z[:20], 1e9)) == 20 * 19 // 2


def test_frnn_row_agrees_with_frnn(oracle_mod):
    z = I.clustered_points(600, 8, 11)
    pairs = oracle_mod.frnn(z, 0.004)
    for i in (0, 5, 77, 599):
        np.testing.assert_array_equal(oracle_mod.frnn_row(z, 0.004, i), pairs[pairs[:, 0] == i, 1])
