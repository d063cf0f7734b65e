"""Seeded synthetic inputs: hit graphs and interaction-network weights.

This module is shared by the GPU path's tests/benchmark and by the CPU oracle's
tests. It holds no arithmetic of the method itself (no MLP, no LayerNorm, no
aggregation): only random draws, the detector-like geometry used to place hits
and candidate edges, and the packing of weights into the flat fp32 blob that
``gnn_create`` accepts.

The paper (section 1, Introduction) motivates GPUs with event graphs of roughly
300k nodes and 1M edges; its own dataset (section 3) is not available, so every
event here is synthetic, from a recorded seed.

Graph conventions
-----------------
* ``x``: ``[n_nodes, 3]`` float32, features ``(r/1000, phi/pi, z/1000)``
  (r and z in mm, phi in rad).
* ``edge_index``: ``[2, n_edges]`` int32, row 0 = source node, row 1 =
  destination node (the usual graph-learning convention).

Weight blob (float32, in this order; ``W`` is ``[out][in]`` row-major)
----------------------------------------------------------------------
``node_enc`` (F->H->H), ``edge_enc`` (2H->H->H), then ``n_mp_weight_sets`` x
[``edge_mlp`` (3H->H->H), ``node_mlp`` (3H->H->H)], then ``edge_cls``
(3H->H->1).  A hidden layer stores ``W, b, gamma, beta``; the classifier's
last layer stores ``W[1][H], b[1]``.
"""
from __future__ import annotations

import dataclasses
import hashlib
import math

import numpy as np

# Seeds: graph seed 1000+c, weight seed 2000+c; the ragged batch draws its
# node counts from seed 4000 and builds event k from graph seed 4001+k.
GRAPH_SEED_BASE = 1000
WEIGHT_SEED_BASE = 2000
BATCH_EVENT_SEED_BASE = 4000

N_LAYERS = 10
R_MIN_MM = 30.0
R_MAX_MM = 1000.0
Z_SIGMA_MM = 300.0
MAX_OUT_DEGREE = 8
# Written windows of the mid-size geometric event.
DPHI_MID = 0.05
DZ_MID = 100.0
# The full-size event scales both windows by this factor so that the 300k-hit
# event has about 1.0M edges (bisected for graph seed 1002: 1,000,513 edges).
FULL_WINDOW_SCALE = 0.2055


@dataclasses.dataclass
class Graph:
    x: np.ndarray           # [N, 3] float32
    edge_index: np.ndarray  # [2, E] int32
    seed: int
    meta: dict

    @property
    def n_nodes(self) -> int:
        return int(self.x.shape[0])

    @property
    def n_edges(self) -> int:
        return int(self.edge_index.shape[1])

    def digest(self) -> str:
        """SHA-256 over the exact bytes of x and edge_index (reproducibility check)."""
        h = hashlib.sha256()
        h.update(np.ascontiguousarray(self.x, dtype=np.float32).tobytes())
        h.update(np.ascontiguousarray(self.edge_index, dtype=np.int32).tobytes())
        return h.hexdigest()


def _features(r, phi, z) -> np.ndarray:
    return np.stack([r / 1000.0, phi / math.pi, z / 1000.0], axis=1).astype(np.float32)


def uniform_graph(n_nodes: int = 2000, n_edges: int = 8000, seed: int = GRAPH_SEED_BASE) -> Graph:
    """Tiny uniform random graph (2,000 nodes, 8,000 edges by default).

    r ~ U[30,1000] mm, phi ~ U[-pi,pi], z ~ U[-1000,1000] mm; src and dst drawn
    uniformly; self-loops are redrawn (dst only, same generator) until none is
    left; duplicate edges are kept.
    """
    rng = np.random.default_rng(seed)
    r = rng.uniform(30.0, 1000.0, n_nodes)
    phi = rng.uniform(-math.pi, math.pi, n_nodes)
    z = rng.uniform(-1000.0, 1000.0, n_nodes)
    src = rng.integers(0, n_nodes, n_edges)
    dst = rng.integers(0, n_nodes, n_edges)
    if n_nodes > 1:
        loops = np.nonzero(dst == src)[0]
        while loops.size:
            dst[loops] = rng.integers(0, n_nodes, loops.size)
            loops = loops[dst[loops] == src[loops]]
    ei = np.stack([src, dst]).astype(np.int32)
    return Graph(_features(r, phi, z), ei, seed,
                 {"kind": "uniform", "n_nodes": n_nodes, "n_edges": n_edges})


def _wrap(dphi: np.ndarray) -> np.ndarray:
    return (dphi + math.pi) % (2.0 * math.pi) - math.pi


def layered_graph(n_nodes: int, seed: int, dphi: float, dz: float,
                  max_out: int = MAX_OUT_DEGREE) -> Graph:
    """Hits on 10 concentric cylinders, edges between adjacent layers.

    Layer l sits at r_l = 30 * (1000/30)^(l/9) mm and holds n_nodes/10 hits
    (the remainder goes to the last layers), phi ~ U[-pi,pi], z ~ N(0, 300 mm).
    Hit ids are layer-major. For every hit i on layer l < 9 the candidates are
    the hits j on layer l+1 with |wrap(phi_j - phi_i)| < dphi and
    |z_j - z_i| < dz; at most ``max_out`` are kept, those with the smallest
    |dphi|, ties broken by the smaller j. Edges are emitted in (layer, i, rank)
    order, so the edge list is grouped by source.
    """
    rng = np.random.default_rng(seed)
    per = [n_nodes // N_LAYERS] * N_LAYERS
    for k in range(n_nodes - sum(per)):
        per[N_LAYERS - 1 - k] += 1
    offs = np.concatenate([[0], np.cumsum(per)]).astype(np.int64)
    r_layers = R_MIN_MM * (R_MAX_MM / R_MIN_MM) ** (np.arange(N_LAYERS) / (N_LAYERS - 1))
    phi = rng.uniform(-math.pi, math.pi, n_nodes)
    z = rng.normal(0.0, Z_SIGMA_MM, n_nodes)
    r = np.repeat(r_layers, per)

    srcs, dsts = [], []
    for l in range(N_LAYERS - 1):
        a0, a1 = offs[l], offs[l + 1]
        b0, b1 = offs[l + 1], offs[l + 2]
        if a1 == a0 or b1 == b0:
            continue
        phi_b = phi[b0:b1]
        order = np.argsort(phi_b, kind="stable")
        ps = phi_b[order]
        nb = ps.size
        # Tile the sorted phi list three times (-2pi, 0, +2pi) so that a window
        # that wraps around +-pi is one contiguous slice.
        ext = np.concatenate([ps - 2.0 * math.pi, ps, ps + 2.0 * math.pi])
        pa = phi[a0:a1]
        lo = np.searchsorted(ext, pa - dphi, side="right")
        hi = np.searchsorted(ext, pa + dphi, side="left")
        hi = np.minimum(hi, lo + nb)  # a window never covers a hit twice
        cnt = hi - lo
        tot = int(cnt.sum())
        if tot == 0:
            continue
        ia = np.repeat(np.arange(a1 - a0), cnt)
        start = np.repeat(lo - np.concatenate([[0], np.cumsum(cnt)[:-1]]), cnt)
        pos = np.arange(tot) + start
        jb = order[pos % nb]
        gi = ia + a0
        gj = jb + b0
        adphi = np.abs(_wrap(phi[gj] - phi[gi]))
        keep = (adphi < dphi) & (np.abs(z[gj] - z[gi]) < dz)
        gi, gj, adphi = gi[keep], gj[keep], adphi[keep]
        if gi.size == 0:
            continue
        o = np.lexsort((gj, adphi, gi))
        gi, gj = gi[o], gj[o]
        # rank of each candidate within its source hit
        first = np.concatenate([[True], gi[1:] != gi[:-1]])
        grp_start = np.maximum.accumulate(np.where(first, np.arange(gi.size), 0))
        rank = np.arange(gi.size) - grp_start
        sel = rank < max_out
        srcs.append(gi[sel])
        dsts.append(gj[sel])
    if srcs:
        src = np.concatenate(srcs)
        dst = np.concatenate(dsts)
    else:
        src = dst = np.zeros(0, np.int64)
    ei = np.stack([src, dst]).astype(np.int32)
    return Graph(_features(r, phi, z), ei, seed,
                 {"kind": "layered", "n_nodes": n_nodes, "dphi": dphi, "dz": dz,
                  "max_out": max_out, "n_edges": int(src.size)})


def shuffled(g: Graph, seed: int) -> tuple[Graph, np.ndarray]:
    """The same graph with its edge list in a seeded random order.

    Returns the new graph and ``p`` such that new edge k is old edge p[k].
    """
    p = np.random.default_rng(seed).permutation(g.n_edges)
    return Graph(g.x, np.ascontiguousarray(g.edge_index[:, p]), g.seed,
                 dict(g.meta, shuffled_with=seed)), p


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    n_nodes: int
    hidden: int
    n_iters: int
    dtype: str  # "fp32" | "bf16"
    kind: str   # "uniform" | "layered" | "batch"
    graph_seed: int
    weight_seed: int
    n_edges: int = 0            # uniform graphs only
    window_scale: float = 1.0   # layered graphs only
    n_events: int = 1           # ragged batch only


CONFIGS = {
    # 2,000 nodes / 8,000 edges, H=64, T=2
    "tiny": Config("tiny", 2000, 64, 2, "fp32", "uniform", 1000, 2000, n_edges=8000),
    # 50k hits, written windows, H=128, T=8
    "mid": Config("mid", 50_000, 128, 8, "fp32", "layered", 1001, 2001),
    # 300k hits, windows scaled to ~1.0M edges, H=128, T=8
    "full": Config("full", 300_000, 128, 8, "fp32", "layered", 1002, 2002,
                   window_scale=FULL_WINDOW_SCALE),
    # the full-size event and the same model, run with bf16 weights and
    # activations (compared with the fp32 definition of that same model)
    "full_bf16": Config("full_bf16", 300_000, 128, 8, "bf16", "layered", 1002, 2002,
                        window_scale=FULL_WINDOW_SCALE),
    # 8 independent events, N ~ U{240k..360k}, full-size windows
    "batch": Config("batch", 0, 128, 8, "fp32", "batch", BATCH_EVENT_SEED_BASE, 2004,
                    window_scale=FULL_WINDOW_SCALE, n_events=8),
}


def make_graph(cfg: Config) -> Graph:
    if cfg.kind == "uniform":
        return uniform_graph(cfg.n_nodes, cfg.n_edges, cfg.graph_seed)
    if cfg.kind == "layered":
        return layered_graph(cfg.n_nodes, cfg.graph_seed, DPHI_MID * cfg.window_scale,
                             DZ_MID * cfg.window_scale)
    raise ValueError(f"config {cfg.name} is a batch; use make_batch")


def batch_sizes(cfg: Config) -> list[int]:
    """Node counts of the ragged batch, N_k ~ U{240000..360000}."""
    rng = np.random.default_rng(cfg.graph_seed)
    return [int(v) for v in rng.integers(240_000, 360_001, cfg.n_events)]


def make_batch(cfg: Config) -> list[Graph]:
    return [layered_graph(n, cfg.graph_seed + 1 + k, DPHI_MID * cfg.window_scale,
                          DZ_MID * cfg.window_scale)
            for k, n in enumerate(batch_sizes(cfg))]


# ---------------------------------------------------------------- weights ---

def layer_shapes(in_features: int, hidden: int, n_mp_weight_sets: int):
    """(name, fan_in, fan_out, hidden_layer) for every Linear, in blob order."""
    F, H = in_features, hidden
    out = []

    def mlp(name, fin, last_out=None):
        out.append((name + ".0", fin, H, True))
        if last_out is None:
            out.append((name + ".1", H, H, True))
        else:
            out.append((name + ".1", H, last_out, False))

    mlp("node_enc", F)
    mlp("edge_enc", 2 * H)
    for s in range(n_mp_weight_sets):
        mlp(f"edge_mlp{s}", 3 * H)
        mlp(f"node_mlp{s}", 3 * H)
    mlp("edge_cls", 3 * H, last_out=1)
    return out


def weight_count(in_features: int, hidden: int, n_mp_weight_sets: int) -> int:
    n = 0
    for _, fin, fout, hid in layer_shapes(in_features, hidden, n_mp_weight_sets):
        n += fin * fout + fout + (2 * fout if hid else 0)
    return n


def make_weights(in_features: int, hidden: int, n_mp_weight_sets: int, seed: int,
                 affine_noise: float = 0.0) -> np.ndarray:
    """Packed fp32 blob: Xavier-uniform (gain 1) W, zero b, gamma=1, beta=0.

    Draws come from one PCG64 stream in blob order. With ``affine_noise`` > 0
    the biases, gammas and betas are perturbed too (b, beta ~ U[-a,a],
    gamma ~ U[1-a,1+a]) so that tests exercise every parameter.
    """
    rng = np.random.default_rng(seed)
    parts = []
    for _, fin, fout, hid in layer_shapes(in_features, hidden, n_mp_weight_sets):
        a = math.sqrt(6.0 / (fin + fout))
        parts.append(rng.uniform(-a, a, fin * fout))
        if affine_noise > 0:
            parts.append(rng.uniform(-affine_noise, affine_noise, fout))
        else:
            parts.append(np.zeros(fout))
        if hid:
            if affine_noise > 0:
                parts.append(rng.uniform(1 - affine_noise, 1 + affine_noise, fout))
                parts.append(rng.uniform(-affine_noise, affine_noise, fout))
            else:
                parts.append(np.ones(fout))
                parts.append(np.zeros(fout))
    blob = np.concatenate(parts).astype(np.float32)
    assert blob.size == weight_count(in_features, hidden, n_mp_weight_sets)
    return blob


def blob_views(blob: np.ndarray, in_features: int, hidden: int, n_mp_weight_sets: int) -> dict:
    """Named views into a blob (for tests that set individual parameters)."""
    views, off = {}, 0
    for name, fin, fout, hid in layer_shapes(in_features, hidden, n_mp_weight_sets):
        views[name + ".W"] = blob[off:off + fin * fout].reshape(fout, fin); off += fin * fout
        views[name + ".b"] = blob[off:off + fout]; off += fout
        if hid:
            views[name + ".g"] = blob[off:off + fout]; off += fout
            views[name + ".beta"] = blob[off:off + fout]; off += fout
    assert off == blob.size
    return views


# ---------------------------------------------------------- edge filter ---

def filter_layer_shapes(in_features: int, hidden: int):
    """(name, fan_in, fan_out, hidden_layer) of the edge-filter MLP, in blob
    order: [x_src; x_dst] (2F) -> H -> H -> 1."""
    return [("filter.0", 2 * in_features, hidden, True), ("filter.1", hidden, hidden, True),
            ("filter.2", hidden, 1, False)]


def filter_weight_count(in_features: int, hidden: int) -> int:
    return sum(fin * fout + fout + (2 * fout if hid else 0)
               for _, fin, fout, hid in filter_layer_shapes(in_features, hidden))


def make_filter_weights(in_features: int, hidden: int, seed: int,
                        affine_noise: float = 0.0) -> np.ndarray:
    """Packed fp32 filter blob, drawn like make_weights (Xavier W, zero b,
    gamma 1, beta 0; perturbed b/gamma/beta with affine_noise > 0)."""
    rng = np.random.default_rng(seed)
    parts = []
    for _, fin, fout, hid in filter_layer_shapes(in_features, hidden):
        a = math.sqrt(6.0 / (fin + fout))
        parts.append(rng.uniform(-a, a, fin * fout))
        parts.append(rng.uniform(-affine_noise, affine_noise, fout) if affine_noise > 0
                     else np.zeros(fout))
        if hid:
            if affine_noise > 0:
                parts.append(rng.uniform(1 - affine_noise, 1 + affine_noise, fout))
                parts.append(rng.uniform(-affine_noise, affine_noise, fout))
            else:
                parts.append(np.ones(fout))
                parts.append(np.zeros(fout))
    return np.concatenate(parts).astype(np.float32)


def filter_blob_views(blob: np.ndarray, in_features: int, hidden: int) -> dict:
    views, off = {}, 0
    for name, fin, fout, hid in filter_layer_shapes(in_features, hidden):
        views[name + ".W"] = blob[off:off + fin * fout].reshape(fout, fin); off += fin * fout
        views[name + ".b"] = blob[off:off + fout]; off += fout
        if hid:
            views[name + ".g"] = blob[off:off + fout]; off += fout
            views[name + ".beta"] = blob[off:off + fout]; off += fout
    assert off == blob.size
    return views


# ------------------------------------------------- graph construction ---

def embed_layer_shapes(in_features: int, hidden: int, out_dim: int):
    """(name, fan_in, fan_out, hidden_layer) of the embedding MLP, in blob
    order: x (F) -> H -> H -> D; the output layer has no LayerNorm."""
    return [("embed.0", in_features, hidden, True), ("embed.1", hidden, hidden, True),
            ("embed.2", hidden, out_dim, False)]


def embed_weight_count(in_features: int, hidden: int, out_dim: int) -> int:
    return sum(fin * fout + fout + (2 * fout if hid else 0)
               for _, fin, fout, hid in embed_layer_shapes(in_features, hidden, out_dim))


def make_embed_weights(in_features: int, hidden: int, out_dim: int, seed: int,
                       affine_noise: float = 0.0) -> np.ndarray:
    """Packed fp32 embedding blob, drawn like make_weights (Xavier W, zero b,
    gamma 1, beta 0; perturbed b/gamma/beta with affine_noise > 0)."""
    rng = np.random.default_rng(seed)
    parts = []
    for _, fin, fout, hid in embed_layer_shapes(in_features, hidden, out_dim):
        a = math.sqrt(6.0 / (fin + fout))
        parts.append(rng.uniform(-a, a, fin * fout))
        parts.append(rng.uniform(-affine_noise, affine_noise, fout) if affine_noise > 0
                     else np.zeros(fout))
        if hid:
            if affine_noise > 0:
                parts.append(rng.uniform(1 - affine_noise, 1 + affine_noise, fout))
                parts.append(rng.uniform(-affine_noise, affine_noise, fout))
            else:
                parts.append(np.ones(fout))
                parts.append(np.zeros(fout))
    return np.concatenate(parts).astype(np.float32)


def embed_blob_views(blob: np.ndarray, in_features: int, hidden: int, out_dim: int) -> dict:
    views, off = {}, 0
    for name, fin, fout, hid in embed_layer_shapes(in_features, hidden, out_dim):
        views[name + ".W"] = blob[off:off + fin * fout].reshape(fout, fin); off += fin * fout
        views[name + ".b"] = blob[off:off + fout]; off += fout
        if hid:
            views[name + ".g"] = blob[off:off + fout]; off += fout
            views[name + ".beta"] = blob[off:off + fout]; off += fout
    assert off == blob.size
    return views


def clustered_points(n: int, dim: int, seed: int, n_clusters: int = 0, sigma: float = 0.02,
                     background: float = 0.2) -> np.ndarray:
    """Synthetic embedded space points (fp32 [n][dim]): a fraction
    `background` uniform in [0, 1]^dim, the rest in isotropic Gaussian
    clusters of width sigma around uniform centres (track-like groups in an
    embedding space).  n_clusters = 0 picks n / 10."""
    rng = np.random.default_rng(seed)
    k = n_clusters if n_clusters > 0 else max(1, n // 10)
    centres = rng.uniform(0.0, 1.0, (k, dim))
    nb = int(round(background * n))
    which = rng.integers(0, k, n - nb)
    pts = np.concatenate([rng.uniform(0.0, 1.0, (nb, dim)),
                          centres[which] + rng.normal(0.0, sigma, (n - nb, dim))])
    return pts[rng.permutation(n)].astype(np.float32)
