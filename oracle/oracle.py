"""ctypes wrapper around the fp64 C oracle (``gnn_oracle.c``).

TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the
benchmark's CPU baseline; never by the product path. See ``gnn_oracle.c`` for
the model it evaluates (paper section 2.1: an interaction network scores the
edges of the hit graph).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "gnn_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

# Portable x86-64 server baseline (the library may be built on one machine and
# run on another).
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-mavx2", "-mfma"]


def build() -> str:
    """Compile the oracle with gcc into ``oracle/liboracle.so``."""
    tmp = LIB + ".tmp"
    subprocess.run(["gcc", *CFLAGS, SRC, "-o", tmp, "-lm"], check=True)
    os.replace(tmp, LIB)
    return LIB


_lib = None

_dp = ctypes.POINTER(ctypes.c_double)
_fp = ctypes.POINTER(ctypes.c_float)
_ip = ctypes.POINTER(ctypes.c_int32)


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = ctypes.CDLL(LIB)
        L.oracle_weight_count.restype = ctypes.c_long
        L.oracle_weight_count.argtypes = [ctypes.c_int] * 3
        L.oracle_csr.restype = ctypes.c_int
        L.oracle_csr.argtypes = [ctypes.c_long, ctypes.c_long, _ip, _ip, _ip]
        L.oracle_hidden_layer.restype = ctypes.c_int
        L.oracle_hidden_layer.argtypes = [_fp, _fp, _fp, _fp, ctypes.c_int, ctypes.c_int,
                                          ctypes.c_double, _dp, ctypes.c_long, _dp]
        L.oracle_forward.restype = ctypes.c_int
        L.oracle_forward.argtypes = [_fp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                     ctypes.c_double, _fp, _ip, ctypes.c_long, ctypes.c_long,
                                     _dp, _dp, ctypes.c_int, _dp, _dp, _dp, _dp]
        L.oracle_wcc.restype = ctypes.c_int
        L.oracle_wcc.argtypes = [ctypes.c_long, ctypes.c_long, _ip, _fp, ctypes.c_float, _ip]
        L.oracle_filter_weight_count.restype = ctypes.c_long
        L.oracle_filter_weight_count.argtypes = [ctypes.c_int, ctypes.c_int]
        L.oracle_filter.restype = ctypes.c_int
        L.oracle_filter.argtypes = [_fp, ctypes.c_int, ctypes.c_int, ctypes.c_double, _fp, _ip,
                                    ctypes.c_long, ctypes.c_long, ctypes.c_double, _dp,
                                    ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64)]
        L.oracle_embed_weight_count.restype = ctypes.c_long
        L.oracle_embed_weight_count.argtypes = [ctypes.c_int] * 3
        L.oracle_embed.restype = ctypes.c_int
        L.oracle_embed.argtypes = [_fp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                   _fp, ctypes.c_long, _dp]
        L.oracle_frnn.restype = ctypes.c_int
        L.oracle_frnn.argtypes = [_fp, ctypes.c_long, ctypes.c_int, ctypes.c_float,
                                  ctypes.POINTER(ctypes.c_int64), ctypes.c_long,
                                  ctypes.POINTER(ctypes.c_int64)]
        L.oracle_frnn_row.restype = ctypes.c_long
        L.oracle_frnn_row.argtypes = [_fp, ctypes.c_long, ctypes.c_int, ctypes.c_float,
                                      ctypes.c_long, ctypes.POINTER(ctypes.c_int64), ctypes.c_long]
        L.oracle_max_threads.restype = ctypes.c_int
        L.oracle_set_threads.argtypes = [ctypes.c_int]
        _lib = L
    return _lib


def _ptr(a, t):
    return a.ctypes.data_as(t) if a is not None else None


def weight_count(F: int, H: int, S: int) -> int:
    return int(lib().oracle_weight_count(F, H, S))


def max_threads() -> int:
    return int(lib().oracle_max_threads())


def set_threads(n: int) -> None:
    lib().oracle_set_threads(int(n))


def csr(keys: np.ndarray, n_nodes: int):
    """Stable counting sort of edge ids by key -> (row_ptr[N+1], perm[E])."""
    keys = np.ascontiguousarray(keys, dtype=np.int32)
    rp = np.zeros(n_nodes + 1, np.int32)
    perm = np.zeros(max(keys.size, 1), np.int32)
    rc = lib().oracle_csr(n_nodes, keys.size, _ptr(keys, _ip), _ptr(rp, _ip), _ptr(perm, _ip))
    if rc:
        raise ValueError(f"oracle_csr failed ({rc})")
    return rp, perm[:keys.size]


def hidden_layer(W, b, g, beta, x, eps=1e-5):
    """Linear + LayerNorm + ReLU on the rows of x (fp64 in, fp64 out)."""
    W = np.ascontiguousarray(W, np.float32)
    fout, fin = W.shape
    x = np.ascontiguousarray(x, np.float64).reshape(-1, fin)
    out = np.zeros((x.shape[0], fout), np.float64)
    args = [np.ascontiguousarray(a, np.float32) for a in (b, g, beta)]
    rc = lib().oracle_hidden_layer(_ptr(W, _fp), *[_ptr(a, _fp) for a in args], fin, fout,
                                   float(eps), _ptr(x, _dp), x.shape[0], _ptr(out, _dp))
    if rc:
        raise ValueError(f"oracle_hidden_layer failed ({rc})")
    return out


def forward(weights, x, edge_index, hidden, n_iters, n_mp_weight_sets=1, eps=1e-5,
            dump_iter=-1):
    """Run the oracle. Returns dict with 'logits', 'scores' (fp64, [E]) and,
    when dump_iter >= 0, 'h', 'e' (and 'agg_in', 'agg_out' for dump_iter > 0)."""
    x = np.ascontiguousarray(x, np.float32)
    n_nodes, F = x.shape
    ei = np.ascontiguousarray(edge_index, np.int32).reshape(2, -1)
    E = ei.shape[1]
    w = np.ascontiguousarray(weights, np.float32)
    if w.size != weight_count(F, hidden, n_mp_weight_sets):
        raise ValueError("weight blob has the wrong size")
    z = np.zeros(E, np.float64)
    s = np.zeros(E, np.float64)
    out = {"logits": z, "scores": s}
    hd = ed = ai = ao = None
    if dump_iter >= 0:
        hd = out["h"] = np.zeros((n_nodes, hidden))
        ed = out["e"] = np.zeros((E, hidden))
        if dump_iter > 0:
            ai = out["agg_in"] = np.zeros((n_nodes, hidden))
            ao = out["agg_out"] = np.zeros((n_nodes, hidden))
    rc = lib().oracle_forward(_ptr(w, _fp), F, hidden, n_iters, n_mp_weight_sets, float(eps),
                              _ptr(x, _fp), _ptr(ei, _ip), n_nodes, E, _ptr(z, _dp),
                              _ptr(s, _dp), int(dump_iter), _ptr(hd, _dp), _ptr(ed, _dp),
                              _ptr(ai, _dp), _ptr(ao, _dp))
    if rc:
        raise ValueError(f"oracle_forward failed ({rc})")
    return out


def wcc(edge_index, n_nodes, scores=None, threshold=0.5):
    """Component label (smallest node id of the component) of every node, over
    the undirected graph of edges with score > threshold (all if scores=None)."""
    ei = np.ascontiguousarray(edge_index, np.int32).reshape(2, -1)
    sc = None if scores is None else np.ascontiguousarray(scores, np.float32)
    lab = np.zeros(max(n_nodes, 1), np.int32)
    rc = lib().oracle_wcc(n_nodes, ei.shape[1], _ptr(ei, _ip), _ptr(sc, _fp), float(threshold),
                          _ptr(lab, _ip))
    if rc:
        raise ValueError(f"oracle_wcc failed ({rc})")
    return lab[:n_nodes]


def filter_weight_count(F: int, H: int) -> int:
    return int(lib().oracle_filter_weight_count(F, H))


def filter_edges(weights, x, edge_index, hidden, threshold=0.5, eps=1e-5):
    """Filter-MLP scores of every candidate edge (fp64) and the ids of the
    edges scoring above `threshold`, in input order."""
    x = np.ascontiguousarray(x, np.float32)
    n_nodes, F = x.shape
    ei = np.ascontiguousarray(edge_index, np.int32).reshape(2, -1)
    E = ei.shape[1]
    w = np.ascontiguousarray(weights, np.float32)
    if w.size != filter_weight_count(F, hidden):
        raise ValueError("filter weight blob has the wrong size")
    sc = np.zeros(max(E, 1))
    kept = np.zeros(max(E, 1), np.int64)
    nk = ctypes.c_int64(0)
    rc = lib().oracle_filter(_ptr(w, _fp), F, hidden, float(eps), _ptr(x, _fp), _ptr(ei, _ip),
                             n_nodes, E, float(threshold), _ptr(sc, _dp),
                             kept.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), ctypes.byref(nk))
    if rc:
        raise ValueError(f"oracle_filter failed ({rc})")
    return sc[:E], kept[:nk.value]


def embed_weight_count(F: int, H: int, D: int) -> int:
    return int(lib().oracle_embed_weight_count(F, H, D))


def embed(weights, x, hidden, out_dim, eps=1e-5):
    """Embedding z [N][D] (fp64) of every row of x."""
    x = np.ascontiguousarray(x, np.float32)
    n, F = x.shape
    w = np.ascontiguousarray(weights, np.float32)
    if w.size != embed_weight_count(F, hidden, out_dim):
        raise ValueError("embedding weight blob has the wrong size")
    z = np.zeros((max(n, 1), out_dim))
    rc = lib().oracle_embed(_ptr(w, _fp), F, hidden, out_dim, float(eps), _ptr(x, _fp), n,
                            _ptr(z, _dp))
    if rc:
        raise ValueError(f"oracle_embed failed ({rc})")
    return z[:n]


def frnn(z, r2):
    """All pairs i < j of rows of the fp32 matrix z with fp32 squared
    distance < r2, as an int64 [n_pairs][2] array in ascending (i, j) order."""
    z = np.ascontiguousarray(z, np.float32)
    n, D = z.shape
    cnt = ctypes.c_int64(0)
    P = ctypes.POINTER(ctypes.c_int64)
    rc = lib().oracle_frnn(_ptr(z, _fp), n, D, float(np.float32(r2)), None, 0, ctypes.byref(cnt))
    if rc:
        raise ValueError(f"oracle_frnn failed ({rc})")
    pairs = np.zeros((max(cnt.value, 1), 2), np.int64)
    rc = lib().oracle_frnn(_ptr(z, _fp), n, D, float(np.float32(r2)), pairs.ctypes.data_as(P),
                           cnt.value, ctypes.byref(cnt))
    if rc:
        raise ValueError(f"oracle_frnn failed ({rc})")
    return pairs[:cnt.value]


def frnn_row(z, r2, i):
    """The partners j > i of row i (ascending) under the same test as frnn."""
    z = np.ascontiguousarray(z, np.float32)
    n, D = z.shape
    P = ctypes.POINTER(ctypes.c_int64)
    c = lib().oracle_frnn_row(_ptr(z, _fp), n, D, float(np.float32(r2)), int(i), None, 0)
    out = np.zeros(max(c, 1), np.int64)
    lib().oracle_frnn_row(_ptr(z, _fp), n, D, float(np.float32(r2)), int(i),
                          out.ctypes.data_as(P), c)
    return out[:c]
