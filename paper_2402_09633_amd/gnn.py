"""Thin ctypes binding of libgnn.so (include/gnn.h), with the same names.

Argument marshalling only: every step of the inference runs in the HIP
kernels of libgnn.so.  Device buffers are passed as torch tensors (or raw
integer addresses); torch is used for device memory and streams, nothing
else.  There is no fallback: if the library is missing, importing this
module raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch  # imported first so that libgnn.so binds to the HIP runtime torch loaded

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgnn.so")

GNN_OK = 0
GNN_E_INVALID_ARG = -1
GNN_E_NO_DEVICE = -2
GNN_E_OOM = -3
GNN_E_INDEX = -4
GNN_E_HIP = -5
GNN_E_UNSUPPORTED = -6
GNN_FP32 = 0
GNN_BF16 = 1
GNN_VALIDATE_INDICES = 1
GNN_LITERAL_GATHER = 2
GNN_FP32_MFMA = 4
GNN_F16_WEIGHTS = 8
GNN_PROFILE_SAMPLE = 2

EXPORTS = ("gnn_weight_count", "gnn_create", "gnn_infer", "gnn_infer_logits", "gnn_infer_noalloc",
           "gnn_filter_weight_count", "gnn_filter_create", "gnn_filter_apply",
           "gnn_filter_destroy", "gnn_wcc", "gnn_infer_labels", "gnn_destroy",
           "gnn_release_workspaces", "gnn_last_error",
           "gnn_profile_enable", "gnn_profile_read", "gnn_debug_csr", "gnn_debug_stages",
           "gnn_server_create", "gnn_server_submit", "gnn_server_wait", "gnn_server_wait_info",
           "gnn_server_destroy", "gnn_set_workspace_limit",
           "gnn_embed_weight_count", "gnn_embed_create", "gnn_embed_apply", "gnn_embed_destroy",
           "gnn_frnn", "gnn_hbm_probe")
STAGES = ("csr", "node_enc", "edge_enc", "edge_update", "aggregate", "node_update",
          "classifier", "total")


class gnn_embed_dims(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("in_features", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("out_dim", ctypes.c_int32),
                ("ln_eps", ctypes.c_float)]


class gnn_dims(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("in_features", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("n_iters", ctypes.c_int32),
                ("n_mp_weight_sets", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("ln_eps", ctypes.c_float), ("flags", ctypes.c_uint32)]


def make_dims(in_features=3, hidden=128, n_iters=8, n_mp_weight_sets=1, dtype=GNN_FP32,
              ln_eps=1e-5, flags=0) -> gnn_dims:
    return gnn_dims(ctypes.sizeof(gnn_dims), in_features, hidden, n_iters, n_mp_weight_sets,
                    dtype, ln_eps, flags)


class gnn_filter_dims(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("in_features", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("ln_eps", ctypes.c_float)]


def make_filter_dims(in_features=3, hidden=64, ln_eps=1e-5) -> gnn_filter_dims:
    return gnn_filter_dims(ctypes.sizeof(gnn_filter_dims), in_features, hidden, ln_eps)


class gnn_profile_stats(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("n_calls", ctypes.c_int32),
                ("launches", ctypes.c_int64 * 8), ("ms", ctypes.c_double * 8)]


class gnn_request_info(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("status", ctypes.c_int32),
                ("latency_ms", ctypes.c_double), ("device_start_ms", ctypes.c_double),
                ("device_end_ms", ctypes.c_double)]


class GnnError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libgnn error {code}: {msg}")
        self.code = code


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    dp = ctypes.POINTER(gnn_dims)
    L.gnn_weight_count.restype = ctypes.c_size_t
    L.gnn_weight_count.argtypes = [dp]
    L.gnn_create.restype = vp
    L.gnn_create.argtypes = [vp, dp]
    for name in ("gnn_infer", "gnn_infer_logits", "gnn_infer_noalloc"):
        f = getattr(L, name)
        f.restype = ctypes.c_int
        f.argtypes = [vp, vp, vp, i64, i64, vp, vp]
    fdp = ctypes.POINTER(gnn_filter_dims)
    L.gnn_filter_weight_count.restype = ctypes.c_size_t
    L.gnn_filter_weight_count.argtypes = [fdp]
    L.gnn_filter_create.restype = vp
    L.gnn_filter_create.argtypes = [vp, fdp]
    L.gnn_filter_destroy.restype = None
    L.gnn_filter_destroy.argtypes = [vp]
    L.gnn_filter_apply.restype = ctypes.c_int
    L.gnn_filter_apply.argtypes = [vp, vp, vp, i64, i64, ctypes.c_float, vp, vp,
                                   ctypes.POINTER(ctypes.c_int64), vp]
    L.gnn_wcc.restype = ctypes.c_int
    L.gnn_wcc.argtypes = [vp, vp, ctypes.c_float, i64, i64, vp, vp]
    L.gnn_infer_labels.restype = ctypes.c_int
    L.gnn_infer_labels.argtypes = [vp, vp, vp, i64, i64, ctypes.c_float, vp, vp, vp]
    L.gnn_destroy.restype = None
    L.gnn_destroy.argtypes = [vp]
    L.gnn_release_workspaces.restype = ctypes.c_int64
    L.gnn_release_workspaces.argtypes = [vp]
    L.gnn_set_workspace_limit.restype = ctypes.c_int
    L.gnn_set_workspace_limit.argtypes = [vp, i64]
    L.gnn_last_error.restype = ctypes.c_char_p
    L.gnn_last_error.argtypes = []
    L.gnn_profile_enable.restype = ctypes.c_int
    L.gnn_profile_enable.argtypes = [vp, ctypes.c_int]
    L.gnn_profile_read.restype = ctypes.c_int
    L.gnn_profile_read.argtypes = [vp, ctypes.POINTER(gnn_profile_stats)]
    L.gnn_hbm_probe.restype = ctypes.c_int
    L.gnn_hbm_probe.argtypes = [ctypes.c_int, vp, vp, i64, i32, i32, ctypes.POINTER(ctypes.c_float),
                                vp]
    L.gnn_debug_csr.restype = ctypes.c_int
    L.gnn_debug_csr.argtypes = [vp, vp, i64, i64, vp, vp, vp, vp, vp]
    L.gnn_debug_stages.restype = ctypes.c_int
    L.gnn_debug_stages.argtypes = [vp, vp, vp, i64, i64, i32, vp, vp, vp, vp, vp]
    edp = ctypes.POINTER(gnn_embed_dims)
    L.gnn_embed_weight_count.restype = ctypes.c_size_t
    L.gnn_embed_weight_count.argtypes = [edp]
    L.gnn_embed_create.restype = vp
    L.gnn_embed_create.argtypes = [vp, edp]
    L.gnn_embed_apply.restype = ctypes.c_int
    L.gnn_embed_apply.argtypes = [vp, vp, i64, vp, vp]
    L.gnn_embed_destroy.restype = None
    L.gnn_embed_destroy.argtypes = [vp]
    L.gnn_frnn.restype = ctypes.c_int
    L.gnn_frnn.argtypes = [vp, i64, i32, ctypes.c_float, vp, i64, ctypes.POINTER(ctypes.c_int64),
                           vp]
    L.gnn_server_create.restype = vp
    L.gnn_server_create.argtypes = [vp, ctypes.c_int]
    L.gnn_server_submit.restype = i64
    L.gnn_server_submit.argtypes = [vp, vp, vp, i64, i64, vp]
    L.gnn_server_wait.restype = ctypes.c_int
    L.gnn_server_wait.argtypes = [vp, i64, ctypes.POINTER(ctypes.c_double)]
    L.gnn_server_wait_info.restype = ctypes.c_int
    L.gnn_server_wait_info.argtypes = [vp, i64, ctypes.POINTER(gnn_request_info)]
    L.gnn_server_destroy.restype = None
    L.gnn_server_destroy.argtypes = [vp]
    return L


lib = _load()


def _addr(t) -> int | None:
    """Device address of a tensor (checked contiguous), an int, or None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if isinstance(t, torch.Tensor):
        if not t.is_contiguous():
            raise ValueError("tensor arguments must be contiguous")
        return t.data_ptr()
    raise TypeError(f"expected a tensor, an int address or None, got {type(t)}")


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _check(rc: int) -> int:
    if rc != GNN_OK:
        raise GnnError(rc, gnn_last_error())
    return rc


def gnn_last_error() -> str:
    return lib.gnn_last_error().decode()


def gnn_weight_count(dims: gnn_dims) -> int:
    return int(lib.gnn_weight_count(ctypes.byref(dims)))


def gnn_create(weights: np.ndarray, dims: gnn_dims) -> int:
    """Upload a host fp32 weight blob; returns the handle (an address)."""
    w = np.ascontiguousarray(weights, dtype=np.float32)
    n = gnn_weight_count(dims)
    if n == 0:
        raise GnnError(GNN_E_INVALID_ARG, gnn_last_error())
    if w.size != n:
        raise ValueError(f"weight blob has {w.size} floats, dims need {n}")
    h = lib.gnn_create(w.ctypes.data, ctypes.byref(dims))
    if not h:
        raise GnnError(GNN_E_INVALID_ARG, gnn_last_error())
    return h


def gnn_destroy(handle) -> None:
    lib.gnn_destroy(handle)


def gnn_release_workspaces(handle) -> int:
    """Frees the handle's idle cached workspaces; returns the bytes freed."""
    r = lib.gnn_release_workspaces(handle)
    if r < 0:
        raise GnnError(int(r), gnn_last_error())
    return int(r)


def gnn_set_workspace_limit(handle, n_bytes: int) -> int:
    """Caps the handle's inference workspace bytes (0 = no cap)."""
    return _check(lib.gnn_set_workspace_limit(handle, int(n_bytes)))


def _check_io(node_feat, edge_index, out):
    for t, dt in ((node_feat, torch.float32), (edge_index, torch.int32), (out, torch.float32)):
        if isinstance(t, torch.Tensor):
            if t.dtype != dt:
                raise TypeError(f"expected {dt}, got {t.dtype}")
            if not t.is_cuda:
                raise ValueError("inputs and outputs must be device tensors")


def gnn_infer(handle, node_feat, edge_index, n_nodes: int, n_edges: int, edge_scores,
              stream=None) -> int:
    _check_io(node_feat, edge_index, edge_scores)
    return _check(lib.gnn_infer(handle, _addr(node_feat), _addr(edge_index), n_nodes, n_edges,
                                _addr(edge_scores), _stream(stream)))


def gnn_infer_logits(handle, node_feat, edge_index, n_nodes: int, n_edges: int, edge_logits,
                     stream=None) -> int:
    _check_io(node_feat, edge_index, edge_logits)
    return _check(lib.gnn_infer_logits(handle, _addr(node_feat), _addr(edge_index), n_nodes,
                                       n_edges, _addr(edge_logits), _stream(stream)))


def gnn_infer_noalloc(handle, node_feat, edge_index, n_nodes: int, n_edges: int, edge_scores,
                      stream=None) -> int:
    """gnn_infer in the library's fixed scratch array: allocates nothing."""
    _check_io(node_feat, edge_index, edge_scores)
    return _check(lib.gnn_infer_noalloc(handle, _addr(node_feat), _addr(edge_index), n_nodes,
                                        n_edges, _addr(edge_scores), _stream(stream)))


def gnn_filter_weight_count(dims: gnn_filter_dims) -> int:
    return int(lib.gnn_filter_weight_count(ctypes.byref(dims)))


def gnn_filter_create(weights: np.ndarray, dims: gnn_filter_dims) -> int:
    w = np.ascontiguousarray(weights, dtype=np.float32)
    n = gnn_filter_weight_count(dims)
    if n == 0:
        raise GnnError(GNN_E_INVALID_ARG, gnn_last_error())
    if w.size != n:
        raise ValueError(f"filter blob has {w.size} floats, dims need {n}")
    h = lib.gnn_filter_create(w.ctypes.data, ctypes.byref(dims))
    if not h:
        raise GnnError(GNN_E_INVALID_ARG, gnn_last_error())
    return h


def gnn_filter_destroy(handle) -> None:
    lib.gnn_filter_destroy(handle)


def gnn_filter_apply(handle, node_feat, edge_index, n_nodes: int, n_edges: int,
                     threshold: float, edge_scores, edge_index_out, stream=None) -> int:
    """Returns n_kept; edge_index_out[: 2 * n_kept] holds the kept edges as [2][n_kept]."""
    nk = ctypes.c_int64(0)
    _check(lib.gnn_filter_apply(handle, _addr(node_feat), _addr(edge_index), n_nodes, n_edges,
                                float(threshold), _addr(edge_scores), _addr(edge_index_out),
                                ctypes.byref(nk), _stream(stream)))
    return int(nk.value)


def gnn_wcc(edge_index, edge_scores, threshold: float, n_nodes: int, n_edges: int, labels,
            stream=None) -> int:
    """Component labels (smallest node id per component) of the edges scoring
    above `threshold`; edge_scores may be None (every edge kept)."""
    for t, dt in ((edge_index, torch.int32), (edge_scores, torch.float32), (labels, torch.int32)):
        if isinstance(t, torch.Tensor) and t.dtype != dt:
            raise TypeError(f"expected {dt}, got {t.dtype}")
    return _check(lib.gnn_wcc(_addr(edge_index), _addr(edge_scores), float(threshold), n_nodes,
                              n_edges, _addr(labels), _stream(stream)))


def gnn_infer_labels(handle, node_feat, edge_index, n_nodes: int, n_edges: int,
                     threshold: float, edge_scores, labels, stream=None) -> int:
    return _check(lib.gnn_infer_labels(handle, _addr(node_feat), _addr(edge_index), n_nodes,
                                       n_edges, float(threshold), _addr(edge_scores),
                                       _addr(labels), _stream(stream)))


def gnn_profile_enable(handle, enable=True) -> int:
    """enable: False/0 off, True/1 every stage, GNN_PROFILE_SAMPLE."""
    mode = int(enable) if not isinstance(enable, bool) else (1 if enable else 0)
    return _check(lib.gnn_profile_enable(handle, mode))


def gnn_profile_read(handle) -> dict:
    """{'n_calls': n, stage: {'launches': k, 'ms': total_ms}} per stage."""
    st = gnn_profile_stats()
    st.struct_size = ctypes.sizeof(gnn_profile_stats)
    _check(lib.gnn_profile_read(handle, ctypes.byref(st)))
    out = {"n_calls": st.n_calls}
    for i, name in enumerate(STAGES):
        out[name] = {"launches": int(st.launches[i]), "ms": float(st.ms[i])}
    return out


GNN_PROBE_READ, GNN_PROBE_WRITE, GNN_PROBE_COPY = 0, 1, 2


def gnn_hbm_probe(kind: int, buf, buf2, nbytes: int, grid: int = 0, reps: int = 5,
                  stream=None) -> float:
    """Fastest of `reps` timed launches of the streaming probe, in ms."""
    ms = ctypes.c_float(0.0)
    _check(lib.gnn_hbm_probe(kind, _addr(buf), _addr(buf2), nbytes, grid, reps, ctypes.byref(ms),
                             _stream(stream)))
    return float(ms.value)


def gnn_debug_csr(handle, edge_index, n_nodes: int, n_edges: int, row_ptr_in=None, perm_in=None,
                  row_ptr_out=None, perm_out=None, stream=None) -> int:
    return _check(lib.gnn_debug_csr(handle, _addr(edge_index), n_nodes, n_edges,
                                    _addr(row_ptr_in), _addr(perm_in), _addr(row_ptr_out),
                                    _addr(perm_out), _stream(stream)))


def gnn_debug_stages(handle, node_feat, edge_index, n_nodes: int, n_edges: int, stop_iter: int,
                     h_out=None, e_out=None, agg_in_out=None, agg_out_out=None,
                     stream=None) -> int:
    return _check(lib.gnn_debug_stages(handle, _addr(node_feat), _addr(edge_index), n_nodes,
                                       n_edges, stop_iter, _addr(h_out), _addr(e_out),
                                       _addr(agg_in_out), _addr(agg_out_out), _stream(stream)))


def make_embed_dims(in_features=3, hidden=64, out_dim=8, ln_eps=1e-5) -> gnn_embed_dims:
    return gnn_embed_dims(ctypes.sizeof(gnn_embed_dims), in_features, hidden, out_dim, ln_eps)


def gnn_embed_weight_count(dims: gnn_embed_dims) -> int:
    return int(lib.gnn_embed_weight_count(ctypes.byref(dims)))


def gnn_embed_create(weights: np.ndarray, dims: gnn_embed_dims):
    w = np.ascontiguousarray(weights, np.float32)
    if w.size != gnn_embed_weight_count(dims):
        raise ValueError("embedding weight blob has the wrong size")
    m = lib.gnn_embed_create(w.ctypes.data, ctypes.byref(dims))
    if not m:
        raise GnnError(GNN_E_INVALID_ARG, gnn_last_error())
    return m


def gnn_embed_apply(embedder, node_feat, n_nodes: int, z, stream=None) -> int:
    return _check(lib.gnn_embed_apply(embedder, _addr(node_feat), n_nodes, _addr(z),
                                      _stream(stream)))


def gnn_embed_destroy(embedder) -> None:
    lib.gnn_embed_destroy(embedder)


def gnn_frnn(z, n_nodes: int, dim: int, r2: float, edge_index=None, max_pairs: int = 0,
             stream=None) -> int:
    """Fixed-radius pairs of the rows of z; returns the pair count (and
    fills edge_index [2][count] when given and large enough)."""
    cnt = ctypes.c_int64(0)
    rc = lib.gnn_frnn(_addr(z), n_nodes, dim, float(r2), _addr(edge_index), int(max_pairs),
                      ctypes.byref(cnt), _stream(stream))
    if rc != GNN_OK:
        raise GnnError(rc, gnn_last_error())
    return int(cnt.value)


class Embedder:
    """Owns one embedding model: ``Embedder(w, dims)(x) -> z``."""

    def __init__(self, weights: np.ndarray, dims: gnn_embed_dims):
        self.dims = dims
        self.handle = gnn_embed_create(weights, dims)

    def __call__(self, x: torch.Tensor, z=None, stream=None) -> torch.Tensor:
        if z is None:
            z = torch.empty(x.shape[0], self.dims.out_dim, dtype=torch.float32, device=x.device)
        gnn_embed_apply(self.handle, x, x.shape[0], z, stream)
        return z

    def close(self):
        if self.handle:
            gnn_embed_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def radius_graph(z: torch.Tensor, r2: float, stream=None) -> torch.Tensor:
    """[2][n_pairs] int32 edge list of the pairs i < j of rows of z with
    fp32 squared distance < r2 (count first, then fill)."""
    n, d = z.shape
    cap = max(16 * n, 1)  # one call when the pairs fit, a second one otherwise
    out = torch.empty(2 * cap, dtype=torch.int32, device=z.device)
    try:
        cnt = gnn_frnn(z, n, d, r2, out, cap, stream)
    except GnnError as e:
        if e.code != GNN_E_INVALID_ARG:
            raise
        cnt = gnn_frnn(z, n, d, r2, None, 0, stream)
        out = torch.empty(2 * max(cnt, 1), dtype=torch.int32, device=z.device)
        cnt = gnn_frnn(z, n, d, r2, out, cnt, stream)
    return out[:2 * cnt].view(2, cnt)


def gnn_server_create(handle, n_instances: int):
    s = lib.gnn_server_create(handle, int(n_instances))
    if not s:
        raise GnnError(GNN_E_INVALID_ARG, gnn_last_error())
    return s


def gnn_server_submit(server, node_feat, edge_index, n_nodes: int, n_edges: int,
                      edge_scores) -> int:
    """Queue one event; returns the request id."""
    _check_io(node_feat, edge_index, edge_scores)
    rid = lib.gnn_server_submit(server, _addr(node_feat), _addr(edge_index), n_nodes, n_edges,
                                _addr(edge_scores))
    if rid < 0:
        raise GnnError(int(rid), gnn_last_error())
    return int(rid)


def gnn_server_wait(server, request_id: int) -> float:
    """Wait for one request; returns its latency (ms, queueing included)."""
    lat = ctypes.c_double(0.0)
    _check(lib.gnn_server_wait(server, int(request_id), ctypes.byref(lat)))
    return lat.value


def gnn_server_wait_info(server, request_id: int) -> dict:
    """Wait for one request; returns its status, latency and device interval (ms)."""
    info = gnn_request_info(ctypes.sizeof(gnn_request_info), 0, 0.0, -1.0, -1.0)
    _check(lib.gnn_server_wait_info(server, int(request_id), ctypes.byref(info)))
    return {"status": info.status, "latency_ms": info.latency_ms,
            "device_start_ms": info.device_start_ms, "device_end_ms": info.device_end_ms}


def gnn_server_destroy(server) -> None:
    lib.gnn_server_destroy(server)


class Server:
    """A request queue served by ``n_instances`` streams of one model."""

    def __init__(self, model: "Model", n_instances: int):
        self.model = model
        self.server = gnn_server_create(model.handle, n_instances)

    def submit(self, x: torch.Tensor, edge_index: torch.Tensor, out: torch.Tensor) -> int:
        return gnn_server_submit(self.server, x, edge_index, x.shape[0], edge_index.shape[1], out)

    def wait(self, request_id: int) -> float:
        return gnn_server_wait(self.server, request_id)

    def wait_info(self, request_id: int) -> dict:
        return gnn_server_wait_info(self.server, request_id)

    def close(self):
        if self.server:
            gnn_server_destroy(self.server)
            self.server = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Model:
    """Owns one handle: ``Model(weights, dims)(x, edge_index) -> scores``."""

    def __init__(self, weights: np.ndarray, dims: gnn_dims):
        self.dims = dims
        self.handle = gnn_create(weights, dims)

    def __call__(self, x: torch.Tensor, edge_index: torch.Tensor, out=None, logits=False,
                 stream=None) -> torch.Tensor:
        E = edge_index.shape[1]
        if out is None:
            out = torch.empty(E, dtype=torch.float32, device=x.device)
        f = gnn_infer_logits if logits else gnn_infer
        f(self.handle, x, edge_index, x.shape[0], E, out, stream)
        return out

    def close(self):
        if self.handle:
            gnn_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
