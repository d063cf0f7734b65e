"""Host-side checks of libgnn.so that need no GPU.

The library loads, exports every function include/gnn.h declares, sizes the
weight blob like the generator, rejects bad dims and bad arguments, and
reports a missing device instead of faulting.  No compute call is made.
"""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

from paper_2402_09633_amd import inputs as I

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gnn.h")
CSRC = os.path.join(ROOT, "paper_2402_09633_amd", "csrc")


@pytest.fixture(scope="module")
def G():
    from paper_2402_09633_amd import gnn
    return gnn


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gnn_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("gnn_create", "gnn_infer", "gnn_destroy", "gnn_weight_count", "gnn_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol(G):
    names = declared_functions()
    assert set(names) == set(G.EXPORTS)
    for n in names:
        assert hasattr(G.lib, n), n


@pytest.mark.parametrize("F,H,T,S", [(3, 64, 2, 1), (3, 128, 8, 1), (3, 128, 8, 8), (5, 64, 3, 3),
                                     (1, 128, 0, 1)])
def test_weight_count_matches_generator(G, F, H, T, S):
    d = G.make_dims(F, H, T, S)
    assert G.gnn_weight_count(d) == I.weight_count(F, H, S)


@pytest.mark.parametrize("kw", [dict(hidden=48), dict(hidden=96), dict(hidden=0),
                                dict(n_iters=-1), dict(n_iters=8, n_mp_weight_sets=3),
                                dict(dtype=7), dict(ln_eps=0.0), dict(in_features=0),
                                dict(in_features=17), dict(flags=16)])
def test_bad_dims_are_rejected(G, kw):
    d = G.make_dims(**kw)
    assert G.gnn_weight_count(d) == 0
    assert G.gnn_last_error() != ""


def test_wrong_struct_size_is_rejected(G):
    d = G.make_dims()
    d.struct_size = 12
    assert G.gnn_weight_count(d) == 0
    assert "struct_size" in G.gnn_last_error()


def test_null_arguments(G):
    d = G.make_dims()
    assert G.lib.gnn_create(None, ctypes.byref(d)) is None
    assert G.lib.gnn_infer(None, None, None, 10, 10, None, None) == G.GNN_E_INVALID_ARG
    assert G.lib.gnn_infer_logits(None, None, None, 10, 10, None, None) == G.GNN_E_INVALID_ARG
    assert G.lib.gnn_debug_csr(None, None, 10, 10, None, None, None, None, None) == \
        G.GNN_E_INVALID_ARG
    G.lib.gnn_destroy(None)  # NULL-safe


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="a GPU is visible")
def test_create_without_device_reports_no_device(G):
    d = G.make_dims(3, 64, 2)
    w = I.make_weights(3, 64, 1, 0)
    assert G.lib.gnn_create(w.ctypes.data, ctypes.byref(d)) is None
    assert "device" in G.gnn_last_error()


def test_no_float_atomics_in_kernels():
    # Aggregation must be deterministic: the only atomics are integer ones --
    # the radix sort's uint32 digit histograms (LDS `h`, global `totals`),
    # its tile counters and error word, its uint32 look-back words (`st`),
    # the components' int32 parent array (atomicMin, relaxed loads) and the
    # relaxed loads of their int32 round flags.
    allowed = ("atomicAdd(&h[", "atomicAdd(&totals[", "atomicAdd(&O.ctr[", "atomicOr(O.err",
               "__hip_atomic_store(st", "__hip_atomic_load(st", "atomicMin(&parent[",
               "__hip_atomic_load(parent", "__hip_atomic_load(prev", "__hip_atomic_load(changed")
    for f in os.listdir(CSRC):
        text = open(os.path.join(CSRC, f)).read()
        for line in text.splitlines():
            code = line.split("//")[0]
            if "atomic" in code:
                assert any(a in code for a in allowed), f"{f}: {line.strip()}"
    csr = open(os.path.join(CSRC, "csr.hip")).read()
    assert "uint32_t h[" in csr and "uint32_t *totals" in csr and "uint32_t *status" in csr
    wcc = open(os.path.join(CSRC, "wcc.hip")).read()
    assert "int32_t *parent" in wcc and "float *parent" not in wcc


def test_product_path_never_touches_the_oracle():
    pkg = os.path.join(ROOT, "paper_2402_09633_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in text.lower() or f == "inputs.py", f


@pytest.mark.parametrize("F,H", [(3, 64), (3, 128), (5, 64)])
def test_filter_weight_count_matches_generator(G, F, H):
    assert G.gnn_filter_weight_count(G.make_filter_dims(F, H)) == I.filter_weight_count(F, H)
    assert G.gnn_filter_weight_count(G.make_filter_dims(F, 96)) == 0


@pytest.mark.parametrize("value", ["12x", "", "-5", "1.5g", "k", "99999999999999999999999"])
def test_malformed_workspace_limit_rejected_at_create(G, value, monkeypatch):
    # The workspace cap is read from GNN_WORKSPACE_LIMIT before any device
    # call, so a malformed value fails gnn_create on any machine.
    monkeypatch.setenv("GNN_WORKSPACE_LIMIT", value)
    d = G.make_dims(3, 64, 2)
    w = I.make_weights(3, 64, 1, 0)
    assert G.lib.gnn_create(w.ctypes.data, ctypes.byref(d)) is None
    assert "GNN_WORKSPACE_LIMIT" in G.gnn_last_error()


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="a GPU is visible")
@pytest.mark.parametrize("value", ["0", "1048576", "64k", "512M", "2G"])
def test_wellformed_workspace_limit_passes_parsing(G, value, monkeypatch):
    # a valid cap is accepted; without a device the call then stops there
    monkeypatch.setenv("GNN_WORKSPACE_LIMIT", value)
    d = G.make_dims(3, 64, 2)
    w = I.make_weights(3, 64, 1, 0)
    assert G.lib.gnn_create(w.ctypes.data, ctypes.byref(d)) is None
    assert "device" in G.gnn_last_error()


def test_workspace_limit_and_server_calls_reject_null(G):
    assert G.lib.gnn_set_workspace_limit(None, 0) == G.GNN_E_INVALID_ARG
    assert "NULL" in G.gnn_last_error()
    info = G.gnn_request_info(ctypes.sizeof(G.gnn_request_info), 0, 0.0, -1.0, -1.0)
    assert G.lib.gnn_server_wait_info(None, 0, ctypes.byref(info)) == G.GNN_E_INVALID_ARG
    bad = G.gnn_request_info(4, 0, 0.0, -1.0, -1.0)
    assert G.lib.gnn_server_wait_info(None, 0, ctypes.byref(bad)) == G.GNN_E_INVALID_ARG
    assert "struct_size" in G.gnn_last_error()
    assert G.lib.gnn_server_wait(None, 0, None) == G.GNN_E_INVALID_ARG
    assert G.lib.gnn_server_submit(None, None, None, 1, 1, None) == G.GNN_E_INVALID_ARG


@pytest.mark.parametrize("kind,nbytes,grid,reps,null", [(3, 1024, 0, 1, False), (0, 1000, 0, 1, False),
                                                         (0, 0, 0, 1, False), (1, 1024, -1, 1, False),
                                                         (2, 1024, 0, 0, False), (2, 1024, 0, 1001, False),
                                                         (0, 1024, 0, 1, True)])
def test_hbm_probe_rejects_bad_arguments(G, kind, nbytes, grid, reps, null):
    # checked before any device call (no GPU needed)
    buf = None if null else 16
    ms = ctypes.c_float(-1.0)
    rc = G.lib.gnn_hbm_probe(kind, buf, 16, nbytes, grid, reps, ctypes.byref(ms), None)
    assert rc == G.GNN_E_INVALID_ARG
    assert ms.value == 0.0
    assert G.gnn_last_error() != ""


@pytest.mark.parametrize("dtype,flags", [(0, 8), (1, 8 | 2), (1, 8 | 4)])
def test_f16_weights_flag_only_with_bf16_regrouped(G, dtype, flags):
    d = G.make_dims(dtype=dtype, flags=flags)
    assert G.gnn_weight_count(d) == 0
    assert "GNN_F16_WEIGHTS" in G.gnn_last_error()
    assert G.gnn_weight_count(G.make_dims(dtype=1, flags=8)) > 0
