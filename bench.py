"""Throughput of the interaction-network edge classifier on one MI355X.

A step is one complete gnn_infer call (CSR build, encoders, 8 message-passing
iterations, classifier) on one synthetic event whose inputs are already in
HBM.  Default workload: the 300k-hit / ~1.0M-edge layered event, H=128,
T=8, fp32, seeded Xavier weights (the event scale of paper section 1).

Prints one JSON line: edges/s (value), ms/event, the roofline position of
the dominant kernel (the fused edge-update kernel, timed with HIP events on
the launch stream by the library's sampled profiler over the timed region),
the node-update and aggregation rooflines, and, outside the timed region:
  parity       the timed path's logits against the fp64 oracle on every edge
               (the process exits with status 3 when they disagree);
  bf16         the same event with the bf16 model (timed the same way) and
               its scores against the oracle's;
  batch        the ragged 8-event service batch on 8 streams, and the request
               queue with 1/2/4/8 instances (throughput, latency, GPU
               utilisation);
  cpu_baseline the oracle timed on this host's cores.
"""
from __future__ import annotations

import argparse
import json
import os
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "edges/sec and ms/event, 8-iter interaction network, 300k nodes/1M edges"
PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"fp32": 157.3, "bf16": 2500.0, "fp16": 2500.0}
FP32_LOGIT_RTOL = 1e-4   # |z - z_ref| <= 1e-4 max(1, |z_ref|)
BF16_SCORE_ATOL = 2e-2   # |s - s_ref| <= 2e-2 against the oracle of the fp32 weights

# HBM bytes per launch of the edge-update kernel on the full event, from
# rocprofv3 FETCH_SIZE / WRITE_SIZE passes scaled by a plain-copy calibration
# (profiles/full_event_fp32_kernels_and_counters.md, profiles/full_event_bf16_kernels_and_counters.md,
# profiles/full_event_bf16_f16_weights_kernels_and_counters.md).
# Valid only for the kernel sources they were measured on (hash of the files of that path).
TRAFFIC_SOURCES = {
    "split": ["paper_2402_09633_amd/csrc/split.hip", "paper_2402_09633_amd/csrc/device_common.h"],
    "bf16": ["paper_2402_09633_amd/csrc/split.hip", "paper_2402_09633_amd/csrc/device_common.h"],
    "f16w": ["paper_2402_09633_amd/csrc/split.hip", "paper_2402_09633_amd/csrc/device_common.h"],
    "fp32_mfma": ["paper_2402_09633_amd/csrc/factored.hip",
                  "paper_2402_09633_amd/csrc/device_common.h"],
}
# (path, source hash) -> (HBM bytes read, written) per edge-update launch on
# the full event
MEASURED_TRAFFIC = {("split", "393e70c466c8f0c6"): (1.131e9, 0.651e9),    # edge_split<4,3>
                    ("bf16", "393e70c466c8f0c6"): (0.551e9, 0.342e9),     # edge_split<4,3,bf16>
                    ("f16w", "393e70c466c8f0c6"): (0.593e9, 0.347e9)}     # edge_split<4,3,f16w>


def kernel_source_hash(path):
    import hashlib
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES[path]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def edge_update_flops(E, H, factored):
    """Algorithmic multiply-adds x 2 of one edge-update launch (fp32 model).

    Per-edge form: layer 1 over [h_src; h_dst; e] (3H -> H) and layer 2
    (H -> H).  Regrouped form: the launch computes W_e e (H -> H) and layer 2;
    the W_s h and W_d h products run once per node inside the node kernel.
    """
    return 2.0 * E * ((1 if factored else 3) * H * H + H * H)


def proj_bytes(s):
    """Bytes per element of the node projections P: fp32 in the fp32 model,
    fp16 in the bf16 model (s = 2)."""
    return 4 if s == 4 else 2


def edge_update_bytes(N, E, H, s=4, n_src=0):
    """Algorithmic HBM bytes of one regrouped edge-update launch, gathered
    rows counted per edge: e read and written (s bytes per element), the
    P[src][0:H] and P[dst][H:2H] half-rows and both indices; with the fused
    out-sums (n_src > 0), one agg_out row (s bytes per element) per node
    that has out-edges."""
    return E * (2 * H * s + 2 * H * proj_bytes(s) + 8) + n_src * H * s


def edge_update_rw(N, E, H, s=4, n_src=0):
    """edge_update_bytes split into (read, written)."""
    return (E * (H * s + 2 * H * proj_bytes(s) + 8), E * H * s + n_src * H * s)


def node_update_rw(N, H, s=4, T=1):
    """node_update_bytes split into (read, written)."""
    return (N * 3 * H * s, N * 2 * H * proj_bytes(s) + N * H * s * (T - 1) / T)


def node_update_sampled_rw(N, H, s=4, T=1):
    """(read, written) bytes of the node-update launch the sampled profiler
    times, that of iteration T // 2 (0-based): it stores h unless it is the
    last of the T iterations."""
    writes_h = T // 2 != T - 1
    return (N * 3 * H * s, N * 2 * H * proj_bytes(s) + (N * H * s if writes_h else 0))


def aggregate_rw(N, E, H, s, n_src):
    """aggregate_bytes after the fused edge update, split into (read, written)."""
    return (E * H * s + E * 4 + 2.0 * (N + 1) * 4, N * H * s + (N - n_src) * H * s)


def practical(rw, seconds, ceil):
    """The launch's HBM rate against what plain streaming kernels reach on
    this device: a launch that reads R and writes W bytes needs at least
    R / read_rate + W / write_rate."""
    if not ceil:
        return None
    r, w = rw
    t_min = r / (ceil["read_gbs"] * 1e9) + w / (ceil["write_gbs"] * 1e9)
    return {"read_bytes": r, "write_bytes": w,
            "ceiling_gbs": round((r + w) / t_min / 1e9, 1),
            "achieved_gbs": round((r + w) / seconds / 1e9, 1),
            "frac": round(t_min / seconds, 4)}


def hbm_ceiling(G, torch):
    """Fastest read, write and copy rates of the library's streaming probe
    (1 GiB, nontemporal 16-byte accesses) over a few grid sizes."""
    nb = 1 << 30
    a = torch.empty(nb // 4, dtype=torch.float32, device="cuda")
    b = torch.empty(nb // 4, dtype=torch.float32, device="cuda")
    a.zero_()
    out = {"bytes": nb}
    for kind, name, moved in ((G.GNN_PROBE_READ, "read_gbs", nb), (G.GNN_PROBE_WRITE, "write_gbs", nb),
                              (G.GNN_PROBE_COPY, "copy_gbs", 2 * nb)):
        best = min(G.gnn_hbm_probe(kind, a, b, nb, grid, 5) for grid in (512, 1024, 2048, 4096))
        out[name] = round(moved / (best / 1000.0) / 1e9, 1)
    del a, b
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    out["note"] = ("plain grid-stride kernels (gnn_hbm_probe), best of 5 launches at 512-4096 "
                   "workgroups of 256 threads; copy_gbs counts bytes read plus written")
    return out


def node_update_bytes(N, H, s=4, T=1):
    """Average per launch over the T launches of one event: h, agg_in,
    agg_out read (s bytes per element) and the projection row of 2H
    elements written every time; h written by all but the last launch,
    whose h feeds the classifier only through its projections."""
    return N * (3 * H * s + 2 * H * proj_bytes(s)) + N * H * s * (T - 1) / T


def split_mfma_flops(N, E, H, bf16=False):
    """Matrix-core work the regrouped kernels execute per launch (each
    partial product counted).  fp32 split: 3 fp16 products per fp32 product
    (W_e e and W2 in the edge update; layer 1 (3H -> H), layer 2 and the
    2H x H projection in the node update).  bf16 model: 2 products (hi/lo
    weights) throughout."""
    k = 2 if bf16 else 3
    return {"edge_update": k * 2.0 * E * 2 * H * H, "node_update": k * 2.0 * N * 6 * H * H}


def aggregate_bytes(N, E, H, act_bytes, n_src=0):
    """Both directions: every message row read once per direction, both
    aggregates written, perm and row pointers read per direction.  After the
    fused edge update (n_src > 0): the in-direction only, both row-pointer
    arrays, and a zero agg_out row per node without out-edges."""
    if n_src:
        return (E * H * act_bytes + N * H * act_bytes + E * 4 + 2.0 * (N + 1) * 4
                + (N - n_src) * H * act_bytes)
    return 2.0 * E * H * act_bytes + 2.0 * N * H * act_bytes + 2.0 * E * 4 + 2.0 * (N + 1) * 4


def union_ms(intervals):
    """Total length of the union of closed intervals [a, b]."""
    tot, cur_a, cur_b = 0.0, None, None
    for a, b in sorted(intervals):
        if cur_b is None or a > cur_b:
            if cur_b is not None:
                tot += cur_b - cur_a
            cur_a, cur_b = a, b
        else:
            cur_b = max(cur_b, b)
    if cur_b is not None:
        tot += cur_b - cur_a
    return tot


def max_scaled_err(got, ref):
    import numpy as np
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if got.size == 0:
        return 0.0
    return float(np.max(np.abs(got - ref) / np.maximum(1.0, np.abs(ref))))


# ------------------------------------------------------------------ host ---

def _run(cmd):
    try:
        return subprocess.run(cmd, capture_output=True, text=True, timeout=30).stdout
    except Exception:  # a missing tool leaves the field empty
        return ""


def host_info():
    """CPU model, physical cores available to this process, the cgroup CPU
    quota, compilers and the build's source revision."""
    info = {}
    for line in _run(["lscpu"]).splitlines():
        k, _, v = line.partition(":")
        if k.strip() in ("Model name", "Socket(s)", "Core(s) per socket", "Thread(s) per core"):
            info[k.strip()] = v.strip()
    aff = sorted(os.sched_getaffinity(0))
    cores = set()
    for line in _run(["lscpu", "-p=CPU,CORE,SOCKET"]).splitlines():
        if line.startswith("#"):
            continue
        p = line.split(",")
        if len(p) >= 3 and p[0].isdigit() and int(p[0]) in aff:
            cores.add((p[1], p[2]))
    quota = None
    try:
        q, per = open("/sys/fs/cgroup/cpu.max").read().split()
        if q != "max":
            quota = float(q) / float(per)
    except Exception:  # no cgroup v2 quota visible
        pass
    gcc = (_run(["gcc", "--version"]).splitlines() or [""])[0]
    bi = {}
    try:
        with open(os.path.join(ROOT, "paper_2402_09633_amd", "build_info.json")) as f:
            bi = json.load(f)
    except Exception:  # built without git metadata
        pass
    return {"cpu_model": info.get("Model name", ""), "logical_cpus_in_affinity": len(aff),
            "physical_cores_in_affinity": len(cores) or len(aff),
            "cgroup_cpu_quota": quota, "omp_num_threads_env": os.environ.get("OMP_NUM_THREADS"),
            "gcc": gcc, "hipcc": bi.get("hipcc", ""), "libgnn_build": bi}


# ------------------------------------------------------------ GPU legs ---

def timed_leg(G, torch, np, g, w, H, T, dtype, flags, steps, warmup):
    """Warm-up, then `steps` gnn_infer calls timed on the wall clock with the
    library's sampled profiler on (GNN_PROFILE_SAMPLE: each call times the
    edge update, aggregation and node update of its iteration T/2 with events
    bound to their dispatches, which costs about 0.02 ms per event; timing
    every stage costs about 0.12 ms).  Afterwards, outside the timed region:
    10 calls with every stage timed (the per-stage breakdown) and one
    gnn_infer_logits call.  Returns the figures, the outputs and the open
    model with its device inputs."""
    dims = G.make_dims(3, H, T, 1, dtype, flags=flags)
    x = torch.as_tensor(g.x).cuda()
    ei = torch.as_tensor(g.edge_index).cuda()
    out = torch.empty(g.n_edges, dtype=torch.float32, device="cuda")
    m = G.Model(w, dims)
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        m(x, ei, out)
    torch.cuda.synchronize()
    G.gnn_profile_enable(m.handle, G.GNN_PROFILE_SAMPLE)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for a, b in evs:
        a.record(stream)
        m(x, ei, out)
        b.record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    prof = G.gnn_profile_read(m.handle)
    G.gnn_profile_enable(m.handle, True)
    for _ in range(10):
        m(x, ei, out)
    prof_all = G.gnn_profile_read(m.handle)
    G.gnn_profile_enable(m.handle, False)
    per = np.array([a.elapsed_time(b) for a, b in evs])
    scores = out.cpu().numpy()
    zt = torch.empty_like(out)
    m(x, ei, zt, logits=True)
    torch.cuda.synchronize()
    ms = (t1 - t0) * 1000.0 / steps
    return {"ms_per_step": ms, "per": per, "prof": prof, "prof_all": prof_all, "scores": scores,
            "logits": zt.cpu().numpy(), "model": m, "x": x, "ei": ei, "out": out}


def f16w_rooflines(roof, roof_node):
    """The fp16-weight kernels execute one fp16 product per weight, half
    the hi/lo bf16 kernels' matrix work (rooflines() counts the latter)."""
    roof["kernel"] = "edge_split<4,3,f16w> (fp16 weights in LDS, bf16 rows converted exactly)"
    for r in (roof, roof_node):
        if r and "mfma" in r:
            r["mfma"]["executed_tflop_per_launch"] /= 2.0
            r["mfma"]["achieved"] = round(r["mfma"]["achieved"] / 2.0, 1)
            r["mfma"]["frac"] = round(r["mfma"]["frac"] / 2.0, 4)
            r["mfma"]["dtype"] = "fp16"
    if roof_node:
        roof_node["kernel"] = "node_split<4,false,1,f16w> (fp16 weights streamed through LDS; " \
                              "fp16 projections)"


def rooflines(prof, N, E, H, T, bf16, split, factored, n_src, traffic, ceil=None):
    """Edge-update (dominant), node-update and aggregation rooflines from the
    library's per-stage HIP-event times over the timed region (the sampled
    profiler: one launch of each per event, that of iteration T // 2).  The
    events bracket the dispatch, so each launch reads about 4 us above the
    kernel's own duration in a kernel trace."""
    act_bytes = 2 if bf16 else 4
    eu = prof["edge_update"]
    eu_ms = eu["ms"] / max(eu["launches"], 1)
    eu_flops = edge_update_flops(E, H, factored)
    ag = prof["aggregate"]
    ag_ms = ag["ms"] / max(ag["launches"], 1)
    ag_bytes = aggregate_bytes(N, E, H, act_bytes, n_src)
    ag_gbs = ag_bytes / (ag_ms / 1000.0) / 1e9
    nu = prof["node_update"]
    nu_ms = nu["ms"] / max(nu["launches"], 1)
    roof_node = None
    if split:
        eb = edge_update_bytes(N, E, H, act_bytes, n_src)
        gbs = eb / (eu_ms / 1000.0) / 1e9
        mf = split_mfma_flops(N, E, H, bf16)
        eu_mfma = mf["edge_update"] / (eu_ms / 1000.0) / 1e12
        mdt = "bf16" if bf16 else "fp16"
        roof = {"kernel": ("edge_split<4,3,bf16> (gathers fp16 node projections, W_e e, layer "
                           "2 transposed, per-source sums of its rows; hi/lo bf16 weights in "
                           "LDS)") if bf16 else
                          ("edge_split<4,3> (gathers node projections, W_e e, layer 2 "
                           "transposed, per-source sums of its rows; f16x2 weights in LDS)"),
                "bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": sum(traffic) if traffic else None,
                "bytes_per_launch": eb, "avg_launch_ms": round(eu_ms, 4),
                "mfma": {"dtype": mdt, "executed_tflop_per_launch": mf["edge_update"] / 1e12,
                         "achieved": round(eu_mfma, 1), "peak": PEAK_TFLOPS[mdt],
                         "unit": "TFLOP/s", "frac": round(eu_mfma / PEAK_TFLOPS[mdt], 4),
                         "fp32_equivalent_tflops": round(eu_flops / (eu_ms / 1000.0) / 1e12, 1)}}
        if traffic:
            # the counter-measured HBM stream of the same launch, beside the
            # algorithmic rate (on-die reuse of the gathered rows makes it lower)
            tg = sum(traffic) / (eu_ms / 1000.0) / 1e9
            roof["traffic_gbs"] = round(tg, 1)
            roof["traffic_frac"] = round(tg / PEAK_HBM_GBS, 4)
        # against the measured streaming ceilings: the counter split when the
        # counters match these sources, else the algorithmic one (gathered
        # rows counted per edge, an upper bound of the bytes moved)
        pr = practical(traffic or edge_update_rw(N, E, H, act_bytes, n_src), eu_ms / 1000.0, ceil)
        if pr:
            pr["bytes"] = "counters" if traffic else "algorithmic"
            roof["practical"] = pr
        # the sampled launch (iteration T // 2), not the average over T
        nb = sum(node_update_sampled_rw(N, H, act_bytes, T))
        nu_gbs = nb / (nu_ms / 1000.0) / 1e9
        nu_mfma = mf["node_update"] / (nu_ms / 1000.0) / 1e12
        roof_node = {"kernel": ("node_split<4,false,1,bf16> (hi/lo bf16 weights streamed "
                                "through LDS; fp16 projections)") if bf16 else
                               ("node_split<4,false,1> (f16x2 products, per-node row scale in "
                                "layer 1; weights streamed through LDS)"),
                     "bound": "hbm", "achieved": round(nu_gbs, 1), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(nu_gbs / PEAK_HBM_GBS, 4),
                     "bytes_per_launch": nb, "avg_launch_ms": round(nu_ms, 4),
                     "mfma": {"dtype": "bf16" if bf16 else "fp16",
                              "executed_tflop_per_launch": mf["node_update"] / 1e12,
                              "achieved": round(nu_mfma, 1), "peak": PEAK_TFLOPS["fp16"],
                              "unit": "TFLOP/s", "frac": round(nu_mfma / PEAK_TFLOPS["fp16"], 4)}}
        pr = practical(node_update_sampled_rw(N, H, act_bytes, T), nu_ms / 1000.0, ceil)
        if pr:
            roof_node["practical"] = pr
    else:
        achieved = eu_flops / (eu_ms / 1000.0) / 1e12
        peak = PEAK_TFLOPS["fp32"]
        roof = {"kernel": ("edge_f32<4,1> (gathers node projections, W_e e, layer 2; "
                           "weights in LDS)") if factored else
                          ("gmlp edge update (gathers [h_src; h_dst; e], 3H->H->H)"),
                "bound": "mfma", "achieved": round(achieved, 2), "peak": peak,
                "unit": "TFLOP/s", "frac": round(achieved / peak, 4), "traffic": sum(traffic) if traffic else None,
                "flops_per_launch": eu_flops, "avg_launch_ms": round(eu_ms, 4)}
    roof_agg = {"kernel": ("aggregate (in-direction CSR sums; out-direction rows the edge update "
                           "left in pieces completed, empty rows zeroed)") if n_src else
                          "aggregate (CSR segmented sums, in and out)",
                "bound": "hbm", "achieved": round(ag_gbs, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(ag_gbs / PEAK_HBM_GBS, 4),
                "bytes_per_launch": ag_bytes, "avg_launch_ms": round(ag_ms, 4)}
    if n_src:
        pr = practical(aggregate_rw(N, E, H, act_bytes, n_src), ag_ms / 1000.0, ceil)
        if pr:
            roof_agg["practical"] = pr
    return roof, roof_node, roof_agg


def stages(prof):
    """ms per event of every stage (a profile of calls with every stage timed)."""
    return {k: round(v["ms"] / max(prof["n_calls"], 1), 4) for k, v in prof.items()
            if k != "n_calls"}


def bench_filter(G, I, cfg):
    """The step before the GNN: filter MLP + threshold compaction over the
    candidate edges of the same hits (wide windows, ~2.1M candidates)."""
    import torch
    g = I.layered_graph(cfg.n_nodes, cfg.graph_seed, I.DPHI_MID, I.DZ_MID)
    f = G.gnn_filter_create(I.make_filter_weights(3, 64, 77), G.make_filter_dims(3, 64))
    x = torch.as_tensor(g.x).cuda()
    ei = torch.as_tensor(g.edge_index).cuda()
    sc = torch.empty(g.n_edges, device="cuda")
    out = torch.empty(2 * g.n_edges, dtype=torch.int32, device="cuda")
    kept = G.gnn_filter_apply(f, x, ei, g.n_nodes, g.n_edges, 0.5, sc, out)
    torch.cuda.synchronize()
    t = time.perf_counter()
    for _ in range(5):
        kept = G.gnn_filter_apply(f, x, ei, g.n_nodes, g.n_edges, 0.5, sc, out)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t) * 1000.0 / 5
    G.gnn_filter_destroy(f)
    # multiply-adds x 2 per candidate: layer 1 (2F -> 64, VALU), layer 2
    # (64 -> 64, fp32 matrix cores), head (64 -> 1)
    flop = 2.0 * g.n_edges * (2 * 3 * 64 + 64 * 64 + 64)
    tf = flop / (ms / 1000.0) / 1e12
    return {"ms_per_event": round(ms, 4), "candidates": g.n_edges, "kept": kept,
            "candidate_edges_per_s": round(g.n_edges / (ms / 1000.0), 1),
            "roofline": {"bound": "mfma", "achieved": round(tf, 2), "peak": PEAK_TFLOPS["fp32"],
                         "unit": "TFLOP/s", "frac": round(tf / PEAK_TFLOPS["fp32"], 4),
                         "flops_per_call": flop,
                         "note": "algorithmic fp32 FLOP over the wall time of the whole call "
                                 "(scoring, compaction, count read-back); layer 2 runs on the "
                                 "fp16 matrix cores from split operands"},
            "note": "filter MLP (2F->64->64->1) + stable compaction at 0.5 on the same hits "
                    "with the wide windows (wall time incl. the count read-back); not part "
                    "of value"}


def bench_graph_construction(G, I, g):
    """Embedding MLP (F -> 128 -> 128 -> 8) on the event's hits and the
    fixed-radius pair search on 300k clustered points in 8 dimensions (a
    stand-in for a trained embedding space: 80% of the points in tight
    groups)."""
    import torch
    w = I.make_embed_weights(3, 128, 8, 3000)
    m = G.Embedder(w, G.make_embed_dims(3, 128, 8))
    x = torch.as_tensor(g.x).cuda()
    z = m(x)
    torch.cuda.synchronize()
    t = time.perf_counter()
    for _ in range(10):
        m(x, z)
    torch.cuda.synchronize()
    embed_ms = (time.perf_counter() - t) * 100.0
    m.close()
    pts = torch.as_tensor(I.clustered_points(300_000, 8, 977, sigma=0.005)).cuda()
    r2 = 0.02 ** 2
    ei = G.radius_graph(pts, r2)
    torch.cuda.synchronize()
    t = time.perf_counter()
    for _ in range(5):
        ei = G.radius_graph(pts, r2)
    torch.cuda.synchronize()
    frnn_ms = (time.perf_counter() - t) * 200.0
    # multiply-adds x 2 per point: 3 -> 128 (VALU), 128 -> 128 (fp32 matrix
    # cores), 128 -> 8 (VALU)
    eflop = 2.0 * g.n_nodes * (3 * 128 + 128 * 128 + 128 * 8)
    etf = eflop / (embed_ms / 1000.0) / 1e12
    return {"embed_ms": round(embed_ms, 4), "embed_points": int(g.n_nodes),
            "embed_roofline": {"bound": "mfma", "achieved": round(etf, 2),
                               "peak": PEAK_TFLOPS["fp32"], "unit": "TFLOP/s",
                               "frac": round(etf / PEAK_TFLOPS["fp32"], 4),
                               "flops_per_call": eflop,
                               "note": "algorithmic fp32 FLOP; layer 2 runs on the fp16 matrix "
                                       "cores from split operands"},
            "frnn_ms": round(frnn_ms, 4), "frnn_points": 300_000, "frnn_dim": 8,
            "frnn_pairs": int(ei.shape[1]),
            "note": "embedding MLP 3->128->128->8 on the event's hits; fixed-radius pairs "
                    "(r = 0.02) on 300k clustered 8-d points, count + fill passes with the "
                    "count read-back (wall time); not part of value"}


def batch_leg(G, I, cfg, steps, warmup):
    """Ragged service batch: 8 independent events, one stream each, one
    handle; then the library's request queue with 1, 2, 4 and 8 instances
    (paper section 3.2, Fig. 4b: throughput and GPU utilisation against the
    number of model instances)."""
    import numpy as np
    import torch

    events = I.make_batch(cfg)
    H, T = cfg.hidden, cfg.n_iters
    w = I.make_weights(3, H, 1, cfg.weight_seed)
    m = G.Model(w, G.make_dims(3, H, T))
    xs = [torch.as_tensor(g.x).cuda() for g in events]
    eis = [torch.as_tensor(g.edge_index).cuda() for g in events]
    outs = [torch.empty(g.n_edges, device="cuda") for g in events]
    streams = [torch.cuda.Stream() for _ in events]
    total_e = sum(g.n_edges for g in events)

    def one_batch(evs=None):
        for k, st in enumerate(streams):
            if evs is not None:
                evs[k][0].record(st)
            G.gnn_infer(m.handle, xs[k], eis[k], xs[k].shape[0], eis[k].shape[1], outs[k], st)
            if evs is not None:
                evs[k][1].record(st)

    for _ in range(warmup):
        one_batch()
    torch.cuda.synchronize()
    samples = []
    t0 = time.perf_counter()
    for _ in range(steps):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in streams]
        one_batch(evs)
        samples.append(evs)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    per = np.array([a.elapsed_time(b) for evs in samples for a, b in evs])

    # The request queue serves 16 requests (the 8 events twice, all submitted
    # at once) with k worker streams sharing one handle.  Utilisation: the
    # union of the requests' device intervals over the wall time from the
    # first submit to the last completion.
    sweep = []
    for k in (1, 2, 4, 8):
        srv = G.Server(m, k)
        ids = [srv.submit(xs[i % 8], eis[i % 8], outs[i % 8]) for i in range(8)]
        for i in ids:
            srv.wait(i)  # warm-up round
        ts = time.perf_counter()
        ids = [srv.submit(xs[i % 8], eis[i % 8], outs[i % 8]) for i in range(16)]
        infos = [srv.wait_info(i) for i in ids]
        ms = (time.perf_counter() - ts) * 1000.0
        srv.close()
        lats = [i["latency_ms"] for i in infos]
        busy = union_ms([(i["device_start_ms"], i["device_end_ms"]) for i in infos])
        sweep.append({"instances": k, "ms_per_16_requests": round(ms, 3),
                      "edges_per_s": round(2 * total_e / (ms / 1000.0), 1),
                      "latency_ms_p50": round(float(np.percentile(lats, 50)), 3),
                      "latency_ms_p99": round(float(np.percentile(lats, 99)), 3),
                      "gpu_busy_ms": round(busy, 3),
                      "gpu_utilisation": round(busy / ms, 4)})
    m.close()
    ms_per_batch = (t1 - t0) * 1000.0 / steps
    return {
        "edges_per_s": round(total_e / (ms_per_batch / 1000.0), 1),
        "ms_per_batch": round(ms_per_batch, 4), "batches": steps, "warmup": warmup,
        "n_events": len(events), "n_nodes": [g.n_nodes for g in events],
        "n_edges": [g.n_edges for g in events], "total_edges": total_e,
        "ms_per_event_p50": round(float(np.percentile(per, 50)), 3),
        "ms_per_event_p99": round(float(np.percentile(per, 99)), 3),
        "server_instances": sweep,
        "note": "8 events on 8 streams of one handle (H=128, T=8, fp32); per-event times overlap "
                "across streams, the aggregate rate is the sum of edges over the wall time of "
                "the batch.  server_instances: the request queue with k worker streams, 16 "
                "requests submitted at once; gpu_utilisation = union of the requests' device "
                "intervals (events on the worker streams) over the wall time",
    }


# ------------------------------------------------------------- CPU leg ---

def cpu_baseline(O, I, g, w, cfg, full):
    """The fp64 oracle as it stands, timed on this host: the measured event
    three times on the cores available to this process (median), and for the
    full event also the tiny and mid workloads on one thread and on all of
    them.  Returns the record and the oracle output of the measured event."""
    import numpy as np
    host = host_info()
    n = host["physical_cores_in_affinity"]
    if host["cgroup_cpu_quota"]:
        n = min(n, max(1, int(host["cgroup_cpu_quota"])))
    if host["omp_num_threads_env"] and host["omp_num_threads_env"].isdigit():
        n = min(n, int(host["omp_num_threads_env"]))
    n = max(1, n)
    O.set_threads(n)
    times, ref = [], None
    for _ in range(3):
        t = time.perf_counter()
        r = O.forward(w, g.x, g.edge_index, cfg.hidden, cfg.n_iters)
        times.append(time.perf_counter() - t)
        ref = ref or r
    med = float(np.median(times))
    rec = {"value": round(g.n_edges / med, 1), "unit": "edges/s", "cores": n, "kind": "oracle",
           "sample": f"median of 3 complete fp64 oracle inferences of the same "
                     f"{g.n_nodes}-node / {g.n_edges}-edge event (H={cfg.hidden}, "
                     f"T={cfg.n_iters}) on {n} threads: "
                     + ", ".join(f"{t:.2f}" for t in times) + " s",
           "host": {k: v for k, v in host.items() if k != "libgnn_build"},
           "oracle_cflags": " ".join(O.CFLAGS)}
    if full:
        sweep = {}
        for name in ("tiny", "mid"):
            c = I.CONFIGS[name]
            gg = I.make_graph(c)
            ww = I.make_weights(3, c.hidden, 1, c.weight_seed)
            for th in (1, n):
                O.set_threads(th)
                reps = 3 if (name == "tiny" or th > 1) else 1
                ts = []
                for _ in range(reps):
                    t = time.perf_counter()
                    O.forward(ww, gg.x, gg.edge_index, c.hidden, c.n_iters)
                    ts.append(time.perf_counter() - t)
                s = float(np.median(ts))
                sweep[f"{name}_{th}_threads"] = {
                    "n_nodes": gg.n_nodes, "n_edges": gg.n_edges, "hidden": c.hidden,
                    "n_iters": c.n_iters, "runs": reps, "seconds_median": round(s, 4),
                    "edges_per_s": round(gg.n_edges / s, 1)}
        O.set_threads(n)
        rec["other_workloads"] = sweep
    return rec, ref


# ---------------------------------------------------------------- main ---

def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="full",
                    choices=["full", "full_bf16", "mid", "tiny", "batch"])
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle (no cpu_baseline and no parity check)")
    ap.add_argument("--no-extra-legs", action="store_true",
                    help="full workload: skip the bf16 and batch legs and the side figures")
    ap.add_argument("--literal", action="store_true",
                    help="evaluate the edge MLPs' first layer per edge (GNN_LITERAL_GATHER)")
    ap.add_argument("--fp32-mfma", action="store_true",
                    help="fp32 products on the fp32 matrix cores (GNN_FP32_MFMA) instead of "
                         "split fp16/bf16 products")
    ap.add_argument("--f16-weights", action="store_true",
                    help="with --workload full_bf16: fp16 weights (GNN_F16_WEIGHTS)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy 3 times (reference "
                         "kernel of known traffic for scaling HBM byte counters)")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        n = (1 << 30) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "copies": 3}))
        return
    if args.f16_weights and (args.workload != "full_bf16" or args.literal or args.fp32_mfma):
        print("--f16-weights needs --workload full_bf16 on the regrouped kernels (no --literal, "
              "no --fp32-mfma)", file=sys.stderr)
        sys.exit(2)
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(events are independent: one process per GPU serves them). Use --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2402_09633_amd import gnn as G
    from paper_2402_09633_amd import inputs as I

    cfg = I.CONFIGS[args.workload]
    torch.cuda.set_device(0)
    if cfg.kind == "batch":
        b = batch_leg(G, I, cfg, args.steps, args.warmup)
        rec = {"metric": "aggregate edges/sec and p50/p99 ms/event, ragged batch of 8 events "
                         "on 8 streams",
               "value": b["edges_per_s"], "unit": "edges/s", "n_gpus": 1, "steps": args.steps,
               "warmup": args.warmup, "ms_per_step": b["ms_per_batch"],
               "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
               "dtype": "f32", "data": "synthetic",
               "config": {"workload": f"batch: 8 events, N={b['n_nodes']}, E={b['n_edges']}, "
                                      f"H={cfg.hidden}, T={cfg.n_iters}, fp32"},
               "batch": b}
        print(json.dumps(rec), flush=True)
        return

    g = I.make_graph(cfg)
    N, E, H, T = g.n_nodes, g.n_edges, cfg.hidden, cfg.n_iters
    w = I.make_weights(3, H, 1, cfg.weight_seed)
    bf16 = cfg.dtype == "bf16"
    dtype = G.GNN_BF16 if bf16 else G.GNN_FP32
    flags = (G.GNN_LITERAL_GATHER if args.literal else 0) | \
        (G.GNN_FP32_MFMA if args.fp32_mfma else 0) | \
        (G.GNN_F16_WEIGHTS if args.f16_weights else 0)
    factored = not args.literal
    split = factored and (bf16 or not args.fp32_mfma)
    path = (("f16w" if args.f16_weights else "bf16") if bf16 else "split") if split else \
        ("fp32_mfma" if factored else "literal")
    extra = cfg.name == "full" and not args.no_extra_legs
    print(f"# workload {cfg.name}: N={N} E={E} H={H} T={T} {cfg.dtype}", file=sys.stderr,
          flush=True)

    leg = timed_leg(G, torch, np, g, w, H, T, dtype, flags, args.steps, args.warmup)
    m, x, ei, out = leg["model"], leg["x"], leg["ei"], leg["out"]
    ms_per_step = leg["ms_per_step"]
    value = E / (ms_per_step / 1000.0)
    print(f"# timed: {ms_per_step:.4f} ms/event", file=sys.stderr, flush=True)

    # Next pipeline step, measured on its own: connected components of the
    # edges scoring above 0.5 (labels = smallest hit id per component).
    labels = torch.empty(N, dtype=torch.int32, device="cuda")
    G.gnn_wcc(ei, out, 0.5, N, E, labels)
    torch.cuda.synchronize()
    tw = time.perf_counter()
    for _ in range(5):
        G.gnn_wcc(ei, out, 0.5, N, E, labels)
    torch.cuda.synchronize()
    wcc_ms = (time.perf_counter() - tw) * 1000.0 / 5
    n_comp = int(torch.unique(labels).numel())
    # The same event with its edge list in a seeded random order (the
    # generator emits edges grouped by source, which favours the gathers).
    gs, _ = I.shuffled(g, 7)
    eis_ = torch.as_tensor(gs.edge_index).cuda()
    m(x, eis_, out)
    torch.cuda.synchronize()
    ts = time.perf_counter()
    for _ in range(5):
        m(x, eis_, out)
    torch.cuda.synchronize()
    shuf_ms = (time.perf_counter() - ts) * 1000.0 / 5
    del eis_
    m.close()

    n_src = int(np.unique(g.edge_index[0]).size) if split else 0
    traffic = None
    if factored and cfg.name in ("full", "full_bf16") and path in TRAFFIC_SOURCES:
        traffic = MEASURED_TRAFFIC.get((path, kernel_source_hash(path)))
    ceil = hbm_ceiling(G, torch)
    roof, roof_node, roof_agg = rooflines(leg["prof"], N, E, H, T, bf16, split, factored,
                                          n_src, traffic, ceil)
    if path == "f16w":
        f16w_rooflines(roof, roof_node)
    per = leg["per"]
    rec = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "edges/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if cfg.dtype == "fp32" else "bf16",
        "data": "synthetic (seeded layered hit graph, seeded Xavier weights)",
        "config": {"workload": f"{cfg.name}: {N}-hit / {E}-edge layered event, H={H}, T={T}, "
                               f"{cfg.dtype}", "n_nodes": N, "n_edges": E, "hidden": H,
                   "n_iters": T, "parallelism": "single GPU",
                   "products": {"split": "fp32 operands split into fp16 pairs on the fp16 "
                                         "matrix cores, fp32 accumulation",
                                "fp32_mfma": "fp32 matrix cores",
                                "literal": "per-edge first layer",
                                "bf16": "bf16 activations on the bf16 matrix cores, hi/lo "
                                        "bf16 weights, fp32 accumulation",
                                "f16w": "bf16 activations converted exactly to fp16, fp16 "
                                        "weights, fp16 matrix cores, fp32 accumulation"}[path]},
        "ms_per_event_p50": round(float(np.percentile(per, 50)), 4),
        "ms_per_event_p99": round(float(np.percentile(per, 99)), 4),
        "ms_per_event_min": round(float(per.min()), 4),
        "roofline": roof,
        "roofline_aggregate": roof_agg,
        "hbm_ceiling": ceil,
        "stages_ms_per_event": stages(leg["prof_all"]),
        "components": {"ms_per_event": round(wcc_ms, 4), "threshold": 0.5,
                       "n_components": n_comp,
                       "note": "weakly-connected components of the edges scoring above the "
                               "threshold, after inference (wall time, host-checked rounds); "
                               "not part of value"},
    }
    if roof_node:
        rec["roofline_node_update"] = roof_node
    rec["shuffled_edge_order"] = {
        "ms_per_event": round(shuf_ms, 4), "edges_per_s": round(E / shuf_ms * 1e3, 1),
        "note": "same event, edge list in a seeded random order (seed 7), 5 events after the "
                "timed region; not part of value"}
    bleg = fleg = None
    if extra:
        # The same event on the fp32 matrix cores (reported for comparison only).
        m2 = G.Model(w, G.make_dims(3, H, T, 1, dtype, flags=G.GNN_FP32_MFMA))
        m2(x, ei, out)
        torch.cuda.synchronize()
        ts = time.perf_counter()
        for _ in range(5):
            m2(x, ei, out)
        torch.cuda.synchronize()
        side_ms = (time.perf_counter() - ts) * 1000.0 / 5
        m2.close()
        rec["fp32_mfma_path"] = {
            "ms_per_event": round(side_ms, 4), "edges_per_s": round(E / side_ms * 1e3, 1),
            "note": "same event with GNN_FP32_MFMA (products on the fp32 matrix cores), "
                    "5 events after the timed region; not part of value"}
        # The bf16 model on the same event and weights, timed like the main leg.
        bleg = timed_leg(G, torch, np, g, w, H, T, G.GNN_BF16, 0, args.steps, args.warmup)
        bleg["model"].close()
        btraffic = MEASURED_TRAFFIC.get(("bf16", kernel_source_hash("bf16")))
        broof, broof_node, broof_agg = rooflines(bleg["prof"], N, E, H, T, True, True, True,
                                                 n_src, btraffic, ceil)
        rec["bf16"] = {
            "ms_per_event": round(bleg["ms_per_step"], 4),
            "edges_per_s": round(E / (bleg["ms_per_step"] / 1000.0), 1),
            "steps": args.steps, "warmup": args.warmup,
            "ms_per_event_p50": round(float(np.percentile(bleg["per"], 50)), 4),
            "ms_per_event_p99": round(float(np.percentile(bleg["per"], 99)), 4),
            "roofline": broof, "roofline_node_update": broof_node,
            "roofline_aggregate": broof_agg, "stages_ms_per_event": stages(bleg["prof_all"]),
            "weights": "each weight carried as two bf16 terms hi = bf16(W), lo = bf16(W - hi) "
                       "(two products per weight): with plain bf16 weights the full event's "
                       "score error measured 2.20e-2, above the 2e-2 bound",
            "note": "same event and fp32 weights, bf16 activations in HBM and as matrix "
                    "operands, fp32 accumulation; timed like the main leg, after it; not part "
                    "of value"}
        # The same model with GNN_F16_WEIGHTS: one fp16 number per weight.
        fleg = timed_leg(G, torch, np, g, w, H, T, G.GNN_BF16, G.GNN_F16_WEIGHTS, args.steps,
                         args.warmup)
        fleg["model"].close()
        ftraffic = MEASURED_TRAFFIC.get(("f16w", kernel_source_hash("f16w")))
        froof, froof_node, froof_agg = rooflines(fleg["prof"], N, E, H, T, True, True, True,
                                                 n_src, ftraffic, ceil)
        f16w_rooflines(froof, froof_node)
        rec["bf16"]["f16_weights"] = {
            "ms_per_event": round(fleg["ms_per_step"], 4),
            "edges_per_s": round(E / (fleg["ms_per_step"] / 1000.0), 1),
            "ms_per_event_p50": round(float(np.percentile(fleg["per"], 50)), 4),
            "ms_per_event_p99": round(float(np.percentile(fleg["per"], 99)), 4),
            "roofline": froof, "roofline_node_update": froof_node,
            "roofline_aggregate": froof_agg, "stages_ms_per_event": stages(fleg["prof_all"]),
            "weights": "GNN_F16_WEIGHTS: each weight one fp16 number times a power of two (one "
                       "fp16 product per weight); activations bf16 in HBM, rounded to bf16 "
                       "where they feed a product and converted exactly to fp16",
            "note": "the bf16 model with the other 16-bit weight format; the edge encoder "
                    "runs inside the first edge update's kernel (its three weight matrices "
                    "fit in LDS together; stages_ms_per_event counts it there); timed like the "
                    "main leg, after the bf16 leg; not part of value"}
        del x, ei, out
        torch.cuda.empty_cache()
        rec["filter"] = bench_filter(G, I, cfg)
        rec["graph_construction"] = bench_graph_construction(G, I, g)
        print("# batch leg", file=sys.stderr, flush=True)
        bc = I.CONFIGS["batch"]
        rec["batch"] = batch_leg(G, I, bc, min(args.steps, 10), min(args.warmup, 2))

    info = host_info()
    rec["host"] = {"cpu_model": info["cpu_model"], "hipcc": info["hipcc"],
                   "libgnn_build": info["libgnn_build"]}
    status = 0
    if not args.no_cpu_baseline:
        from oracle import oracle as O
        print("# cpu baseline (oracle)", file=sys.stderr, flush=True)
        cpu, ref = cpu_baseline(O, I, g, w, cfg, extra)
        rec["cpu_baseline"] = cpu
        if bf16:
            serr = float(np.max(np.abs(leg["scores"] - ref["scores"]))) if E else 0.0
            ok = serr <= BF16_SCORE_ATOL
            rec["parity"] = {"max_score_err": serr, "n_edges_compared": E,
                             "tol": BF16_SCORE_ATOL, "pass": ok}
        else:
            zerr = max_scaled_err(leg["logits"], ref["logits"])
            serr = float(np.max(np.abs(leg["scores"] - ref["scores"]))) if E else 0.0
            ok = zerr <= FP32_LOGIT_RTOL
            rec["parity"] = {"max_scaled_logit_err": zerr, "max_score_err": serr,
                             "n_edges_compared": E, "tol": FP32_LOGIT_RTOL, "pass": ok}
        if bleg is not None:
            berr = float(np.max(np.abs(bleg["scores"] - ref["scores"])))
            rec["bf16"]["max_score_err"] = berr
            rec["bf16"]["n_edges_compared"] = E
            rec["bf16"]["parity_pass"] = berr <= BF16_SCORE_ATOL
            ok = ok and berr <= BF16_SCORE_ATOL
            if fleg is not None:
                ferr = float(np.max(np.abs(fleg["scores"] - ref["scores"])))
                fw = rec["bf16"]["f16_weights"]
                fw["max_score_err"] = ferr
                fw["n_edges_compared"] = E
                fw["parity_pass"] = ferr <= BF16_SCORE_ATOL
                ok = ok and ferr <= BF16_SCORE_ATOL
        rec["parity"]["note"] = ("the timed path's output (and the bf16 leg's scores) against "
                                 "the fp64 oracle on every edge of the event; computed after "
                                 "the timed region")
        if not ok:
            status = 3
    print(json.dumps(rec), flush=True)
    if status:
        print("bench.py: the GPU output disagrees with the oracle beyond the tolerance",
              file=sys.stderr)
        sys.exit(status)


if __name__ == "__main__":
    main()
