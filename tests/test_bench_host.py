"""Host-side logic of bench.py (no GPU): the one-GPU guard and the
algorithmic byte and matrix-work counts behind its roofline figures, each
checked against the per-unit definition written out by hand for the full
event (300,000 hits, 1,000,513 edges, H = 128, T = 8; 247,893 hits have
out-edges)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

N, E, H, T, N_SRC = 300_000, 1_000_513, 128, 8, 247_893


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_edge_update_bytes_per_launch():
    # per edge: e row read and written (2 x 512 B), the two gathered
    # projection half-rows (2 x 512 B), two int32 indices; per source node
    # one agg_out row (512 B)
    per_edge = 2 * 512 + 2 * 512 + 8
    assert bench.edge_update_bytes(N, E, H, 4, N_SRC) == E * per_edge + N_SRC * 512
    assert bench.edge_update_bytes(N, E, H, 4, N_SRC) == 2_183_975_944
    # bf16 model: e and agg_out rows in bf16, the projections in fp16
    assert bench.edge_update_bytes(N, E, H, 2, N_SRC) == E * (2 * 256 + 2 * 256 + 8) + N_SRC * 256


def test_aggregate_bytes_per_launch():
    # fused form: message rows (in-direction) and their int32 positions,
    # agg_in rows, both row-pointer arrays, a zero agg_out row per hit
    # without out-edges
    want = E * 512 + E * 4 + N * 512 + 2 * (N + 1) * 4 + (N - N_SRC) * 512
    assert bench.aggregate_bytes(N, E, H, 4, N_SRC) == want == 698_943_500
    # unfused form: both directions of everything
    assert bench.aggregate_bytes(N, E, H, 4) == 2 * (E * 512 + N * 512 + E * 4 + (N + 1) * 4)


def test_node_update_bytes_average_launch():
    # h, agg_in, agg_out read and the 2H-float projection row written every
    # launch; h written in 7 of the 8 launches
    want = N * (3 * 512 + 1024) + N * 512 * 7 / 8
    assert bench.node_update_bytes(N, H, 4, T) == pytest.approx(want, rel=0, abs=1e-6)
    assert bench.node_update_bytes(N, H, 4, T) == 902_400_000
    # bf16 model: 256-byte rows, the fp16 projection row 512 bytes
    assert bench.node_update_bytes(N, H, 2, T) == N * (3 * 256 + 512) + N * 256 * 7 / 8


def test_matrix_work_per_launch():
    # split fp32: three fp16 products per fp32 product; the edge update runs
    # W_e e and layer 2 (2 H^2 per edge), the node update layer 1 (3 H^2),
    # layer 2 (H^2) and the projections (2 H^2)
    f = bench.split_mfma_flops(N, E, H)
    assert f["edge_update"] == 3 * 2 * E * 2 * H * H == 196_708_859_904
    assert f["node_update"] == 3 * 2 * N * 6 * H * H
    b = bench.split_mfma_flops(N, E, H, bf16=True)
    assert b["edge_update"] == 2 * 2 * E * 2 * H * H
    # the fp32 model's algorithmic work: regrouped 2 H^2 per edge, per-edge 4 H^2
    assert bench.edge_update_flops(E, H, True) == 2 * E * 2 * H * H
    assert bench.edge_update_flops(E, H, False) == 2 * E * 4 * H * H


def test_union_of_device_intervals():
    # the utilisation figure: overlapping requests count once, gaps not at all
    assert bench.union_ms([]) == 0.0
    assert bench.union_ms([(0.0, 1.0)]) == 1.0
    assert bench.union_ms([(0.0, 1.0), (0.5, 2.0), (3.0, 4.0), (3.5, 3.6)]) == 3.0
    assert bench.union_ms([(3.0, 4.0), (0.0, 1.0), (1.0, 2.0)]) == 3.0  # order-free, touching


def test_max_scaled_error_definition():
    # |z - z_ref| / max(1, |z_ref|): absolute below 1, relative above
    assert bench.max_scaled_err([0.5, 10.0], [0.5, 10.0]) == 0.0
    assert bench.max_scaled_err([0.0], [1e-3]) == pytest.approx(1e-3)
    assert bench.max_scaled_err([101.0], [100.0]) == pytest.approx(1e-2)
    assert bench.max_scaled_err([], []) == 0.0


def test_practical_ceiling_is_the_serial_read_write_bound():
    # 1 GB read at 8 GB/s and 0.5 GB written at 4 GB/s need at least
    # 0.125 + 0.125 s: a launch of 0.5 s reaches half of that ceiling
    ceil = {"read_gbs": 8.0, "write_gbs": 4.0}
    pr = bench.practical((1e9, 0.5e9), 0.5, ceil)
    assert pr["ceiling_gbs"] == pytest.approx(1.5e9 / 0.25 / 1e9)
    assert pr["achieved_gbs"] == pytest.approx(3.0)
    assert pr["frac"] == pytest.approx(0.5)
    assert bench.practical((1e9, 0.5e9), 0.5, None) is None


def test_read_write_splits_add_up_to_the_byte_counts():
    for s in (4, 2):
        r, w = bench.edge_update_rw(N, E, H, s, N_SRC)
        assert r + w == pytest.approx(bench.edge_update_bytes(N, E, H, s, N_SRC))
        r, w = bench.node_update_rw(N, H, s, T)
        assert r + w == pytest.approx(bench.node_update_bytes(N, H, s, T))
        r, w = bench.aggregate_rw(N, E, H, s, N_SRC)
        assert r + w == pytest.approx(bench.aggregate_bytes(N, E, H, s, N_SRC))


@pytest.mark.parametrize("extra", [["--workload", "full"], ["--workload", "full_bf16", "--literal"]])
def test_f16_weights_needs_the_regrouped_bf16_workload(extra):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--f16-weights", *extra],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "--f16-weights needs" in r.stderr
    assert r.stdout == ""


def test_sampled_node_update_launch_bytes():
    # the profiler times iteration T // 2 = 4 of 8, which stores h: reads h,
    # agg_in, agg_out, writes the projection row and h
    r, w = bench.node_update_sampled_rw(N, H, 4, T)
    assert (r, w) == (N * 3 * 512, N * (1024 + 512))
    # T = 1 and T = 2: the sampled launch is the last one and stores no h
    assert bench.node_update_sampled_rw(N, H, 4, 1)[1] == N * 1024
    assert bench.node_update_sampled_rw(N, H, 4, 2)[1] == N * 1024
    assert bench.node_update_sampled_rw(N, H, 2, 3)[1] == N * (512 + 256)
