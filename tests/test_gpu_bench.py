"""bench.py on the smallest workload (GPU): one JSON line with the keys and
types the benchmark contract fixes, a value consistent with its own step
time, and the roofline and CPU-baseline objects."""
import json
import os
import subprocess
import sys

import pytest

from paper_2402_09633_amd import inputs as I

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_json_line_tiny_workload():
    cmd = [sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", "tiny",
           "--steps", "3", "--warmup", "1"]
    print("running", " ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, r.stdout[-3000:]
    rec = json.loads(lines[0])
    types = {"metric": str, "value": (int, float), "unit": str, "n_gpus": int, "steps": int,
             "warmup": int, "ms_per_step": (int, float), "higher_is_better": bool,
             "scaling": str, "dtype": str, "data": str, "config": dict}
    for k, t in types.items():
        assert isinstance(rec[k], t), k
    assert rec["n_gpus"] == 1 and rec["steps"] == 3 and rec["warmup"] == 1
    assert rec["vs_baseline"] is None and rec["higher_is_better"] is True
    assert rec["unit"] == "edges/s" and rec["dtype"] == "f32"
    assert "workload" in rec["config"]
    g = I.make_graph(I.CONFIGS["tiny"])
    assert rec["config"]["n_edges"] == g.n_edges
    want = g.n_edges / (rec["ms_per_step"] / 1000.0)
    assert abs(rec["value"] - want) <= 1e-3 * want + 1.0
    roof = rec["roofline"]
    assert roof["bound"] in ("hbm", "mfma", "alu")
    assert roof["unit"] in ("GB/s", "TFLOP/s")
    assert roof["achieved"] > 0 and roof["peak"] > 0
    assert abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-3
    assert "traffic" in roof
    cb = rec["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0
    assert cb["unit"] == "edges/s" and cb["sample"]
    assert cb["host"]["physical_cores_in_affinity"] >= 1
    par = rec["parity"]
    assert par["n_edges_compared"] == g.n_edges and par["pass"] is True
    assert par["max_scaled_logit_err"] <= 1e-4
