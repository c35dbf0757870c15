"""The benchmark's output line: a short run of bench.py (its own process) must print one
JSON object with the fields the benchmark reports, consistent with each other."""
import json
import os
import subprocess
import sys

import pytest

from gpu_helpers import log

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_json_line():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cmd = [sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--steps", "3", "--warmup", "1",
           "--alt-steps", "0", "--cold-reps", "2", "--no-copy-ceiling", "--cpu-seconds", "0.5"]
    log("bench: " + " ".join(cmd[2:]))
    res = subprocess.run(cmd, cwd=ROOT, capture_output=True, text=True, timeout=110)
    assert res.returncode == 0, res.stderr[-2000:]
    lines = [l for l in res.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1, res.stdout[-2000:]
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["unit"] == "RoIs/s" and d["higher_is_better"] is True
    assert d["value"] > 0 and d["ms_per_step"] > 0
    K = d["config"]["num_rois"]
    assert abs(d["value"] - K / (d["ms_per_step"] * 1e-3)) <= 1e-3 * d["value"]
    assert "workload" in d["config"]
    r = d["roofline"]
    for key in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in r, key
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert abs(r["frac"] - r["achieved"] / r["peak"]) <= 1e-3
    assert r["achieved"] == pytest.approx(r["bytes_per_launch"] / (r["launch_ms"] * 1e-3) / 1e9,
                                          rel=1e-3)
    if r["kernel"] == "roi_align_bwd_gather":
        # the same kernel against the effective bytes of the workload (a scatter's
        # read-modify-write included): larger bytes, the same launch time
        assert r["frac_effective"] == pytest.approx(
            r["effective_bytes_per_launch"] / (r["launch_ms"] * 1e-3) / 1e9 / 8000.0, rel=1e-3)
        assert r["effective_bytes_per_launch"] > r["bytes_per_launch"]
    for kind in ("warm", "cold"):
        w = d[kind]
        assert w["unit"] == "RoIs/s" and w["ms_per_step"] > 0
        assert abs(w["value"] - K / (w["ms_per_step"] * 1e-3)) <= 1e-3 * w["value"]
        assert 0 < w["frac_effective_fwd_bwd"] < 2
    assert d["warm"]["ms_per_step"] == d["ms_per_step"]
    c = d["cpu_baseline"]
    for key in ("value", "unit", "cores", "kind", "sample"):
        assert key in c, key
    assert c["kind"] == "oracle" and c["value"] > 0 and c["cores"] >= 1
