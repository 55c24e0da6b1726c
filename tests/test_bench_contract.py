"""bench.py's output contract: one JSON line with the required fields, and a
clear refusal of more than one GPU (checked without touching a GPU)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


@pytest.mark.gpu
def test_json_line_has_the_required_fields():
    print("bench.py --workload tiny --steps 2 --warmup 1 --workloads tiny,clusters-e64",
          flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny",
                        "--steps", "2", "--warmup", "1", "--workloads", "tiny,clusters-e64"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.startswith("{")]
    assert len(lines) == 1, r.stdout[-2000:]
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 2 and d["warmup"] == 1
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["higher_is_better"] is True
    assert d["vs_baseline"] is None and "workload" in d["config"]
    roof = d["roofline"]
    for key in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in roof, key
    assert roof["bound"] == "hbm" and roof["peak"] == 8000.0 and roof["unit"] == "GB/s"
    assert abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-9
    cpu = d["cpu_baseline"]
    for key in ("value", "unit", "cores", "kind", "sample"):
        assert key in cpu, key
    assert cpu["kind"] == "oracle" and cpu["cores"] >= 1 and cpu["value"] > 0
    # one summary per workload: throughput, HBM fractions, and Eq. 1's V for
    # Algorithm 1 against both owner-only baselines
    assert set(d["workloads"]) == {"tiny", "clusters-e64"}
    for name, e in d["workloads"].items():
        assert e["tokens_per_s"] > 0 and e["ms_per_step"] > 0, name
        assert 0 < e["pack_combine_hbm_frac"] and 0 < e["step_hbm_frac"]
        r_ = e["routing"]
        for k in ("alg1", "owner_only", "contiguous_ep_owner_only"):
            assert r_[k]["V"] >= 0 and 0 <= r_[k]["cross_pair_frac"] <= 1
        # Algorithm 1 picks a minimum cover per token (Section 3.3)
        assert r_["alg1"]["V"] <= r_["owner_only"]["V"]
