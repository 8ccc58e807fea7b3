"""bench.py on the GPU: each path runs a few steps and prints one JSON line with
the fields its consumers read (a child process, as the benchmark is run)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("args", [[], ["--path", "mesh"], ["--path", "p2s"], ["--path", "emd"]],
                         ids=["chamfer", "mesh", "p2s", "emd"])
def test_bench_prints_one_json_line(args):
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "3", "--warmup", "2",
           "--no-cpu-baseline"] + args
    print("[bench test]", " ".join(cmd[1:]), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=240, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, r.stdout
    out = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config"):
        assert key in out, key
    assert out["n_gpus"] == 1 and out["steps"] == 3 and out["warmup"] == 2
    assert out["value"] > 0 and out["ms_per_step"] > 0
    # The clock-settle phase ran before the warm-up and is reported.
    assert out["settle_steps"] >= 5 and out["settle_ms"] > 0
    assert "workload" in out["config"]
    calls = out["ms_per_call"]
    assert all(v > 0 for k, v in calls.items() if isinstance(v, float)), calls
    if "roofline" in out:
        rl = out["roofline"]
        assert rl["bound"] == "alu" and rl["unit"] == "TFLOP/s" and rl["peak"] == 157.3
        # Algorithmic flops over the peak: it can pass 1 where a kernel does
        # less work than the count credits (the fused Chamfer search), never by much.
        assert 0 < rl["frac"] < 1.5 and abs(rl["frac"] - rl["achieved"] / rl["peak"]) < 1e-9
    if not args:
        # The Chamfer path: what the chip executes stays under its peak, and
        # every workload has its figures.
        rl = out["roofline"]
        assert 0 < rl["executed_frac"] < 1.0
        assert abs(rl["executed_frac"] / rl["frac"] - 10.0 / 18.0) < 1e-9
        assert rl["valu_issue_frac"] is None or 0 < rl["valu_issue_frac"] < 1.0
        pc = out["per_config"]
        assert sorted(pc) == sorted(["uniform_b1_n1024", "sphere_b32_n2048", "mesh_b16_n16384",
                                     "gmm_b4_n100000_m10000", "griddup_b8_n65536"])
        for name, c in pc.items():
            assert c["ms_per_step"] > 0 and c["pair_evals_per_s"] > 0, name
            assert all(v > 0 for v in c["ms_per_call"].values()), name
            assert 0 < c["executed_frac"] < 1.0, name
            assert c["valu_issue_frac"] is None or 0 < c["valu_issue_frac"] < 1.0, name
            # Every receiver count is at least 1 somewhere and at most the senders.
            deg = c["max_in_degree"]
            assert 1 <= deg["onto_x"] <= c["M"] and 1 <= deg["onto_y"] <= c["N"], (name, deg)
