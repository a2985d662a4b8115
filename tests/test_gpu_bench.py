"""The bench.py contract on the small workload: one JSON line with the metric,
the per-stage times, the roofline object and the CPU baseline; the stage
clock the roofline is timed with leaves the output unchanged (GPU)."""
import json
import os
import subprocess
import sys

import pytest
import torch

from paper_2608_07001_amd import gracekv as gk
from synth.workloads import CONFIGS, make_case

import gpu_harness as H

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_json_line_on_the_small_workload():
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--config", "tiny", "--steps", "2",
                          "--warmup", "1", "--cpu-budget-s", "1", "--no-decode"],
                         cwd=ROOT, capture_output=True, text=True, timeout=240)
    assert out.returncode == 0, out.stderr[-2000:]
    r = json.loads(out.stdout.strip().splitlines()[-1])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
              "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline", "stages_ms", "multi_hop"):
        assert k in r, k
    assert r["n_gpus"] == 1 and r["steps"] == 2 and r["warmup"] == 1 and r["value"] > 0
    ro = r["roofline"]
    assert ro["bound"] == "hbm" and ro["unit"] == "GB/s" and ro["peak"] == 8000.0
    assert abs(ro["frac"] - ro["achieved"] / ro["peak"]) < 1e-9
    assert 0 < ro["ms_per_launch"] < r["ms_per_step"] and ro["copy_gbs"] > 0
    ks = r["kernels"]
    assert ro["kernel"] == max((v for k, v in ks.items() if k != "segment"), key=lambda v: v["ms"])["kernel"]
    for k in ("segment", "root", "root_split", "pack"):
        assert ks[k]["ms"] > 0 and ks[k]["bytes"] > 0, k
    cb = r["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0
    st = r["stages_ms"]
    assert abs(sum(st[k] for k in ("segment", "build", "score", "select", "pack")) - r["ms_per_step"]) < 0.05 * r["ms_per_step"]
    assert r["multi_hop"]["ms_per_step"] > 0
    fl = r["alpha_floor"]
    assert fl["ms_per_step"] > 0 and 0 < fl["B_floor"] <= fl["cap"] and fl["floor_candidates_ms"] > 0


def test_stage_clock_leaves_the_output_unchanged():
    case = H.to_dev(make_case(CONFIGS["tiny"], 4, with_hidden=True))
    gk.stage_times()
    g0 = H.gpu_run(case, prune=True)
    assert all(n == 0 for _, n in gk.stage_times().values())       # off: nothing recorded
    g1 = H.gpu_run(case, prune=True, flags=gk.FLAG_STAGE_TIMES)
    t = gk.stage_times()
    for k in ("tok_R", "offsets", "K_out", "V_out", "pos_out", "logm_out"):
        assert torch.equal(g0[k], g1[k]), k
    assert g0["b_used"] == g1["b_used"]
    for s in ("segment", "rowstats", "root", "root_split", "refine", "pack"):
        assert t[s][1] == 1 and t[s][0] > 0, (s, t[s])
    assert t["token_relevance"][1] == 0                                  # fp32: relevance inside the root pass
    assert all(n == 0 for _, n in gk.stage_times().values())           # read once
