"""Host-side logic of bench.py (no GPU): the FLOP count the step roofline uses
and the refusal of more than one GPU."""
import os
import subprocess
import sys

import pytest

import synthetic

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("name,tflop", [("small", 14.0), ("xl", 69.4), ("6.7b", 170.0), ("13b", 162.9)])
def test_step_flops_match_the_configuration_table(name, tflop):
    # algorithmic FLOPs per step (C = 1) of the GPT-3 configurations, as
    # tabulated from their shapes: 6 per linear-layer parameter per token
    # (blocks and untied head) plus the causal half of attention
    assert round(bench.step_flops(synthetic.CONFIGS[name]) / 1e12, 1) == tflop


def test_step_flops_scale_with_micro_batches():
    cfg = synthetic.CONFIGS["xl"]
    assert bench.step_flops(cfg.with_(accum=4)) == 4 * bench.step_flops(cfg)


def test_more_than_one_gpu_is_refused_before_any_gpu_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""
