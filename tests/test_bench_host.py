"""Host-side checks of the benchmark's work figures (no GPU): the multiply-add count behind every
roofline fraction, and the one-GPU refusal of the command line."""
import math
import os
import subprocess
import sys

import pytest

import bench
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (l, r, s) of every generation workload the benchmark runs
SHAPES = sorted({(w.n_layers, w.r, w.s) for w in synth.WORKLOADS.values()})


@pytest.mark.parametrize("L,r,s", SHAPES)
def test_macs_follow_the_papers_performance_model(L, r, s):
    """Appendix "Performance model": per layer the two dilated-convolution halves cost
    2 x (2r . 2r) FLOPs and the residual product 2r . r, i.e. 10 r^2 of matrix-vector FLOPs; the
    skip sum over all layers (l . 2r) . s; the head 2s . a and 2a . a.  Those product terms are
    twice the multiply-adds the benchmark counts when the last layer's residual product is kept."""
    a = synth.A_CLASSES
    paper_matvec_flops = L * 10 * r * r + (L * 2 * r) * s + 2 * s * a + 2 * a * a
    assert 2 * bench.macs_per_sample(L, r, s, a, last_res=True) == paper_matvec_flops
    # the kernels skip the last layer's residual product (its x feeds no later layer)
    assert bench.macs_per_sample(L, r, s, a) == bench.macs_per_sample(L, r, s, a, last_res=True) - r * r


@pytest.mark.parametrize("L,r,s", SHAPES)
def test_macs_equal_the_weight_matrices_touched_per_sample(L, r, s):
    """Every weight matrix element (not the embedding tables, which are gathered, nor the biases)
    enters exactly one multiply-add per generated sample; counted from the parameter shapes the
    weights are built from."""
    a = synth.A_CLASSES
    shapes = synth.weight_shapes(L, r, s, a)
    matrices = ("w_prev", "w_cur", "w_res", "w_skip", "w_relu", "w_out")
    touched = sum(math.prod(shapes[k]) for k in matrices)
    assert bench.macs_per_sample(L, r, s, a, last_res=True) == touched


def test_spot_totals():
    """Spot values: l = 20, r = 64, s = 256 touches 868,352 weights per sample with every residual
    product (864,256 without the last one); l = 4, r = 16, s = 32 touches 80,896."""
    assert bench.macs_per_sample(20, 64, 256, last_res=True) == 868352
    assert bench.macs_per_sample(20, 64, 256) == 864256
    assert bench.macs_per_sample(4, 16, 32, last_res=True) == 80896


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout == ""
