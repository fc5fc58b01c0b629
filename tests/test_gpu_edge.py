"""Degenerate inputs of the layer on the GPU vs the float64 oracle: fewer eligible
selection blocks than k* (-1 slots), clouds that are mostly padding (empty balls,
compression blocks and selection blocks), and a single real point (no eligible block at
all: the selection branch outputs zeros with LSE -inf). Forward outputs and gradients at
the bars of the regular tests."""
import numpy as np
import pytest

from parity import TOL, gpu_forward, oracle_params, valid_from_tree
from test_gpu_backward import run_case
from test_gpu_forward import _check_head
from workloads import Config, make_inputs

pytestmark = pytest.mark.gpu

CASES = {
    # 128 slots, balls of 64, selection blocks of 16: 4 eligible blocks for top-8
    "few_candidates": Config("few_cand", 1, 128, 128, 2, 64, "bf16", 64, 8, 8, 16, 8, 16, "uniform", "fwdbwd"),
    # 70 real points in 1024 slots per cloud: most balls and blocks hold no real token
    "sparse_cloud": Config("sparse", 2, 70, 1024, 2, 32, "bf16", 64, 8, 8, 16, 4, 8, "uniform", "fwdbwd"),
    # one real point: its own ball holds every block, so nothing is eligible for selection
    "single_point": Config("single", 1, 1, 64, 2, 32, "f32", 64, 4, 4, 16, 2, 8, "uniform", "fwdbwd"),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_degenerate_forward(name):
    cfg = CASES[name]
    print(f"degenerate forward {name}", flush=True)
    inp = make_inputs(cfg, seed=13, layout="ball", with_grad=False)
    valid = valid_from_tree(cfg, seed=13)
    g, _ = gpu_forward(cfg, inp, valid)
    P = oracle_params(cfg)
    for b in range(cfg.batch):
        for h in range(cfg.heads):
            _check_head(cfg, inp, valid, g, b, h, P, TOL[cfg.dtype])
    if name == "few_candidates":
        assert np.all(g["sel"][..., 4:] == -1) and np.all(g["sel"][..., :4] >= 0)
    if name == "single_point":
        assert np.all(g["sel"] == -1)
        assert np.all(np.isneginf(g["lse"][2]))


@pytest.mark.parametrize("name", sorted(CASES))
def test_degenerate_backward(name):
    print(f"degenerate backward {name}", flush=True)
    run_case(CASES[name], seed=13)
