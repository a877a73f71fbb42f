"""Randomized parity cases through the C ABI: each case draws, from its own seed, one to three
matrices of random shapes (multiples of 256 give or take 3, or any size up to 1300), the
parameter dtype, Nesterov momentum, the Newton-Schulz step count (1-5) and the Gram-space segment
length (1-3), and sometimes a few hot rows, then runs two steps of Algorithm "MeqMuon" with every
stage checked against the oracle (tests/gpu_support.check_matrix_step). The cases cover schedules,
shape groups and tile edges that the hand-picked tests do not combine.
"""
import numpy as np
import pytest
import torch

import workloads
from gpu_support import Run, check_matrix_step, log
from paper_2609_35701_amd import meq

pytestmark = pytest.mark.gpu
LR = 0.02
N_CASES = 24


def draw_case(case: int):
    rng = np.random.default_rng(20261202 + case)

    def dim():
        if rng.random() < 0.4:
            return int(256 * rng.integers(1, 6) + rng.integers(-3, 4))
        return int(rng.integers(1, 1301))

    shapes = [(max(1, dim()), max(1, dim())) for _ in range(int(rng.integers(1, 4)))]
    dtype = "bf16" if rng.random() < 0.7 else "f32"
    kw = dict(nesterov=int(rng.random() < 0.3), ns_gram_steps=int(rng.integers(1, 4)), ns_steps=int(rng.integers(1, 6)))
    hot = 0.05 if rng.random() < 0.3 else 0.0
    return shapes, dtype, kw, int(rng.integers(0, 10000)), hot


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_case(case):
    shapes, dtype, kw, seed, hot = draw_case(case)
    label = f"sweep case {case}: {shapes} {dtype} {kw} seed {seed} hot {hot}"
    log(f"[case] {label}")
    wl = workloads.custom(shapes, dtype, name=f"sweep-{case}", seed=seed, hot_row_frac=hot, hot_row_gain=10.0)
    run = Run(wl, range(len(shapes)), meq.default_hparams(**kw))
    for step in range(2):
        w_before = [run.params[k].detach().to("cpu", torch.float64).numpy() for k in range(len(shapes))]
        b_before = [run.upd.momenta[k].detach().to("cpu", torch.float64).numpy() for k in range(len(shapes))]
        grads = run.step(LR)
        stats = run.upd.stats()
        for k in range(len(shapes)):
            check_matrix_step(run, k, w_before[k], b_before[k], grads[k].astype(np.float64), LR, stats,
                              f"{label} step {step} matrix {k}")
