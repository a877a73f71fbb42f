"""The seeded input generator: determinism, shapes, storage exactness, imbalance structure."""
import numpy as np
import torch

import workloads


def test_shapes_of_named_workloads():
    counts = {"single-256x512": 1, "llama-130m": 84, "llama-350m": 168, "llama-1b": 112,
              "llama-7b-block-x4": 28}
    for name, n in counts.items():
        assert workloads.workload(name).count == n
    wl = workloads.workload("llama-1b")
    shapes = {(m.rows, m.cols) for m in wl.matrices}
    assert shapes == {(2048, 2048), (512, 2048), (8192, 2048), (2048, 8192)}
    assert wl.elements == 973_078_528


def test_deterministic_and_independent_streams():
    wl = workloads.workload("single-256x512")
    g0 = workloads.grad_at_step(wl, 0, 0)
    np.testing.assert_array_equal(g0, workloads.grad_at_step(wl, 0, 0))
    assert not np.array_equal(g0, workloads.grad_at_step(wl, 0, 1))
    np.testing.assert_array_equal(workloads.weight_init(wl, 0), workloads.weight_init(wl, 0))


def test_storage_values_are_exact_in_bf16():
    wl = workloads.custom([(64, 96)], "bf16")
    g = workloads.grad_at_step(wl, 0, 0)
    t = torch.from_numpy(g)
    assert torch.equal(t.to(torch.bfloat16).to(torch.float32), t)


def test_row_and_column_imbalance_present():
    wl = workloads.workload("single-256x512")
    g = workloads.grad_at_step(wl, 0, 0).astype(np.float64)
    r = np.sqrt((g * g).mean(1))
    c = np.sqrt((g * g).mean(0))
    assert r.std() / r.mean() > 0.5 and c.std() / c.mean() > 0.5
    wl4 = workloads.custom([(400, 64)], sigma=2.0, hot_row_frac=0.01, hot_row_gain=100.0)
    g4 = workloads.grad_at_step(wl4, 0, 0).astype(np.float64)
    assert np.isfinite(g4).all()
