"""Plans side by side on one stream, and the learning-rate edge: the C ABI keeps every plan's
state in its own workspace and momenta, and lr = 0 leaves the parameters untouched
(eq. "meqmuon-update" with eta = 0 applies neither the decay nor the step)."""
import numpy as np
import pytest
import torch

import workloads

from gpu_support import Run, log, oracle_hp, to_dev, to_np

pytestmark = pytest.mark.gpu


def test_zero_learning_rate_leaves_parameters_and_advances_momentum():
    log("[case] lr = 0")
    for dtype in ("f32", "bf16"):
        wl = workloads.custom([(200, 96), (96, 640)], dtype, name=f"lr0-{dtype}", seed=31)
        run = Run(wl, [0, 1])
        w0 = [p.clone() for p in run.params]
        for _ in range(2):
            grads = run.step(0.0)
        for k in range(2):
            assert torch.equal(run.params[k], w0[k]), f"{dtype}: parameter {k} changed with lr = 0"
        # momentum after two steps: mu G_0 + G_1 in fp32 (one fused multiply-add: within half an
        # fp32 ulp of the exact value, which float64 holds here up to its own rounding)
        hp = oracle_hp(run.hp)
        for k in range(2):
            g0 = workloads.grad_at_step(wl, k, 0).astype(np.float32)
            g1 = grads[k].astype(np.float32)
            if dtype == "bf16":
                g0 = to_np(to_dev(g0, "bf16"))
                g1 = to_np(to_dev(g1, "bf16"))
            want = hp.mu * g0.astype(np.float64) + g1.astype(np.float64)
            np.testing.assert_allclose(to_np(run.upd.momenta[k]), want, rtol=6.1e-8, atol=0)


def test_two_plans_interleaved_on_one_stream_match_sequential_runs():
    log("[case] two plans interleaved")
    wl_a = workloads.custom([(256, 1024), (300, 100)], "bf16", name="plan-a", seed=41)
    wl_b = workloads.custom([(512, 512), (1024, 256), (7, 5)], "bf16", name="plan-b", seed=42)

    def fresh():
        return Run(wl_a, [0, 1]), Run(wl_b, [0, 1, 2])

    grads = {name: [[to_dev(workloads.grad_at_step(wl, i, s), "bf16") for i in range(wl.count)]
                    for s in range(3)] for name, wl in (("a", wl_a), ("b", wl_b))}
    # one plan after the other, synchronized
    ra, rb = fresh()
    for s in range(3):
        ra.upd.step(grads["a"][s], 0.02)
    torch.cuda.synchronize()
    for s in range(3):
        rb.upd.step(grads["b"][s], 0.02)
    torch.cuda.synchronize()
    # interleaved step by step on the same stream, no synchronization in between
    ia, ib = fresh()
    for s in range(3):
        ia.upd.step(grads["a"][s], 0.02)
        ib.upd.step(grads["b"][s], 0.02)
    torch.cuda.synchronize()
    for x, y in ((ra, ia), (rb, ib)):
        for k in range(len(x.params)):
            assert torch.equal(x.params[k], y.params[k])
            assert torch.equal(x.upd.momenta[k], y.upd.momenta[k])
        assert x.upd.stats() == y.upd.stats()


def test_capped_plan_matches_the_uncapped_plan_bitwise():
    """A workspace-capped plan runs its matrices in several passes that reuse one Newton-Schulz
    region; every matrix's arithmetic is the same, so parameters, momenta and statistics match the
    uncapped plan bit for bit over several steps (mixed shapes, tall and wide, fp32 and bf16)."""
    from paper_2609_35701_amd import meq

    for dtype, shapes, cap in (("bf16", [(m.rows, m.cols) for m in workloads.workload("llama-130m").matrices[:14]],
                                32 << 20),
                               ("f32", [(300, 100), (1024, 256), (256, 1024), (96, 640), (7, 5), (512, 512)],
                                4 << 20)):
        wl = workloads.custom(shapes, dtype, name=f"capped-{dtype}", seed=57)
        log(f"[case] capped plan {dtype} {len(shapes)} matrices cap {cap >> 20} MiB")
        w0 = [to_dev(workloads.weight_init(wl, i), dtype) for i in range(wl.count)]
        ref = meq.HiddenWeightUpdate([w.clone() for w in w0])
        cap_upd = meq.HiddenWeightUpdate([w.clone() for w in w0], max_workspace_bytes=cap)
        assert cap_upd.plan.passes >= 3 and cap_upd.plan.workspace_bytes <= cap
        assert ref.plan.passes == 1
        for s in range(3):
            g = [to_dev(workloads.grad_at_step(wl, i, s), dtype) for i in range(wl.count)]
            ref.step(g, 0.02)
            cap_upd.step(g, 0.02)
        torch.cuda.synchronize()
        for k in range(wl.count):
            assert torch.equal(ref.params[k], cap_upd.params[k]), f"{dtype}: parameter {k}"
            assert torch.equal(ref.momenta[k], cap_upd.momenta[k]), f"{dtype}: momentum {k}"
        assert ref.stats() == cap_upd.stats()


def test_capped_1b_plan_at_full_size_matches_uncapped_and_static_step():
    """The 1B-shape step (112 matrices) capped to the static scratch size runs in 30 passes; with a
    caller workspace and through meq_step_static it matches the uncapped step bit for bit."""
    from paper_2609_35701_amd import meq

    wl = workloads.workload("llama-1b")
    log(f"[case] llama-1b capped to {meq.MEQ_STATIC_SCRATCH_BYTES >> 20} MiB against uncapped")
    params, grads, _ = workloads.device_inputs(wl, "cuda:0")
    ref = meq.HiddenWeightUpdate([p.clone() for p in params])
    cap = meq.HiddenWeightUpdate([p.clone() for p in params], max_workspace_bytes=meq.MEQ_STATIC_SCRATCH_BYTES)
    assert cap.plan.passes >= 20 and cap.plan.workspace_bytes <= meq.MEQ_STATIC_SCRATCH_BYTES
    static_plan = meq.Plan([tuple(p.shape) for p in params], "bf16", max_workspace_bytes=meq.MEQ_STATIC_SCRATCH_BYTES)
    sp = [p.clone() for p in params]
    sb = [torch.zeros(p.shape, dtype=torch.float32, device=p.device) for p in params]
    for _ in range(2):
        ref.step(grads, 0.02)
        cap.step(grads, 0.02)
        static_plan.step_static_ptrs([p.data_ptr() for p in sp], [g.data_ptr() for g in grads],
                                     [b.data_ptr() for b in sb], 0.02, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    for k in range(wl.count):
        assert torch.equal(ref.params[k], cap.params[k]) and torch.equal(ref.params[k], sp[k]), f"parameter {k}"
        assert torch.equal(ref.momenta[k], cap.momenta[k]) and torch.equal(ref.momenta[k], sb[k]), f"momentum {k}"
    assert ref.stats() == cap.stats()
