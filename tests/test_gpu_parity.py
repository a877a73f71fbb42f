"""GPU parity of the HIP path against the fp64 oracle (through the C ABI).

Each case prints its name and shapes before the first launch.  Tolerances are
stated in ``gpu_support``: 1e-5 relative Frobenius for fp32 stages, 3e-2 for the
bf16 Newton-Schulz output and the final parameter delta, bf16 weights within
one ulp of the rounded oracle value (>= 99.9% exact), directions equal except
within a stated CV tie band.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_support import (DEV, TOL_DELTA, TOL_NS, Run, check_matrix_step, log, oracle_hp, relerr, schedule_of,
                         to_dev, to_np)
from paper_2609_35701_amd import meq

pytestmark = pytest.mark.gpu
LR = 0.02


def run_and_check(wl, idxs, steps=1, hp=None, lr=LR, label=""):
    log(f"[case] {label or wl.name}: matrices {[(wl.matrices[i].rows, wl.matrices[i].cols) for i in idxs]} "
        f"steps={steps}")
    run = Run(wl, idxs, hp)
    results = []
    for s in range(steps):
        w_before = [to_np(p) for p in run.params]
        b_before = [to_np(b) for b in run.upd.momenta]
        grads = run.step(lr)
        stats = run.upd.stats()
        for k in range(len(idxs)):
            results.append(check_matrix_step(run, k, w_before[k], b_before[k], grads[k].astype(np.float64), lr,
                                             stats, f"{label or wl.name} step {s} matrix {idxs[k]}"))
    log(f"[case] {label or wl.name}: max NS err {max(r['ns'] for r in results):.4g}, "
        f"max delta err {max(r['delta'] for r in results):.4g}, ties {sum(r['tie'] for r in results)}")
    return run, results


def test_single_matrix_256x512_fp32():
    run_and_check(workloads.workload("single-256x512"), [0], label="single-256x512")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_one_ns_step_keeps_x0(dtype):
    """With K = 1 the bf16 V buffer survives: V within one bf16 ulp of the rounded oracle V,
    and one Newton-Schulz step on exactly that X_0 matches the oracle."""
    wl = workloads.custom([(200, 72), (72, 200), (256, 512)], dtype, name=f"one-step-{dtype}")
    run_and_check(wl, [0, 1, 2], steps=2, hp=meq.default_hparams(ns_steps=1), label=wl.name)


@pytest.mark.parametrize("steps,gram", [(5, 1), (5, 2), (4, 3), (3, 3), (7, 3), (2, 3), (1, 3)])
def test_newton_schulz_schedules(steps, gram):
    """Schedules other than the default 3 + 2 (eq. "ns" as printed; 2 + 2 + 1, 3 + 1, one
    segment of 3, 3 + 3 + 1, one segment of 2 and a single step) against the printed iteration in
    fp64; X_0 is checked bit for bit when a schedule has one segment."""
    wl = workloads.custom([(256, 768), (1376, 512), (300, 100), (512, 512)], "bf16", name=f"sched-{steps}-{gram}")
    hp = meq.default_hparams(ns_steps=steps, ns_gram_steps=gram)
    run, _ = run_and_check(wl, range(4), steps=2, hp=hp, label=f"schedule K={steps} g={gram}")
    segs = [run.upd.plan.schedule(g) for g in range(len(run.upd.plan.groups()))]
    log(f"[case] schedules {segs}")
    assert all(sum(sg) == steps for sg in segs)


@pytest.mark.parametrize("coeffs", [(2.0, -0.5, 0.0), (1.5, -0.5, 0.0)])
def test_other_ns_coefficients(coeffs):
    """Coefficients other than the paper's: the cubic step (bounded, fp16 Gram-space segments) and
    one that grows singular values past the fp16 range check (every matrix through the printed
    iteration in bf16), against the oracle's iteration with the same coefficients."""
    a, b, c = coeffs
    wl = workloads.custom([(256, 768), (1376, 512), (512, 512)], "bf16", name=f"coeffs-{a}-{b}-{c}")
    hp = meq.default_hparams(ns_a=a, ns_b=b, ns_c=c)
    run, _ = run_and_check(wl, range(3), steps=2, hp=hp, label=f"coefficients {coeffs}")
    log(f"[case] schedules {[run.upd.plan.schedule(g) for g in range(len(run.upd.plan.groups()))]}")


def test_llama130m_subset_ten_steps():
    wl = workloads.workload("llama-130m")
    # q, k, v, o, gate, up, down of layer 0 and the down projection of the last layer
    run, res = run_and_check(wl, [0, 1, 2, 3, 4, 5, 6, 83], steps=10, label="llama-130m 10 steps")
    assert len(res) == 80


@pytest.mark.parametrize("shape", [(192, 576), (1376, 512), (2736, 1024), (320, 960), (128, 896), (7, 5),
                                   (1, 300), (300, 1), (65, 257), (513, 100)])
def test_odd_shapes(shape):
    wl = workloads.custom([shape], "bf16", name=f"odd-{shape[0]}x{shape[1]}")
    run_and_check(wl, [0], steps=2, label=wl.name)


def test_odd_shapes_fp32_and_mixed_groups():
    wl = workloads.custom([(96, 40), (40, 96), (256, 256), (33, 700), (700, 33)], "f32", name="mixed-f32")
    run_and_check(wl, range(5), steps=2, label=wl.name)


def test_nesterov_flag():
    wl = workloads.custom([(256, 768), (768, 256)], "bf16", name="nesterov")
    run_and_check(wl, [0, 1], steps=3, hp=meq.default_hparams(nesterov=1), label="nesterov")


def test_nesterov_fp32_cancelling_entries():
    """fp32 gradients with Nesterov, where G + mu B cancels almost exactly at a few entries of the
    second step: the bf16 V still matches V formed from the GPU's own momentum within one ulp."""
    wl = workloads.custom([(253, 2559)], "f32", seed=9107, name="nesterov-f32-cancel")
    run_and_check(wl, [0], steps=2, hp=meq.default_hparams(nesterov=1, ns_gram_steps=1, ns_steps=1),
                  label=wl.name)


def test_extreme_imbalance_block():
    wl = workloads.custom([(512, 1376), (1376, 512)], "bf16", sigma=2.0, hot_row_frac=0.01, hot_row_gain=100.0,
                          name="extreme")
    run_and_check(wl, [0, 1], steps=2, label="extreme imbalance")


def test_zero_gradient_is_pure_decay():
    log("[case] zero gradient")
    wl = workloads.custom([(96, 200), (200, 96)], "f32", name="zero")
    run = Run(wl, [0, 1])
    w0 = [to_np(p) for p in run.params]
    run.step(LR, [np.zeros((96, 200), np.float32), np.zeros((200, 96), np.float32)])
    hp = oracle_hp(run.hp)
    decay = np.float32(1.0 - np.float64(np.float32(LR)) * np.float64(hp.weight_decay))
    for k in range(2):
        np.testing.assert_array_equal(to_np(run.params[k]), (np.float32(w0[k]) * decay).astype(np.float64))
        assert not torch.any(run.upd.view(k, meq.BUF_U).float() != 0)
    gr, gc, d = run.upd.stats()
    assert gr == [0.0, 0.0] and gc == [0.0, 0.0] and d == [0, 0]


@pytest.mark.parametrize("shape", [(256, 256), (128, 512), (512, 128)])
def test_signed_permutation_closed_form(shape):
    """G = alpha Q with Q a signed (partial) permutation: every quantity stays exact in bf16, so
    U~ = sqrt(n) Q and W' = (1 - lr lambda) W - rho lr sqrt(n) Q for any NS coefficients."""
    log(f"[case] signed permutation {shape}")
    m, n = shape
    rng = np.random.default_rng(5)
    q = np.zeros(shape, np.float32)
    k = min(m, n)
    rows = rng.permutation(m)[:k]
    cols = rng.permutation(n)[:k]
    q[rows, cols] = rng.choice([-1.0, 1.0], k)
    wl = workloads.custom([shape], "f32", name="perm")
    run = Run(wl, [0])
    w0 = to_np(run.params[0])
    run.step(LR, [np.float32(0.25) * q])
    gr, gc, d = run.upd.stats()
    # both CVs vanish (up to the rounding of a mean of equal values): a tie, where rows and
    # columns are both correct choices; U~ = sqrt(n) Q for rows, sqrt(m) Q for columns
    assert max(gr[0], gc[0]) < 1e-12
    hp = oracle_hp(run.hp)
    scale = np.sqrt(n) if d[0] == oracle.ROW else np.sqrt(m)
    want = oracle.write_back(w0, scale * q.astype(np.float64), LR, hp.rho, hp.weight_decay)
    assert relerr(to_np(run.params[0]) - w0, want - w0) <= 1e-5


def test_zero_rows_and_columns_stay_zero():
    log("[case] zero rows/cols")
    wl = workloads.custom([(160, 416)], "f32", name="zrows")
    g = workloads.grad_at_step(wl, 0, 0)
    g[[3, 77]] = 0
    g[:, 100:130] = 0
    run = Run(wl, [0])
    w0 = to_np(run.params[0])
    run.step(LR, [g])
    u = to_np(run.upd.view(0, meq.BUF_U))
    assert not np.any(u[[3, 77]]) and not np.any(u[:, 100:130])
    hp = oracle_hp(run.hp)
    decay = np.float32(1.0 - np.float64(np.float32(LR)) * np.float64(hp.weight_decay))
    decayed = (np.float32(w0) * decay).astype(np.float64)
    w1 = to_np(run.params[0])
    # zero rows/columns of U are zero in either direction's U~, so only decay reaches them
    np.testing.assert_array_equal(w1[[3, 77]], decayed[[3, 77]])
    np.testing.assert_array_equal(w1[:, 100:130], decayed[:, 100:130])


def test_bitwise_determinism():
    log("[case] determinism")
    wl = workloads.custom([(512, 1536), (1536, 512), (768, 768)], "bf16", name="det")
    outs = []
    for _ in range(2):
        run = Run(wl, [0, 1, 2])
        run.step(LR)
        run.step(LR)
        outs.append([p.clone() for p in run.params] + [b.clone() for b in run.upd.momenta])
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def test_checkpoint_resume_equivalence():
    """k + j steps == k steps, save momentum and weights, restore into a fresh plan, j steps."""
    log("[case] resume")
    wl = workloads.custom([(256, 640), (640, 256)], "bf16", name="resume")
    full = Run(wl, [0, 1])
    for _ in range(3):
        full.step(LR)
    part = Run(wl, [0, 1])
    part.step(LR)
    saved_w = [p.clone() for p in part.params]
    saved_b = [b.clone() for b in part.upd.momenta]
    resumed = Run(wl, [0, 1])
    for k in range(2):
        resumed.params[k].copy_(saved_w[k])
        resumed.upd.momenta[k].copy_(saved_b[k])
    resumed.step_no = 1
    resumed.step(LR)
    resumed.step(LR)
    for a, b in zip(full.params + full.upd.momenta, resumed.params + resumed.upd.momenta):
        assert torch.equal(a, b)


def test_timing_events_report_every_kernel():
    log("[case] timing")
    wl = workloads.custom([(512, 2048), (2048, 512)], "bf16", name="timing")
    run = Run(wl, [0, 1])
    hidden_kinds = list(range(8))
    run.upd.plan.set_timing(hidden_kinds)
    run.step(LR)
    segs = run.upd.plan.schedule(0)
    assert segs == [3, 2]
    for kind in hidden_kinds:
        ms, n = run.upd.plan.get_timing(kind)
        if kind == meq.K_ROWCOL:
            # the step's row/column sums come from the last X product's epilogue
            assert n == 0, "rowcol"
            continue
        assert n >= 1 and ms > 0, meq.KERNEL_NAMES[kind]
    ms, n = run.upd.plan.get_timing(meq.K_APPLY)
    assert n == len(segs)  # one X product per segment for the single shape group
    ms, n = run.upd.plan.get_timing(meq.K_POLY)
    assert n == 5
    ms, n = run.upd.plan.get_timing(meq.K_GRAM, reset=True)
    # X X^T once per segment; P A and P T at every step but a segment's last, P Q at every step
    # but a segment's first (sharing its launch with P A where both run)
    assert n == len(segs) + 5 + 3
    assert run.upd.plan.get_timing(meq.K_APPLY) == (0.0, 0)
    # the row/column sums kernel of its own still runs in the CV trace (no apply before X_0)
    run.upd.plan.set_timing([meq.K_ROWCOL])
    meq.ns_cv_trace(run.upd, [p.clone() for p in run.params], 1)
    ms, n = run.upd.plan.get_timing(meq.K_ROWCOL, reset=True)
    assert n >= 2 and ms > 0


@pytest.mark.parametrize("name", ["llama-130m", "llama-350m", "llama-1b", "llama-7b-block-x4"])
def test_full_launch_sampled_parity(name):
    """A full-size workload in one meq_step (the 1B one is the benchmark's launch
    configuration; the 7B block carries the extreme row/column imbalance); the first, middle and
    last matrix of each shape group are seeded from the numpy generator and checked against the
    oracle, the rest carry device-drawn inputs of the same recipe."""
    wl = workloads.workload(name)
    shapes = [(m.rows, m.cols) for m in wl.matrices]
    groups = {}
    for i, s in enumerate(shapes):
        groups.setdefault((min(s), max(s)), []).append(i)
    sample = sorted({g[0] for g in groups.values()} | {g[len(g) // 2] for g in groups.values()} |
                    {g[-1] for g in groups.values()})
    log(f"[case] {name} full launch, sampled matrices {sample}")
    params, grads, _ = workloads.device_inputs(wl, DEV)
    w_np, g_np = {}, {}
    for i in sample:
        w_np[i] = workloads.weight_init(wl, i)
        g_np[i] = workloads.grad_at_step(wl, i, 0)
        params[i].copy_(to_dev(w_np[i], "bf16"))
        grads[i].copy_(to_dev(g_np[i], "bf16"))
    upd = meq.HiddenWeightUpdate(params)
    upd.step(grads, LR)
    torch.cuda.synchronize()
    gr, gc, d = upd.stats()
    hp = oracle_hp(upd.plan.hparams)
    for i in sample:
        log(f"[case]   oracle on matrix {i} {shapes[i]}")
        w0 = w_np[i].astype(np.float64)
        full = oracle.meq_step(w0, g_np[i].astype(np.float64), np.zeros_like(w0), hp, LR, wide=True)
        if d[i] != full["dir"]:
            assert abs(full["gamma_r"] - full["gamma_c"]) <= 0.05 * max(full["gamma_r"], full["gamma_c"])
            full = oracle.meq_step(w0, g_np[i].astype(np.float64), np.zeros_like(w0), hp, LR, force_dir=d[i],
                                   wide=True)
        u = to_np(upd.view(i, meq.BUF_U))
        u = u.T if shapes[i][0] > shapes[i][1] else u
        e_ns, e_dw = relerr(u, full["U"]), relerr(to_np(params[i]) - w0, full["W"] - w0)
        log(f"[case]   matrix {i} {shapes[i]} schedule {schedule_of(upd.plan, shapes[i])}: NS error {e_ns:.4g}, "
            f"delta error {e_dw:.4g}")
        assert e_ns <= TOL_NS
        assert e_dw <= TOL_DELTA
    # properties at full size for every matrix: finite weights, CVs non-negative, momentum == grad (first step)
    for i in range(wl.count):
        assert torch.isfinite(params[i].float()).all()
        assert gr[i] >= 0 and gc[i] >= 0
    assert torch.equal(upd.momenta[5], grads[5].float())


@pytest.mark.parametrize("shape", [(16384, 49152), (30000, 10000)])
def test_largest_shapes_properties(shape):
    """Shapes far beyond the workloads (the wide one at the 2^31-byte buffer limit's scale, the
    tall one ragged on both sides), checked through properties that hold at any size, since the
    fp64 oracle cannot run there: after one step from zero momentum B = G exactly; W stays finite;
    the balance condition (every nonzero row of U~ has RMS 1 for the row direction, every
    nonzero column for the column direction) holds for the applied update
    (W' - (1 - lr lambda) W) / (-rho lr) up to the rounding of W'; U's largest singular value and
    mean squared singular value lie in the band the quintic maps normalized singular values to."""
    m, n = shape
    log(f"[case] largest shapes {shape}")
    wl = workloads.custom([shape], "bf16", name=f"large-{m}x{n}")
    params, grads, _ = workloads.device_inputs(wl, DEV)
    w0 = params[0].clone()
    upd = meq.HiddenWeightUpdate(params)
    log(f"[case]   schedule {upd.plan.schedule(0)}, workspace {upd.plan.workspace_bytes / 2**30:.2f} GiB")
    upd.step(grads, LR)
    torch.cuda.synchronize()
    gr, gc, d = upd.stats()
    assert torch.equal(upd.momenta[0], grads[0].float())
    w1 = params[0].float()
    assert torch.isfinite(w1).all()
    hp = oracle_hp(upd.plan.hparams)
    decay = float(np.float32(1.0 - np.float64(np.float32(LR)) * np.float64(hp.weight_decay)))
    step = float(np.float32(np.float64(hp.rho) * np.float64(np.float32(LR))))
    ut = (w1.double() - decay * w0.double()) / (-step)  # U~ plus the rounding of W'
    dim = 1 if d[0] == meq.MEQ_DIR_ROW else 0
    rms = ut.pow(2).mean(dim=dim).sqrt()
    nz = rms > 0.5
    log(f"[case]   direction {d[0]}, CVs {gr[0]:.4f} / {gc[0]:.4f}, nonzero lines {int(nz.sum())} of {rms.numel()}, "
        f"RMS range {float(rms[nz].min()):.5f} .. {float(rms[nz].max()):.5f}")
    assert int(nz.sum()) == rms.numel()
    assert float((rms[nz] - 1.0).abs().max()) < 1e-2
    # singular values of U (wide orientation, bf16 buffer): power iteration in fp32 for the largest
    u = upd.view(0, meq.BUF_U).float()
    v = torch.randn(u.shape[1], 1, device=DEV, generator=torch.Generator(device=DEV).manual_seed(3))
    for _ in range(30):
        v = u.T @ (u @ v)
        v = v / v.norm()
    smax = float((u @ v).norm())
    msq = float(u.pow(2).sum() / u.shape[0])
    log(f"[case]   U: largest singular value {smax:.4f}, mean squared singular value {msq:.4f}")
    assert 0.68 <= smax <= 1.21
    assert 0.4 <= msq <= 1.45
