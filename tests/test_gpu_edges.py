"""GPU edge cases the oracle defines, through the C ABI:

- the delta band of eqs. "cv" and "operators": rows or columns whose RMS lies strictly between 0
  and delta count as zero (left out of the CV, scale 0) while those just above delta do not, for
  hidden weights (row and column directions) and for the two-sided normalization of eq. "aux";
- non-finite gradients (the paper is silent): a NaN or Inf in one matrix's gradient poisons that
  matrix only -- its momentum entry and all of its weights become non-finite, as the iteration
  mixes every entry -- while the other matrices of the same launches match the oracle;
- the full 84-matrix 130M-shape plan over 10 steps of Algorithm "MeqMuon", with the first, middle and
  last matrix of each shape group checked against the oracle at every step;
- the Gram-space schedule on hard spectra (rank 8 plus noise, a geometric spectrum) of segmented
  shapes: finite, and no further from the printed iteration's fp64 result than the printed bf16
  iteration itself (plus 0.01; tests/test_ns_emulation.py pins the same margin on the CPU);
- invariance to the gradient's scale: the iteration starts from V / ||V||_F (eq. "ns"), so
  gradients multiplied by 2^k give bitwise the same weights, both schedules, both dtypes.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_support import (DEV, TOL_FP32, TOL_NS, Run, check_matrix_step, log, oracle_hp, relerr, to_dev, to_np,
                         ulp_bf16)
from paper_2609_35701_amd import meq

pytestmark = pytest.mark.gpu
LR = 0.02


def _band_grad(shape, dtype, seed, lines, axis):
    """A gradient with row (axis 0) or column (axis 1) imbalance, the given lines scaled by their factor."""
    rng = np.random.default_rng(seed)
    m, n = shape
    imb = rng.lognormal(0, 1.0, (m, 1)) if axis == 0 else rng.lognormal(0, 1.0, (1, n))
    g = rng.standard_normal((m, n)) * imb * 1e-3
    for i, f in lines.items():
        if axis == 0:
            g[i] *= f
        else:
            g[:, i] *= f
    return workloads.to_storage(g, dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("axis", [0, 1])
def test_delta_band_hidden(dtype, axis):
    """Tall 416 x 160 (row direction) with small rows, wide 160 x 416 (column direction) with small
    columns: U's RMS of the lines scaled by 1e-6 lies in (0, delta] (about 1e-8 to 5e-8 in the fp64
    oracle), of the one scaled by 1e-5 above it (7 to 25 delta)."""
    shape = (416, 160) if axis == 0 else (160, 416)
    lines = {5: 1e-6, 200 if axis == 0 else 100: 1e-6, 77: 1e-5}
    log(f"[case] delta band hidden {shape} {dtype} lines {lines}")
    wl = workloads.custom([shape], dtype, name="band", seed=13)
    g = _band_grad(shape, dtype, 21 + axis, lines, axis)
    run = Run(wl, [0])
    w0 = to_np(run.params[0])
    b0 = np.zeros(shape)
    run.step(LR, [g])
    stats = run.upd.stats()
    res = check_matrix_step(run, 0, w0, b0, g.astype(np.float64), LR, stats, f"band {shape} {dtype}")
    hp = oracle_hp(run.hp)
    assert res["dir"] == axis, f"expected the {'row' if axis == 0 else 'column'} direction"
    rms = to_np(run.upd.view(0, meq.BUF_ROW_RMS if axis == 0 else meq.BUF_COL_RMS))
    sc = to_np(run.upd.view(0, meq.BUF_SCALE))
    small = [i for i, f in lines.items() if f == 1e-6]
    for i in small:
        assert 0 < rms[i] <= hp.delta, f"line {i}: RMS {rms[i]} not inside (0, delta]"
        assert sc[i] == 0, f"line {i}: scale {sc[i]} for an RMS at or below delta"
    assert rms[77] > hp.delta and sc[77] == np.float32(1.0 / rms[77]), "line 77 just above delta"
    # the CVs leave the band's lines out: the oracle's CV of the GPU's U with them excluded
    u = to_np(run.upd.view(0, meq.BUF_U))
    u = u.T if shape[0] > shape[1] else u
    r, c = oracle.row_col_rms(u)
    keep = np.ones(len(r if axis == 0 else c), bool)
    keep[small] = False
    want = oracle.coeff_of_variation((r if axis == 0 else c)[keep], 0.0)
    got = stats[0][0] if axis == 0 else stats[1][0]
    assert abs(got - want) <= TOL_FP32 * want


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_delta_band_aux(dtype):
    """Two-sided normalization: rows of V with RMS in (0, delta] get row scale 0; columns of N_r(V)
    with RMS in (0, delta] get column scale 0; lines just above delta keep their scales."""
    shape = (300, 256)
    log(f"[case] delta band aux {shape} {dtype}")
    hp = meq.default_hparams()
    ohp = oracle_hp(hp)
    rng = np.random.default_rng(31)
    g = rng.standard_normal(shape) * 1e-3
    g[[4, 150]] *= 5e-5    # row RMS about 5e-8
    g[9] *= 5e-4           # row RMS about 5e-7, just above
    g[:, 30] *= 2e-8       # column RMS of N_r(V) about 2e-8
    g[:, 31] *= 3e-7       # about 3e-7, just above
    g = workloads.to_storage(g, dtype).astype(np.float64)
    wl = workloads.custom([shape], dtype, seed=33)
    w = workloads.weight_init(wl, 0).astype(np.float64)
    param = to_dev(w, dtype)
    upd = meq.AuxUpdate([param], hp)
    upd.step([to_dev(g, dtype)], LR)
    torch.cuda.synchronize()
    lr32 = float(np.float32(LR))
    out = oracle.aux_step(w, g, np.zeros(shape), ohp, lr32)
    r_gpu = to_np(upd.view(0, meq.BUF_ROW_RMS))
    c_gpu = to_np(upd.view(0, meq.BUF_COL_RMS))
    assert relerr(r_gpu, out["r"]) <= TOL_FP32 and relerr(c_gpu, out["c"]) <= TOL_FP32
    for i in (4, 150):
        assert 0 < r_gpu[i] <= ohp.delta and 0 < out["r"][i] <= ohp.delta
    assert r_gpu[9] > ohp.delta
    assert 0 < c_gpu[30] <= ohp.delta and c_gpu[31] > ohp.delta
    # the written parameters: band lines receive decay only, the rest the oracle's update
    w_gpu = to_np(param)
    if dtype == "bf16":
        w_rne = oracle.round_bf16(out["W"])
        off = np.abs(w_gpu - w_rne)
        bound = ulp_bf16(w_rne) + 2.0 ** -21 * (np.abs(w) + ohp.rho * lr32 * np.abs(out["Ut"]))
        assert np.all(off <= bound)
    else:
        assert relerr(w_gpu - w, out["W"] - w) <= TOL_FP32
    assert not np.any(out["Ut"][[4, 150]]) and not np.any(out["Ut"][:, 30])
    decay = np.float32(1.0 - np.float64(np.float32(LR)) * np.float64(ohp.weight_decay))
    decayed = (np.float32(w) * decay).astype(np.float64)
    if dtype == "bf16":
        decayed = oracle.round_bf16(decayed)
    np.testing.assert_array_equal(w_gpu[[4, 150]], decayed[[4, 150]])
    np.testing.assert_array_equal(w_gpu[:, 30], decayed[:, 30])


@pytest.mark.parametrize("bad", [float("nan"), float("inf")])
def test_nonfinite_gradient_stays_in_its_matrix(bad):
    shapes = [(256, 768), (768, 256), (256, 768), (300, 100)]
    log(f"[case] non-finite gradient {bad} in matrix 1 of {shapes}")
    wl = workloads.custom(shapes, "bf16", name="nonfinite", seed=61)
    run = Run(wl, range(len(shapes)))
    for step in range(2):
        w_before = [to_np(p) for p in run.params]
        b_before = [to_np(b) for b in run.upd.momenta]
        grads = run.grads(step)
        grads[1] = grads[1].copy()
        grads[1][17, 33] = bad
        run.step(LR, grads)
        stats = run.upd.stats()
        for k in (0, 2, 3):
            check_matrix_step(run, k, w_before[k], b_before[k], grads[k].astype(np.float64), LR, stats,
                              f"non-finite step {step} clean matrix {k}")
        b1 = to_np(run.upd.momenta[1])
        mask = np.ones(b1.shape, bool)
        mask[17, 33] = False
        assert not np.isfinite(b1[17, 33])
        if step == 0:
            assert np.all(np.isfinite(b1[mask]))
            np.testing.assert_array_equal(b1[mask], grads[1].astype(np.float64)[mask])
        assert not np.any(np.isfinite(to_np(run.params[1]))), "every weight of the poisoned matrix"


def test_llama130m_full_plan_ten_steps():
    wl = workloads.workload("llama-130m")
    groups = {}
    for i, m in enumerate(wl.matrices):
        groups.setdefault((min(m.rows, m.cols), max(m.rows, m.cols)), []).append(i)
    sample = sorted({g[0] for g in groups.values()} | {g[len(g) // 2] for g in groups.values()} |
                    {g[-1] for g in groups.values()})
    log(f"[case] llama-130m all {wl.count} matrices, 10 steps, checked {sample}")
    run = Run(wl, range(wl.count))
    worst = 0.0
    for step in range(10):
        w_before = {k: to_np(run.params[k]) for k in sample}
        b_before = {k: to_np(run.upd.momenta[k]) for k in sample}
        grads = run.step(LR)
        stats = run.upd.stats()
        for k in sample:
            res = check_matrix_step(run, k, w_before[k], b_before[k], grads[k].astype(np.float64), LR, stats,
                                    f"llama-130m step {step} matrix {k}")
            worst = max(worst, res["delta"])
        assert all(torch.isfinite(p.float()).all() for p in run.params)
        log(f"[case]   step {step}: worst delta error so far {worst:.4g}")


@pytest.mark.parametrize("shape", [(256, 768), (512, 2048)])
def test_segmented_schedule_on_hard_spectra(shape):
    s, l = shape
    rng = np.random.default_rng(11)
    cases = {"rank 8 + noise": rng.standard_normal((s, 8)) @ rng.standard_normal((8, l))
             + 1e-3 * rng.standard_normal((s, l))}
    qa, _ = np.linalg.qr(rng.standard_normal((s, s)))
    qb, _ = np.linalg.qr(rng.standard_normal((l, s)))
    cases["geometric spectrum"] = qa @ np.diag(np.geomspace(1.0, 1e-4, s)) @ qb.T
    for what, v in cases.items():
        g = workloads.to_storage(v * 1e-3, "f32").astype(np.float64)
        log(f"[case] segmented schedule {shape} {what}")
        x0 = oracle.round_bf16(g)
        hpo = oracle_hp(meq.default_hparams())
        ref = oracle.newton_schulz(x0, hpo.ns_a, hpo.ns_b, hpo.ns_c, hpo.ns_steps)
        errs = {}
        for gram in (3, 1):
            hp = meq.default_hparams(ns_gram_steps=gram)
            upd = meq.HiddenWeightUpdate([torch.zeros(shape, dtype=torch.float32, device=DEV)], hp)
            assert len(upd.plan.schedule(0)) == (2 if gram == 3 else 5)
            upd.step([to_dev(g, "f32")], LR)
            torch.cuda.synchronize()
            u = to_np(upd.view(0, meq.BUF_U))
            assert np.all(np.isfinite(u))
            errs[gram] = relerr(u, ref)
        log(f"[case]   NS error: Gram-space schedule {errs[3]:.4g}, printed iteration {errs[1]:.4g}")
        assert errs[3] <= errs[1] + 0.01


class _Plan:
    """The attributes of a Run that check_matrix_step reads, for a plan built by hand."""

    def __init__(self, wl, params, upd, hp):
        self.wl, self.params, self.upd, self.hp = wl, params, upd, hp


@pytest.mark.parametrize("dtype,nesterov", [("f32", 0), ("bf16", 0), ("bf16", 1)])
def test_update_is_invariant_to_gradient_scale(dtype, nesterov):
    """Five copies of one matrix in one plan, with gradients multiplied by 2^-24 .. 2^24: every
    kernel step scales exactly by a power of two while its values stay in fp32's normal range (the
    bf16 rounding of V, the fp32 tile sums of squares, 1/||V||^2 and 1/||V|| from a correctly
    rounded square root, the folded prescale), so the weights, U and the statistics are bitwise
    those of the unscaled copy, which is checked against the oracle; the momenta scale exactly."""
    exps = [-24, -12, 0, 12, 24]
    ref = exps.index(0)
    hp = meq.default_hparams(nesterov=nesterov)
    for shape in [(384, 1000), (700, 700)]:  # Gram-space segments (L >= 2S after padding) and printed steps
        log(f"[case] gradient scale 2^{exps} {shape} {dtype} nesterov {nesterov}")
        wl = workloads.custom([shape], dtype, seed=71, name="scale")
        w0 = workloads.weight_init(wl, 0)
        params = [to_dev(w0, dtype) for _ in exps]
        upd = meq.HiddenWeightUpdate(params, hp)
        plan = _Plan(wl, params, upd, hp)
        for step in range(2):
            g = workloads.grad_at_step(wl, 0, step)
            w_before = to_np(params[ref])
            b_before = to_np(upd.momenta[ref])
            upd.step([to_dev(g * np.float32(2.0 ** k), dtype) for k in exps], LR)
            torch.cuda.synchronize()
            stats = upd.stats()
            check_matrix_step(plan, ref, w_before, b_before, g.astype(np.float64), LR, stats,
                              f"scale {shape} {dtype} step {step}")
            for i, k in enumerate(exps):
                assert torch.equal(params[i], params[ref]), f"{shape} 2^{k} step {step}: weights differ"
                assert torch.equal(upd.view(i, meq.BUF_U), upd.view(ref, meq.BUF_U)), f"2^{k}: U differs"
                assert torch.equal(upd.momenta[i], upd.momenta[ref] * 2.0 ** k), f"2^{k}: momentum"
                assert (stats[0][i], stats[1][i], stats[2][i]) == (stats[0][ref], stats[1][ref], stats[2][ref])
