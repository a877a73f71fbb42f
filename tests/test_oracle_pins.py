"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these re-types the oracle's formulas: each checks it against an
independent fact (a closed form, an SVD, an invariance, brute force on tiny
inputs, or a number the paper prints), chosen so that a dropped term, a wrong
sign or index, or a transposed operand in the oracle fails at least one.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import COL, ROW, HParams

HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "paper_tables.json")))
HP = HParams()
A, B, C = HP.ns_a, HP.ns_b, HP.ns_c


def phi(x, a=A, b=B, c=C):
    """The scalar quintic a x + b x^3 + c x^5 that eq. 'ns' applies to each singular value."""
    return a * x + b * x ** 3 + c * x ** 5


def phi_k(x, k, **kw):
    for _ in range(k):
        x = phi(x, **kw)
    return x


def rng(seed):
    return np.random.default_rng(seed)


def cv_brute(v):
    """Population CV by explicit loops (definition of eq. 'cv')."""
    v = [float(t) for t in v]
    n = len(v)
    mean = 0.0
    for t in v:
        mean += t
    mean /= n
    var = 0.0
    for t in v:
        var += (t - mean) * (t - mean)
    return math.sqrt(var / n) / mean


# ---------------------------------------------------------------- golden numbers
def test_golden_hyperparameters_match_defaults():
    g = GOLD["hyperparameters"]
    assert (HP.mu, HP.ns_steps, HP.ns_a, HP.ns_b, HP.ns_c, HP.rho, HP.weight_decay, HP.delta) == (
        g["mu"], g["ns_steps"], g["ns_a"], g["ns_b"], g["ns_c"], g["rho"], g["weight_decay"], g["delta"])


def test_golden_state_is_one_fp32_value_per_parameter():
    """P12: the paper's MeqMuon memory equals 4 bytes x parameters (fp32 momentum, one per element)."""
    for row in GOLD["optimizer_state_memory_mib"]["models"]:
        mib = row["params_m"] * 1e6 * 4 / 2 ** 20
        assert abs(mib - row["meqmuon_mib"]) < 0.011, row


def test_golden_llama130m_hidden_shapes_reproduce_muon_memory():
    """The 84 hidden matrices of the llama-130m workload reproduce the Muon/NorMuon memory figures."""
    import workloads

    wl = workloads.workload("llama-130m")
    n_h = wl.elements
    r_h = sum(m.rows for m in wl.matrices)
    g = GOLD["llama130m_hidden_elements"]
    n_a = g["params_m"] * 1e6 - n_h
    assert n_h == 84_934_656 and wl.count == 84
    assert abs((n_h + 2 * n_a) * 4 / 2 ** 20 - g["muon_mib"]) < 0.011
    assert abs((n_h + 2 * n_a + r_h) * 4 / 2 ** 20 - g["normuon_mib"]) < 0.011


def test_golden_cv_hand_example():
    g = GOLD["cv_hand_example"]
    assert oracle.coeff_of_variation(np.array(g["values"]), 1e-7) == pytest.approx(g["cv"], abs=1e-15)


# --------------------------------------------------------------------- momentum
def test_P1_momentum_closed_form():
    r = rng(1)
    gs = [r.standard_normal((7, 5)) for _ in range(9)]
    b = np.zeros((7, 5))
    for k, g in enumerate(gs):
        b = oracle.momentum(b, g, HP.mu)
        closed = sum(HP.mu ** (k - i) * gs[i] for i in range(k + 1))
        np.testing.assert_allclose(b, closed, rtol=1e-13, atol=1e-13)


def test_P1_nesterov_closed_form():
    r = rng(2)
    gs = [r.standard_normal((4, 6)) for _ in range(5)]
    b = np.zeros((4, 6))
    for k, g in enumerate(gs):
        b = oracle.momentum(b, g, HP.mu)
        v = oracle.ns_input(b, g, HP.mu, True)
        closed = gs[k] + HP.mu * sum(HP.mu ** (k - i) * gs[i] for i in range(k + 1))
        np.testing.assert_allclose(v, closed, rtol=1e-13, atol=1e-13)
        np.testing.assert_array_equal(oracle.ns_input(b, g, HP.mu, False), b)


# --------------------------------------------------------------- Newton-Schulz
@pytest.mark.parametrize("shape", [(5, 8), (9, 4), (6, 6), (1, 7), (7, 1)])
def test_P2_ns_is_spectral_polynomial(shape):
    """With H = P S Q^T, K steps of eq. 'ns' give P phi^K(S / ||S||_2) Q^T (numpy SVD as the pin)."""
    h = rng(3).standard_normal(shape)
    u = oracle.newton_schulz(h, A, B, C, 5)
    p, s, qt = np.linalg.svd(h, full_matrices=False)
    expect = (p * phi_k(s / np.linalg.norm(s), 5)) @ qt
    np.testing.assert_allclose(u, expect, rtol=0, atol=1e-13)


def test_P2_band_and_polar_distance():
    """Normalized singular values >= 1.51e-3 land in [0.6818, 1.2024] after 5 steps; ||U - PQ^T||_2 <= 0.32."""
    xs = np.concatenate([np.geomspace(1.51e-3, 1.0, 20001), np.linspace(1.51e-3, 1.0, 20001)])
    ys = phi_k(xs, 5)
    assert ys.min() >= 0.6818 and ys.max() <= 1.2025
    r = rng(4)
    for shape in [(12, 20), (20, 12), (16, 16)]:
        p, _ = np.linalg.qr(r.standard_normal((shape[0], min(shape))))
        q, _ = np.linalg.qr(r.standard_normal((shape[1], min(shape))))
        sig = np.geomspace(1.0, 0.05, min(shape))
        h = (p * sig) @ q.T
        u = oracle.newton_schulz(h, A, B, C, 5)
        sv = np.linalg.svd(u, compute_uv=False)
        assert sv.min() >= 0.6818 and sv.max() <= 1.2025
        assert np.linalg.norm(u - p @ q.T, 2) <= 0.32


def test_P2_zero_input_gives_zero():
    assert not np.any(oracle.newton_schulz(np.zeros((3, 4)), A, B, C, 5))


def test_P3_transpose_equivariance_and_wide_form():
    r = rng(5)
    for shape in [(11, 4), (4, 11), (8, 8)]:
        h = r.standard_normal(shape)
        np.testing.assert_allclose(oracle.newton_schulz(h.T, A, B, C, 5),
                                   oracle.newton_schulz(h, A, B, C, 5).T, atol=1e-13)
        np.testing.assert_allclose(oracle.newton_schulz(h, A, B, C, 5, wide=True),
                                   oracle.newton_schulz(h, A, B, C, 5), atol=1e-13)


def test_P10_convergent_ns_gives_one_sided_balance():
    """With a convergent quintic (15/8, -10/8, 3/8) NS reaches Orth: tall => gamma_c = 0 -> rows; wide => cols."""
    r = rng(6)
    a, b, c = 15 / 8, -10 / 8, 3 / 8
    for shape, want in [((24, 8), ROW), ((8, 24), COL)]:
        p, _ = np.linalg.qr(r.standard_normal((shape[0], 8)))
        q, _ = np.linalg.qr(r.standard_normal((shape[1], 8)))
        h = (p * np.linspace(1.0, 0.5, 8)) @ q.T
        u = oracle.newton_schulz(h, a, b, c, 40)
        np.testing.assert_allclose(u, p @ q.T, atol=1e-10)
        _, gr, gc, d = oracle.equilibrate(u, 1e-7)
        assert d == want
        assert (gc if want == ROW else gr) < 1e-10
        assert (gr if want == ROW else gc) > 1e-2


# ------------------------------------------------------------- statistics / CV
def test_P11_cv_matches_brute_force_and_threshold():
    r = rng(7)
    v = r.lognormal(0, 1, 37)
    assert oracle.coeff_of_variation(v, 1e-7) == pytest.approx(cv_brute(v), rel=1e-13)
    # entries at or below delta are excluded (strict >), zero CV for <= 1 surviving entry
    assert oracle.coeff_of_variation(np.array([1e-7, 1.0, 2.0, 0.0]), 1e-7) == pytest.approx(1 / 3)
    assert oracle.coeff_of_variation(np.array([1e-7, 0.0]), 1e-7) == 0.0
    assert oracle.coeff_of_variation(np.array([0.0, 3.0]), 1e-7) == 0.0
    # dimensionless: invariant to uniform scaling
    assert oracle.coeff_of_variation(5 * v, 1e-7) == pytest.approx(oracle.coeff_of_variation(v, 1e-7), rel=1e-13)


def test_row_col_rms_brute_force():
    x = rng(8).standard_normal((3, 5))
    r, c = oracle.row_col_rms(x)
    for i in range(3):
        assert r[i] == pytest.approx(math.sqrt(sum(x[i, j] ** 2 for j in range(5)) / 5), rel=1e-14)
    for j in range(5):
        assert c[j] == pytest.approx(math.sqrt(sum(x[i, j] ** 2 for i in range(3)) / 3), rel=1e-14)


def test_P6_balance_condition():
    """After row (column) selection every nonzero row (column) has RMS 1; ||U~||_F^2 = m_+ n (n_+ m)."""
    r = rng(9)
    for shape in [(16, 40), (40, 16), (24, 24)]:
        g = r.standard_normal(shape) * r.lognormal(0, 1, (shape[0], 1)) * r.lognormal(0, 1, (1, shape[1]))
        g[3] = 0.0
        u = oracle.newton_schulz(g, A, B, C, 5)
        for d in (ROW, COL):
            ut, _, _, _ = oracle.equilibrate(u, 1e-7, force_dir=d)
            rr, cc = oracle.row_col_rms(ut)
            side = rr if d == ROW else cc
            nz = side > 1e-7
            np.testing.assert_allclose(side[nz], 1.0, atol=1e-12)
            other = shape[1] if d == ROW else shape[0]
            assert np.sum(ut * ut) == pytest.approx(nz.sum() * other, rel=1e-12)
            assert oracle.coeff_of_variation(side, 1e-7) < 1e-12
        assert not np.any(oracle.equilibrate(u, 1e-7)[0][3])  # zero row stays zero


def test_P7_rank_one_closed_form():
    r = rng(10)
    m, n = 9, 14
    uu = r.standard_normal(m) * r.lognormal(0, 1, m)
    vv = r.standard_normal(n) * r.lognormal(0, 0.3, n)
    g = np.outer(uu, vv)
    u = oracle.newton_schulz(g, A, B, C, 5)
    np.testing.assert_allclose(u, phi_k(1.0, 5) * np.outer(uu / np.linalg.norm(uu), vv / np.linalg.norm(vv)),
                               atol=1e-14)
    ut, gr, gc, d = oracle.equilibrate(u, 1e-7)
    assert gr == pytest.approx(cv_brute(np.abs(uu)), rel=1e-12)
    assert gc == pytest.approx(cv_brute(np.abs(vv)), rel=1e-12)
    assert d == ROW  # CV(|u|) > CV(|v|) by construction of the spreads
    np.testing.assert_allclose(ut, np.outer(np.sign(uu), vv * math.sqrt(n) / np.linalg.norm(vv)), atol=1e-12)
    # swap the roles: now the column spread dominates
    ut2, gr2, gc2, d2 = oracle.equilibrate(u.T, 1e-7)
    assert d2 == COL
    np.testing.assert_allclose(ut2, np.outer(vv * math.sqrt(n) / np.linalg.norm(vv), np.sign(uu)), atol=1e-12)
    # write-back from zero weights is exactly -rho * lr * U~
    lr = 0.02
    w = oracle.write_back(np.zeros((m, n)), ut, lr, HP.rho, HP.weight_decay)
    np.testing.assert_allclose(w, -HP.rho * lr * np.outer(np.sign(uu), vv * math.sqrt(n) / np.linalg.norm(vv)),
                               atol=1e-14)


def test_P8_orthogonal_input():
    r = rng(11)
    q, _ = np.linalg.qr(r.standard_normal((12, 12)))
    perm = np.eye(12)[r.permutation(12)] * r.choice([-1.0, 1.0], 12)[:, None]
    for mat in (q, perm):
        u = oracle.newton_schulz(3.7 * mat, A, B, C, 5)
        for d in (None, ROW, COL):
            ut, gr, gc, dd = oracle.equilibrate(u, 1e-7, force_dir=d)
            np.testing.assert_allclose(ut, math.sqrt(12) * mat, atol=1e-12)
    # an exact tie (identical row and column RMS values) selects rows: eq. 'hidden' uses >=
    perm4 = np.array([[0, 2.0, 0, 0], [0, 0, 0, -2.0], [2.0, 0, 0, 0], [0, 0, -2.0, 0]])
    ut, gr, gc, d = oracle.equilibrate(perm4, 1e-7)
    assert gr == gc == 0.0 and d == ROW
    ut, gr, gc, d = oracle.equilibrate(np.array([[1.0, 2.0], [2.0, 1.0]]), 1e-7)
    assert gr == gc and d == ROW


def test_P4_permutation_and_sign_equivariance():
    r = rng(12)
    m, n = 10, 17
    g = r.standard_normal((m, n)) * r.lognormal(0, 1, (m, 1))
    w = r.standard_normal((m, n)) * 0.02
    p1 = np.eye(m)[r.permutation(m)] * r.choice([-1.0, 1.0], m)[:, None]
    p2 = (np.eye(n)[r.permutation(n)] * r.choice([-1.0, 1.0], n)[:, None]).T
    out = oracle.meq_step(w, g, np.zeros((m, n)), HP, 0.02)
    out2 = oracle.meq_step(p1 @ w @ p2, p1 @ g @ p2, np.zeros((m, n)), HP, 0.02)
    np.testing.assert_allclose(out2["W"], p1 @ out["W"] @ p2, atol=1e-14)
    assert out2["gamma_r"] == pytest.approx(out["gamma_r"], rel=1e-10)
    assert out2["gamma_c"] == pytest.approx(out["gamma_c"], rel=1e-10)
    assert out2["dir"] == out["dir"]


def test_P5_scale_invariance():
    r = rng(13)
    g = r.standard_normal((8, 13)) * r.lognormal(0, 1, (1, 13))
    base = oracle.meq_step(np.zeros((8, 13)), g, np.zeros((8, 13)), HP, 0.02)["Ut"]
    for alpha, sign in [(1e-3, 1), (250.0, 1), (-0.7, -1)]:
        ut = oracle.meq_step(np.zeros((8, 13)), alpha * g, np.zeros((8, 13)), HP, 0.02)["Ut"]
        np.testing.assert_allclose(ut, sign * base, atol=1e-11)


def test_P9_zero_gradient_and_zero_rows():
    r = rng(14)
    w = r.standard_normal((6, 9))
    out = oracle.meq_step(w, np.zeros((6, 9)), np.zeros((6, 9)), HP, 0.02)
    np.testing.assert_allclose(out["W"] - w, -0.02 * HP.weight_decay * w, rtol=1e-12, atol=0)
    assert not np.any(out["Ut"])
    assert out["dir"] == ROW and out["gamma_r"] == 0.0 and out["gamma_c"] == 0.0
    g = r.standard_normal((6, 9))
    g[[1, 4]] = 0.0
    g[:, 7] = 0.0
    out = oracle.meq_step(w, g, np.zeros((6, 9)), HP, 0.02)
    assert not np.any(out["U"][[1, 4]]) and not np.any(out["U"][:, 7])
    assert not np.any(out["Ut"][[1, 4]]) and not np.any(out["Ut"][:, 7])
    r_, c_ = oracle.row_col_rms(out["U"])
    assert out["gamma_r"] == pytest.approx(cv_brute(r_[[0, 2, 3, 5]]), rel=1e-12)
    assert out["gamma_c"] == pytest.approx(cv_brute(np.delete(c_, 7)), rel=1e-12)


def test_P11_brute_force_tiny():
    g = np.array([[0.3, -1.2, 2.0, -0.05]])
    out = oracle.meq_step(np.zeros((1, 4)), g, np.zeros((1, 4)), HP, 0.02)
    np.testing.assert_allclose(out["U"], phi_k(1.0, 5) * g / np.linalg.norm(g), atol=1e-15)
    assert out["dir"] == COL and out["gamma_r"] == 0.0
    np.testing.assert_allclose(out["Ut"], np.sign(g), atol=1e-14)
    d = np.diag([3.0, 4.0])
    np.testing.assert_allclose(oracle.newton_schulz(d, A, B, C, 5),
                               np.diag([phi_k(0.6, 5), phi_k(0.8, 5)]), atol=1e-15)


def test_write_back_decay_and_step():
    w = np.array([[1.0, -2.0]])
    ut = np.array([[0.5, 3.0]])
    out = oracle.write_back(w, ut, 0.5, 0.2, 0.1)
    np.testing.assert_allclose(out, [[0.95 * 1.0 - 0.1 * 0.5, 0.95 * -2.0 - 0.1 * 3.0]], atol=1e-15)


# ------------------------------------------------------------------- bf16 rounding
def test_round_bf16_against_torch_and_ties():
    r = rng(15)
    x = np.concatenate([r.standard_normal(20000) * 10.0 ** r.integers(-30, 30, 20000),
                        r.standard_normal(1000) * 1e-39]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.round_bf16(x.astype(np.float64)), ref)
    one = 1.0
    assert oracle.round_bf16(np.array([one + 2 ** -8]))[0] == 1.0            # tie -> even
    assert oracle.round_bf16(np.array([one + 3 * 2 ** -8]))[0] == 1.0 + 2 ** -6
    assert oracle.round_bf16(np.array([one + 2 ** -8 + 2 ** -30]))[0] == 1.0 + 2 ** -7
    assert oracle.round_bf16(np.array([-(one + 2 ** -8)]))[0] == -1.0


def _gram_space_ns(h, a, b, c, segs):
    """The Gram-space regrouping of eq. "ns" (reading R21), written out in fp64 for this test
    only: per segment A = X X^T, then for each step P = a I + b A + c A A, A <- P (P A) and
    Q <- P Q, and finally X <- Q X."""
    x = np.asarray(h, np.float64) / np.linalg.norm(h)
    eye = np.eye(x.shape[0])
    for seg in segs:
        am = x @ x.T
        q = eye
        for j in range(seg):
            p = a * eye + b * am + c * (am @ am)
            q = p @ q
            if j + 1 < seg:
                am = p @ (p @ am)
        x = q @ x
    return x


@pytest.mark.parametrize("segs", [[1] * 5, [2, 2, 1], [3, 2], [2, 3], [5], [4, 1]])
@pytest.mark.parametrize("shape", [(24, 96), (40, 40), (7, 300)])
def test_R21_gram_space_regrouping_is_exact(shape, segs):
    """Every segmentation of the five steps equals the printed iteration up to fp64 rounding:
    the factors of a segment are polynomials of its first Gram matrix, so they commute and
    X_{k+1} X_{k+1}^T = P_k A_k P_k.  A wrong update (A <- P A instead of P (P A), or Q
    accumulated as Q P with a non-commuting factor) breaks it on the wide shapes."""
    g = rng(31).standard_normal(shape) * np.exp(rng(32).standard_normal((shape[0], 1)))
    want = oracle.newton_schulz(g, A, B, C, 5)
    got = _gram_space_ns(g, A, B, C, segs)
    assert np.linalg.norm(got - want) <= 1e-10 * np.linalg.norm(want)


def test_R21_planted_mistakes_fail():
    g = rng(33).standard_normal((24, 96)) * np.exp(rng(34).standard_normal((24, 1)))
    want = oracle.newton_schulz(g, A, B, C, 5)

    def wrong_update(h, segs):  # A <- P A: one factor of P missing
        x = h / np.linalg.norm(h)
        eye = np.eye(x.shape[0])
        for seg in segs:
            am, q = x @ x.T, eye
            for j in range(seg):
                p = A * eye + B * am + C * (am @ am)
                q = p @ q
                if j + 1 < seg:
                    am = p @ am
            x = q @ x
        return x

    assert np.linalg.norm(wrong_update(g, [3, 2]) - want) > 1e-2 * np.linalg.norm(want)
    assert np.linalg.norm(_gram_space_ns(g, A, B, C, [3, 2]) - want) <= 1e-10 * np.linalg.norm(want)
