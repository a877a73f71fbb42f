"""Pins of the oracle's other parameter kinds (eqs. "aux", "vector", "moonlight-update").

As for the hidden-weight pins, each test checks the oracle against an independent
fact: a hand-worked example, a closed form, brute force, an invariance or an SVD.
The order of the two-sided normalization (rows first, then columns) is pinned by
facts that the reverse order violates.
"""
import math

import numpy as np
import pytest

import oracle
from oracle import HParams

HP = HParams()


def rng(seed):
    return np.random.default_rng(seed)


def rms_rows_cols_loops(x):
    """Row and column RMS by explicit loops (definition of eq. 'row-col-rms')."""
    m, n = len(x), len(x[0])
    r = []
    for i in range(m):
        s = 0.0
        for j in range(n):
            s += float(x[i][j]) ** 2
        r.append(math.sqrt(s / n))
    c = []
    for j in range(n):
        s = 0.0
        for i in range(m):
            s += float(x[i][j]) ** 2
        c.append(math.sqrt(s / m))
    return r, c


# ------------------------------------------------------------------------ eq. "aux"
def test_two_sided_hand_worked_2x2():
    # V = [[3, 4], [0, 1]]: row RMS 5/sqrt2 and 1/sqrt2; N_r(V) = [[3 sqrt2/5, 4 sqrt2/5], [0, sqrt2]];
    # its column RMS 3/5 and sqrt41/5; so U~ = [[sqrt2, 4 sqrt2/sqrt41], [0, 5 sqrt2/sqrt41]].
    v = np.array([[3.0, 4.0], [0.0, 1.0]])
    ut, r, c = oracle.two_sided(v, HP.delta)
    s2, s41 = math.sqrt(2.0), math.sqrt(41.0)
    np.testing.assert_allclose(r, [5 / s2, 1 / s2], rtol=1e-15)
    np.testing.assert_allclose(c, [3 / 5, s41 / 5], rtol=1e-15)
    np.testing.assert_allclose(ut, [[s2, 4 * s2 / s41], [0.0, 5 * s2 / s41]], rtol=1e-15, atol=1e-16)


def test_two_sided_columns_exactly_unit_rows_not():
    # columns are normalized last, so every nonzero column has RMS 1; the rows keep the
    # imbalance the column step reintroduces (the reverse order would give unit rows)
    v = rng(1).standard_normal((40, 24)) * np.exp(rng(2).standard_normal((40, 1))) * np.exp(
        rng(3).standard_normal((1, 24)))
    ut, _, _ = oracle.two_sided(v, HP.delta)
    r, c = rms_rows_cols_loops(ut)
    np.testing.assert_allclose(c, 1.0, rtol=1e-13)
    assert max(abs(t - 1.0) for t in r) > 1e-3


def test_two_sided_rank1_closed_form():
    # V = u v^T with nonzero entries: both normalizations leave sign(u_i) sign(v_j)
    u = rng(4).standard_normal(13)
    w = rng(5).standard_normal(7)
    ut, _, _ = oracle.two_sided(np.outer(u, w), HP.delta)
    np.testing.assert_allclose(ut, np.outer(np.sign(u), np.sign(w)), rtol=1e-13)


def test_two_sided_invariances():
    v = rng(6).standard_normal((9, 11))
    ut, _, _ = oracle.two_sided(v, HP.delta)
    # positive scale
    np.testing.assert_allclose(oracle.two_sided(3.7e-4 * v, HP.delta)[0], ut, rtol=1e-12)
    # row and column sign flips and permutations carry through
    pr, pc = rng(7).permutation(9), rng(8).permutation(11)
    sr, sc = np.sign(rng(9).standard_normal(9)), np.sign(rng(10).standard_normal(11))
    vt = (sr[:, None] * v * sc[None, :])[pr][:, pc]
    expect = (sr[:, None] * ut * sc[None, :])[pr][:, pc]
    np.testing.assert_allclose(oracle.two_sided(vt, HP.delta)[0], expect, rtol=1e-12, atol=1e-15)


def test_two_sided_zero_rows_and_columns_stay_zero():
    v = rng(11).standard_normal((6, 5))
    v[2, :] = 0.0
    v[:, 3] = 0.0
    v[4, :] = 1e-9  # RMS <= delta: treated as a zero row
    ut, r, c = oracle.two_sided(v, HP.delta)
    assert np.all(ut[2] == 0) and np.all(ut[4] == 0) and np.all(ut[:, 3] == 0)
    assert r[4] <= HP.delta and c[3] == 0
    keep = [0, 1, 3, 5]
    _, cc = rms_rows_cols_loops(ut[keep])
    for j in (0, 1, 2, 4):  # remaining columns have unit RMS over all 6 rows
        assert abs(math.sqrt(sum(ut[i, j] ** 2 for i in range(6)) / 6) - 1.0) < 1e-13


def test_aux_step_write_back_and_momentum():
    hp = HParams()
    w = rng(12).standard_normal((8, 6))
    g1, g2 = rng(13).standard_normal((8, 6)), rng(14).standard_normal((8, 6))
    b1 = oracle.aux_step(w, g1, np.zeros_like(w), hp, 0.02)["B"]
    out = oracle.aux_step(w, g2, b1, hp, 0.02)
    np.testing.assert_allclose(out["B"], 0.95 * g1 + g2, rtol=1e-15)
    ut, _, _ = oracle.two_sided(0.95 * g1 + g2, hp.delta)
    np.testing.assert_allclose(out["W"], (1 - 0.02 * 0.1) * w - 0.2 * 0.02 * ut, rtol=1e-14)
    # Nesterov: the normalized matrix is G + mu B
    hn = HParams(nesterov=True)
    outn = oracle.aux_step(w, g2, b1, hn, 0.02)
    np.testing.assert_allclose(outn["V"], g2 + 0.95 * (0.95 * g1 + g2), rtol=1e-15)


# --------------------------------------------------------------------- eq. "vector"
def test_global_rms_hand_worked():
    np.testing.assert_allclose(oracle.global_rms_normalize(np.array([3.0, 4.0])),
                               [3 * math.sqrt(2) / 5, 4 * math.sqrt(2) / 5], rtol=1e-15)


def test_global_rms_unit_rms_and_direction():
    v = rng(15).standard_normal(1000) * 1e-5
    ut = oracle.global_rms_normalize(v)
    s = 0.0
    for t in ut:
        s += float(t) ** 2
    assert abs(math.sqrt(s / 1000) - 1.0) < 1e-13
    ratio = ut / v
    np.testing.assert_allclose(ratio, ratio[0], rtol=1e-13)
    assert ratio[0] > 0


def test_global_rms_special_cases():
    assert np.all(oracle.global_rms_normalize(np.zeros(17)) == 0)
    np.testing.assert_array_equal(oracle.global_rms_normalize(np.array([-2.5])), [-1.0])
    np.testing.assert_allclose(oracle.global_rms_normalize(np.full(9, 7.0)), np.ones(9), rtol=1e-15)


def test_vec_step_write_back():
    hp = HParams()
    w = rng(16).standard_normal(33)
    g = rng(17).standard_normal(33)
    bp = rng(18).standard_normal(33)
    out = oracle.vec_step(w, g, bp, hp, 0.01)
    b = 0.95 * bp + g
    np.testing.assert_allclose(out["B"], b, rtol=1e-15)
    ut = b * math.sqrt(33) / math.sqrt(float(np.sum(b * b)))
    np.testing.assert_allclose(out["W"], (1 - 0.01 * 0.1) * w - 0.2 * 0.01 * ut, rtol=1e-14)


# ---------------------------------------------------------- eq. "moonlight-update"
def phi(x, a=HP.ns_a, b=HP.ns_b, c=HP.ns_c):
    return a * x + b * x ** 3 + c * x ** 5


@pytest.mark.parametrize("shape", [(12, 20), (20, 12)])
def test_moonlight_spectral_closed_form(shape):
    m, n = shape
    hp = HParams()
    w = rng(19).standard_normal(shape)
    g = rng(20).standard_normal(shape)
    out = oracle.moonlight_step(w, g, np.zeros(shape), hp, 0.02)
    p, s, qt = np.linalg.svd(g, full_matrices=False)
    x = s / np.linalg.norm(s)
    for _ in range(hp.ns_steps):
        x = phi(x)
    u = (p * x) @ qt
    np.testing.assert_allclose(out["U"], u, atol=1e-12)
    np.testing.assert_allclose(out["W"], (1 - 0.02 * 0.1) * w - 0.02 * 0.2 * math.sqrt(max(m, n)) * u,
                               atol=1e-13)


def test_moonlight_update_rms_matches_rho_for_orthogonal_u():
    # with a convergent quintic U -> Orth(G), whose RMS is sqrt(min/(m n)); the sqrt(max)
    # factor then makes the update RMS exactly rho * eta regardless of shape
    hp = HParams(ns_a=15 / 8, ns_b=-10 / 8, ns_c=3 / 8, ns_steps=60, weight_decay=0.0)
    for shape in [(16, 48), (48, 16), (30, 30)]:
        g = rng(21).standard_normal(shape)
        w = np.zeros(shape)
        out = oracle.moonlight_step(w, g, np.zeros(shape), hp, 0.5)
        upd_rms = math.sqrt(float(np.mean(out["W"] ** 2)))
        assert abs(upd_rms - 0.2 * 0.5) < 1e-9


# ------------------------------------------------------------- NS CV trajectories
def test_ns_cv_trace_start_and_end_points():
    hp = HParams()
    v = rng(30).standard_normal((24, 40)) * np.exp(rng(31).standard_normal((24, 1)))
    gr, gc = oracle.ns_cv_trace(v, hp, 6)
    assert len(gr) == len(gc) == 7
    # k = 0 is the input itself (CVs are scale free): brute force
    rr, cc = rms_rows_cols_loops(v)
    for got, vals in ((gr[0], rr), (gc[0], cc)):
        mean = sum(vals) / len(vals)
        want = math.sqrt(sum((t - mean) ** 2 for t in vals) / len(vals)) / mean
        assert abs(got - want) < 1e-12
    # k = K is what the update equilibrates
    hp5 = HParams(ns_steps=5)
    out = oracle.meq_step(np.zeros_like(v), v, np.zeros_like(v), hp5, 0.0)
    assert abs(gr[5] - out["gamma_r"]) < 1e-12 and abs(gc[5] - out["gamma_c"]) < 1e-12


@pytest.mark.parametrize("shape,zero_side", [((20, 50), "rows"), ((50, 20), "cols"), ((30, 30), "both")])
def test_ns_cv_trace_orthogonality_constraints(shape, zero_side):
    # exact orthogonalization equalizes the short side's magnitudes (Y Y^T = I for m < n,
    # Y^T Y = I for m > n, both when square); a convergent quintic reaches it
    hp = HParams(ns_a=15 / 8, ns_b=-10 / 8, ns_c=3 / 8)
    v = rng(32).standard_normal(shape) * np.exp(rng(33).standard_normal((shape[0], 1)))
    gr, gc = oracle.ns_cv_trace(v, hp, 60)
    if zero_side in ("rows", "both"):
        assert gr[-1] < 1e-9
    if zero_side in ("cols", "both"):
        assert gc[-1] < 1e-9
    if zero_side == "rows":
        assert gc[-1] > 0.05
    if zero_side == "cols":
        assert gr[-1] > 0.05
