"""fp64 CPU oracle of the MeqMuon update (hidden 2D weights, remaining 2D parameters,
1-D parameters) and of the Moonlight-Muon update it is compared with.

TEST INFRASTRUCTURE ONLY.  This module is the plain, slow definition that the
HIP path is checked against.  Only the tests, the package's ``smoke()`` check
and the benchmark's CPU-baseline leg may import it; the product path never
does.  It shares no code with the HIP path: both sides only read inputs from
the ``workloads`` generator.

Everything is float64 numpy; matrix products use numpy's ``@``.  Each function
names the passage of the paper (arxiv 2609.35701, "MeqMuon") that it follows.

Readings where the paper is silent (all listed, with reasons, in the design notes):
* momentum is the heavy-ball form of eq. "momentum" (no (1 - mu) factor);
  the experiments' "Nesterov momentum" is offered as the flag ``nesterov``,
  taken as V = G + mu * B (not printed in the paper);
* X_0 = H / ||H||_F without an epsilon; a zero matrix gives U = 0 (the
  iteration is defined only for nonzero input, Section "Preliminaries");
* RMS values at or below delta count as zero both in the CVs (eq. "cv") and in
  the row/column operators (eq. "operators"), i.e. such a row gets scale 0;
* a CV over no nonzero entry is 0;
* the direction tie gamma_r == gamma_c selects rows (eq. "hidden" uses >=);
* remaining 2D parameters and 1-D parameters use the same momentum as the hidden
  weights (Algorithm "MeqMuon" has one momentum rule); ``nesterov`` applies to them
  only if set, since the paper states Nesterov momentum for the hidden weights only;
* decoupled weight decay applies to every parameter kind, as the algorithm's last
  line does;
* a zero 1-D momentum gives a zero update (the global RMS is then 0).

Parity pins: every function here is pinned by tests in ``tests/test_oracle_pins.py``
against closed forms, SVD, invariances and brute force; none is "parity unpinned".
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Optional

import numpy as np

ROW = 0
COL = 1


@dataclass(frozen=True)
class HParams:
    """Hyperparameters of the update.

    Defaults are the paper's experimental settings (Section "Experiments"):
    mu = 0.95, K = 5 Newton-Schulz steps with (a, b, c) = (3.4445, -4.7750, 2.0315),
    rho = 0.2, decoupled weight decay 0.1; delta = 1e-7 from Section
    "Imbalance patterns".  ``nesterov`` defaults to off, as in Algorithm "MeqMuon".
    """

    mu: float = 0.95
    rho: float = 0.2
    weight_decay: float = 0.1
    ns_steps: int = 5
    ns_a: float = 3.4445
    ns_b: float = -4.7750
    ns_c: float = 2.0315
    delta: float = 1e-7
    nesterov: bool = False

    def as_f32(self) -> "HParams":
        """The same values rounded to float32, as the C boundary stores them."""
        f = lambda v: float(np.float32(v))  # noqa: E731
        return HParams(f(self.mu), f(self.rho), f(self.weight_decay), int(self.ns_steps),
                       f(self.ns_a), f(self.ns_b), f(self.ns_c), f(self.delta), bool(self.nesterov))


# --------------------------------------------------------------------------- momentum
def momentum(b_prev: np.ndarray, g: np.ndarray, mu: float) -> np.ndarray:
    """B_t = mu * B_{t-1} + G_t  (eq. "momentum"; B_{-1} = 0)."""
    return mu * np.asarray(b_prev, np.float64) + np.asarray(g, np.float64)


def ns_input(b: np.ndarray, g: np.ndarray, mu: float, nesterov: bool) -> np.ndarray:
    """The matrix handed to orthogonalization.

    Algorithm "MeqMuon" orthogonalizes B_t itself.  With ``nesterov`` it uses the
    look-ahead G_t + mu * B_t instead (the experiments state Nesterov momentum with
    mu = 0.95 without printing its form).
    """
    b = np.asarray(b, np.float64)
    return np.asarray(g, np.float64) + mu * b if nesterov else b


# --------------------------------------------------------------------- Newton-Schulz
def frobenius(h: np.ndarray) -> float:
    """||H||_F = sqrt(sum of squared entries)."""
    h = np.asarray(h, np.float64)
    return math.sqrt(float(np.sum(h * h)))


def newton_schulz(h: np.ndarray, a: float, b: float, c: float, steps: int,
                  wide: bool = False) -> np.ndarray:
    """K quintic Newton-Schulz steps approximating Orth(H) (eq. "ns").

    X_0 = H / ||H||_F;  A_k = X_k X_k^T;  X_{k+1} = a X_k + (b A_k + c A_k A_k) X_k.
    A zero H returns zeros (the iteration is stated for nonzero inputs).

    ``wide=True`` runs the same iteration on H^T when H has more rows than
    columns and transposes the result back.  That is an exact identity,
    (X X^T)^j X = X (X^T X)^j, checked by the transpose-equivariance pin; it only
    makes the oracle cheaper on tall matrices.
    """
    h = np.asarray(h, np.float64)
    if wide and h.shape[0] > h.shape[1]:
        return newton_schulz(h.T, a, b, c, steps, wide=False).T
    nrm = frobenius(h)
    if nrm == 0.0:
        return np.zeros_like(h)
    x = h / nrm
    for _ in range(steps):
        am = x @ x.T
        x = a * x + (b * am + c * (am @ am)) @ x
    return x


# ------------------------------------------------------------- row / column statistics
def row_col_rms(x: np.ndarray):
    """r_i = ||X_{i,:}||_2 / sqrt(n),  c_j = ||X_{:,j}||_2 / sqrt(m)  (eq. "row-col-rms")."""
    x = np.asarray(x, np.float64)
    m, n = x.shape
    r = np.sqrt(np.sum(x * x, axis=1) / n)
    c = np.sqrt(np.sum(x * x, axis=0) / m)
    return r, c


def coeff_of_variation(v: np.ndarray, delta: float) -> float:
    """Population std / mean over the entries strictly above delta (eq. "cv").

    Entries at or below delta count as zero rows/columns and are excluded.
    With no such entry the CV is taken as 0.
    """
    v = np.asarray(v, np.float64)
    pos = v[v > delta]
    if pos.size == 0:
        return 0.0
    mean = float(np.sum(pos)) / pos.size
    var = float(np.sum((pos - mean) ** 2)) / pos.size
    return math.sqrt(var) / mean


def row_normalize(x: np.ndarray, delta: float) -> np.ndarray:
    """N_r(X) = diag(r^{-1}) X; rows with RMS <= delta are treated as zero (eq. "operators")."""
    x = np.asarray(x, np.float64)
    r, _ = row_col_rms(x)
    s = np.zeros_like(r)
    nz = r > delta
    s[nz] = 1.0 / r[nz]
    return x * s[:, None]


def col_normalize(x: np.ndarray, delta: float) -> np.ndarray:
    """N_c(X) = X diag(c^{-1}); columns with RMS <= delta are treated as zero (eq. "operators")."""
    x = np.asarray(x, np.float64)
    _, c = row_col_rms(x)
    s = np.zeros_like(c)
    nz = c > delta
    s[nz] = 1.0 / c[nz]
    return x * s[None, :]


def equilibrate(u: np.ndarray, delta: float, force_dir: Optional[int] = None):
    """Adaptive one-sided normalization of an orthogonalized update (eq. "hidden").

    Rows are normalized when gamma_r(U) >= gamma_c(U), columns otherwise.
    ``force_dir`` (ROW / COL) overrides the choice; tests use it where two
    directions are both correct within a stated CV tolerance.
    Returns (U_tilde, gamma_r, gamma_c, direction).
    """
    r, c = row_col_rms(u)
    gr = coeff_of_variation(r, delta)
    gc = coeff_of_variation(c, delta)
    d = (ROW if gr >= gc else COL) if force_dir is None else int(force_dir)
    ut = row_normalize(u, delta) if d == ROW else col_normalize(u, delta)
    return ut, gr, gc, d


# ------------------------------------------------------------------------ write-back
def write_back(w: np.ndarray, ut: np.ndarray, lr: float, rho: float, weight_decay: float) -> np.ndarray:
    """W_{t+1} = (1 - eta_t lambda) W_t - rho eta_t U_tilde_t  (eq. "meqmuon-update")."""
    w = np.asarray(w, np.float64)
    return (1.0 - lr * weight_decay) * w - (rho * lr) * np.asarray(ut, np.float64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (8 significant bits), ties to even.

    Written from the definition: x = m * 2**e with 0.5 <= |m| < 1; keep 8 bits
    of m with numpy's half-to-even rounding.  Values below bfloat16's normal
    range are rounded on the subnormal grid (spacing 2**-133).
    """
    x = np.asarray(x, np.float64)
    m, e = np.frexp(x)
    e = np.maximum(e, -125)           # bfloat16 min normal is 2**-126 = 0.5 * 2**-125
    q = np.round(np.ldexp(x, 8 - e))  # x scaled so that 8 significant bits sit above the point
    return np.ldexp(q, e - 8)


# -------------------------------------------------------------------------- full step
def meq_step(w: np.ndarray, g: np.ndarray, b_prev: np.ndarray, hp: HParams, lr: float,
             force_dir: Optional[int] = None, wide: bool = False) -> dict:
    """One MeqMuon step for one 2D hidden-layer weight (Algorithm "MeqMuon", hidden branch).

    momentum -> Orth by K Newton-Schulz steps -> adaptive one-sided normalization
    -> decoupled-weight-decay write-back.  ``w`` is returned in float64 (not rounded).
    """
    b = momentum(b_prev, g, hp.mu)
    v = ns_input(b, g, hp.mu, hp.nesterov)
    u = newton_schulz(v, hp.ns_a, hp.ns_b, hp.ns_c, hp.ns_steps, wide=wide)
    ut, gr, gc, d = equilibrate(u, hp.delta, force_dir)
    w_new = write_back(w, ut, lr, hp.rho, hp.weight_decay)
    return {"W": w_new, "B": b, "V": v, "normsq": frobenius(v) ** 2, "U": u, "Ut": ut,
            "gamma_r": gr, "gamma_c": gc, "dir": d}


# ------------------------------------------------- remaining 2D parameters (eq. "aux")
def two_sided(v: np.ndarray, delta: float):
    """U~ = N_c(N_r(V))  (eq. "aux").

    Rows of V are scaled to unit RMS first; the column RMS is then taken of that
    row-normalized matrix.  Rows or columns with RMS <= delta stay zero.
    Returns (U~, r of V, c of N_r(V)).
    """
    v = np.asarray(v, np.float64)
    r, _ = row_col_rms(v)
    vr = row_normalize(v, delta)
    _, c = row_col_rms(vr)
    return col_normalize(vr, delta), r, c


def aux_step(w: np.ndarray, g: np.ndarray, b_prev: np.ndarray, hp: HParams, lr: float) -> dict:
    """One MeqMuon step for a remaining 2D parameter such as a token embedding or an LM
    head (Algorithm "MeqMuon", second branch): momentum -> two-sided normalization of the
    momentum itself (no orthogonalization) -> decoupled-weight-decay write-back."""
    b = momentum(b_prev, g, hp.mu)
    v = ns_input(b, g, hp.mu, hp.nesterov)
    ut, r, c = two_sided(v, hp.delta)
    w_new = write_back(w, ut, lr, hp.rho, hp.weight_decay)
    return {"W": w_new, "B": b, "V": v, "r": r, "c": c, "Ut": ut}


# ------------------------------------------------------------ 1-D parameters (eq. "vector")
def global_rms_normalize(v: np.ndarray) -> np.ndarray:
    """U~ = V / (||V||_2 / sqrt(d))  (eq. "vector"); a zero V gives a zero update."""
    v = np.asarray(v, np.float64).ravel()
    nrm = math.sqrt(float(np.sum(v * v)))
    if nrm == 0.0:
        return np.zeros_like(v)
    return v / (nrm / math.sqrt(v.size))


def vec_step(w: np.ndarray, g: np.ndarray, b_prev: np.ndarray, hp: HParams, lr: float) -> dict:
    """One MeqMuon step for a 1-D parameter such as an RMSNorm weight or a bias
    (Algorithm "MeqMuon", last branch)."""
    b = momentum(np.ravel(b_prev), np.ravel(g), hp.mu)
    v = ns_input(b, np.ravel(g), hp.mu, hp.nesterov)
    ut = global_rms_normalize(v)
    w_new = write_back(np.ravel(w), ut, lr, hp.rho, hp.weight_decay)
    return {"W": w_new, "B": b, "V": v, "normsq": float(np.sum(v * v)), "Ut": ut}


# ------------------------------------------------------- Moonlight-Muon (eq. "moonlight-update")
def moonlight_step(w: np.ndarray, g: np.ndarray, b_prev: np.ndarray, hp: HParams, lr: float,
                   wide: bool = False) -> dict:
    """One Muon step in the Moonlight form the paper compares with (eq. "moonlight-update"):
    U = Orth(B) by the same K Newton-Schulz steps, then
    W_{t+1} = (1 - eta lambda) W - eta rho sqrt(max(m, n)) U, with no equilibration."""
    b = momentum(b_prev, g, hp.mu)
    v = ns_input(b, g, hp.mu, hp.nesterov)
    u = newton_schulz(v, hp.ns_a, hp.ns_b, hp.ns_c, hp.ns_steps, wide=wide)
    m, n = u.shape
    ut = math.sqrt(max(m, n)) * u
    w_new = write_back(w, ut, lr, hp.rho, hp.weight_decay)
    return {"W": w_new, "B": b, "V": v, "normsq": frobenius(v) ** 2, "U": u, "Ut": ut}


# ------------------------------------------- NS trajectories (Section "Imbalance patterns")
def ns_cv_trace(v: np.ndarray, hp: HParams, kmax: int, wide: bool = False):
    """Row and column CVs of X_k for k = 0 .. kmax, where X_0 = V / ||V||_F and X_k follows
    eq. "ns"; the replay behind the paper's figure of CV trajectories during the NS iterations.
    Returns two lists of kmax + 1 values (gamma_r, gamma_c)."""
    gr, gc = [], []
    for k in range(kmax + 1):
        x = (np.asarray(v, np.float64) / frobenius(v) if k == 0 else
             newton_schulz(v, hp.ns_a, hp.ns_b, hp.ns_c, k, wide=wide))
        r, c = row_col_rms(x)
        gr.append(coeff_of_variation(r, hp.delta))
        gc.append(coeff_of_variation(c, hp.delta))
    return gr, gc
