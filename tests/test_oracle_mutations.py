"""Mutation check of the oracle's pins: each test plants one plausible mistake in the oracle (a
dropped term, a wrong sign, swapped indices or operands, an off-by-one, a wrong rounding) and
runs every pin of tests/test_oracle_pins.py and tests/test_oracle_pins_other.py against the
planted version; at least one pin has to fail, so the pins can tell the oracle from a
plausible wrong one.  Mistakes are planted on the CPU only, in this process."""
import math

import numpy as np
import pytest

import oracle
import oracle.meq_oracle as om
import test_oracle_pins as P
import test_oracle_pins_other as PO

F64 = np.float64


def _ns(h, a, b, c, steps, wide=False, *, drop_c=False, no_prescale=False, neg_b=False, off_by_one=False,
        sq_norm=False):
    h = np.asarray(h, F64)
    if wide and h.shape[0] > h.shape[1]:
        return _ns(h.T, a, b, c, steps, False, drop_c=drop_c, no_prescale=no_prescale, neg_b=neg_b,
                   off_by_one=off_by_one, sq_norm=sq_norm).T
    nrm = math.sqrt(float(np.sum(h * h)))
    if nrm == 0.0:
        return np.zeros_like(h)
    x = h if no_prescale else h / (nrm * nrm if sq_norm else nrm)
    for _ in range(steps - 1 if off_by_one else steps):
        am = x @ x.T
        x = a * x + ((-b if neg_b else b) * am + (0.0 if drop_c else c) * (am @ am)) @ x
    return x


def _rms_swapped(x):
    x = np.asarray(x, F64)
    m, n = x.shape
    return np.sqrt(np.sum(x * x, axis=1) / m), np.sqrt(np.sum(x * x, axis=0) / n)


def _cv_sample(v, delta):
    pos = np.asarray(v, F64)[np.asarray(v, F64) > delta]
    if pos.size < 2:
        return 0.0
    return float(np.std(pos, ddof=1)) / float(np.mean(pos))


def _cv_threshold_ge(v, delta):
    pos = np.asarray(v, F64)[np.asarray(v, F64) >= delta]
    if pos.size == 0:
        return 0.0
    return float(np.std(pos)) / float(np.mean(pos))


def _equilibrate(u, delta, force_dir=None, *, tie_cols=False, swapped=False):
    r, c = om.row_col_rms(u)
    gr, gc = om.coeff_of_variation(r, delta), om.coeff_of_variation(c, delta)
    rows = (gr > gc) if tie_cols else (gr >= gc)
    d = (om.ROW if rows else om.COL) if force_dir is None else int(force_dir)
    use_rows = (d != om.ROW) if swapped else (d == om.ROW)
    ut = om.row_normalize(u, delta) if use_rows else om.col_normalize(u, delta)
    return ut, gr, gc, d


def _two_sided_cols_first(v, delta):
    v = np.asarray(v, F64)
    r, _ = om.row_col_rms(v)
    vc = om.col_normalize(v, delta)
    _, c = om.row_col_rms(vc)
    return om.row_normalize(vc, delta), r, c


def _two_sided_colrms_of_v(v, delta):
    v = np.asarray(v, F64)
    r, c = om.row_col_rms(v)
    vr = om.row_normalize(v, delta)
    s = np.zeros_like(c)
    s[c > delta] = 1.0 / c[c > delta]
    return vr * s[None, :], r, c


def _global_rms_no_sqrt_d(v):
    v = np.asarray(v, F64).ravel()
    nrm = math.sqrt(float(np.sum(v * v)))
    return np.zeros_like(v) if nrm == 0.0 else v / nrm


def _moonlight_sqrt_min(w, g, b_prev, hp, lr, wide=False):
    b = om.momentum(b_prev, g, hp.mu)
    v = om.ns_input(b, g, hp.mu, hp.nesterov)
    u = om.newton_schulz(v, hp.ns_a, hp.ns_b, hp.ns_c, hp.ns_steps, wide=wide)
    ut = math.sqrt(min(u.shape)) * u
    w_new = om.write_back(w, ut, lr, hp.rho, hp.weight_decay)
    return {"W": w_new, "B": b, "V": v, "normsq": om.frobenius(v) ** 2, "U": u, "Ut": ut}


def _round_truncate(x):
    x = np.asarray(x, F64)
    m, e = np.frexp(x)
    return np.ldexp(np.trunc(m * 256.0), e - 8)


MUTATIONS = {
    "momentum drops mu B": ("momentum", lambda b, g, mu: np.asarray(g, F64) + 0.0 * np.asarray(b, F64)),
    "momentum as a (1 - mu) average": ("momentum", lambda b, g, mu: mu * np.asarray(b, F64) + (1 - mu) * np.asarray(g, F64)),
    "Nesterov with the wrong sign": ("ns_input", lambda b, g, mu, nest: np.asarray(g, F64) - mu * b if nest else b),
    "NS drops the c A A term": ("newton_schulz", lambda *a, **k: _ns(*a, **k, drop_c=True)),
    "NS without the prescale": ("newton_schulz", lambda *a, **k: _ns(*a, **k, no_prescale=True)),
    "NS prescale by ||H||^2": ("newton_schulz", lambda *a, **k: _ns(*a, **k, sq_norm=True)),
    "NS with the sign of b flipped": ("newton_schulz", lambda *a, **k: _ns(*a, **k, neg_b=True)),
    "NS one step short": ("newton_schulz", lambda *a, **k: _ns(*a, **k, off_by_one=True)),
    "row/column RMS with m and n swapped": ("row_col_rms", _rms_swapped),
    "CV with the sample std": ("coeff_of_variation", _cv_sample),
    "CV counting entries equal to delta": ("coeff_of_variation", _cv_threshold_ge),
    "direction tie goes to columns": ("equilibrate", lambda u, d, f=None: _equilibrate(u, d, f, tie_cols=True)),
    "direction applied to the other side": ("equilibrate", lambda u, d, f=None: _equilibrate(u, d, f, swapped=True)),
    "write-back adds the step": ("write_back", lambda w, ut, lr, rho, wd: (1 - lr * wd) * np.asarray(w, F64) + rho * lr * np.asarray(ut, F64)),
    "write-back without decay": ("write_back", lambda w, ut, lr, rho, wd: np.asarray(w, F64) - rho * lr * np.asarray(ut, F64)),
    "write-back decay without lr": ("write_back", lambda w, ut, lr, rho, wd: (1 - wd) * np.asarray(w, F64) - rho * lr * np.asarray(ut, F64)),
    "two-sided normalization columns first": ("two_sided", _two_sided_cols_first),
    "two-sided column RMS of V": ("two_sided", _two_sided_colrms_of_v),
    "global RMS without sqrt(d)": ("global_rms_normalize", _global_rms_no_sqrt_d),
    "Moonlight with sqrt(min(m, n))": ("moonlight_step", _moonlight_sqrt_min),
    "bf16 rounding by truncation": ("round_bf16", _round_truncate),
}

# the four mistakes in the other parameter kinds the design notes name, each caught twice
TWICE = {"two-sided normalization columns first", "two-sided column RMS of V", "global RMS without sqrt(d)",
         "Moonlight with sqrt(min(m, n))"}


def _pins():
    """Every pin with fixed arguments (the R21 planted-mistake test plants its own and is left out)."""
    out = []
    for mod in (P, PO):
        for name in sorted(dir(mod)):
            if not name.startswith("test_") or name == "test_R21_planted_mistakes_fail":
                continue
            fn = getattr(mod, name)
            if name == "test_P2_ns_is_spectral_polynomial":
                out += [(f"{name}{s}", lambda fn=fn, s=s: fn(s)) for s in [(5, 8), (9, 4), (1, 7)]]
            elif name == "test_R21_gram_space_regrouping_is_exact":
                out += [(f"{name}{a}", lambda fn=fn, a=a: fn(*a)) for a in [((24, 96), [3, 2]), ((40, 40), [1] * 5)]]
            elif name == "test_moonlight_spectral_closed_form":
                out += [(f"{name}{s}", lambda fn=fn, s=s: fn(s)) for s in [(12, 20), (20, 12)]]
            elif name == "test_ns_cv_trace_orthogonality_constraints":
                out += [(f"{name}{a}", lambda fn=fn, a=a: fn(*a))
                        for a in [((20, 50), "rows"), ((50, 20), "cols"), ((30, 30), "both")]]
            else:
                out.append((name, fn))
    return out


def test_every_pin_passes_on_the_oracle_itself():
    failed = []
    for name, fn in _pins():
        try:
            fn()
        except Exception as e:  # noqa: BLE001 - any failure counts
            failed.append(f"{name}: {type(e).__name__}")
    assert not failed, failed


@pytest.mark.filterwarnings("ignore::RuntimeWarning")  # planted mistakes may overflow or divide by zero
@pytest.mark.parametrize("mutation", list(MUTATIONS))
def test_a_planted_mistake_fails_a_pin(mutation, monkeypatch):
    attr, fn = MUTATIONS[mutation]
    monkeypatch.setattr(om, attr, fn)
    if hasattr(oracle, attr):
        monkeypatch.setattr(oracle, attr, fn)
    caught = []
    for name, pin in _pins():
        try:
            pin()
        except Exception:  # noqa: BLE001 - a failing pin is what is asked for
            caught.append(name)
    need = 2 if mutation in TWICE else 1
    assert len(caught) >= need, f"{mutation}: caught by {caught}"
