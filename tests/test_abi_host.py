"""Host-side checks of the C ABI (no GPU needed: meq_init touches no device and
meq_step validates every argument before enqueuing anything)."""
import ctypes
import os
import re

import pytest

import workloads
from paper_2609_35701_amd import meq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "meq.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(meq_[a-z_]+)\s*\(", text)))


def test_library_exports_every_header_symbol():
    L = meq.lib()
    names = header_functions()
    assert len(names) >= 12
    for name in names:
        assert hasattr(L, name), name
    assert sorted(meq.EXPORTED) == names


def test_default_hparams_are_the_papers():
    hp = meq.default_hparams()
    assert hp.ns_steps == 5 and hp.nesterov == 0
    for got, want in [(hp.mu, 0.95), (hp.rho, 0.2), (hp.weight_decay, 0.1), (hp.ns_a, 3.4445),
                      (hp.ns_b, -4.7750), (hp.ns_c, 2.0315), (hp.zero_rms_delta, 1e-7)]:
        assert got == pytest.approx(want, rel=1e-6)


def _init(descs, hp=None):
    L = meq.lib()
    arr = (meq.MatrixDesc * max(len(descs), 1))(*[meq.MatrixDesc(*d) for d in descs])
    h = ctypes.c_void_p()
    hp = hp or meq.default_hparams()
    st = L.meq_init(arr, len(descs), ctypes.byref(hp), ctypes.byref(h))
    if h.value:
        L.meq_destroy(h)
    return st


@pytest.mark.parametrize("desc,status", [
    ((4, 8, meq.MEQ_BF16, meq.MEQ_BF16), meq.MEQ_OK),
    ((4, 8, meq.MEQ_F32, meq.MEQ_F32), meq.MEQ_OK),
    ((0, 8, meq.MEQ_BF16, meq.MEQ_BF16), meq.MEQ_ERR_INVALID_ARG),
    ((4, -1, meq.MEQ_BF16, meq.MEQ_BF16), meq.MEQ_ERR_INVALID_ARG),
    ((65537, 8, meq.MEQ_BF16, meq.MEQ_BF16), meq.MEQ_ERR_INVALID_ARG),
    ((4, 8, 7, meq.MEQ_BF16), meq.MEQ_ERR_INVALID_ARG),
    ((4, 8, meq.MEQ_BF16, meq.MEQ_F32), meq.MEQ_ERR_UNSUPPORTED),
    ((65536, 65536, meq.MEQ_BF16, meq.MEQ_BF16), meq.MEQ_ERR_UNSUPPORTED),
])
def test_init_validates_descriptors(desc, status):
    assert _init([desc]) == status


@pytest.mark.parametrize("field,value", [("mu", 1.0), ("mu", -0.1), ("mu", float("nan")), ("rho", 0.0),
                                         ("weight_decay", -1.0), ("ns_steps", 0), ("ns_steps", 65),
                                         ("ns_a", float("inf")), ("zero_rms_delta", -1e-7), ("nesterov", 2)])
def test_init_validates_hparams(field, value):
    hp = meq.default_hparams(**{field: value})
    assert _init([(4, 8, meq.MEQ_BF16, meq.MEQ_BF16)], hp) == meq.MEQ_ERR_INVALID_ARG


def test_init_null_arguments_and_empty_plan():
    L = meq.lib()
    hp = meq.default_hparams()
    h = ctypes.c_void_p(1234)
    assert L.meq_init(None, 1, ctypes.byref(hp), ctypes.byref(h)) == meq.MEQ_ERR_INVALID_ARG
    assert h.value is None
    assert L.meq_init(None, -1, ctypes.byref(hp), ctypes.byref(h)) == meq.MEQ_ERR_INVALID_ARG
    assert L.meq_init(None, 0, ctypes.byref(hp), None) == meq.MEQ_ERR_INVALID_ARG
    assert L.meq_init(None, 0, ctypes.byref(hp), ctypes.byref(h)) == meq.MEQ_OK
    assert L.meq_workspace_bytes(h) == 0
    # an empty plan's step is a no-op that needs no device
    assert L.meq_step(h, None, None, None, ctypes.c_float(0.02), None, 0, None) == meq.MEQ_OK
    L.meq_destroy(h)
    L.meq_destroy(None)
    assert L.meq_workspace_bytes(None) == 0


def test_grouping_of_the_1b_shapes():
    wl = workloads.workload("llama-1b")
    plan = meq.Plan([(m.rows, m.cols) for m in wl.matrices], "bf16")
    assert sorted(plan.groups()) == sorted([(2048, 2048, 32), (512, 2048, 32), (2048, 8192, 48)])
    # two bf16 s x l buffers per matrix dominate the workspace
    assert plan.workspace_bytes > 4 * wl.elements


def test_step_rejects_bad_arguments_before_any_device_work():
    plan = meq.Plan([(4, 8), (16, 3)], "f32")
    L = meq.lib()
    n = 2
    fake = [0x1000, 0x2000]
    P = (ctypes.c_void_p * n)(*fake)
    Z = (ctypes.c_void_p * n)(0, 0x3000)
    ws = plan.workspace_bytes

    def step(params=P, grads=P, moms=P, lr=0.02, w=0x100000, wb=ws):
        return L.meq_step(plan.handle, params, grads, moms, ctypes.c_float(lr), ctypes.c_void_p(w), wb, None)

    assert step(params=None) == meq.MEQ_ERR_INVALID_ARG
    assert step(grads=Z) == meq.MEQ_ERR_INVALID_ARG
    assert step(lr=float("nan")) == meq.MEQ_ERR_INVALID_ARG
    assert step(lr=-1.0) == meq.MEQ_ERR_INVALID_ARG
    assert step(w=0) == meq.MEQ_ERR_WORKSPACE
    assert step(wb=ws - 1) == meq.MEQ_ERR_WORKSPACE
    assert step(w=0x100000 + 128) == meq.MEQ_ERR_WORKSPACE
    assert L.meq_step(None, P, P, P, ctypes.c_float(0.02), ctypes.c_void_p(0x100000), ws, None) == \
        meq.MEQ_ERR_INVALID_ARG


def test_debug_regions_and_timing_kinds():
    plan = meq.Plan([(300, 100), (64, 64)], "bf16")
    off_x0, r, c, ld = plan.debug_region(0, meq.BUF_X0)
    assert (r, c, ld) == (100, 300, 512)  # wide orientation, long side padded to 256
    off_u, *_ = plan.debug_region(0, meq.BUF_U)
    assert off_u != off_x0  # five (odd) steps end in the second buffer
    for k in range(6):
        off, *_ = plan.debug_region(1, k)
        assert off % 8 == 0 and off < plan.workspace_bytes
    with pytest.raises(meq.MeqError):
        plan.debug_region(2, meq.BUF_U)
    with pytest.raises(meq.MeqError):
        plan.debug_region(0, 99)
    plan.set_timing([meq.K_APPLY, meq.K_GRAM])
    assert plan.get_timing(meq.K_APPLY) == (0.0, 0)
    with pytest.raises(meq.MeqError):
        plan.get_timing(8)
