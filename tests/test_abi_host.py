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
    assert hp.ns_steps == 5 and hp.nesterov == 0 and hp.ns_gram_steps == 3
    for got, want in [(hp.mu, 0.95), (hp.rho, 0.2), (hp.weight_decay, 0.1), (hp.ns_a, 3.4445),
                      (hp.ns_b, -4.7750), (hp.ns_c, 2.0315), (hp.zero_rms_delta, 1e-7)]:
        assert got == pytest.approx(want, rel=1e-6)


def test_status_strings_cover_every_status():
    header = open(os.path.join(ROOT, "include", "meq.h")).read()
    codes = {int(v) for v in re.findall(r"MEQ_(?:OK|ERR_[A-Z_]+) = (-?\d+)", header)}
    assert codes == {0, -1, -2, -3, -4, -5, -6}
    texts = {meq.status_string(c) for c in codes}
    assert len(texts) == len(codes) and "unknown status" not in texts
    assert meq.status_string(-99) == "unknown status"
    assert meq.MEQ_ERR_NO_MEMORY == -5 and meq.MEQ_ERR_INTERNAL == -6


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
                                         ("ns_a", float("inf")), ("zero_rms_delta", -1e-7), ("nesterov", 2),
                                         ("ns_gram_steps", 0), ("ns_gram_steps", 4)])
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


@pytest.mark.parametrize("shape,steps,gram,segs", [
    ((256, 512), 5, 3, [3, 2]),          # padded long side 2x the short side: Gram-space segments
    ((512, 256), 5, 3, [3, 2]),          # tall matrices run in wide orientation
    ((512, 512), 5, 3, [1] * 5),         # square: eq. "ns" as printed
    ((256, 300), 5, 3, [3, 2]),          # the padded sizes decide: 256 x 512
    ((256, 257), 5, 3, [3, 2]),
    ((2048, 3840), 5, 3, [1] * 5),       # 1.875x: not worth it
    ((2048, 8192), 5, 1, [1] * 5),       # ns_gram_steps 1: the printed iteration everywhere
    ((2048, 8192), 5, 2, [2, 2, 1]),
    ((2048, 8192), 4, 3, [3, 1]),
    ((2048, 8192), 3, 3, [3]),
    ((2048, 8192), 7, 3, [3, 3, 1]),
    ((2048, 8192), 2, 3, [2]),
    ((1, 300), 1, 3, [1]),
])
def test_newton_schulz_schedule(shape, steps, gram, segs):
    plan = meq.Plan([shape], "bf16", hparams=meq.default_hparams(ns_steps=steps, ns_gram_steps=gram))
    got = plan.schedule(0)
    assert got == segs and sum(got) == steps


@pytest.mark.parametrize("coeffs,segs", [
    ((3.4445, -4.7750, 2.0315), [3, 2]),   # the paper's quintic: singular values stay below 1.21
    ((1.5, -0.5, 0.0), [3, 2]),            # the cubic Newton-Schulz step: bounded by 1
    ((2.0, -0.5, 0.0), [1] * 5),           # grows singular values to about 1.57: fp16 unsafe
    ((3.0, 0.0, 0.0), [1] * 5),            # divergent
])
def test_schedule_falls_back_when_fp16_is_unsafe(coeffs, segs):
    a, b, c = coeffs
    plan = meq.Plan([(256, 512)], "bf16", hparams=meq.default_hparams(ns_a=a, ns_b=b, ns_c=c))
    assert plan.schedule(0) == segs


def test_schedule_of_the_1b_shapes_and_workspace():
    wl = workloads.workload("llama-1b")
    shapes = [(m.rows, m.cols) for m in wl.matrices]
    plan = meq.Plan(shapes, "bf16")
    sched = {plan.groups()[g][:2]: plan.schedule(g) for g in range(len(plan.groups()))}
    assert sched == {(2048, 2048): [1] * 5, (512, 2048): [3, 2], (2048, 8192): [3, 2]}
    literal = meq.Plan(shapes, "bf16", hparams=meq.default_hparams(ns_gram_steps=1))
    assert all(literal.schedule(g) == [1] * 5 for g in range(3))
    # four more s x s 16-bit buffers per matrix of the two segmented groups (P', T, Q, Q')
    extra = 4 * 2 * (48 * 2048 * 2048 + 32 * 512 * 512)
    assert plan.workspace_bytes - literal.workspace_bytes == pytest.approx(extra, abs=64 * 256)
    L = meq.lib()
    n = ctypes.c_int32()
    assert L.meq_plan_group_schedule(plan.handle, 3, None, 0, ctypes.byref(n)) == meq.MEQ_ERR_INVALID_ARG
    assert L.meq_plan_group_schedule(plan.handle, 0, None, 1, ctypes.byref(n)) == meq.MEQ_ERR_INVALID_ARG
    assert L.meq_plan_group_schedule(None, 0, None, 0, ctypes.byref(n)) == meq.MEQ_ERR_INVALID_ARG
    one = (ctypes.c_int32 * 1)()
    assert L.meq_plan_group_schedule(plan.handle, 1, one, 1, ctypes.byref(n)) == meq.MEQ_OK
    assert n.value == len(plan.schedule(1)) and one[0] == plan.schedule(1)[0]


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
    assert plan.schedule(0) == [3, 2]
    assert off_u == off_x0  # two segments: the second one writes back into the first buffer
    off_x0, *_ = plan.debug_region(1, meq.BUF_X0)
    off_u, *_ = plan.debug_region(1, meq.BUF_U)
    assert plan.schedule(1) == [1] * 5
    assert off_u != off_x0  # five (odd) single steps end in the second buffer
    for k in range(6):
        off, *_ = plan.debug_region(1, k)
        assert off % 8 == 0 and off < plan.workspace_bytes
    with pytest.raises(meq.MeqError):
        plan.debug_region(2, meq.BUF_U)
    with pytest.raises(meq.MeqError):
        plan.debug_region(0, 99)
    plan.set_timing([meq.K_APPLY, meq.K_GRAM])
    assert plan.get_timing(meq.K_APPLY) == (0.0, 0)
    assert plan.get_timing(meq.K_VECTOR) == (0.0, 0)
    with pytest.raises(meq.MeqError):
        plan.get_timing(len(meq.KERNEL_NAMES))


# ------------------------------------------------------------------ parameter kinds
def _init_kind(kind, descs, hp=None):
    L = meq.lib()
    arr = (meq.MatrixDesc * max(len(descs), 1))(*[meq.MatrixDesc(*d) for d in descs])
    h = ctypes.c_void_p()
    hp = hp or meq.default_hparams()
    st = L.meq_init_kind(kind, arr, len(descs), ctypes.byref(hp), ctypes.byref(h))
    if h.value:
        L.meq_destroy(h)
    return st


BF = (meq.MEQ_BF16, meq.MEQ_BF16)
F32 = (meq.MEQ_F32, meq.MEQ_F32)


@pytest.mark.parametrize("kind,desc,status", [
    (meq.PARAM_AUX, (32000, 2048, *BF), meq.MEQ_OK),
    (meq.PARAM_AUX, (151936, 896, *BF), meq.MEQ_OK),          # a large-vocabulary embedding
    (meq.PARAM_AUX, (7, 3, *F32), meq.MEQ_OK),
    (meq.PARAM_AUX, (1 << 24, 8, *BF), meq.MEQ_OK),
    ((meq.PARAM_AUX), ((1 << 24) + 1, 8, *BF), meq.MEQ_ERR_UNSUPPORTED),
    (meq.PARAM_AUX, (8, 65537, *BF), meq.MEQ_ERR_UNSUPPORTED),
    (meq.PARAM_AUX, (1 << 20, 4096, *BF), meq.MEQ_ERR_UNSUPPORTED),  # 2^32 elements
    (meq.PARAM_AUX, (0, 8, *BF), meq.MEQ_ERR_INVALID_ARG),
    (meq.PARAM_AUX, (8, 8, meq.MEQ_BF16, meq.MEQ_F32), meq.MEQ_ERR_UNSUPPORTED),
    (meq.PARAM_VECTOR, (1, 2048, *BF), meq.MEQ_OK),
    (meq.PARAM_VECTOR, (1, 1, *F32), meq.MEQ_OK),
    (meq.PARAM_VECTOR, (3, 5, *F32), meq.MEQ_OK),              # any shape is one flat vector
    (meq.PARAM_VECTOR, (1, (1 << 31) - 1, *F32), meq.MEQ_OK),
    (meq.PARAM_VECTOR, (2, 1 << 30, *F32), meq.MEQ_ERR_UNSUPPORTED),
    (meq.PARAM_VECTOR, (1, 0, *F32), meq.MEQ_ERR_INVALID_ARG),
    (meq.PARAM_VECTOR, (1, 8, 5, meq.MEQ_F32), meq.MEQ_ERR_INVALID_ARG),
])
def test_init_kind_validates_descriptors(kind, desc, status):
    assert _init_kind(kind, [desc]) == status


def test_init_kind_rejects_unknown_kind_and_moonlight_outside_hidden():
    assert _init_kind(3, [(4, 8, *BF)]) == meq.MEQ_ERR_INVALID_ARG
    assert _init_kind(-1, [(4, 8, *BF)]) == meq.MEQ_ERR_INVALID_ARG
    moon = meq.default_hparams(update_rule=meq.RULE_MOONLIGHT)
    assert _init_kind(meq.PARAM_HIDDEN, [(4, 8, *BF)], moon) == meq.MEQ_OK
    assert _init_kind(meq.PARAM_AUX, [(4, 8, *BF)], moon) == meq.MEQ_ERR_INVALID_ARG
    assert _init_kind(meq.PARAM_VECTOR, [(1, 8, *BF)], moon) == meq.MEQ_ERR_INVALID_ARG
    assert _init_kind(meq.PARAM_HIDDEN, [(4, 8, *BF)], meq.default_hparams(update_rule=2)) == \
        meq.MEQ_ERR_INVALID_ARG
    # meq_init is the hidden kind
    assert _init([(4, 8, *BF)], moon) == meq.MEQ_OK


def test_aux_and_vector_plans_layout_and_regions():
    aux = meq.Plan([(32000, 2048), (300, 7)], "bf16", kind=meq.PARAM_AUX)
    assert aux.groups() == []
    # r, c (double), their reciprocals (float) and 128-row column partials (double)
    want = 0
    for m, n in [(32000, 2048), (300, 7)]:
        for nbytes in (8 * m, 8 * n, 4 * m, 4 * n, 8 * ((m + 127) // 128) * n):
            want += (nbytes + 255) // 256 * 256
    assert aux.workspace_bytes == want
    off_r, r, c, _ = aux.debug_region(1, meq.BUF_ROW_RMS)
    off_c, r2, c2, _ = aux.debug_region(1, meq.BUF_COL_RMS)
    assert (r, c, r2, c2) == (1, 300, 1, 7) and off_c > off_r
    for k in (meq.BUF_X0, meq.BUF_U, meq.BUF_NORMSQ, meq.BUF_SCALE):
        with pytest.raises(meq.MeqError):
            aux.debug_region(0, k)
    vec = meq.Plan([(2048,), (1, 5), (3, 4)], "f32", kind=meq.PARAM_VECTOR)
    assert vec.workspace_bytes == 3 * 256
    assert vec.debug_region(2, meq.BUF_NORMSQ)[0] == 512
    with pytest.raises(meq.MeqError):
        vec.debug_region(0, meq.BUF_ROW_RMS)


def test_stats_only_for_meqmuon_hidden_plans():
    L = meq.lib()
    for plan in (meq.Plan([(4, 8)], "f32", kind=meq.PARAM_AUX), meq.Plan([(8,)], "f32", kind=meq.PARAM_VECTOR),
                 meq.Plan([(4, 8)], "f32", hparams=meq.default_hparams(update_rule=meq.RULE_MOONLIGHT))):
        st = L.meq_get_stats(plan.handle, ctypes.c_void_p(0x100000), None, None, None, None)
        assert st == meq.MEQ_ERR_UNSUPPORTED


@pytest.mark.parametrize("kind", [meq.PARAM_AUX, meq.PARAM_VECTOR])
def test_kind_step_rejects_bad_arguments_before_any_device_work(kind):
    plan = meq.Plan([(4, 8), (16, 3)], "f32", kind=kind)
    L = meq.lib()
    P = (ctypes.c_void_p * 2)(0x1000, 0x2000)
    Z = (ctypes.c_void_p * 2)(0x1000, 0)
    ws = plan.workspace_bytes

    def step(params=P, grads=P, moms=P, lr=0.02, w=0x100000, wb=ws):
        return L.meq_step(plan.handle, params, grads, moms, ctypes.c_float(lr), ctypes.c_void_p(w), wb, None)

    assert step(moms=Z) == meq.MEQ_ERR_INVALID_ARG
    assert step(lr=float("inf")) == meq.MEQ_ERR_INVALID_ARG
    assert step(w=0) == meq.MEQ_ERR_WORKSPACE
    assert step(wb=ws - 1) == meq.MEQ_ERR_WORKSPACE


def test_ns_cv_trace_rejects_bad_arguments_before_any_device_work():
    L = meq.lib()
    hid = meq.Plan([(4, 8), (16, 3)], "f32")
    aux = meq.Plan([(4, 8)], "f32", kind=meq.PARAM_AUX)
    X = (ctypes.c_void_p * 2)(0x1000, 0x2000)
    Z = (ctypes.c_void_p * 2)(0x1000, 0)
    gr = (ctypes.c_double * 64)()
    gc = (ctypes.c_double * 64)()
    ws = hid.workspace_bytes

    def trace(plan=hid.handle, inputs=X, kmax=3, w=0x100000, wb=ws, r=gr, c=gc):
        return L.meq_ns_cv_trace(plan, inputs, kmax, ctypes.c_void_p(w), wb, r, c, None)

    assert trace(plan=aux.handle) == meq.MEQ_ERR_INVALID_ARG
    assert trace(kmax=-1) == meq.MEQ_ERR_INVALID_ARG
    assert trace(kmax=65) == meq.MEQ_ERR_INVALID_ARG
    assert trace(inputs=Z) == meq.MEQ_ERR_INVALID_ARG
    assert trace(r=None) == meq.MEQ_ERR_INVALID_ARG
    assert trace(w=0) == meq.MEQ_ERR_WORKSPACE
    assert trace(wb=ws - 1) == meq.MEQ_ERR_WORKSPACE


def test_split_parameters_classifies_kinds():
    import torch
    from paper_2609_35701_amd.optim import split_parameters

    class Tiny(torch.nn.Module):
        def __init__(self, tied):
            super().__init__()
            self.embed = torch.nn.Embedding(50, 16)
            self.q = torch.nn.Linear(16, 16, bias=False)
            self.up = torch.nn.Linear(16, 40, bias=True)
            self.norm = torch.nn.Parameter(torch.ones(16))
            self.lm_head = torch.nn.Linear(16, 50, bias=False)
            if tied:
                self.lm_head.weight = self.embed.weight

    hidden, aux, vec = split_parameters(Tiny(tied=False))
    assert [tuple(p.shape) for p in hidden] == [(16, 16), (40, 16)]
    assert [tuple(p.shape) for p in aux] == [(50, 16), (50, 16)]
    assert sorted(tuple(p.shape) for p in vec) == [(16,), (40,)]
    _, aux_t, _ = split_parameters(Tiny(tied=True))
    assert len(aux_t) == 1  # a tied embedding / LM head is one parameter

    class Conv(torch.nn.Module):
        def __init__(self):
            super().__init__()
            self.c = torch.nn.Conv2d(3, 4, 3)

    with pytest.raises(ValueError):
        split_parameters(Conv())


def test_capped_plans_fit_their_cap_and_split_into_passes():
    shapes = [(m.rows, m.cols) for m in workloads.workload("llama-1b").matrices]
    full = meq.Plan(shapes, "bf16")
    assert full.passes == 1
    same = meq.Plan(shapes, "bf16", max_workspace_bytes=0)
    assert same.workspace_bytes == full.workspace_bytes and same.groups() == full.groups()
    for cap in (4 << 30, 1 << 30, 256 << 20):
        p = meq.Plan(shapes, "bf16", max_workspace_bytes=cap)
        assert p.workspace_bytes <= cap and p.passes >= 2
        # slices of the shape groups add up to the groups, each with its group's schedule
        tot = {}
        for g, (s_, l_, c) in enumerate(p.groups()):
            tot[(s_, l_)] = tot.get((s_, l_), 0) + c
            assert p.schedule(g) == full.schedule([x[:2] for x in full.groups()].index((s_, l_)))
        assert tot == {(s_, l_): c for s_, l_, c in full.groups()}
    # a cap above the uncapped workspace changes nothing
    big = meq.Plan(shapes, "bf16", max_workspace_bytes=full.workspace_bytes + 4096)
    assert big.passes == 1 and big.workspace_bytes == full.workspace_bytes


def test_capped_plans_reject_caps_too_small():
    for shapes, cap in (([(2048, 8192)], 64 << 20), ([(256, 512)] * 4, 4096)):
        with pytest.raises(meq.MeqError) as e:
            meq.Plan(shapes, "bf16", max_workspace_bytes=cap)
        assert e.value.status == meq.MEQ_ERR_WORKSPACE
    with pytest.raises(meq.MeqError) as e:
        meq.Plan([(32000, 2048)], "bf16", kind=meq.PARAM_AUX, max_workspace_bytes=1024)
    assert e.value.status == meq.MEQ_ERR_WORKSPACE
    assert meq.Plan([(32000, 2048)], "bf16", kind=meq.PARAM_AUX, max_workspace_bytes=64 << 20).passes == 0


def test_step_static_rejects_plans_beyond_its_scratch_before_any_device_work():
    L = meq.lib()
    assert meq.MEQ_STATIC_SCRATCH_BYTES == 256 << 20
    header = open(os.path.join(ROOT, "include", "meq.h")).read()
    assert "#define MEQ_STATIC_SCRATCH_BYTES ((size_t)256 << 20)" in header
    big = meq.Plan([(m.rows, m.cols) for m in workloads.workload("llama-1b").matrices], "bf16")
    assert big.workspace_bytes > meq.MEQ_STATIC_SCRATCH_BYTES
    n = big.count
    ptrs = (ctypes.c_void_p * n)(*([0x1000] * n))
    assert L.meq_step_static(big.handle, ptrs, ptrs, ptrs, ctypes.c_float(0.02), None) == meq.MEQ_ERR_WORKSPACE
    assert L.meq_step_static(None, ptrs, ptrs, ptrs, ctypes.c_float(0.02), None) == meq.MEQ_ERR_INVALID_ARG
    capped = meq.Plan([(m.rows, m.cols) for m in workloads.workload("llama-1b").matrices], "bf16",
                      max_workspace_bytes=meq.MEQ_STATIC_SCRATCH_BYTES)
    assert capped.workspace_bytes <= meq.MEQ_STATIC_SCRATCH_BYTES


C_PROGRAM = r"""
#include <stdio.h>
#include "meq.h"

/* plain C against the C ABI: plan the 1B shapes (one of each, tall included) on the host */
int main(void) {
  meq_hparams hp;
  meq_default_hparams(&hp);
  const meq_matrix_desc mats[4] = {{2048, 2048, MEQ_BF16, MEQ_BF16}, {512, 2048, MEQ_BF16, MEQ_BF16},
                                   {2048, 8192, MEQ_BF16, MEQ_BF16}, {8192, 2048, MEQ_BF16, MEQ_BF16}};
  meq_plan* plan = NULL;
  meq_status st = meq_init(mats, 4, &hp, &plan);
  if (st != MEQ_OK) {
    printf("init %d %s\n", (int)st, meq_status_string(st));
    return 1;
  }
  printf("steps %d gram %d groups %d ws %zu\n", (int)hp.ns_steps, (int)hp.ns_gram_steps,
         (int)meq_plan_num_groups(plan), meq_workspace_bytes(plan));
  meq_destroy(plan);
  st = meq_init(mats, 4, &hp, NULL);
  printf("null %s\n", meq_status_string(st));
  return 0;
}
"""


def test_header_compiles_and_links_as_c(tmp_path):
    """The header is plain C: a C11 program built with gcc against include/meq.h and linked with the
    built library plans the 1B shapes on the host, and agrees with the Python binding."""
    import shutil
    import subprocess

    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "use_meq.c"
    src.write_text(C_PROGRAM)
    exe = tmp_path / "use_meq"
    libdir = os.path.dirname(meq.LIB_PATH)
    cmd = [gcc, "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           "-I" + os.path.join(ROOT, "include"), str(src), "-L" + libdir, "-lmeq", "-Wl,-rpath," + libdir,
           "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True, timeout=60).stdout.split("\n")
    plan = meq.Plan([(2048, 2048), (512, 2048), (2048, 8192), (8192, 2048)], "bf16")
    assert out[0] == f"steps 5 gram 3 groups {len(plan.groups())} ws {plan.workspace_bytes}", out[0]
    assert out[1] == "null " + meq.status_string(meq.MEQ_ERR_INVALID_ARG), out[1]
