"""ctypes binding of libmeq.so (the MeqMuon optimizer update on MI355X).

Argument marshalling only: every step of the update runs in the library's HIP
kernels.  The names follow the C ABI in ``include/meq.h``.  If the library has
not been built, loading raises ``MeqLibraryMissing``; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Iterable, List, Optional, Sequence, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmeq.so")

(MEQ_OK, MEQ_ERR_INVALID_ARG, MEQ_ERR_UNSUPPORTED, MEQ_ERR_HIP, MEQ_ERR_WORKSPACE, MEQ_ERR_NO_MEMORY,
 MEQ_ERR_INTERNAL) = 0, -1, -2, -3, -4, -5, -6
MEQ_F32, MEQ_BF16 = 0, 1
MEQ_STATIC_SCRATCH_BYTES = 256 << 20
MEQ_DIR_ROW, MEQ_DIR_COL = 0, 1
PARAM_HIDDEN, PARAM_AUX, PARAM_VECTOR = 0, 1, 2
RULE_MEQMUON, RULE_MOONLIGHT = 0, 1
BUF_X0, BUF_U, BUF_NORMSQ, BUF_ROW_RMS, BUF_COL_RMS, BUF_SCALE = range(6)
(K_MOMENTUM, K_NORM, K_GRAM, K_POLY, K_APPLY, K_ROWCOL, K_SELECT, K_UPDATE,
 K_AUX_ROWS, K_AUX_COLS, K_AUX_UPDATE, K_VECTOR) = range(12)
KERNEL_NAMES = ("momentum", "norm", "gram", "poly", "apply", "rowcol", "select", "update",
                "aux_rows", "aux_cols", "aux_update", "vector")

EXPORTED = ("meq_default_hparams", "meq_init", "meq_init_kind", "meq_init_capped", "meq_workspace_bytes", "meq_step",
            "meq_get_stats", "meq_ns_cv_trace", "meq_destroy", "meq_status_string", "meq_plan_num_groups",
            "meq_plan_num_passes", "meq_plan_group", "meq_plan_group_schedule", "meq_debug_region", "meq_set_timing",
            "meq_get_timing", "meq_step_static")


class MeqLibraryMissing(RuntimeError):
    pass


class MeqError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)} ({status})")
        self.status = status


class HParams(ctypes.Structure):
    _fields_ = [("mu", ctypes.c_float), ("rho", ctypes.c_float), ("weight_decay", ctypes.c_float),
                ("ns_steps", ctypes.c_int32), ("ns_a", ctypes.c_float), ("ns_b", ctypes.c_float),
                ("ns_c", ctypes.c_float), ("zero_rms_delta", ctypes.c_float), ("nesterov", ctypes.c_int32),
                ("update_rule", ctypes.c_int32), ("ns_gram_steps", ctypes.c_int32)]


class MatrixDesc(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int64), ("cols", ctypes.c_int64), ("param_dtype", ctypes.c_int32),
                ("grad_dtype", ctypes.c_int32)]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise MeqLibraryMissing(f"{LIB_PATH} is not built; run `python -m paper_2609_35701_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, c_i32, c_i64, c_sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    L.meq_default_hparams.argtypes = [ctypes.POINTER(HParams)]
    L.meq_default_hparams.restype = None
    L.meq_init.argtypes = [ctypes.POINTER(MatrixDesc), c_i32, ctypes.POINTER(HParams), ctypes.POINTER(vp)]
    L.meq_init.restype = c_i32
    L.meq_init_kind.argtypes = [c_i32, ctypes.POINTER(MatrixDesc), c_i32, ctypes.POINTER(HParams), ctypes.POINTER(vp)]
    L.meq_init_kind.restype = c_i32
    L.meq_init_capped.argtypes = [c_i32, ctypes.POINTER(MatrixDesc), c_i32, ctypes.POINTER(HParams), c_sz,
                                  ctypes.POINTER(vp)]
    L.meq_init_capped.restype = c_i32
    L.meq_workspace_bytes.argtypes = [vp]
    L.meq_workspace_bytes.restype = c_sz
    L.meq_step.argtypes = [vp, ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.c_float, vp,
                           c_sz, vp]
    L.meq_step.restype = c_i32
    L.meq_step_static.argtypes = [vp, ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.c_float, vp]
    L.meq_step_static.restype = c_i32
    L.meq_get_stats.argtypes = [vp, vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                ctypes.POINTER(c_i32), vp]
    L.meq_get_stats.restype = c_i32
    L.meq_ns_cv_trace.argtypes = [vp, ctypes.POINTER(vp), c_i32, vp, c_sz, ctypes.POINTER(ctypes.c_double),
                                  ctypes.POINTER(ctypes.c_double), vp]
    L.meq_ns_cv_trace.restype = c_i32
    L.meq_destroy.argtypes = [vp]
    L.meq_destroy.restype = None
    L.meq_status_string.argtypes = [c_i32]
    L.meq_status_string.restype = ctypes.c_char_p
    L.meq_plan_num_groups.argtypes = [vp]
    L.meq_plan_num_groups.restype = c_i32
    L.meq_plan_num_passes.argtypes = [vp]
    L.meq_plan_num_passes.restype = c_i32
    L.meq_plan_group.argtypes = [vp, c_i32, ctypes.POINTER(c_i64), ctypes.POINTER(c_i64), ctypes.POINTER(c_i32)]
    L.meq_plan_group.restype = c_i32
    L.meq_plan_group_schedule.argtypes = [vp, c_i32, ctypes.POINTER(c_i32), c_i32, ctypes.POINTER(c_i32)]
    L.meq_plan_group_schedule.restype = c_i32
    L.meq_debug_region.argtypes = [vp, c_i32, c_i32, ctypes.POINTER(c_sz), ctypes.POINTER(c_i64),
                                   ctypes.POINTER(c_i64), ctypes.POINTER(c_i64)]
    L.meq_debug_region.restype = c_i32
    L.meq_set_timing.argtypes = [vp, ctypes.c_uint32]
    L.meq_set_timing.restype = c_i32
    L.meq_get_timing.argtypes = [vp, c_i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(c_i64), c_i32]
    L.meq_get_timing.restype = c_i32
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().meq_status_string(int(status)).decode()


def _check(status: int, what: str) -> None:
    if status != MEQ_OK:
        raise MeqError(status, what)


def default_hparams(**overrides) -> HParams:
    hp = HParams()
    lib().meq_default_hparams(ctypes.byref(hp))
    for k, v in overrides.items():
        if not hasattr(hp, k):
            raise AttributeError(k)
        setattr(hp, k, v)
    return hp


def _dtype_code(dtype) -> int:
    name = str(dtype)
    if name in ("f32", "float32", "torch.float32"):
        return MEQ_F32
    if name in ("bf16", "bfloat16", "torch.bfloat16"):
        return MEQ_BF16
    raise ValueError(f"unsupported dtype {dtype}")


class Plan:
    """A validated set of parameters of one kind plus hyperparameters (``meq_init_capped``).

    ``kind`` is PARAM_HIDDEN (2D hidden weights), PARAM_AUX (remaining 2D parameters)
    or PARAM_VECTOR (1-D parameters; a shape (1, d) or (d,) each).  ``max_workspace_bytes``
    caps the plan's workspace (0: no cap)."""

    def __init__(self, shapes: Sequence[Tuple[int, ...]], param_dtype="bf16", grad_dtype=None,
                 hparams: Optional[HParams] = None, kind: int = PARAM_HIDDEN, max_workspace_bytes: int = 0):
        L = lib()
        self.kind = int(kind)
        self.shapes = [(1, int(sh[0])) if len(sh) == 1 else (int(sh[0]), int(sh[1])) for sh in shapes]
        pd = _dtype_code(param_dtype)
        gd = pd if grad_dtype is None else _dtype_code(grad_dtype)
        n = len(self.shapes)
        descs = (MatrixDesc * max(n, 1))()
        for i, (r, c) in enumerate(self.shapes):
            descs[i] = MatrixDesc(r, c, pd, gd)
        self.hparams = hparams if hparams is not None else default_hparams()
        handle = ctypes.c_void_p()
        _check(L.meq_init_capped(self.kind, descs, n, ctypes.byref(self.hparams), ctypes.c_size_t(max_workspace_bytes),
                                 ctypes.byref(handle)), "meq_init_capped")
        self._h = handle
        self.count = n

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.meq_destroy(h)
            self._h = None

    @property
    def handle(self) -> ctypes.c_void_p:
        return self._h

    @property
    def workspace_bytes(self) -> int:
        return int(lib().meq_workspace_bytes(self._h))

    @property
    def passes(self) -> int:
        return int(lib().meq_plan_num_passes(self._h))

    def groups(self) -> List[Tuple[int, int, int]]:
        L = lib()
        out = []
        for g in range(L.meq_plan_num_groups(self._h)):
            s, l, c = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int32()
            _check(L.meq_plan_group(self._h, g, ctypes.byref(s), ctypes.byref(l), ctypes.byref(c)), "meq_plan_group")
            out.append((s.value, l.value, c.value))
        return out

    def schedule(self, group: int) -> List[int]:
        """Steps per Newton-Schulz segment of shape group ``group`` (``meq_plan_group_schedule``)."""
        L = lib()
        n = ctypes.c_int32()
        _check(L.meq_plan_group_schedule(self._h, group, None, 0, ctypes.byref(n)), "meq_plan_group_schedule")
        segs = (ctypes.c_int32 * max(n.value, 1))()
        _check(L.meq_plan_group_schedule(self._h, group, segs, n.value, ctypes.byref(n)), "meq_plan_group_schedule")
        return list(segs)[:n.value]

    def debug_region(self, matrix: int, kind: int):
        """(byte offset, rows, cols, ld) of a workspace buffer (``meq_debug_region``)."""
        off, r, c, ld = ctypes.c_size_t(), ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        _check(lib().meq_debug_region(self._h, matrix, kind, ctypes.byref(off), ctypes.byref(r), ctypes.byref(c),
                                      ctypes.byref(ld)), "meq_debug_region")
        return off.value, r.value, c.value, ld.value

    def step_ptrs(self, params: Sequence[int], grads: Sequence[int], moms: Sequence[int], lr: float,
                  workspace: int, workspace_bytes: int, stream: int = 0) -> None:
        """``meq_step`` on raw device addresses (integers)."""
        n = self.count
        P = (ctypes.c_void_p * max(n, 1))(*params)
        G = (ctypes.c_void_p * max(n, 1))(*grads)
        B = (ctypes.c_void_p * max(n, 1))(*moms)
        _check(lib().meq_step(self._h, P, G, B, ctypes.c_float(lr), ctypes.c_void_p(workspace),
                              ctypes.c_size_t(workspace_bytes), ctypes.c_void_p(stream)), "meq_step")

    def step_static_ptrs(self, params: Sequence[int], grads: Sequence[int], moms: Sequence[int], lr: float,
                         stream: int = 0) -> None:
        """``meq_step_static`` (the library's own scratch as the workspace) on raw device addresses."""
        n = self.count
        P = (ctypes.c_void_p * max(n, 1))(*params)
        G = (ctypes.c_void_p * max(n, 1))(*grads)
        B = (ctypes.c_void_p * max(n, 1))(*moms)
        _check(lib().meq_step_static(self._h, P, G, B, ctypes.c_float(lr), ctypes.c_void_p(stream)), "meq_step_static")

    def stats_ptr(self, workspace: int, stream: int = 0):
        n = self.count
        gr = (ctypes.c_double * max(n, 1))()
        gc = (ctypes.c_double * max(n, 1))()
        d = (ctypes.c_int32 * max(n, 1))()
        _check(lib().meq_get_stats(self._h, ctypes.c_void_p(workspace), gr, gc, d, ctypes.c_void_p(stream)),
               "meq_get_stats")
        return list(gr)[:n], list(gc)[:n], list(d)[:n]

    def ns_cv_trace_ptr(self, inputs: Sequence[int], kmax: int, workspace: int, workspace_bytes: int,
                        stream: int = 0):
        """Row and column CVs of X_0 .. X_kmax per matrix (``meq_ns_cv_trace``)."""
        n = self.count
        X = (ctypes.c_void_p * max(n, 1))(*inputs)
        gr = (ctypes.c_double * max(n * (kmax + 1), 1))()
        gc = (ctypes.c_double * max(n * (kmax + 1), 1))()
        _check(lib().meq_ns_cv_trace(self._h, X, int(kmax), ctypes.c_void_p(workspace),
                                     ctypes.c_size_t(workspace_bytes), gr, gc, ctypes.c_void_p(stream)),
               "meq_ns_cv_trace")
        w = kmax + 1
        return [list(gr)[i * w:(i + 1) * w] for i in range(n)], [list(gc)[i * w:(i + 1) * w] for i in range(n)]

    def set_timing(self, kinds: Iterable[int]) -> None:
        mask = 0
        for k in kinds:
            mask |= 1 << int(k)
        _check(lib().meq_set_timing(self._h, mask), "meq_set_timing")

    def get_timing(self, kind: int, reset: bool = False) -> Tuple[float, int]:
        ms, n = ctypes.c_double(), ctypes.c_int64()
        _check(lib().meq_get_timing(self._h, kind, ctypes.byref(ms), ctypes.byref(n), int(reset)), "meq_get_timing")
        return ms.value, n.value


class ParamUpdate:
    """Torch glue: owns fp32 momenta and the workspace for a list of parameters of one kind.

    ``step(grads, lr)`` enqueues one MeqMuon update of every parameter on the
    current torch stream.  Hidden and aux parameters are 2D tensors; vector
    parameters are 1-D (or any shape, taken as one flat vector).
    """

    kind = PARAM_HIDDEN

    def __init__(self, params, hparams: Optional[HParams] = None, kind: Optional[int] = None,
                 max_workspace_bytes: int = 0):
        import torch

        if kind is not None:
            self.kind = int(kind)
        self.params = list(params)
        if not self.params:
            raise ValueError("no parameters")
        dev = self.params[0].device
        pdt = self.params[0].dtype
        for p in self.params:
            if not p.is_contiguous() or p.device != dev or p.dtype != pdt:
                raise ValueError("parameters must be contiguous tensors of one dtype on one device")
            if self.kind != PARAM_VECTOR and p.dim() != 2:
                raise ValueError("hidden and aux parameters must be 2D")
        shapes = [tuple(p.shape) if self.kind != PARAM_VECTOR else (p.numel(),) for p in self.params]
        self.plan = Plan(shapes, str(pdt), hparams=hparams, kind=self.kind, max_workspace_bytes=max_workspace_bytes)
        self.momenta = [torch.zeros(p.shape, dtype=torch.float32, device=dev) for p in self.params]
        self.workspace = torch.empty(max(self.plan.workspace_bytes, 256), dtype=torch.uint8, device=dev)

    def step(self, grads, lr: float, stream=None) -> None:
        import torch

        grads = list(grads)
        if len(grads) != len(self.params):
            raise ValueError("one gradient per parameter is required")
        for g, p in zip(grads, self.params):
            if g.shape != p.shape or g.dtype != p.dtype or not g.is_contiguous() or g.device != p.device:
                raise ValueError("gradients must match their parameters in shape, dtype and device")
        st = torch.cuda.current_stream(self.params[0].device) if stream is None else stream
        self.plan.step_ptrs([p.data_ptr() for p in self.params], [g.data_ptr() for g in grads],
                            [b.data_ptr() for b in self.momenta], lr, self.workspace.data_ptr(),
                            self.workspace.numel(), st.cuda_stream)

    def stats(self, stream=None):
        import torch

        st = torch.cuda.current_stream(self.params[0].device) if stream is None else stream
        return self.plan.stats_ptr(self.workspace.data_ptr(), st.cuda_stream)

    def view(self, matrix: int, kind: int):
        """A torch view of a workspace buffer of one parameter (valid until the next step)."""
        import torch

        off, rows, cols, ld = self.plan.debug_region(matrix, kind)
        if kind in (BUF_X0, BUF_U):
            t = self.workspace[off:off + 2 * rows * ld].view(torch.bfloat16).view(rows, ld)
            return t[:, :cols]
        if kind in (BUF_NORMSQ, BUF_ROW_RMS, BUF_COL_RMS):
            return self.workspace[off:off + 8 * cols].view(torch.float64)
        return self.workspace[off:off + 4 * cols].view(torch.float32)


class HiddenWeightUpdate(ParamUpdate):
    """2D hidden-layer weights: Newton-Schulz + adaptive one-sided normalization (or the
    Moonlight-Muon rule with ``hparams.update_rule = RULE_MOONLIGHT``)."""

    kind = PARAM_HIDDEN


def ns_cv_trace(upd: "HiddenWeightUpdate", inputs, kmax: int = 20, stream=None):
    """CV trajectories of the Newton-Schulz iterates for ``inputs`` (one tensor per matrix of a
    hidden update, shaped and typed like its parameters), using that update's plan and workspace."""
    import torch

    inputs = list(inputs)
    if len(inputs) != len(upd.params):
        raise ValueError("one input per parameter is required")
    for x, p in zip(inputs, upd.params):
        if x.shape != p.shape or x.dtype != p.dtype or not x.is_contiguous() or x.device != p.device:
            raise ValueError("inputs must match their parameters in shape, dtype and device")
    st = torch.cuda.current_stream(upd.params[0].device) if stream is None else stream
    return upd.plan.ns_cv_trace_ptr([x.data_ptr() for x in inputs], kmax, upd.workspace.data_ptr(),
                                    upd.workspace.numel(), st.cuda_stream)


class AuxUpdate(ParamUpdate):
    """Remaining 2D parameters (token embedding, LM head): two-sided normalization."""

    kind = PARAM_AUX


class VectorUpdate(ParamUpdate):
    """1-D parameters (norm weights, biases): global-RMS normalization."""

    kind = PARAM_VECTOR
