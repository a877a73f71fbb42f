"""Address-range checks of every kernel launch the planner enqueues (test infrastructure).

`check_plan` builds a plan in the host-check library (the planner linked with recording
launchers), runs meq_step once with fake device addresses, and checks the recorded ranges:

- every range lies inside one buffer: the workspace (below meq_workspace_bytes) or the caller's
  parameter, gradient or momentum of the right matrix and kind;
- within one launch no written range overlaps any other range of that launch (no read/write
  or write/write race between matrices, groups or operands);
- every workspace byte a launch reads was written earlier in the same step (no stale or
  uninitialized workspace is read, which the zero-padding argument of the GEMMs relies on);
- the momentum kernel writes the whole zero-padded wide buffer of every matrix (S x L).
"""
from __future__ import annotations

import ctypes
from typing import Sequence, Tuple

from paper_2609_35701_amd import meq

WS_BASE = 1 << 44
PARAM_BASE, GRAD_BASE, MOM_BASE = 2 << 44, 3 << 44, 4 << 44
SLOT = 1 << 34  # address space per caller buffer (16 GiB: the largest matrix, 1024 matrices per kind)

READ, WRITE, READ_WRITE, BOUND = 0, 1, 2, 3  # BOUND: a direction-dependent extent, buffer check only
WHAT = ("G", "B", "X", "part", "scal", "fold", "A", "Bop", "C", "E", "rpart", "cpart", "U", "rrms", "crms",
        "scale", "W", "rscale", "cscale", "normsq")
CALLER = {"G": GRAD_BASE, "B": MOM_BASE, "W": PARAM_BASE}


def load(path: str) -> ctypes.CDLL:
    L = ctypes.CDLL(path)
    vp, i32, i64, u64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_size_t
    L.meq_init_kind.argtypes = [i32, ctypes.POINTER(meq.MatrixDesc), i32, ctypes.POINTER(meq.HParams),
                                ctypes.POINTER(vp)]
    L.meq_init_kind.restype = i32
    L.meq_init_capped.argtypes = [i32, ctypes.POINTER(meq.MatrixDesc), i32, ctypes.POINTER(meq.HParams), sz,
                                  ctypes.POINTER(vp)]
    L.meq_init_capped.restype = i32
    L.meq_plan_num_passes.argtypes = [vp]
    L.meq_plan_num_passes.restype = i32
    L.meq_workspace_bytes.argtypes = [vp]
    L.meq_workspace_bytes.restype = sz
    L.meq_step.argtypes = [vp, ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.c_float, vp, sz, vp]
    L.meq_step.restype = i32
    L.meq_destroy.argtypes = [vp]
    L.meq_destroy.restype = None
    L.meq_default_hparams.argtypes = [ctypes.POINTER(meq.HParams)]
    L.meq_default_hparams.restype = None
    L.meq_plan_num_groups.argtypes = [vp]
    L.meq_plan_num_groups.restype = i32
    L.meq_plan_group.argtypes = [vp, i32, ctypes.POINTER(i64), ctypes.POINTER(i64), ctypes.POINTER(i32)]
    L.meq_plan_group.restype = i32
    L.meq_hc_clear.argtypes = []
    L.meq_hc_clear.restype = None
    L.meq_hc_num_ranges.restype = i32
    L.meq_hc_num_launches.restype = i32
    L.meq_hc_range.argtypes = [i32, ctypes.POINTER(i32), ctypes.POINTER(u64), ctypes.POINTER(u64)]
    L.meq_hc_range.restype = i32
    L.meq_hc_num_covers.restype = i32
    L.meq_hc_cover.argtypes = [i32, ctypes.POINTER(i32), ctypes.POINTER(u64), ctypes.POINTER(i64)]
    L.meq_hc_cover.restype = i32
    return L


def _hparams(L, **over) -> meq.HParams:
    hp = meq.HParams()
    L.meq_default_hparams(ctypes.byref(hp))
    for k, v in over.items():
        setattr(hp, k, v)
    return hp


def _ranges(L):
    out = []
    f = (ctypes.c_int32 * 5)()
    lo, hi = ctypes.c_uint64(), ctypes.c_uint64()
    for i in range(L.meq_hc_num_ranges()):
        assert L.meq_hc_range(i, f, ctypes.byref(lo), ctypes.byref(hi)) == 0
        out.append((f[0], f[1], f[2], f[3], WHAT[f[4]], lo.value, hi.value))
    return out


def _covers(L):
    out = []
    li = (ctypes.c_int32 * 2)()
    base = ctypes.c_uint64()
    rcl = (ctypes.c_int64 * 3)()
    for i in range(L.meq_hc_num_covers()):
        assert L.meq_hc_cover(i, li, ctypes.byref(base), rcl) == 0
        out.append((li[0], li[1], base.value, rcl[0], rcl[1], rcl[2]))
    return out


def _merge(intervals):
    out = []
    for lo, hi in sorted(intervals):
        if out and lo <= out[-1][1]:
            out[-1][1] = max(out[-1][1], hi)
        else:
            out.append([lo, hi])
    return out


def _covered(merged, lo, hi) -> bool:
    import bisect

    i = bisect.bisect_right([m[0] for m in merged], lo) - 1
    return i >= 0 and merged[i][0] <= lo and hi <= merged[i][1]


def record_step(L, kind: int, shapes: Sequence[Tuple[int, int]], dtype: str = "bf16", max_ws: int = 0,
                **hp_over) -> dict:
    """Build a plan in the host-check library (workspace capped at max_ws bytes unless 0) and record
    one meq_step with fake device addresses."""
    dt = meq.MEQ_BF16 if dtype == "bf16" else meq.MEQ_F32
    n = len(shapes)
    descs = (meq.MatrixDesc * max(n, 1))(*[meq.MatrixDesc(r, c, dt, dt) for r, c in shapes])
    hp = _hparams(L, **hp_over)
    h = ctypes.c_void_p()
    st = L.meq_init_capped(kind, descs, n, ctypes.byref(hp), max_ws, ctypes.byref(h))
    assert st == meq.MEQ_OK, f"init {st}"
    try:
        ws_bytes = L.meq_workspace_bytes(h)
        passes = L.meq_plan_num_passes(h)
        assert max_ws == 0 or ws_bytes <= max_ws, f"workspace {ws_bytes} above the cap {max_ws}"
        params = (ctypes.c_void_p * n)(*[PARAM_BASE + i * SLOT for i in range(n)])
        grads = (ctypes.c_void_p * n)(*[GRAD_BASE + i * SLOT for i in range(n)])
        moms = (ctypes.c_void_p * n)(*[MOM_BASE + i * SLOT for i in range(n)])
        L.meq_hc_clear()
        st = L.meq_step(h, params, grads, moms, ctypes.c_float(0.02), ctypes.c_void_p(WS_BASE), ws_bytes, None)
        assert st == meq.MEQ_OK, f"step {st}"
        return {"kind": kind, "shapes": list(shapes), "esz": 2 if dtype == "bf16" else 4, "ws_bytes": ws_bytes,
                "passes": passes,
                "ranges": _ranges(L), "covers": _covers(L), "launches": L.meq_hc_num_launches()}
    finally:
        L.meq_destroy(h)


def check_record(rec: dict, label: str = "") -> dict:
    """Check a recorded step (see the module docstring); raises AssertionError on the first violation."""
    shapes, esz, ws_bytes, n = rec["shapes"], rec["esz"], rec["ws_bytes"], len(rec["shapes"])
    ranges, covers, launches = rec["ranges"], rec["covers"], rec["launches"]

    def owner(r):
        lo, hi = r[5], r[6]
        if WS_BASE <= lo and hi <= WS_BASE + ws_bytes:
            return ("ws", None)
        for name, base in CALLER.items():
            if base <= lo < base + n * SLOT:
                i = (lo - base) // SLOT
                m, c = shapes[i]
                size = m * c * (4 if name == "B" else esz)
                start = base + i * SLOT
                if lo >= start and hi <= start + size:
                    return (name, i)
        return None

    by_launch = {}
    for r in ranges:
        o = owner(r)
        assert o is not None, f"{label}: launch {r[0]} kernel {r[1]} operand {r[4]} item {r[3]} " \
                              f"[{r[5]:#x}, {r[6]:#x}) outside every buffer (workspace {ws_bytes} bytes)"
        assert r[6] > r[5], f"{label}: empty range {r}"
        if o[0] != "ws":
            assert r[4] == o[0], f"{label}: operand {r[4]} touches the caller's {o[0]} buffer"
        if r[2] != BOUND:
            by_launch.setdefault(r[0], []).append((r, o))
    # no write overlaps another range of the same launch
    for lid, rs in by_launch.items():
        for w, _ in rs:
            if w[2] == READ:
                continue
            for r, _ in rs:
                if r is not w and r[5] < w[6] and w[5] < r[6]:
                    raise AssertionError(f"{label}: launch {lid}: {w[4]} of item {w[3]} (written) overlaps "
                                         f"{r[4]} of item {r[3]}")
    # reads of the workspace only after writes within the step
    written, stale = [], []
    for lid in range(launches):
        merged = _merge(written)
        for r, o in by_launch.get(lid, []):
            if o[0] == "ws" and r[2] != WRITE and not _covered(merged, r[5], r[6]):
                stale.append((lid, r[4], r[3]))
        for r, o in by_launch.get(lid, []):
            if o[0] == "ws" and r[2] != READ:
                written.append((r[5], r[6]))
    assert not stale, f"{label}: workspace read before written: {stale[:5]}"
    # the padded wide buffers are written whole
    if rec["kind"] == meq.PARAM_HIDDEN:
        assert len(covers) == n, f"{label}: {len(covers)} momentum covers for {n} matrices"
        want = sorted((-(-min(r, c) // 256) * 256, -(-max(r, c) // 256) * 256) for r, c in shapes)
        got = sorted((rows, cols) for _, _, _, rows, cols, _ in covers)
        assert got == want, f"{label}: padded covers {got[:4]} vs {want[:4]}"
        for _, _, _, rows, cols, ld in covers:
            assert ld == cols, f"{label}: leading dimension {ld} of a {rows} x {cols} buffer"
    # every matrix's parameter is written exactly once per step, whatever the passes
    if rec["kind"] == meq.PARAM_HIDDEN:
        wr = sorted((r[5] - PARAM_BASE) // SLOT for r in ranges if r[4] == "W" and r[2] != READ)
        assert wr == list(range(n)), f"{label}: parameters written {wr[:8]}... for {n} matrices"
    return {"launches": launches, "ranges": len(ranges), "ws_bytes": ws_bytes}


def check_plan(L, kind: int, shapes: Sequence[Tuple[int, int]], dtype: str = "bf16", label: str = "",
               max_ws: int = 0, **hp_over) -> dict:
    """Record one step of a plan and check every launch's ranges; returns a summary."""
    rec = record_step(L, kind, shapes, dtype, max_ws, **hp_over)
    out = check_record(rec, label)
    out["passes"] = rec["passes"]
    return out
