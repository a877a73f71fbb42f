"""Benchmark: MeqMuon steps/s over all hidden 2D weights of the 1B shape on one MI355X.

One step = one meq_step over all 112 hidden matrices of the 1B-shape Llama
(16 layers, d 2048, ffn 8192, GQA 32/8 heads of dim 64): momentum, Newton-Schulz
(5 steps, bf16 MFMA), row/column equilibration and the write-back, bf16 weights
and gradients, fp32 momentum, inputs resident in HBM.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "MeqMuon steps/sec over all hidden 2D weights (1B shape); NS MFMA %, norm GB/s"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
GEMM_SOURCE = os.path.join(ROOT, "paper_2609_35701_amd", "csrc", "k_ns_gemm.hip")
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "k_ns_gemm_apply_llama1b_traffic.md")
CALIBRATION_BYTES = 256 << 20  # the plain copy kernel of known size: 256 MiB read + 256 MiB written
CALIBRATION_KERNEL = "neg_kernel"  # torch.neg on fp32 is the copy (one read, one write per element)
# Kernel instantiations of the NS products: template mode (0 symmetric NT, 1 poly, 2 apply) and
# operand format (fp16 for the Gram-space products).
APPLY_KERNEL = "k_ns_gemm<2, false>"
NS_KERNELS = ("k_ns_gemm<0, false>", "k_ns_gemm<0, true>", "k_ns_gemm<1, false>", "k_ns_gemm<1, true>",
              APPLY_KERNEL)


def gemm_source_hash() -> str:
    with open(GEMM_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def recorded_traffic(workload: str):
    """HBM bytes per apply launch from the committed counter summary, or None when that summary
    is missing, was taken on another workload or on another version of the GEMM source."""
    if workload != "llama-1b" or not os.path.exists(TRAFFIC_PROFILE):
        return None
    fields = {}
    with open(TRAFFIC_PROFILE) as f:
        for line in f:
            m = re.match(r"^- (\w+): (\S+)\s*$", line)
            if m:
                fields[m.group(1)] = m.group(2)
    if fields.get("kernel_source_sha256") != gemm_source_hash():
        return None
    try:
        return float(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _kernel_key(name: str) -> str:
    if CALIBRATION_KERNEL in name:
        return CALIBRATION_KERNEL
    m = re.search(r"meq::(?:\(anonymous namespace\)::)?(k_\w+(<[^>]*>)?)\(", name)
    if m:
        return m.group(1)
    return "torch: " + name.split("<")[0][:50]


def _counter_means(run_dir: str, counter: str):
    """Mean value of one rocprofv3 --pmc counter per dispatch, by kernel."""
    path = os.path.join(run_dir, "run_counter_collection.csv")
    tot, disp = {}, {}
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            k = _kernel_key(r["Kernel_Name"])
            tot[k] = tot.get(k, 0.0) + float(r["Counter_Value"])
            disp.setdefault(k, set()).add(r["Dispatch_Id"])
    return {k: (tot[k] / len(disp[k]), len(disp[k])) for k in tot}


def summarize_traffic(fetch_dir: str, write_dir: str, out: str, fetch_cmd: str, write_cmd: str) -> None:
    """Write the apply kernel's HBM traffic summary from two counter runs (FETCH_SIZE, WRITE_SIZE).

    Both counters are in KiB per dispatch.  Each is divided by what it reads, per byte, for the
    calibration copy of known size, so the result is in bytes the copy would have moved."""
    fe = _counter_means(fetch_dir, "FETCH_SIZE")
    wr = _counter_means(write_dir, "WRITE_SIZE")
    cf = fe[CALIBRATION_KERNEL][0] * 1024 / CALIBRATION_BYTES
    cw = wr[CALIBRATION_KERNEL][0] * 1024 / CALIBRATION_BYTES
    rows = []
    for k in sorted(set(fe) | set(wr)):
        f_kib, n = fe.get(k, (float("nan"), 0))
        w_kib, _ = wr.get(k, (float("nan"), 0))
        rows.append((k, n, f_kib, w_kib, f_kib * 1024 / cf + w_kib * 1024 / cw))
    apply = [r for r in rows if r[0] == APPLY_KERNEL][0]
    lines = [
        "# HBM traffic per dispatch (rocprofv3 FETCH_SIZE / WRITE_SIZE), llama-1b step\n\n",
        "Commands (from the repository root on one MI355X; each counter in a run of its own):\n\n",
        f"    {fetch_cmd}\n    {write_cmd}\n\n",
        "Summarised with `python bench.py --summarize-traffic <fetch dir> <write dir> --out <this file>`.\n",
        f"Calibration: torch.neg over {CALIBRATION_BYTES >> 20} MiB of fp32 (one read and one write of "
        f"{CALIBRATION_BYTES >> 20} MiB) reads FETCH_SIZE {fe[CALIBRATION_KERNEL][0]:.0f} KiB and WRITE_SIZE "
        f"{wr[CALIBRATION_KERNEL][0]:.0f} KiB, i.e. factors {cf:.4f} (fetch) and {cw:.4f} (write) per byte moved; "
        "kernel figures below are divided by these factors.\n\n",
        "| kernel | dispatches | FETCH_SIZE KiB/dispatch | WRITE_SIZE KiB/dispatch | calibrated bytes/dispatch |\n",
        "|---|---|---|---|---|\n",
    ]
    for k, n, f_kib, w_kib, b in rows:
        lines.append(f"| {k} | {n} | {f_kib:.0f} | {w_kib:.0f} | {b:.4g} |\n")
    lines += [
        f"\nRecorded for the benchmark's roofline (apply product, {APPLY_KERNEL}):\n\n",
        f"- traffic_bytes_per_launch: {apply[4]:.6g}\n",
        f"- kernel_source_sha256: {gemm_source_hash()}\n",
    ]
    with open(out, "w") as f:
        f.write("".join(lines))


def breakdown_steps(steps: int) -> int:
    """Steps of the per-kernel breakdown pass that follows the timed region."""
    return max(1, min(steps, 10))


def timed_region_average(trace_csv: str, line: dict, kernel: str = APPLY_KERNEL) -> tuple:
    """Average duration (ms) and count of `kernel`'s dispatches inside the benchmark's timed region,
    from a rocprofv3 kernel trace of the same run: the main plan runs warmup + steps steps first,
    with roofline.launches_per_step launches of the kernel each; later legs follow them."""
    with open(trace_csv) as f:
        rows = [r for r in csv.DictReader(f) if _kernel_key(r["Kernel_Name"]) == kernel]
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    per = int(round(line["roofline"]["launches_per_step"]))
    lo, hi = line["warmup"] * per, (line["warmup"] + line["steps"]) * per
    durs = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e6 for r in rows[lo:hi]]
    return sum(durs) / len(durs), len(durs)


def summarize_stats(stats_csv: str, out: str, command: str, note: str, trace_csv: str = None,
                    bench_json: str = None) -> None:
    """Markdown table of a rocprofv3 --kernel-trace --stats run; with the run's kernel trace and
    bench line, also the apply kernel's timed-region average next to the bench's HIP-event figure."""
    with open(stats_csv) as f:
        rows = list(csv.DictReader(f))

    def short(n):
        n = re.sub(r"\(anonymous namespace\)::", "", n)
        if "at::native" in n:
            return "torch: " + n.split("<")[0][:60]
        return n[:90]

    lines = ["# rocprofv3 kernel stats\n\n", "Command (from the repository root on one MI355X):\n\n",
             f"    {command}\n\n"]
    if note:
        lines.append(note + "\n\n")
    if trace_csv and bench_json:
        with open(bench_json) as f:
            line = json.loads([x for x in f if x.startswith("{")][-1])
        avg, n = timed_region_average(trace_csv, line)
        lines.append(
            f"Timed region of the same run (summarised with `python bench.py --summarize-stats <stats csv> "
            f"--trace <trace csv> --bench-json <bench line> --out <this file>`): {line['steps']} steps after "
            f"{line['warmup']} warm-up steps, {line['ms_per_step']:.3f} ms/step under the profiler; the apply "
            f"product {APPLY_KERNEL} launches {line['roofline']['launches_per_step']:g} times per step. Its "
            f"average over the {n} timed-region dispatches in the rocprofv3 trace is {avg:.4f} ms; the "
            f"bench line reports {line['roofline']['avg_launch_ms']:.4f} ms from HIP events on its launch "
            "stream. The table below averages every dispatch of the run, including the legs after the "
            "timed region (other parameter kinds, the Moonlight-Muon rule and the printed iteration on the "
            "same kernels, the library GEMM), so its per-kernel averages mix launch shapes.\n\n")
    lines.append("| kernel | calls | total ms | avg ms | min ms | max ms | % |\n|---|---|---|---|---|---|---|\n")
    for r in rows:
        lines.append(f"| {short(r['Name'])} | {r['Calls']} | {int(r['TotalDurationNs']) / 1e6:.3f} | "
                     f"{float(r['AverageNs']) / 1e6:.4f} | {int(r['MinNs']) / 1e6:.4f} | "
                     f"{int(r['MaxNs']) / 1e6:.4f} | {float(r['Percentage']):.2f} |\n")
    lines.append(f"\nkernel_source_sha256: {gemm_source_hash()}\n")
    with open(out, "w") as f:
        f.write("".join(lines))


MFMA_COUNTERS = ("GRBM_GUI_ACTIVE", "SQ_BUSY_CYCLES", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU_MFMA_MOPS_BF16",
                 "SQ_INSTS_VALU_MFMA_MOPS_F16")
SIMDS = 256 * 4  # MI355X: 256 compute units of 4 SIMDs
XCDS = 8


def ns_launch_flops(wl) -> dict:
    """Per step, for each NS kernel instantiation over all shape groups: (algorithmic symmetric-aware
    flops, flops of the 256 x 256 tiles by count, padding and the lower half of diagonal tiles
    included), under the default schedule and coefficients: X X^T runs in k_ns_gemm<0, false>
    (bf16 X, fp16 output), the Gram-space products in k_ns_gemm<0, true> and every polynomial in
    k_ns_gemm<1, true> (fp16 A); k_ns_gemm<1, false> only runs for coefficients that fail the fp16
    range check."""
    from paper_2609_35701_amd import meq

    plan = meq.Plan([(m.rows, m.cols) for m in wl.matrices], wl.param_dtype)
    segs = {(s, l): plan.schedule(g) for g, (s, l, _) in enumerate(plan.groups())}
    out = {k: [0, 0] for k in NS_KERNELS}
    for m in wl.matrices:
        s, l = min(m.rows, m.cols), max(m.rows, m.cols)
        sp, lp = -(-s // 256) * 256, -(-l // 256) * 256
        tm, tl = sp // 256, lp // 256
        tri = tm * (tm + 1) // 2
        sg = segs[(s, l)]
        nseg = len(sg)
        nsprod = sum(3 * (j - 1) for j in sg)
        poly16 = sum(sg)
        poly_bf = 0
        for k, alg, exe in (("k_ns_gemm<0, false>", nseg * s * s * l, nseg * tri * 2 * 256 * 256 * lp),
                            ("k_ns_gemm<0, true>", nsprod * s ** 3, nsprod * tri * 2 * 256 * 256 * sp),
                            ("k_ns_gemm<1, false>", poly_bf * s ** 3, poly_bf * tri * 2 * 256 * 256 * sp),
                            ("k_ns_gemm<1, true>", poly16 * s ** 3, poly16 * tri * 2 * 256 * 256 * sp),
                            (APPLY_KERNEL, nseg * 2 * s * s * l, nseg * tm * tl * 2 * 256 * 256 * sp)):
            out[k][0] += alg
            out[k][1] += exe
    return out


def _counter_totals(run_dir: str, counter: str):
    """Sum of one rocprofv3 --pmc counter over all dispatches, and the dispatch count, by kernel."""
    return {k: (mean * n, n) for k, (mean, n) in _counter_means(run_dir, counter).items()}


def summarize_mfma(run_dir: str, out: str, command: str, workload: str, note: str, steps: int) -> None:
    """Matrix-core utilisation of the NS products from one rocprofv3 --pmc run of MFMA_COUNTERS
    covering `steps` meq_step calls (warm-up included)."""
    import workloads

    wl = workloads.workload(workload)
    flops = ns_launch_flops(wl)
    tot = {c: _counter_totals(run_dir, c) for c in MFMA_COUNTERS}
    lines = [
        f"# Matrix-core counters of the Newton-Schulz products, {workload} step\n\n",
        "Command (from the repository root on one MI355X):\n\n", f"    {command}\n\n",
        f"Summarised with `python bench.py --summarize-mfma <dir> --profiled-steps {steps} --out <this file>`. "
        f"Per step ({steps} meq_step calls in the run, warm-up included): GRBM_GUI_ACTIVE summed over the 8 XCDs "
        f"(divided by 8: cycles the kernel template was active); SQ_VALU_MFMA_BUSY_CYCLES summed over all {SIMDS} "
        f"SIMDs (divided by {SIMDS} and by the active cycles: fraction of the time a SIMD's matrix core was busy); "
        "SQ_INSTS_VALU_MFMA_MOPS_BF16 (SQ_INSTS_VALU_MFMA_MOPS_F16 for the fp16 instantiations) x 512 = flops "
        "the matrix cores executed, against the flops of the 256 x 256 tiles by count (padding and the "
        "lower half of diagonal tiles of the symmetric products included) and the algorithmic "
        "symmetric-aware flops of the step's schedule. Diagonal tiles of X X^T and of the polynomial's A A "
        "(a matrix times its own transpose) run only the 36 of their 64 32 x 32 blocks on or below OUT's "
        "diagonal, so those two instantiations execute about 0.90 of their tile flops. "
        "k_ns_gemm<0, false> runs X X^T, k_ns_gemm<0, true> the fp16 Gram-space products P A, P T, P Q, "
        "k_ns_gemm<1, *> the polynomial of one-step (bf16) and longer (fp16) segments, "
        "k_ns_gemm<2, false> the X products.\n\n",
        (note + "\n\n" if note else ""),
        "| kernel | dispatches per step | active cycles per step | MFMA busy | MOPS x 512 per step | tile flops "
        "per step | algorithmic flops per step | MOPS x 512 / tile flops |\n",
        "|---|---|---|---|---|---|---|---|\n",
    ]
    for k in NS_KERNELS:
        if k not in tot["GRBM_GUI_ACTIVE"] and flops[k][0] == 0:
            continue  # not launched under the default coefficients
        gui, n = tot["GRBM_GUI_ACTIVE"].get(k, (float("nan"), 0))
        cyc = gui / XCDS / steps
        busy = tot["SQ_VALU_MFMA_BUSY_CYCLES"].get(k, (float("nan"), 0))[0] / SIMDS / steps / cyc
        ctr = "SQ_INSTS_VALU_MFMA_MOPS_F16" if k.endswith("true>") else "SQ_INSTS_VALU_MFMA_MOPS_BF16"
        mops = tot[ctr].get(k, (float("nan"), 0))[0] * 512 / steps
        alg, exe = flops[k]
        lines.append(f"| {k} | {n / steps:.4g} | {cyc:.4g} | {busy:.1%} | {mops:.4g} | {exe:.4g} | {alg:.4g} | "
                     f"{mops / exe:.4f} |\n")
    lines.append(f"\nkernel_source_sha256: {gemm_source_hash()}\n")
    with open(out, "w") as f:
        f.write("".join(lines))


def ns_flops(s: int, l: int, segs) -> dict:
    """Algorithmic Newton-Schulz flops of one s x l matrix (wide orientation) under a schedule
    of Gram-space segments (all ones: eq. "ns" as printed), symmetric products counted once:
    per segment one X X^T (s^2 l) and one X product (2 s^2 l); per step one polynomial
    product (s^3); per segment of j steps 3 (j - 1) products P A, P T, P Q (s^3 each).
    "printed" is the printed iteration's symmetric-aware count K (3 s^2 l + s^3) and "dense"
    its literal dense count K (4 s^2 l + 2 s^3), for any schedule."""
    nseg, steps = len(segs), sum(segs)
    out = {"gram": nseg * s * s * l, "poly": steps * s ** 3, "gram_space": sum(3 * (j - 1) for j in segs) * s ** 3,
           "apply": nseg * 2 * s * s * l}
    out["total"] = sum(out.values())
    out["printed"] = steps * (3 * s * s * l + s ** 3)
    out["dense"] = steps * (4 * s * s * l + 2 * s ** 3)
    return out


def stage_bytes(elems: int, param_bytes: int, rowcol_pass: bool):
    """Algorithmic HBM bytes per element of the byte stages: momentum (G, B read+write, bf16 V),
    row/column sums (U, only when they run as a pass of their own rather than in the last
    apply product's epilogue), write-back (U, W read+write)."""
    out = {"momentum": elems * (param_bytes + 4 + 4 + 2), "update": elems * (2 + 2 * param_bytes)}
    if rowcol_pass:
        out["rowcol"] = elems * 2
    return out


def time_steps(upd, grads, lr: float, steps: int, warmup: int, kinds) -> dict:
    """Wall time per step (no timing events), then per-kind kernel time from a separate pass with
    HIP events on the launch stream around the kernels of `kinds`."""
    import torch

    from paper_2609_35701_amd import meq

    for _ in range(warmup):
        upd.step(grads, lr)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        upd.step(grads, lr)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    out = {"ms_per_step": (t1 - t0) * 1e3 / steps}
    nb = breakdown_steps(steps)
    upd.plan.set_timing(kinds)
    for k in kinds:
        upd.plan.get_timing(k, reset=True)
    for _ in range(nb):
        upd.step(grads, lr)
    torch.cuda.synchronize()
    for k in kinds:
        ms, n = upd.plan.get_timing(k)
        out[meq.KERNEL_NAMES[k] + "_ms"] = ms / nb
    upd.plan.set_timing([])
    return out


def extras_leg(params, wl, lr: float, steps: int, warmup: int) -> dict:
    """The other parameter kinds of the same 1B-shape model, and the Moonlight-Muon rule on its
    hidden weights (same Newton-Schulz kernels, no equilibration)."""
    import torch

    from paper_2609_35701_amd import meq

    dev = params[0].device
    out = {}
    # Moonlight-Muon on the same 112 hidden matrices: the difference to the MeqMuon step is the
    # cost of the row/column statistics, CVs and direction choice
    g_hidden = [torch.randn_like(p) * 1e-3 for p in params]
    moon = meq.HiddenWeightUpdate(params, meq.default_hparams(update_rule=meq.RULE_MOONLIGHT))
    out["moonlight_hidden"] = time_steps(moon, g_hidden, lr, steps, warmup,
                                         [meq.K_ROWCOL, meq.K_SELECT, meq.K_UPDATE])
    # the printed iteration everywhere (no Gram-space segments): what the segments save
    literal = meq.HiddenWeightUpdate(params, meq.default_hparams(ns_gram_steps=1))
    out["printed_iteration_hidden"] = time_steps(literal, g_hidden, lr, steps, warmup,
                                                 [meq.K_GRAM, meq.K_POLY, meq.K_APPLY])
    del moon, literal
    # the same step with the workspace capped to the static scratch size: passes that reuse one
    # Newton-Schulz region (what a caller without a large workspace, or meq_step_static, runs)
    capped = meq.HiddenWeightUpdate(params, max_workspace_bytes=meq.MEQ_STATIC_SCRATCH_BYTES)
    out["capped_workspace_hidden"] = time_steps(capped, g_hidden, lr, steps, warmup, [meq.K_APPLY])
    out["capped_workspace_hidden"].update({"workspace_bytes": capped.plan.workspace_bytes,
                                           "passes": capped.plan.passes})
    del capped
    # the NS-CV trajectory (row and column CVs of X_0 .. X_20 of every hidden matrix, the printed
    # iteration replayed step by step): one call, timed around the whole call
    trace_upd = meq.HiddenWeightUpdate(params)
    meq.ns_cv_trace(trace_upd, g_hidden, 2)  # warm-up
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    meq.ns_cv_trace(trace_upd, g_hidden, 20)
    torch.cuda.synchronize()
    out["ns_cv_trace_hidden"] = {"kmax": 20, "matrices": len(params),
                                 "ms_per_call": (time.perf_counter() - t0) * 1e3,
                                 "note": "20 printed Newton-Schulz steps with CVs after each, host copy of the "
                                         "CVs included"}
    del trace_upd, g_hidden
    torch.cuda.empty_cache()
    # remaining 2D parameters: the Llama token embedding and LM head (32000 x 2048, untied), bf16
    aux_p = [torch.randn(32000, 2048, device=dev).mul_(0.02).to(torch.bfloat16) for _ in range(2)]
    aux_g = [(torch.randn(32000, 2048, device=dev) * torch.rand(32000, 1, device=dev).mul_(3).exp_()
              * 1e-4).to(torch.bfloat16) for _ in range(2)]
    aux = meq.AuxUpdate(aux_p, meq.default_hparams())
    t = time_steps(aux, aux_g, lr, steps, warmup, [meq.K_AUX_ROWS, meq.K_AUX_COLS, meq.K_AUX_UPDATE])
    elems = sum(p.numel() for p in aux_p)
    # bytes per element: rows (G 2, B 4 + 4), columns (B 4), write-back (B 4, W 2 + 2)
    bytes_step = elems * (10 + 4 + 8)
    kern_ms = t["aux_rows_ms"] + t["aux_cols_ms"] + t["aux_update_ms"]
    t.update({"shapes": "2 x 32000x2048 bf16", "bytes_per_step": bytes_step,
              "gbs": bytes_step / (kern_ms * 1e-3) / 1e9,
              "roofline": {"bound": "hbm", "achieved": bytes_step / (kern_ms * 1e-3) / 1e9, "peak": PEAK_HBM_GBS,
                           "unit": "GB/s", "frac": bytes_step / (kern_ms * 1e-3) / 1e9 / PEAK_HBM_GBS}})
    out["aux_two_sided"] = t
    del aux, aux_p, aux_g
    # 1-D parameters: the 33 RMSNorm weights (2 per layer + final), bf16
    vec_p = [torch.ones(2048, device=dev, dtype=torch.bfloat16) for _ in range(2 * 16 + 1)]
    vec_g = [torch.randn(2048, device=dev).mul_(1e-3).to(torch.bfloat16) for _ in vec_p]
    vec = meq.VectorUpdate(vec_p, meq.default_hparams())
    t = time_steps(vec, vec_g, lr, steps, warmup, [meq.K_VECTOR])
    t.update({"shapes": "33 x 2048 bf16", "launches_per_step": 2,
              "note": "latency-bound: 67,584 elements in one or two launches"})
    out["vector_global_rms"] = t
    return out


def library_gemm_leg() -> dict:
    """The platform's library GEMM (hipBLASLt through torch.bmm / torch.mm) on the apply
    product's largest shape group of the 1B step (48 x (2048 x 2048 @ 2048 x 8192), bf16 in and
    out) and on one large square product: what a tuned dense kernel reaches on this chip under
    the same clock and power limits."""
    import torch

    dev = torch.device("cuda:0")
    out = {}

    def rate(f, flops, iters):
        for _ in range(3):
            f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            f()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / iters
        return {"ms": ms, "tflops": flops / (ms * 1e-3) / 1e12}

    p = torch.randn(48, 2048, 2048, device=dev, dtype=torch.bfloat16)
    x = torch.randn(48, 2048, 8192, device=dev, dtype=torch.bfloat16)
    out["bmm_48x2048x2048x8192"] = rate(lambda: torch.bmm(p, x), 2.0 * 48 * 2048 * 2048 * 8192, 10)
    del p, x
    a = torch.randn(8192, 8192, device=dev, dtype=torch.bfloat16)
    b = torch.randn(8192, 8192, device=dev, dtype=torch.bfloat16)
    out["mm_8192_cubed"] = rate(lambda: torch.mm(a, b), 2.0 * 8192 ** 3, 10)
    del a, b
    torch.cuda.empty_cache()
    return out


def _layer_runs(wl):
    """Index ranges of the workload's identical transformer layers (7 matrices each, q k v o gate up
    down), or one range over every matrix when the workload is not a layer stack."""
    per = 7
    if wl.count % per == 0 and wl.count > per:
        shapes = [(m.rows, m.cols) for m in wl.matrices]
        if all(shapes[i] == shapes[i % per] for i in range(wl.count)):
            return [range(i, i + per) for i in range(0, wl.count, per)]
    return [range(wl.count)]


def time_oracle_layers(wl, lr: float, budget_s: float, max_layers: int | None = None):
    """Wall time of the fp64 oracle over whole layers of the workload, one full step of each of their
    matrices in order (momentum from zero, the printed Newton-Schulz iteration in wide orientation,
    row/column equilibration, write-back), layer after layer until `budget_s` is spent or
    `max_layers` are done; inputs are generated outside the timed calls.  Returns (seconds, layers
    timed, layers in the step)."""
    import numpy as np

    import oracle
    import workloads

    hp = oracle.HParams()
    layers = _layer_runs(wl)
    spent, done = 0.0, 0
    for lay in layers:
        if max_layers is not None and done >= max_layers:
            break
        inputs = [(workloads.weight_init(wl, i).astype(np.float64), workloads.grad_at_step(wl, i, 0).astype(np.float64))
                  for i in lay]
        t0 = time.perf_counter()
        for w0, g in inputs:
            oracle.meq_step(w0, g, np.zeros_like(w0), hp, lr, wide=True)
        spent += time.perf_counter() - t0
        done += 1
        if spent > budget_s:
            break
    return spent, done, len(layers)


def blas_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        return max([int(i.get("num_threads", 1)) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover - threadpoolctl missing
        return len(os.sched_getaffinity(0))


def cpu_baseline_leg(wl, lr: float, budget_s: float, full_step: bool = False):
    """The fp64 oracle on the host cores: whole layers of the step (every layer of a Llama stack has
    the same seven shapes, so k of the n layers are k/n of the step's work), or with `full_step`
    every matrix of the step."""
    threads = blas_threads()
    spent, done, total = time_oracle_layers(wl, lr, float("inf") if full_step else budget_s)
    sec_per_step = spent * total / done
    what = (f"the full {wl.count}-matrix step timed whole" if done == total else
            f"{done} of the {total} identical {wl.count // total}-matrix layers timed whole ({spent:.1f} s), "
            f"scaled by {total}/{done} to the full {wl.count}-matrix step")
    return {"value": 1.0 / sec_per_step, "unit": "steps/s", "cores": threads, "kind": "oracle",
            "sample": f"fp64 numpy oracle (printed Newton-Schulz iteration, wide orientation), {what}: "
                      f"{sec_per_step:.1f} s/step",
            "seconds_timed": spent, "layers_timed": done, "layers": total,
            "affinity_cores": len(os.sched_getaffinity(0)), "blas_threads": threads,
            "single_core": single_core_leg(lr)}


def single_core_leg(lr: float) -> dict:
    """The oracle with BLAS limited to one thread: the single 256 x 512 fp32 step whole, and two whole
    layers of the 130M-shape step (12 identical layers) scaled to the step."""
    import numpy as np

    import oracle
    import workloads

    try:
        from threadpoolctl import threadpool_limits
    except Exception:  # pragma: no cover - threadpoolctl missing
        return None
    hp = oracle.HParams()
    out = {}
    with threadpool_limits(limits=1, user_api="blas"):
        wl = workloads.workload("single-256x512")
        w0 = workloads.weight_init(wl, 0).astype(np.float64)
        g = workloads.grad_at_step(wl, 0, 0).astype(np.float64)
        t0 = time.perf_counter()
        oracle.meq_step(w0, g, np.zeros_like(w0), hp, lr)
        out["single-256x512_s_per_step"] = time.perf_counter() - t0
        wl = workloads.workload("llama-130m")
        spent, done, total = time_oracle_layers(wl, lr, float("inf"), max_layers=2)
        out["llama-130m_s_per_step"] = spent * total / done
        out["llama-130m_sample"] = f"{done} of {total} layers timed whole ({spent:.2f} s)"
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama-1b")
    ap.add_argument("--lr", type=float, default=0.02)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the other parameter kinds and the Moonlight-Muon comparison")
    ap.add_argument("--cpu-budget", type=float, default=30.0,
                    help="seconds of oracle work at most: whole layers of the step are timed until it is spent")
    ap.add_argument("--cpu-full-step", action="store_true",
                    help="time the oracle on every matrix of the step (about 90 s for the 1B shapes)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one plain copy kernel of known size (torch.neg over 256 MiB of fp32) before the "
                         "warm-up, as the reference for FETCH_SIZE / WRITE_SIZE counter runs")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) into --out and exit")
    ap.add_argument("--summarize-stats", metavar="STATS_CSV",
                    help="summarise a rocprofv3 --kernel-trace --stats run into --out and exit")
    ap.add_argument("--summarize-mfma", metavar="PMC_DIR",
                    help="summarise a rocprofv3 --pmc run of the matrix-core counters into --out and exit")
    ap.add_argument("--trace", help="rocprofv3 kernel trace csv of the --summarize-stats run")
    ap.add_argument("--bench-json", help="the bench line printed by the --summarize-stats run")
    ap.add_argument("--profiled-steps", type=int, default=3,
                    help="meq_step calls (warm-up included) in the run --summarize-mfma reads")
    ap.add_argument("--out")
    ap.add_argument("--command", default="", help="command line(s) recorded in a summary ('|' separates two)")
    ap.add_argument("--note", default="")
    args = ap.parse_args()
    if args.summarize_traffic:
        cmds = args.command.split("|") + ["", ""]
        summarize_traffic(args.summarize_traffic[0], args.summarize_traffic[1], args.out, cmds[0].strip(),
                          cmds[1].strip())
        return 0
    if args.summarize_stats:
        summarize_stats(args.summarize_stats, args.out, args.command, args.note, args.trace, args.bench_json)
        return 0
    if args.summarize_mfma:
        summarize_mfma(args.summarize_mfma, args.out, args.command, args.workload, args.note, args.profiled_steps)
        return 0
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the MeqMuon update is measured on a single MI355X; "
              f"--gpus {args.gpus} is not supported (multi-GPU sharding is a design note, not built)",
              file=sys.stderr)
        return 2

    import torch

    import workloads
    from paper_2609_35701_amd import meq

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    dev = torch.device("cuda:0")
    wl = workloads.workload(args.workload)
    params, grads, _ = workloads.device_inputs(wl, dev)
    calib = None
    if args.copy_calibration:
        def calib():
            src = torch.ones(CALIBRATION_BYTES // 4, dtype=torch.float32, device=dev)
            dst = torch.empty_like(src)
            torch.neg(src, out=dst)
            torch.cuda.synchronize()
            del src, dst
    res = measure_workload(wl, params, grads, args.steps, args.warmup, args.lr, before_warmup=calib)
    extras = None
    if not args.no_extras and wl.name == "llama-1b":
        print("# bench: other parameter kinds and the Moonlight-Muon rule", file=sys.stderr, flush=True)
        extras = extras_leg(params, wl, args.lr, min(args.steps, 20), max(args.warmup, 1))
        extras["equilibration_overhead_ms"] = res["ms_per_step"] - extras["moonlight_hidden"]["ms_per_step"]
        extras["library_gemm"] = library_gemm_leg()
        del params, grads
        torch.cuda.empty_cache()
        extras["configs"] = configs_leg(res, args.lr, min(args.steps, 20), args.warmup)
    cpu = None
    if not args.no_cpu_baseline:
        print("# bench: timing the fp64 oracle on host cores", file=sys.stderr, flush=True)
        cpu = cpu_baseline_leg(wl, args.lr, args.cpu_budget, args.cpu_full_step)
    line = {
        "metric": METRIC, "value": 1e3 / res["ms_per_step"], "unit": "steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": res["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": res["config"],
        "roofline": res["roofline"], "cpu_baseline": cpu, "stages": res["stages"],
        "kernels_ms_per_step": res["kernels_ms_per_step"],
        "kernels_pass": f"{breakdown_steps(args.steps)} steps after the timed region with HIP events around every kernel",
        "extras": extras,
    }
    print(json.dumps(line), flush=True)
    return 0


def measure_workload(wl, params, grads, steps: int, warmup: int, lr: float, before_warmup=None,
                     tag: str = "bench") -> dict:
    """One workload's hidden-weight step on the GPU: wall time per step over `steps` timed steps (HIP
    events around the dominant X products only), then a breakdown pass with events around every
    kernel, and the flop and byte rates of the step's stages."""
    import torch

    from paper_2609_35701_amd import meq

    print(f"# {tag}: workload {wl.name}, {wl.count} matrices, {wl.elements} elements", file=sys.stderr, flush=True)
    upd = meq.HiddenWeightUpdate(params)
    hp = upd.plan.hparams
    print(f"# {tag}: workspace {upd.plan.workspace_bytes / 2**30:.2f} GiB, groups {upd.plan.groups()}",
          file=sys.stderr, flush=True)
    if before_warmup is not None:
        before_warmup()
    for _ in range(warmup):
        upd.step(grads, lr)
    torch.cuda.synchronize()
    # timed region: HIP events on the launch stream around the dominant kernel (the X product)
    # only; events around every kernel cost about 1% of the step, so the per-kernel breakdown
    # comes from a separate pass after the timed region
    apply_kind = meq.KERNEL_NAMES.index("apply")
    upd.plan.set_timing([apply_kind])
    upd.plan.get_timing(apply_kind, reset=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        upd.step(grads, lr)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    upd.plan.set_timing([])
    ms_per_step = (t1 - t0) * 1e3 / steps
    ap_total_ms, ap_n = upd.plan.get_timing(apply_kind)
    nb = breakdown_steps(steps)
    upd.plan.set_timing(range(len(meq.KERNEL_NAMES)))
    for k in range(len(meq.KERNEL_NAMES)):
        upd.plan.get_timing(k, reset=True)
    torch.cuda.synchronize()
    for _ in range(nb):
        upd.step(grads, lr)
    torch.cuda.synchronize()
    upd.plan.set_timing([])
    kern = {}
    for k, name in enumerate(meq.KERNEL_NAMES):
        ms, n = upd.plan.get_timing(k)
        kern[name] = {"ms_per_step": ms / nb, "launches_per_step": n / nb,
                      "avg_launch_ms": ms / n if n else None}
    print(f"# {tag}: {ms_per_step:.3f} ms/step; breakdown over {nb} more steps: " +
          ", ".join(f"{k} {v['ms_per_step']:.3f}" for k, v in kern.items() if v["launches_per_step"]),
          file=sys.stderr, flush=True)

    sched = {(gs, gl): upd.plan.schedule(g) for g, (gs, gl, _) in enumerate(upd.plan.groups())}
    fl = {}
    for m in wl.matrices:
        s, l = min(m.rows, m.cols), max(m.rows, m.cols)
        for k, v in ns_flops(s, l, sched[(s, l)]).items():
            fl[k] = fl.get(k, 0) + v
    pbytes = 2 if wl.param_dtype == "bf16" else 4
    sb = stage_bytes(wl.elements, pbytes, kern["rowcol"]["launches_per_step"] > 0)
    # timing kinds by kernel template: k_ns_gemm<0, *> runs X X^T and the Gram-space products ("gram")
    kflops = {"gram": fl["gram"] + fl["gram_space"], "poly": fl["poly"], "apply": fl["apply"]}
    ns_kinds = ("gram", "poly", "apply")
    ns_ms = sum(kern[k]["ms_per_step"] for k in ns_kinds)
    # the dominant kernel's figures come from the timed region's own events
    ap_ms = ap_total_ms / steps
    ap_per_step = ap_n / steps
    apply_tflops = fl["apply"] / (ap_ms * 1e-3) / 1e12
    roofline = {"bound": "mfma", "kernel": f"{APPLY_KERNEL} (X <- P X, or Q X after a Gram-space segment; bf16 MFMA)",
                "achieved": apply_tflops, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": apply_tflops / PEAK_BF16_TFLOPS, "traffic": recorded_traffic(wl.name),
                "flops_per_launch": fl["apply"] / max(ap_per_step, 1),
                "launches_per_step": ap_per_step,
                "avg_launch_ms": ap_total_ms / ap_n if ap_n else None}
    stages = {
        "ns_tflops": fl["total"] / (ns_ms * 1e-3) / 1e12,
        "ns_frac_of_peak": fl["total"] / (ns_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
        "ns_tflops_by_kernel": {k: kflops[k] / (kern[k]["ms_per_step"] * 1e-3) / 1e12
                                for k in ns_kinds if kern[k]["ms_per_step"] > 0},
        "ns_printed_equiv_tflops": fl["printed"] / (ns_ms * 1e-3) / 1e12,
        "momentum_gbs": sb["momentum"] / (kern["momentum"]["ms_per_step"] * 1e-3) / 1e9,
        "update_gbs": sb["update"] / (kern["update"]["ms_per_step"] * 1e-3) / 1e9,
        "byte_stages_ms": sum(kern[k]["ms_per_step"] for k in sb),
        "byte_stages_gbs": sum(sb.values()) / (sum(kern[k]["ms_per_step"] for k in sb) * 1e-3) / 1e9,
    }
    if "rowcol" in sb:
        stages["rowcol_gbs"] = sb["rowcol"] / (kern["rowcol"]["ms_per_step"] * 1e-3) / 1e9
    config = {"workload": wl.name, "matrices": wl.count, "elements": wl.elements,
              "param_dtype": wl.param_dtype, "grad_dtype": wl.param_dtype, "momentum_dtype": "f32",
              "ns_steps": hp.ns_steps, "ns_gram_steps": hp.ns_gram_steps,
              "ns_operands": "bf16 X and the P or Q multiplying it; fp16 A = X X^T and Gram-space "
                             "matrices; fp32 accumulation",
              "ns_schedules": {f"{k[0]}x{k[1]}": v for k, v in sched.items()},
              "ns_tflop_per_step": fl["total"] / 1e12,
              "ns_tflop_per_step_printed_sym": fl["printed"] / 1e12,
              "ns_tflop_per_step_printed_dense": fl["dense"] / 1e12}
    del upd
    return {"ms_per_step": ms_per_step, "steps_per_s": 1e3 / ms_per_step, "config": config, "roofline": roofline,
            "stages": stages, "kernels_ms_per_step": {k: v["ms_per_step"] for k, v in kern.items()
                                                      if v["launches_per_step"]}}


# The workloads of the benchmark's table besides the headline: the single 256 x 512 fp32 matrix,
# the 130M and 350M Llama shapes and the 7B block x4 with extreme imbalance.
OTHER_CONFIGS = ("single-256x512", "llama-130m", "llama-350m", "llama-7b-block-x4")


def configs_leg(headline: dict, lr: float, steps: int, warmup: int) -> dict:
    """Every workload of the table on the same build and box: steps/s, the executed-flop NS rate and
    fraction of the bf16 peak, the X product's fraction, and the byte stages' GB/s."""
    import torch

    import workloads

    def row(r):
        st = r["stages"]
        return {"steps_per_s": r["steps_per_s"], "ms_per_step": r["ms_per_step"],
                "ns_tflop_per_step": r["config"]["ns_tflop_per_step"],
                "ns_tflops": st["ns_tflops"], "ns_frac_of_peak": st["ns_frac_of_peak"],
                "ns_tflops_by_kernel": st["ns_tflops_by_kernel"],
                "apply_frac": r["roofline"]["frac"],
                "momentum_gbs": st["momentum_gbs"], "update_gbs": st["update_gbs"],
                "byte_stages_gbs": st["byte_stages_gbs"],
                "byte_stages_frac_of_peak": st["byte_stages_gbs"] / PEAK_HBM_GBS,
                "kernels_ms_per_step": r["kernels_ms_per_step"]}

    out = {"llama-1b": row(headline)}
    dev = torch.device("cuda:0")
    for name in OTHER_CONFIGS:
        wl = workloads.workload(name)
        params, grads, _ = workloads.device_inputs(wl, dev)
        out[name] = row(measure_workload(wl, params, grads, steps, warmup, lr, tag=f"config {name}"))
        del params, grads
        torch.cuda.empty_cache()
    return out


if __name__ == "__main__":
    sys.exit(main())
