"""Host-side checks of bench.py: the flop and byte models behind its roofline figures, the
selection of timed-region dispatches from a profiler trace, and the one-GPU contract."""
import csv
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
import workloads  # noqa: E402


def _products(s, l, segs):
    """Every matrix product of a Newton-Schulz schedule as (m, n, k, symmetric output), listed
    step by step: a segment of j steps forms A = X X^T, then per step P = p(A) (A A), the A
    update P (P A) except after the last step, Q <- P Q from the second step on, and at the end
    X <- Q X (eq. "ns" regrouped; a one-step segment is the printed step)."""
    ops = []
    for j in segs:
        ops.append((s, s, l, True))           # A = X X^T
        for t in range(j):
            ops.append((s, s, s, True))       # A A inside p(A)
            if t < j - 1:
                ops.append((s, s, s, True))   # T = P A
                ops.append((s, s, s, True))   # A <- P T
            if t > 0:
                ops.append((s, s, s, True))   # Q <- P Q
        ops.append((s, l, s, False))          # X <- Q X
    return ops


def _count(ops):
    # a symmetric output is counted once: half of the dense 2 m n k
    return sum(m * n * k if sym else 2 * m * n * k for m, n, k, sym in ops)


@pytest.mark.parametrize("s,l,segs", [(2048, 8192, [3, 2]), (512, 2048, [3, 2]), (2048, 2048, [1] * 5),
                                      (64, 640, [2, 2, 1]), (96, 96, [3]), (128, 384, [1, 3, 1])])
def test_ns_flops_matches_enumerated_products(s, l, segs):
    fl = bench.ns_flops(s, l, segs)
    assert fl["total"] == _count(_products(s, l, segs))
    assert fl["gram"] + fl["apply"] == len(segs) * 3 * s * s * l
    # the closed form of a j-step segment, (3 r + 4 j - 3) s^3 with r = l / s
    assert fl["total"] * s == sum((3 * l + (4 * j - 3) * s) * s ** 3 for j in segs)
    # the printed iteration's counts do not depend on the schedule
    steps = sum(segs)
    assert fl["printed"] == _count(_products(s, l, [1] * steps))
    assert fl["dense"] == steps * (4 * s * s * l + 2 * s ** 3)


def test_ns_flops_of_the_1b_step():
    wl = workloads.workload("llama-1b")
    sched = {(2048, 2048): [1] * 5, (512, 2048): [3, 2], (2048, 8192): [3, 2]}
    tot = {"total": 0, "printed": 0, "dense": 0}
    for m in wl.matrices:
        s, l = min(m.rows, m.cols), max(m.rows, m.cols)
        fl = bench.ns_flops(s, l, sched[(s, l)])
        for k in tot:
            tot[k] += fl[k]
    assert round(tot["total"] / 1e12, 2) == 21.33
    assert round(tot["printed"] / 1e12, 2) == 32.58
    assert round(tot["dense"] / 1e12, 2) == 45.74


def test_stage_bytes_per_element():
    n = 1000
    bf = bench.stage_bytes(n, 2, False)
    assert bf == {"momentum": 12 * n, "update": 6 * n}
    f32 = bench.stage_bytes(n, 4, True)
    assert f32 == {"momentum": 14 * n, "update": 10 * n, "rowcol": 2 * n}


def test_breakdown_steps():
    assert [bench.breakdown_steps(k) for k in (1, 3, 10, 20, 100)] == [1, 3, 10, 10, 10]


def test_timed_region_average_takes_the_main_plans_timed_dispatches(tmp_path):
    # 2 warm-up and 3 timed steps with 2 apply launches each, then a later leg; another kernel
    # interleaved; rows deliberately out of order
    rows = []
    t = 0
    for i in range(14):
        rows.append({"Kernel_Name": "void meq::(anonymous namespace)::k_ns_gemm<2, false>(meq::GemmArgs)",
                     "Start_Timestamp": t, "End_Timestamp": t + 1_000_000 * (i + 1)})
        rows.append({"Kernel_Name": "void meq::(anonymous namespace)::k_ns_gemm<0, false>(meq::GemmArgs)",
                     "Start_Timestamp": t + 5, "End_Timestamp": t + 7})
        t += 100_000_000
    path = tmp_path / "trace.csv"
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        w.writerows(reversed(rows))
    line = {"warmup": 2, "steps": 3, "roofline": {"launches_per_step": 2.0}}
    avg, n = bench.timed_region_average(str(path), line)
    assert n == 6
    assert avg == pytest.approx(sum(range(5, 11)) / 6)  # dispatches 4 .. 9 last 5 .. 10 ms


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
