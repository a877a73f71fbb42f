"""The planner on the host, without a GPU: every launch of a step, for every workload and odd or
extreme shape, stays inside the caller's buffers and the workspace, no launch writes what it or a
neighbour reads, and the workspace is never read before it is written (the GEMMs have no bounds
checks and rely on this layout).  The same checks and the ABI host tests also run against a build of
the planner with AddressSanitizer and UndefinedBehaviorSanitizer.

The host-check library is the planner (meq_api.cpp) linked with recording launchers
(tests/hostcheck/launch_record.cpp) instead of the HIP kernels, built with g++."""
import os
import subprocess
import sys

import pytest

import workloads
from paper_2609_35701_amd import meq

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, os.path.join(HERE, "hostcheck"))
import build_hostcheck  # noqa: E402
import footprints  # noqa: E402

ODD_SHAPES = [(7, 5), (1, 300), (300, 1), (65, 257), (257, 65), (1000, 1000), (2736, 1024), (1024, 2736),
              (255, 257), (513, 4097)]
LARGEST = [(256, 65536), (65536, 256), (16384, 65280), (4096, 65536)]


@pytest.fixture(scope="module")
def hc(tmp_path_factory):
    path = str(tmp_path_factory.mktemp("hostcheck") / "libmeq_hostcheck.so")
    build_hostcheck.build(path, sanitize=False)
    return footprints.load(path)


@pytest.mark.parametrize("name", workloads.WORKLOAD_NAMES)
def test_named_workloads(hc, name):
    wl = workloads.workload(name)
    shapes = [(m.rows, m.cols) for m in wl.matrices]
    footprints.check_plan(hc, meq.PARAM_HIDDEN, shapes, wl.param_dtype, name)


@pytest.mark.parametrize("over", [{}, {"ns_gram_steps": 1}, {"ns_gram_steps": 2}, {"nesterov": 1},
                                  {"update_rule": meq.RULE_MOONLIGHT}, {"ns_steps": 7},
                                  {"ns_a": 2.0, "ns_b": -0.5, "ns_c": 0.0}])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_odd_shapes_and_schedules(hc, over, dtype):
    footprints.check_plan(hc, meq.PARAM_HIDDEN, ODD_SHAPES, dtype, f"odd {dtype} {over}", **over)


def test_largest_shapes(hc):
    for shape in LARGEST:
        footprints.check_plan(hc, meq.PARAM_HIDDEN, [shape, shape], "bf16", f"largest {shape}")


def test_many_matrices_span_several_launch_chunks(hc):
    shapes = [(64 + 8 * (i % 5), 96 + 16 * (i % 3)) for i in range(300)]
    footprints.check_plan(hc, meq.PARAM_HIDDEN, shapes, "bf16", "300 matrices")
    footprints.check_plan(hc, meq.PARAM_HIDDEN, shapes[:140] + [(2, 3)] * 140, "f32", "280 matrices")


@pytest.mark.parametrize("name,cap_mib", [("llama-1b", 256), ("llama-1b", 128), ("llama-130m", 64),
                                          ("llama-7b-block-x4", 512), ("llama-350m-ffn2736", 100)])
def test_capped_plans(hc, name, cap_mib):
    wl = workloads.workload(name)
    shapes = [(m.rows, m.cols) for m in wl.matrices]
    out = footprints.check_plan(hc, meq.PARAM_HIDDEN, shapes, wl.param_dtype, f"{name} cap {cap_mib} MiB",
                                max_ws=cap_mib << 20)
    assert out["ws_bytes"] <= cap_mib << 20 and out["passes"] > 1


def test_capped_odd_shapes(hc):
    out = footprints.check_plan(hc, meq.PARAM_HIDDEN, ODD_SHAPES * 3, "f32", "odd capped", max_ws=24 << 20,
                                ns_gram_steps=2)
    assert out["passes"] > 1


def test_aux_and_vector_plans(hc):
    footprints.check_plan(hc, meq.PARAM_AUX, [(32000, 2048), (300, 64), (1, 1), (7, 5)], "bf16", "aux")
    footprints.check_plan(hc, meq.PARAM_AUX, [(129, 65536), (1, 3)], "f32", "aux f32", nesterov=1)
    footprints.check_plan(hc, meq.PARAM_VECTOR, [(1, 2048)] * 33 + [(1, 1), (3, 7)], "bf16", "vector")
    footprints.check_plan(hc, meq.PARAM_VECTOR, [(1, 5)] * 200, "f32", "vector chunks", nesterov=1)


def _plant(rec, pick, change):
    """A copy of a recorded step with one range changed."""
    out = dict(rec)
    rs = list(rec["ranges"])
    i = next(k for k, r in enumerate(rs) if pick(r))
    rs[i] = change(rs[i])
    out["ranges"] = rs
    return out


def test_checker_catches_planted_layout_mistakes(hc):
    """The checker itself, on a recorded 1B-shape step with one planted mistake each."""
    wl = workloads.workload("llama-1b")
    rec = footprints.record_step(hc, meq.PARAM_HIDDEN, [(m.rows, m.cols) for m in wl.matrices], "bf16")
    footprints.check_record(rec, "as recorded")
    ws_end = footprints.WS_BASE + rec["ws_bytes"]
    plants = {
        # the last workspace region read one byte past the end of the workspace
        "past the workspace": _plant(rec, lambda r: r[4] == "scale" and r[2] == footprints.READ,
                                     lambda r: r[:5] + (ws_end - 4, ws_end + 1)),
        # a GEMM output moved onto its own operand
        "output over operand": _plant(rec, lambda r: r[4] == "C" and r[1] == 4,
                                      lambda r: r[:5] + (r[5] - 4096, r[6] - 4096)),
        # the momentum kernel no longer writing a matrix's padded V
        "stale X": _plant(rec, lambda r: r[4] == "X", lambda r: r[:2] + (footprints.READ,) + r[3:]),
        # a gradient read one element past its buffer
        "past a gradient": _plant(rec, lambda r: r[4] == "G", lambda r: r[:6] + (r[6] + 2,)),
    }
    for what, bad in plants.items():
        with pytest.raises(AssertionError):
            footprints.check_record(bad, what)
    short = dict(rec)
    short["covers"] = rec["covers"][:-1] + [rec["covers"][-1][:3] + (rec["covers"][-1][3] - 256,) +
                                            rec["covers"][-1][4:]]
    with pytest.raises(AssertionError):
        footprints.check_record(short, "short cover")


def test_planner_and_abi_tests_under_sanitizers(tmp_path):
    """The ABI host tests and the range checks, against the planner built with AddressSanitizer and
    UndefinedBehaviorSanitizer (errors abort the run)."""
    path = str(tmp_path / "libmeq_hostcheck_asan.so")
    build_hostcheck.build(path, sanitize=True)
    env = dict(os.environ)
    env["LD_PRELOAD"] = build_hostcheck.sanitizer_preload()
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    driver = (
        "import sys; sys.path.insert(0, %r); sys.path.insert(0, %r)\n"
        "from paper_2609_35701_amd import meq\n"
        "meq.LIB_PATH = %r\n"
        "import pytest\n"
        "sys.exit(pytest.main(['-q', '-p', 'no:cacheprovider', %r, '-k', 'not exports_every_header_symbol']))\n"
        "" % (ROOT, os.path.join(HERE, "hostcheck"), path, os.path.join(HERE, "test_abi_host.py")))
    res = subprocess.run([sys.executable, "-c", driver], cwd=ROOT, env=env, stdout=subprocess.PIPE,
                         stderr=subprocess.STDOUT, text=True, timeout=600)
    assert res.returncode == 0, res.stdout[-4000:]
    driver2 = (
        "import sys; sys.path.insert(0, %r); sys.path.insert(0, %r)\n"
        "import footprints, workloads\n"
        "from paper_2609_35701_amd import meq\n"
        "L = footprints.load(%r)\n"
        "for name in ('llama-1b', 'llama-130m', 'single-256x512'):\n"
        "    wl = workloads.workload(name)\n"
        "    footprints.check_plan(L, meq.PARAM_HIDDEN, [(m.rows, m.cols) for m in wl.matrices], wl.param_dtype, name)\n"
        "footprints.check_plan(L, meq.PARAM_HIDDEN, %r, 'bf16', 'odd', ns_gram_steps=2)\n"
        "footprints.check_plan(L, meq.PARAM_AUX, [(300, 64), (7, 5)], 'f32', 'aux')\n"
        "footprints.check_plan(L, meq.PARAM_VECTOR, [(1, 64), (1, 1000)], 'bf16', 'vec')\n"
        "print('sanitized range checks ok')\n" % (ROOT, os.path.join(HERE, "hostcheck"), path, ODD_SHAPES))
    res = subprocess.run([sys.executable, "-c", driver2], cwd=ROOT, env=env, stdout=subprocess.PIPE,
                         stderr=subprocess.STDOUT, text=True, timeout=600)
    assert res.returncode == 0 and "sanitized range checks ok" in res.stdout, res.stdout[-4000:]
