"""meq_step_static, the entry point that allocates nothing (its workspace is the library's own
device scratch array), against meq_step with a caller workspace on the same inputs: two calls in a
row on different plans, the second smaller, then a workspace-capped plan of several passes.  The
kernels are the same, so parameters and momenta must match bit for bit."""
import pytest
import torch

import workloads
from gpu_support import log, to_dev
from paper_2609_35701_amd import meq

pytestmark = pytest.mark.gpu


def _pair(shapes, dtype, seed, cap=0, steps=2):
    wl = workloads.custom(shapes, dtype, name=f"noalloc-{dtype}", seed=seed)
    w0 = [to_dev(workloads.weight_init(wl, i), dtype) for i in range(wl.count)]
    ref = meq.HiddenWeightUpdate([w.clone() for w in w0], max_workspace_bytes=cap)
    plan = meq.Plan(shapes, dtype, max_workspace_bytes=cap)
    assert plan.workspace_bytes <= meq.MEQ_STATIC_SCRATCH_BYTES
    params = [w.clone() for w in w0]
    moms = [torch.zeros(w.shape, dtype=torch.float32, device=w.device) for w in w0]
    stream = torch.cuda.current_stream().cuda_stream
    for s in range(steps):
        g = [to_dev(workloads.grad_at_step(wl, i, s), dtype) for i in range(wl.count)]
        ref.step(g, 0.02)
        plan.step_static_ptrs([p.data_ptr() for p in params], [x.data_ptr() for x in g],
                              [b.data_ptr() for b in moms], 0.02, stream)
    torch.cuda.synchronize()
    for k in range(wl.count):
        assert torch.equal(ref.params[k], params[k]), f"{shapes[k]} {dtype}: parameter"
        assert torch.equal(ref.momenta[k], moms[k]), f"{shapes[k]} {dtype}: momentum"
    return plan


def test_static_step_matches_workspace_step():
    log("[case] no-alloc step: first call, 5 matrices bf16")
    p1 = _pair([(1024, 3000), (3000, 1024), (512, 512), (2048, 512), (7, 5)], "bf16", 71)
    log("[case] no-alloc step: second, smaller call, 2 matrices fp32")
    p2 = _pair([(300, 200), (64, 64)], "f32", 72)
    assert p2.workspace_bytes < p1.workspace_bytes
    log("[case] no-alloc step: capped plan of several passes")
    shapes = [(m.rows, m.cols) for m in workloads.workload("llama-1b").matrices[:7]]
    p3 = _pair(shapes, "bf16", 73, cap=meq.MEQ_STATIC_SCRATCH_BYTES, steps=1)
    assert p3.passes >= 2


def test_static_step_rejects_a_plan_beyond_its_scratch():
    plan = meq.Plan([(m.rows, m.cols) for m in workloads.workload("llama-1b").matrices[:7]], "bf16")
    assert plan.workspace_bytes > meq.MEQ_STATIC_SCRATCH_BYTES
    x = torch.zeros(1, device="cuda:0")
    with pytest.raises(meq.MeqError) as e:
        plan.step_static_ptrs([x.data_ptr()] * 7, [x.data_ptr()] * 7, [x.data_ptr()] * 7, 0.02)
    assert e.value.status == meq.MEQ_ERR_WORKSPACE


def test_static_step_captured_in_a_graph_replays_like_the_workspace_step():
    """The point of the entry point: a step that allocates nothing can be captured into a HIP graph
    and replayed; each replay equals the eager workspace step bitwise."""
    shapes = [(256, 1024), (1024, 256), (300, 100)]
    wl = workloads.custom(shapes, "bf16", name="noalloc-graph", seed=75)
    w0 = [to_dev(workloads.weight_init(wl, i), "bf16") for i in range(wl.count)]
    grads = [[to_dev(workloads.grad_at_step(wl, i, s), "bf16") for i in range(wl.count)] for s in range(3)]
    log("[case] no-alloc step in a graph: 3 replays")
    # the device's scratch address is looked up on a first eager call, outside the capture
    warm = meq.Plan([(7, 5)], "bf16")
    x = [torch.zeros(7, 5, dtype=torch.bfloat16, device="cuda:0")]
    xb = [torch.zeros(7, 5, dtype=torch.float32, device="cuda:0")]
    warm.step_static_ptrs([x[0].data_ptr()], [x[0].data_ptr()], [xb[0].data_ptr()], 0.0,
                          torch.cuda.current_stream().cuda_stream)
    ref = meq.HiddenWeightUpdate([w.clone() for w in w0])
    plan = meq.Plan(shapes, "bf16")
    params = [w.clone() for w in w0]
    moms = [torch.zeros(w.shape, dtype=torch.float32, device=w.device) for w in w0]
    static_g = [torch.zeros_like(g) for g in grads[0]]
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        plan.step_static_ptrs([p.data_ptr() for p in params], [g.data_ptr() for g in static_g],
                              [b.data_ptr() for b in moms], 0.02, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    for p, w in zip(params, w0):
        assert torch.equal(p, w), "capture must not run the step"
    for s in range(3):
        ref.step(grads[s], 0.02)
        for dst, src in zip(static_g, grads[s]):
            dst.copy_(src)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k in range(len(shapes)):
            assert torch.equal(params[k], ref.params[k]), f"replay {s}: parameter {k}"
            assert torch.equal(moms[k], ref.momenta[k]), f"replay {s}: momentum {k}"
    graph.reset()
