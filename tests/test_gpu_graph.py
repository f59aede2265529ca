"""Plans executed inside a captured HIP graph (torch.cuda.CUDAGraph). A plan's work table is
uploaded when the plan is built and an execution is one kernel launch (no memset, copy or
synchronisation), so forward, backward, product and product-with-softmax executions can be captured. Each replay is
checked bit for bit against eager executions on the same inputs, with eager work (new inputs)
between replays."""

import numpy as np
import pytest
import torch

import paper_2002_07062_amd as bsm
import workloads
from gpu_util import covered_mask, to_device

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.view(torch.int32 if t.dtype == torch.float32 else torch.int16)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_captured_graph_replays_match_eager(dtype):
    # ragged slices, one with rows on no 16-byte boundary and one long enough for the
    # workgroup-held path
    w = workloads.custom([40, 7, 3, 25], [512, 1001, 6000, 96], dtype=dtype, sigma=3.0, seed=51,
                         gap=5)
    n = int(w.offsets[-1])
    mask = torch.from_numpy(covered_mask(w.offsets[: w.batch], w.rows, w.cols, n)).cuda()
    plan = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[: w.batch], dtype=dtype,
                               schedule="balanced", device=0)
    batch, m, nn, k = 6, 256, 256, 64
    gplan = bsm.bsm_gemm_plan_create(batch, m, nn, k, "nt", "bf16", "balanced", device=0)
    splan = bsm.bsm_gemm_plan_create(batch, m, nn, k, "nt_softmax", "f32", "balanced", device=0)
    x = to_device(w.x, dtype)
    tdt = x.dtype
    out, dx = torch.zeros_like(x), torch.zeros_like(x)
    dy = torch.randn(n, device="cuda").to(tdt)
    a = torch.randn(batch * m * k, device="cuda").to(torch.bfloat16)
    b = torch.randn(batch * nn * k, device="cuda").to(torch.bfloat16)
    c = torch.zeros(batch * m * nn, device="cuda", dtype=torch.bfloat16)
    p = torch.zeros(batch * m * nn, device="cuda", dtype=torch.float32)

    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):  # one eager run on the capture stream first
        bsm.bsm_plan_execute(plan, x, out)
        bsm.bsm_plan_execute_backward(plan, out, dy, dx)
        bsm.bsm_gemm_execute(gplan, a, b, c, alpha=0.125)
        bsm.bsm_gemm_execute(splan, a, b, p, alpha=0.125)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        bsm.bsm_plan_execute(plan, x, out)
        bsm.bsm_plan_execute_backward(plan, out, dy, dx)
        bsm.bsm_gemm_execute(gplan, a, b, c, alpha=0.125)
        bsm.bsm_gemm_execute(splan, a, b, p, alpha=0.125)

    rng = np.random.default_rng(52)
    for rep in range(4):
        print(f"[graph {dtype} replay {rep}]", flush=True)
        # eager work between replays: new inputs in the captured buffers
        x.copy_(torch.from_numpy(rng.standard_normal(n).astype(np.float32) * 3).cuda().to(tdt))
        dy.normal_()
        a.normal_()
        b.normal_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        ref_out, ref_dx = torch.zeros_like(x), torch.zeros_like(x)
        ref_c, ref_p = torch.zeros_like(c), torch.zeros_like(p)
        bsm.bsm_plan_execute(plan, x, ref_out)
        bsm.bsm_plan_execute_backward(plan, ref_out, dy, ref_dx)
        bsm.bsm_gemm_execute(gplan, a, b, ref_c, alpha=0.125)
        bsm.bsm_gemm_execute(splan, a, b, ref_p, alpha=0.125)
        torch.cuda.synchronize()
        assert torch.equal(_bits(out)[mask], _bits(ref_out)[mask]), rep
        assert torch.equal(_bits(dx)[mask], _bits(ref_dx)[mask]), rep
        assert torch.equal(_bits(c), _bits(ref_c)), rep
        assert torch.equal(_bits(p), _bits(ref_p)), rep
    del graph
    plan.destroy()
    gplan.destroy()
    splan.destroy()
