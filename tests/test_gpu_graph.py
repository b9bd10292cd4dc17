"""ft_moe_forward and ft_moe_forward_noalloc captured once in a HIP graph and replayed with new
inputs copied in eagerly between the replays: every replay's routing must equal an eager call's
on the same inputs bit for bit, and its output the eager output (bit-identical on the streaming
path with the ordered combine, within float32 atomic-order noise on the matrix-core path) and
the oracle within the format's tolerance.  The calls keep every routing-dependent count on the
device (Section 4.1), which is what makes them capturable."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_16157_amd as ftm
import workloads
from tests._util import oracle_inputs
from tests.test_gpu_parity import check_output, check_route

pytestmark = pytest.mark.gpu

ROUTE_FIELDS = ("topk_ids", "topk_w", "topk_slot", "hit_pairs", "miss_pairs", "hit_off", "miss_off",
                "counts")

CASES = {
    # 32 tokens x 128 experts: the split router, the streaming kernels, the ordered combine
    "stream": dict(hidden=256, inter=384, n_experts=128, top_k=8, tokens=32, gating=0,
                   w_dtype=workloads.DT_BF16, n_resident=64, shared=False, zipf_s=1.0),
    # 300 tokens: the multi-block router and the matrix-core GEMM with its atomic combine
    "gemm": dict(hidden=256, inter=256, n_experts=24, top_k=6, tokens=300, gating=1,
                 w_dtype=workloads.DT_FP8, n_resident=15, shared=True, zipf_s=1.0),
}


def _say(msg):
    print(f"[gpu-graph] {msg}", flush=True)


def _eager(desc, lay, logits, x, T):
    ws = ftm.alloc_workspace(desc, T)
    route = ftm.RouteBuffers(T, lay.top_k, lay.n_experts)
    out = torch.full((T, lay.hidden), float("nan"), device="cuda")
    ftm.ft_moe_forward(desc, ftm.banks_of(lay), logits, lay.slot_table, x, T, out, route, ws)
    torch.cuda.synchronize()
    return out, route


@pytest.mark.parametrize("noalloc", [False, True], ids=["forward", "noalloc"])
@pytest.mark.parametrize("kind", list(CASES))
def test_forward_graph_replays(kind, noalloc):
    c = CASES[kind]
    lay = workloads.random_layer(70 + len(kind), device="cuda", **c)
    desc, T = lay.desc(), c["tokens"]
    lg_buf, x_buf = lay.logits.clone(), lay.x.clone()
    route = ftm.RouteBuffers(T, lay.top_k, lay.n_experts)
    out = torch.empty(T, lay.hidden, device="cuda")
    ws = None if noalloc else ftm.alloc_workspace(desc, T)
    if noalloc:   # the array's device address is looked up by a first, uncaptured call
        ftm.ft_moe_forward_noalloc(desc, ftm.banks_of(lay), lg_buf, lay.slot_table, x_buf, T, out, route)
    cap = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=cap, capture_error_mode="relaxed"):
        if noalloc:
            ftm.ft_moe_forward_noalloc(desc, ftm.banks_of(lay), lg_buf, lay.slot_table, x_buf, T, out,
                                       route, stream=cap)
        else:
            ftm.ft_moe_forward(desc, ftm.banks_of(lay), lg_buf, lay.slot_table, x_buf, T, out, route, ws,
                               stream=cap)
    torch.cuda.synchronize()
    g = torch.Generator(device="cpu").manual_seed(5)
    for step in range(3):
        logits = torch.randn(T, lay.n_experts, generator=g)
        if c["zipf_s"] > 0:
            logits -= c["zipf_s"] * torch.log(torch.randperm(lay.n_experts, generator=g).float() + 1)[None, :]
        lg_buf.copy_(logits)
        x_buf.copy_(torch.randn(T, lay.hidden, generator=g).to(x_buf.dtype))
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        _say(f"{kind} noalloc={noalloc} replay {step}")
        graph.replay()
        torch.cuda.synchronize()
        eo, er = _eager(desc, lay, lg_buf, x_buf, T)
        for n in ROUTE_FIELDS:
            assert torch.equal(getattr(route, n), getattr(er, n)), (step, n)
        a, b = out.cpu().numpy(), eo.cpu().numpy()
        if kind == "stream":
            assert np.array_equal(a, b)
        else:
            assert oracle.max_rel_err(a, b) <= 1e-5
        lay.logits, lay.x = lg_buf, x_buf
        ref, r = oracle.moe_partial(*oracle_inputs(lay))
        check_route(route, r, T, lay.top_k)
        check_output(out, ref, lay.w_dtype)
