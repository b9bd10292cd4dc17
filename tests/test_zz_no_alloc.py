"""ft_moe_forward_noalloc (the library's own device scratch array instead of a caller workspace)
against ft_moe_forward on the same inputs, through the C ABI: routing outputs bit-exact, layer
outputs within the float tolerance of each weight format, and both within that tolerance of the
oracle.  Two calls in a row, the second with fewer tokens, so the second reads a scratch array
the first left full of its own data."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_16157_amd as ftm
import workloads
from tests._util import oracle_inputs

pytestmark = pytest.mark.gpu

TOL = {workloads.DT_F32: 1e-3, workloads.DT_BF16: 1e-2, workloads.DT_FP8: 3e-2, workloads.DT_MXFP4: 1e-2}
ROUTE_FIELDS = ("topk_ids", "topk_w", "topk_slot", "hit_pairs", "miss_pairs", "hit_off",
                "miss_off", "counts")


def _layer(kind, T):
    if kind == "stream":     # few tokens: the streaming kernels
        return workloads.random_layer(41, hidden=256, inter=384, n_experts=16, top_k=4, tokens=T,
                                      w_dtype=workloads.DT_BF16, n_resident=10, shared=True,
                                      device="cuda")
    if kind == "gemm":       # many tokens: the matrix-core kernels
        return workloads.random_layer(42, hidden=256, inter=256, n_experts=24, top_k=6, tokens=T,
                                      w_dtype=workloads.DT_FP8, gating=1, n_resident=15, shared=True,
                                      zipf_s=1.0, device="cuda")
    return workloads.make_layer(kind, T, device="cuda")


def _both(lay, T, act_quant=0):
    desc = dict(lay.desc(), act_quant=act_quant)
    banks = ftm.banks_of(lay)
    ra, rb = (ftm.RouteBuffers(T, lay.top_k, lay.n_experts) for _ in range(2))
    oa = torch.full((T, lay.hidden), float("nan"), device="cuda")
    ob = torch.full((T, lay.hidden), float("nan"), device="cuda")
    ws = ftm.alloc_workspace(desc, T)
    ftm.ft_moe_forward(desc, banks, lay.logits, lay.slot_table, lay.x, T, oa, ra, ws)
    ftm.ft_moe_forward_noalloc(desc, banks, lay.logits, lay.slot_table, lay.x, T, ob, rb)
    torch.cuda.synchronize()
    return oa, ra, ob, rb


@pytest.mark.parametrize("kind,T1,T2", [("stream", 40, 7), ("gemm", 700, 300),
                                        ("dsv3_decode", 64, 16), ("qwen3_decode", 32, 1)])
def test_noalloc_matches_forward_twice(kind, T1, T2):
    for T in (T1, T2):
        print(f"noalloc {kind} T={T}", flush=True)
        lay = _layer(kind, T)
        oa, ra, ob, rb = _both(lay, T)
        for n in ROUTE_FIELDS:
            assert torch.equal(getattr(ra, n), getattr(rb, n)), n
        a, b = oa.cpu().numpy(), ob.cpu().numpy()
        assert np.isfinite(b).all()
        assert np.array_equal(~a.any(axis=1), ~b.any(axis=1))
        tol = TOL[lay.w_dtype]
        assert oracle.max_rel_err(b, a) <= tol
        ref, _ = oracle.moe_partial(*oracle_inputs(lay))
        assert oracle.max_rel_err(b, ref) <= tol


@pytest.mark.parametrize("kind,T1,T2", [("gemm", 700, 300), ("dsv3_decode", 64, 16)])
def test_noalloc_fp8_activations_twice(kind, T1, T2):
    """The optional fp8-activation mode through the array: the matrix-core path (codes of x and
    h in the array) and the streaming path (the widened x in the array)."""
    for T in (T1, T2):
        print(f"noalloc fp8 activations {kind} T={T}", flush=True)
        lay = _layer(kind, T)
        oa, ra, ob, rb = _both(lay, T, ftm.FT_ACT_FP8_1x128_POW2)
        for n in ROUTE_FIELDS:
            assert torch.equal(getattr(ra, n), getattr(rb, n)), n
        a, b = oa.cpu().numpy(), ob.cpu().numpy()
        assert np.isfinite(b).all()
        assert np.array_equal(~a.any(axis=1), ~b.any(axis=1))
        # the same kernels on the same inputs: only the order of the float32 atomic adds of the
        # matrix-core down projection may differ
        assert oracle.max_rel_err(b, a) <= 1e-4


def test_noalloc_rejects_a_workspace_beyond_the_array():
    lay = workloads.make_layer("qwen3_prefill", 4096, device="cuda")
    desc = dict(lay.desc())
    big = 8192
    assert ftm.ft_moe_workspace_bytes(desc, big) > ftm.FT_NOALLOC_SCRATCH_BYTES
    assert ftm.ft_moe_workspace_bytes(desc, 4096) <= ftm.FT_NOALLOC_SCRATCH_BYTES
    logits = torch.zeros(big, lay.n_experts, device="cuda")
    x = torch.zeros(big, lay.hidden, dtype=torch.bfloat16, device="cuda")
    out = torch.zeros(big, lay.hidden, device="cuda")
    route = ftm.RouteBuffers(big, lay.top_k, lay.n_experts)
    with pytest.raises(ftm.FtError) as e:
        ftm.ft_moe_forward_noalloc(desc, ftm.banks_of(lay), logits, lay.slot_table, x, big, out, route)
    assert e.value.status == ftm.FT_ERR_CAPACITY
    torch.cuda.synchronize()
    assert not out.any()       # nothing was enqueued
