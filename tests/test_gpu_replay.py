"""Placement replay on the GPU (paper_2608_16157_amd.replay, through ft_route_only and
ft_cache_plan) against oracle.replay: per-step miss counts and the final cache state are
bit-exact for every policy."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from paper_2608_16157_amd import replay as rp

pytestmark = pytest.mark.gpu


def _desc(name):
    c = workloads.CONFIGS[name]
    return dict(hidden=c.hidden, inter=c.inter, n_experts=c.n_experts, top_k=c.top_k, gating=c.gating,
                w_dtype=c.w_dtype, x_dtype=c.x_dtype, n_slots=0, shared_slot=-1)


CASES = [
    # config, prefill tokens, decode tokens, capacity, policy, (B_P, B_H)
    ("qwen3_decode", 64, 150, 47, "lru", (1.0, 1.0)),
    ("qwen3_decode", 64, 150, 47, "split", (53.9, 82.7)),
    ("qwen3_decode", 64, 150, 47, "prefill", (1.0, 1.0)),
    ("qwen3_decode", 64, 150, 47, "blind", (1.0, 1.0)),
    ("dsv3_decode", 48, 120, 28, "lru", (1.0, 1.0)),
    ("dsv3_decode", 48, 120, 28, "split", (55.5, 44.9)),
    ("dsv3_decode", 48, 120, 28, "prefill", (1.0, 1.0)),
    ("dsv3_decode", 48, 120, 8, "split", (10.0, 70.0)),      # capacity == k
]


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-{c[3]}-{c[4]}" for c in CASES])
def test_replay_matches_oracle(case):
    name, P, N, C, policy, (bp, bh) = case
    logits = workloads.routing_trace(name, P, N, layer=C)
    desc = _desc(name)
    print(f"[gpu-replay] {name} C={C} {policy}", flush=True)
    got = rp.replay(desc, logits.cuda(), P, C, policy, bp, bh, k_max=desc["top_k"])
    torch.cuda.synchronize()
    want = oracle.replay(desc, logits.numpy(), P, C, policy, bp, bh, k_max=desc["top_k"])
    assert got["misses"].cpu().numpy().tolist() == want["misses"].tolist()
    assert np.array_equal(got["slot_table"].cpu().numpy(), want["slot_table"])
    assert np.array_equal(got["slot_expert"].cpu().numpy(), want["slot_expert"])
    assert np.array_equal(got["slot_stamp"].cpu().numpy().astype(np.uint32), want["slot_stamp"])
    assert want["misses"].sum() > 0


def test_prefill_placement_matches_oracle():
    desc = _desc("dsv3_decode")
    logits = workloads.routing_trace("dsv3_decode", 500, 0)
    for C in (1, 28, 100, 256):
        got = rp.prefill_placement(dict(desc, n_slots=C), logits.cuda(), C).cpu().tolist()
        assert got == oracle.placement(dict(desc, n_slots=C), logits.numpy(), C, "prefill")
