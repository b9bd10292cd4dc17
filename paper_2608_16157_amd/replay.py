"""Placement replay over a routing trace on the GPU (Section 5, "Expert locality", Figure 4b).

Replays the decode tokens of one layer's routing trace, one token per step, through the
library's routing (ft_route_only) and, for the cache policies, its device-side cache control
(ft_cache_plan), and counts the routed pairs whose expert is not resident when the token is
routed.  Policies, at equal capacity C:

  'lru'     the decode cache seeded with the prefill placement, every miss filled (B_H <= B_P
            makes q = m), least recently demanded expert evicted
  'split'   the same cache with the misses split into fills and CPU executions by
            q* = m B_P / B_H (the CPU share is not cached)
  'prefill' the C experts with the most routed pairs over the prefill tokens (ties to the lower
            id), fixed for the whole decode
  'blind'   experts 0 .. C-1, fixed (a routing-blind split)

Seeding: slot i holds the i-th placed expert with stamp C - i, so the most demanded prefill
expert is evicted last; decode step t (from 0) is stamp C + 1 + t.  Only the cache state is
replayed: no expert weights are involved, so the banks are not needed.
"""
from __future__ import annotations

import torch

from . import (CacheState, FillPlanBuffers, RouteBuffers, alloc_workspace, ft_cache_plan,
               ft_route_only)

POLICIES = ("lru", "split", "prefill", "blind")


def prefill_placement(desc: dict, prefill_logits: torch.Tensor, capacity: int) -> torch.Tensor:
    """The `capacity` experts with the most routed pairs over the prefill tokens, ties to the
    lower id (routing by ft_route_only against an empty cache: every pair is a miss, so the miss
    offsets count each expert's pairs)."""
    E, k = desc["n_experts"], desc["top_k"]
    T = prefill_logits.shape[0]
    d = dict(desc, n_slots=0, shared_slot=-1)
    route = RouteBuffers(T, k, E)
    ws = alloc_workspace(d, T)
    empty = torch.full((E,), -1, dtype=torch.int32, device=prefill_logits.device)
    ft_route_only(d, prefill_logits, empty, T, route, ws)
    counts = route.miss_off[1:] - route.miss_off[:-1]
    # stable sort on descending count keeps ascending ids among equal counts
    order = torch.sort(-counts.long(), stable=True).indices
    return order[:capacity].to(torch.int32)


def replay(desc: dict, logits: torch.Tensor, n_prefill: int, capacity: int, policy: str,
           b_pcie: float = 1.0, b_host: float = 1.0, k_max: int = 64) -> dict:
    """Per-step miss pairs [n_decode] (int32, device) and the final cache state."""
    if policy not in POLICIES:
        raise ValueError(f"policy must be one of {POLICIES}")
    dev = logits.device
    E, k = desc["n_experts"], desc["top_k"]
    d = dict(desc, n_slots=capacity, shared_slot=-1)
    if policy == "blind":
        placed = torch.arange(capacity, dtype=torch.int32, device=dev)
    else:
        placed = prefill_placement(d, logits[:n_prefill].contiguous(), capacity)
    slots = torch.arange(capacity, dtype=torch.int32, device=dev)
    table = torch.full((E,), -1, dtype=torch.int32, device=dev)
    table[placed.long()] = slots
    state = CacheState(placed.clone(), (capacity - slots).contiguous())
    if policy == "lru":
        b_pcie, b_host = 1.0, 1.0
    route = RouteBuffers(1, k, E)
    plan = FillPlanBuffers(k_max, E)
    ws = alloc_workspace(d, 1)
    n_decode = logits.shape[0] - n_prefill
    misses = torch.empty(max(n_decode, 1), dtype=torch.int32, device=dev)
    cached = policy in ("lru", "split")
    for i in range(n_decode):
        row = logits[n_prefill + i:n_prefill + i + 1]
        ft_route_only(d, row, table, 1, route, ws)
        misses[i:i + 1].copy_(route.counts[1:2])
        if cached:
            ft_cache_plan(d, route, 1, table, state, b_pcie, b_host, k_max, capacity + 1 + i, plan)
    return dict(misses=misses[:n_decode], slot_table=table, slot_expert=state.slot_expert,
                slot_stamp=state.slot_stamp)
