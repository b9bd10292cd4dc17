"""Device-side cache control (ft_cache_plan) against the CPU oracle, bit-exact.

The routing comes from the library's own router (ft_route_only) on the same logits and slot
table the oracle routes; the plan, the updated cache state and the rewritten routed slot ids
must equal the oracle's exactly.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2608_16157_amd as ftm

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _say(msg):
    print(f"[gpu-cache] {msg}", flush=True)


def _desc(E, k, n_slots, shared_slot=-1):
    return dict(hidden=128, inter=128, n_experts=E, top_k=k, gating=0, w_dtype=1, x_dtype=1,
                n_slots=n_slots, shared_slot=shared_slot)


class DeviceCache:
    """Cache state on the device plus the buffers one planning step needs."""

    def __init__(self, desc, T, table, sexp, stamp, K):
        self.desc, self.T, self.K = desc, T, K
        E = desc["n_experts"]
        self.table = torch.tensor(np.asarray(table, np.int32), device="cuda")
        self.state = ftm.CacheState(torch.tensor(np.asarray(sexp, np.int32), device="cuda"),
                                    torch.tensor(np.asarray(stamp, np.int64).astype(np.int32),
                                                 device="cuda"))
        self.route = ftm.RouteBuffers(T, desc["top_k"], E)
        self.ws = ftm.alloc_workspace(desc, T)
        self.plan = ftm.FillPlanBuffers(K, E)

    def step(self, logits_np, b_pcie, b_host, step):
        logits = torch.tensor(logits_np, device="cuda")
        ftm.ft_route_only(self.desc, logits, self.table, self.T, self.route, self.ws)
        ftm.ft_cache_plan(self.desc, self.route, self.T, self.table, self.state, b_pcie, b_host,
                          self.K, step, self.plan)
        torch.cuda.synchronize()

    def host_state(self):
        return (self.table.cpu().numpy(), self.state.slot_expert.cpu().numpy(),
                self.state.slot_stamp.cpu().numpy().astype(np.uint32))


def _check_plan(dc, ref, T, k):
    counts = dc.plan.counts.cpu().numpy()
    q, m = ref["q"], ref["m"]
    assert counts.tolist() == [q, m - q, m, ref["status"]]
    K, E = dc.K, dc.desc["n_experts"]
    fe, fs = dc.plan.fill_expert.cpu().numpy(), dc.plan.fill_slot.cpu().numpy()
    ev, cpu = dc.plan.evict_expert.cpu().numpy(), dc.plan.cpu_expert.cpu().numpy()
    assert fe[:q].tolist() == list(ref["fill_expert"])
    assert fs[:q].tolist() == list(ref["fill_slot"])
    assert ev[:q].tolist() == list(ref["evict_expert"])
    assert (fe[q:K] == -1).all() and (fs[q:K] == -1).all() and (ev[q:K] == -1).all()
    assert cpu[:m - q].tolist() == list(ref["cpu_expert"])
    assert (cpu[m - q:E] == -1).all()
    table, sexp, stamp = dc.host_state()
    assert np.array_equal(table, ref["slot_table"])
    assert np.array_equal(sexp, ref["slot_expert"])
    assert np.array_equal(stamp, ref["slot_stamp"])
    tslot = dc.route.topk_slot.cpu().numpy()[:T * k]
    assert np.array_equal(tslot, ref["topk_slot"].ravel())


def _ranked_logits(E, rank_order):
    logits = np.full((len(rank_order), E), -10.0, dtype=np.float32)
    for t, order in enumerate(rank_order):
        for j, e in enumerate(order):
            logits[t, e] = 5.0 - j
    return logits


def test_cache_plan_fig2_golden():
    with open(os.path.join(GOLDEN, "fig2_cache_plan.json")) as f:
        g = json.load(f)
    E, k = g["n_experts"], g["top_k"]
    desc = _desc(E, k, g["n_slots"])
    logits = _ranked_logits(E, g["logits_rank_order"])
    T = logits.shape[0]
    dc = DeviceCache(desc, T, g["slot_table"], g["slot_expert"], g["slot_stamp"], g["max_fill"])
    dc.step(logits, g["b_pcie"], g["b_host"], g["step"])
    r = oracle.route(desc, logits, np.asarray(g["slot_table"], np.int32))
    ref = oracle.cache_plan(desc, r, g["slot_table"], g["slot_expert"], g["slot_stamp"],
                            g["b_pcie"], g["b_host"], g["max_fill"], g["step"])
    _check_plan(dc, ref, T, k)
    assert ref["fill_expert"] == g["expect"]["fill_expert"]


def _random_state(rng, E, n_slots, shared):
    n_res = int(rng.integers(0, min(E, n_slots - (1 if shared else 0)) + 1))
    res = rng.choice(E, n_res, replace=False)
    routed = [s for s in range(n_slots) if not (shared and s == n_slots - 1)]
    slots = rng.choice(routed, n_res, replace=False)
    table = np.full(E, -1, np.int32)
    sexp = np.full(n_slots, -1, np.int32)
    table[res] = slots
    sexp[slots] = res
    stamp = rng.integers(0, 1000, n_slots).astype(np.uint32)
    return table, sexp, stamp


@pytest.mark.parametrize("seed", range(4))
def test_cache_plan_random(seed):
    rng = np.random.default_rng(100 + seed)
    for case in range(30):
        E = int(rng.integers(1, 300))
        k = int(rng.integers(1, min(E, 16) + 1))
        T = int(rng.integers(1, 40))
        shared = bool(rng.integers(0, 2))
        n_slots = int(rng.integers(1, 200)) + (1 if shared else 0)
        K = int(rng.integers(1, 65))
        bp, bh = float(rng.uniform(1, 60)), float(rng.uniform(1, 80))
        _say(f"random seed={seed} case={case} E={E} k={k} T={T} slots={n_slots} K={K}")
        desc = _desc(E, k, n_slots, n_slots - 1 if shared else -1)
        table, sexp, stamp = _random_state(rng, E, n_slots, shared)
        logits = rng.standard_normal((T, E)).astype(np.float32)
        dc = DeviceCache(desc, T, table, sexp, stamp, K)
        dc.step(logits, bp, bh, 2000)
        r = oracle.route(desc, logits, table)
        ref = oracle.cache_plan(desc, r, table, sexp, stamp, bp, bh, K, 2000)
        _check_plan(dc, ref, T, k)


@pytest.mark.parametrize("ratio", [(11.8, 47.5), (52.7, 77.3), (49.0, 53.8), (6.0, 5.0)])
def test_cache_plan_decode_sequence(ratio):
    """Forty decode steps with the state kept on the device, Zipf-skewed routing whose ranking
    shifts halfway; every step must match the oracle carried on the host."""
    rng = np.random.default_rng(7)
    E, k, T, n_slots, K = 64, 4, 4, 16, 8
    desc = _desc(E, k, n_slots)
    table = np.full(E, -1, np.int32)
    sexp = np.full(n_slots, -1, np.int32)
    stamp = np.zeros(n_slots, np.uint32)
    dc = DeviceCache(desc, T, table, sexp, stamp, K)
    rank = rng.permutation(E) + 1
    for step in range(1, 41):
        if step == 21:
            rank = rng.permutation(E) + 1
        logits = (rng.standard_normal((T, E)) - 1.2 * np.log(rank)[None, :]).astype(np.float32)
        _say(f"sequence ratio={ratio} step={step}")
        dc.step(logits, ratio[0], ratio[1], step)
        r = oracle.route(desc, logits, table)
        ref = oracle.cache_plan(desc, r, table, sexp, stamp, ratio[0], ratio[1], K, step)
        _check_plan(dc, ref, T, k)
        table, sexp, stamp = ref["slot_table"], ref["slot_expert"], ref["slot_stamp"]


def test_cache_plan_faulty_table_is_a_noop():
    E, n_slots = 6, 4
    table = np.array([0, 0, 1, -1, -1, -1], np.int32)
    sexp = np.array([0, 2, -1, -1], np.int32)
    stamp = np.array([3, 4, 5, 6], np.uint32)
    desc = _desc(E, 2, n_slots)
    logits = _ranked_logits(E, [[0, 3], [1, 4]])
    dc = DeviceCache(desc, 2, table, sexp, stamp, 4)
    dc.step(logits, 1.0, 2.0, 9)
    r = oracle.route(desc, logits, table)
    ref = oracle.cache_plan(desc, r, table, sexp, stamp, 1.0, 2.0, 4, 9)
    assert ref["status"] != 0 and ref["q"] == 0
    _check_plan(dc, ref, 2, 2)


def test_cache_plan_prefill_scale():
    """DeepSeek-V3-sized expert pool (256 experts, 103 slots with the shared one), 64 tokens of
    top-8, all candidates (K = 64)."""
    rng = np.random.default_rng(3)
    E, k, T, n_slots = 256, 8, 64, 103
    desc = _desc(E, k, n_slots, n_slots - 1)
    table, sexp, stamp = _random_state(rng, E, n_slots, True)
    logits = rng.standard_normal((T, E)).astype(np.float32)
    dc = DeviceCache(desc, T, table, sexp, stamp, 64)
    dc.step(logits, 52.7, 77.3, 5000)
    r = oracle.route(desc, logits, table)
    ref = oracle.cache_plan(desc, r, table, sexp, stamp, 52.7, 77.3, 64, 5000)
    _check_plan(dc, ref, T, k)
    assert ref["q"] > 1


@pytest.mark.parametrize("E,n_slots,shared,K", [(300, 600, True, 64), (1024, 4096, False, 40),
                                                (1024, 700, True, 64)])
def test_cache_plan_large_pools(E, n_slots, shared, K):
    """Pools above 256 slots take the bitonic sort of (age, slot id) keys; up to the 4096-slot
    limit, with random stamps (ties included) and empty slots."""
    rng = np.random.default_rng(E + n_slots)
    k, T = 8, 30
    desc = _desc(E, k, n_slots, n_slots - 1 if shared else -1)
    table, sexp, stamp = _random_state(rng, E, n_slots, shared)
    stamp = (stamp % 50).astype(np.uint32)          # many equal stamps
    logits = rng.standard_normal((T, E)).astype(np.float32)
    _say(f"large pool E={E} slots={n_slots} K={K}")
    dc = DeviceCache(desc, T, table, sexp, stamp, K)
    dc.step(logits, 52.7, 77.3, 9000)
    r = oracle.route(desc, logits, table)
    ref = oracle.cache_plan(desc, r, table, sexp, stamp, 52.7, 77.3, K, 9000)
    _check_plan(dc, ref, T, k)
    assert ref["q"] > 1
