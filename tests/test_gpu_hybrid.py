"""Cache fills and the complete hybrid layer step (GPU hits and fills + CPU branch + exact merge)
against the oracle.

Every step routes once on the current cache, plans, fills the planned slots from the pinned host
pool, evaluates hits and fills on the GPU from the plan's rewritten slot ids and the rest on the
CPU (a host function on a second stream, on a persistent worker pool), and merges: the output must
equal the oracle's output of the full MoE layer (every expert), the cache state must equal the
oracle's plan bit for bit, and every occupied slot must hold its expert's weights bit for bit.
The same step captured in a HIP graph is checked the same way on every replay.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_16157_amd as ftm
import workloads
from tests._util import to_np_bits

pytestmark = pytest.mark.gpu

TOL = {workloads.DT_F32: 1e-3, workloads.DT_BF16: 1e-2, workloads.DT_FP8: 3e-2, workloads.DT_MXFP4: 1e-2}


def _say(msg):
    print(f"[gpu-hybrid] {msg}", flush=True)


class Setup:
    """Host pool (pinned, indexed by expert), device slot banks, cache state and buffers."""

    def __init__(self, seed, wdt, gating, E, R, k, T, H, I, shared, K, clock=False):
        lay = workloads.random_layer(seed, hidden=H, inter=I, n_experts=E, top_k=k, tokens=T,
                                     gating=gating, w_dtype=wdt, n_resident=E, shared=shared)
        st = lay.slot_table.long()
        scaled = lay.s13 is not None
        self.pool = {"w13": lay.w13[st].contiguous().pin_memory(),
                     "w2": lay.w2[st].contiguous().pin_memory(),
                     "s13": lay.s13[st].contiguous().pin_memory() if scaled else None,
                     "s2": lay.s2[st].contiguous().pin_memory() if scaled else None}
        self.E, self.R, self.k, self.T, self.H, self.I, self.K = E, R, k, T, H, I, K
        self.wdt, self.shared = wdt, shared
        n_slots = R + (1 if shared else 0)
        self.desc = dict(hidden=H, inter=I, n_experts=E, top_k=k, gating=gating, w_dtype=wdt,
                         x_dtype=lay.x_dtype, n_slots=n_slots, shared_slot=R if shared else -1)
        # device banks: garbage in every routed slot, the shared expert in its slot
        self.dev = {}
        for name in ("w13", "w2", "s13", "s2"):
            src = getattr(lay, name)
            if src is None:
                self.dev[name] = None
                continue
            d = torch.empty((n_slots,) + tuple(src.shape[1:]), dtype=src.dtype, device="cuda")
            d.view(torch.uint8).fill_(0x5A) if d.dtype != torch.float32 else d.fill_(7.0)
            if shared:
                d[R] = src[lay.shared_slot].cuda()
            self.dev[name] = d
        self.shared_rows = {n: (getattr(lay, n)[lay.shared_slot] if shared and getattr(lay, n) is not None
                                else None) for n in ("w13", "w2", "s13", "s2")}
        self.x_dtype = lay.x.dtype
        self.table = torch.full((E,), -1, dtype=torch.int32, device="cuda")
        self.state = ftm.CacheState(torch.full((n_slots,), -1, dtype=torch.int32, device="cuda"),
                                    torch.zeros(n_slots, dtype=torch.int32, device="cuda"),
                                    torch.zeros(1, dtype=torch.int32, device="cuda") if clock else None)
        self.route = ftm.RouteBuffers(T, k, E)
        self.plan = ftm.FillPlanBuffers(K, E)
        self.ws = ftm.alloc_workspace(self.desc, T)
        self.host = ftm.HybridHostBuffers(T, k, E, H, self.x_dtype)
        self.out = torch.empty(T, H, dtype=torch.float32, device="cuda")

    def oracle_full(self, logits, x):
        """Output of the full layer: every routed expert resident (bank row = expert id), plus the
        shared expert in row E."""
        banks = {}
        for n in ("w13", "w2", "s13", "s2"):
            if self.pool[n] is None:
                continue
            rows = self.pool[n]
            if self.shared:
                rows = torch.cat([rows, self.shared_rows[n][None]], 0)
            banks[n] = to_np_bits(rows)
        d = dict(self.desc, n_slots=self.E + (1 if self.shared else 0),
                 shared_slot=self.E if self.shared else -1)
        ref, _ = oracle.moe_partial(d, banks, logits, np.arange(self.E, dtype=np.int32), to_np_bits(x))
        return ref

    def check_banks(self, sexp):
        for s, e in enumerate(sexp.tolist()):
            if e < 0 or (self.shared and s == self.R):
                continue
            for n in ("w13", "w2", "s13", "s2"):
                if self.pool[n] is None:
                    continue
                got = self.dev[n][s].cpu()
                want = self.pool[n][e]
                assert torch.equal(got.view(torch.uint8), want.view(torch.uint8)), (n, s, e)


def _logits(rng, T, E, rank):
    return (rng.standard_normal((T, E)) - 1.1 * np.log(rank)[None, :]).astype(np.float32)


@pytest.fixture(scope="module")
def workers():
    p = ftm.ft_cpu_pool_create(3, pin=True)
    yield p
    ftm.ft_cpu_pool_destroy(p)


class OracleCache:
    """The oracle's cache state, advanced one step at a time on the oracle's routing."""

    def __init__(self, su, bp, bh, K):
        self.su, self.bp, self.bh, self.K = su, bp, bh, K
        self.table = np.full(su.E, -1, np.int32)
        self.sexp = np.full(su.desc["n_slots"], -1, np.int32)
        self.stamp = np.zeros(su.desc["n_slots"], np.uint32)

    def step_and_check(self, step, logits, x):
        su = self.su
        r = oracle.route(su.desc, logits, self.table)
        plan = oracle.cache_plan(su.desc, r, self.table, self.sexp, self.stamp, self.bp, self.bh,
                                 self.K, step)
        self.table, self.sexp, self.stamp = plan["slot_table"], plan["slot_expert"], plan["slot_stamp"]
        assert np.array_equal(su.table.cpu().numpy(), self.table)
        assert np.array_equal(su.state.slot_expert.cpu().numpy(), self.sexp)
        assert np.array_equal(su.state.slot_stamp.cpu().numpy().astype(np.uint32), self.stamp)
        assert su.plan.counts.cpu().tolist() == [plan["q"], plan["m"] - plan["q"], plan["m"], 0]
        su.check_banks(self.sexp)
        ref = su.oracle_full(logits, x)
        err = oracle.max_rel_err(su.out.cpu().numpy(), ref)
        _say(f"   step {step}: q={plan['q']} cpu={plan['m'] - plan['q']} max_rel_err={err:.2e}")
        assert err <= TOL[su.wdt], step
        return plan


CASES = [
    # seed, w_dtype, gating, E, R (routed slots), k, T, H, I, shared, K, (B_P, B_H)
    (0, workloads.DT_BF16, 0, 16, 5, 4, 3, 256, 256, False, 4, (11.8, 47.5)),
    (1, workloads.DT_FP8, 1, 20, 6, 4, 2, 256, 384, True, 3, (52.7, 77.3)),
    (2, workloads.DT_F32, 0, 8, 3, 2, 4, 128, 128, False, 2, (6.0, 5.0)),
    (3, workloads.DT_BF16, 1, 24, 8, 6, 5, 384, 256, True, 8, (25.1, 63.2)),
    (4, workloads.DT_MXFP4, 1, 20, 6, 4, 3, 256, 384, False, 4, (55.5, 44.9)),
    # a prefill-sized step: the evaluation groups of G = H u F drive the matrix-core GEMM
    (5, workloads.DT_FP8, 1, 16, 6, 4, 300, 256, 256, True, 4, (54.1, 137.2)),
]


@pytest.mark.parametrize("case", CASES, ids=[str(c[0]) for c in CASES])
def test_hybrid_steps_match_full_layer(case, workers):
    seed, wdt, gating, E, R, k, T, H, I, shared, K, (bp, bh) = case
    su = Setup(seed, wdt, gating, E, R, k, T, H, I, shared, K)
    oc = OracleCache(su, bp, bh, K)
    rng = np.random.default_rng(seed)
    rank = rng.permutation(E) + 1
    n_cpu_steps = n_fill_steps = 0
    for step in range(1, 11):
        if step == 6:
            rank = rng.permutation(E) + 1
        logits = _logits(rng, T, E, rank)
        x = torch.randn(T, H, generator=torch.Generator().manual_seed(seed * 100 + step)).to(su.x_dtype)
        _say(f"case {seed} step {step}")
        lg, xd = torch.tensor(logits, device="cuda"), x.cuda()
        # odd steps without a pool: the CPU branch then runs on the runtime's callback thread
        ftm.ft_moe_step_hybrid(su.desc, su.dev, su.pool, lg, su.table, su.state, bp, bh, K, step, xd, T,
                               su.out, su.route, su.plan, su.host, su.ws,
                               workers if step % 2 == 0 else None)
        torch.cuda.synchronize()
        plan = oc.step_and_check(step, logits, x)
        n_cpu_steps += plan["m"] > plan["q"]
        n_fill_steps += plan["q"] > 0
    assert n_fill_steps > 0
    if bh > bp:
        assert n_cpu_steps > 0


@pytest.mark.parametrize("case", [CASES[0], CASES[3]], ids=["0", "3"])
def test_hybrid_step_graph_replays_match_full_layer(case, workers):
    """The step captured once in a HIP graph (fixed input buffers, a device step clock) and
    replayed step after step, with new inputs copied in eagerly between replays: every replay's
    cache state, slot bytes and merged output match the oracle, and the captured CPU branch runs."""
    seed, wdt, gating, E, R, k, T, H, I, shared, K, (bp, bh) = case
    su = Setup(seed, wdt, gating, E, R, k, T, H, I, shared, K, clock=True)
    oc = OracleCache(su, bp, bh, K)
    lg_buf = torch.zeros(T, E, dtype=torch.float32, device="cuda")
    x_buf = torch.zeros(T, H, dtype=su.x_dtype, device="cuda")
    cap = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=cap, capture_error_mode="relaxed"):
        ftm.ft_moe_step_hybrid(su.desc, su.dev, su.pool, lg_buf, su.table, su.state, bp, bh, K, 0,
                               x_buf, T, su.out, su.route, su.plan, su.host, su.ws,
                               workers, stream=cap)
    torch.cuda.synchronize()
    rng = np.random.default_rng(seed + 1000)
    rank = rng.permutation(E) + 1
    n_cpu_steps = n_fill_steps = 0
    for step in range(1, 9):
        if step == 5:
            rank = rng.permutation(E) + 1
        logits = _logits(rng, T, E, rank)
        x = torch.randn(T, H, generator=torch.Generator().manual_seed(seed * 100 + step)).to(su.x_dtype)
        lg_buf.copy_(torch.tensor(logits))
        x_buf.copy_(x)
        su.out.fill_(float("nan"))
        torch.cuda.synchronize()
        _say(f"graph case {seed} replay {step}")
        graph.replay()
        torch.cuda.synchronize()
        assert int(su.state.clock[0]) == step
        plan = oc.step_and_check(step, logits, x)
        n_cpu_steps += plan["m"] > plan["q"]
        n_fill_steps += plan["q"] > 0
    assert n_fill_steps > 0
    if bh > bp:
        assert n_cpu_steps > 0


def test_cache_fill_alone():
    """ft_route_only + ft_cache_plan + ft_cache_fill: filled slots hold their experts, other slots
    keep their bytes."""
    su = Setup(7, workloads.DT_BF16, 0, 12, 6, 3, 4, 256, 128, False, 6)
    rng = np.random.default_rng(7)
    logits = torch.tensor(rng.standard_normal((4, 12)).astype(np.float32), device="cuda")
    before = {n: su.dev[n].clone() for n in ("w13", "w2")}
    ftm.ft_route_only(su.desc, logits, su.table, 4, su.route, su.ws)
    ftm.ft_cache_plan(su.desc, su.route, 4, su.table, su.state, 52.7, 77.3, 6, 1, su.plan)
    ftm.ft_cache_fill(su.desc, su.pool, su.dev, su.plan, 6)
    torch.cuda.synchronize()
    q = int(su.plan.counts[0])
    assert q > 0
    fe = su.plan.fill_expert.cpu().tolist()[:q]
    fs = su.plan.fill_slot.cpu().tolist()[:q]
    for n in ("w13", "w2"):
        for s in range(su.desc["n_slots"]):
            got = su.dev[n][s].cpu()
            if s in fs:
                assert torch.equal(got, su.pool[n][fe[fs.index(s)]])
            else:
                assert torch.equal(got, before[n][s].cpu())
