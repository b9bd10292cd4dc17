"""Full-layer double-buffered prefill (ft_prefill_layers) against the oracle.

Every layer's complete expert set sits in its own pinned host pool; the call loads the layers
through two full-layer device buffers (overlapped or serialised) and evaluates each.  Layer l's
output must equal the oracle's full-layer output (every expert resident) on layer l's weights,
and the buffers must end up holding the last two layers' experts byte for byte.
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
BANKS = ("w13", "w2", "s13", "s2")


def _say(msg):
    print(f"[gpu-prefill] {msg}", flush=True)


def _pool_in_id_order(lay):
    """The layer's experts re-laid out so that row e holds expert e (shared expert in row E),
    in pinned host memory."""
    E = lay.n_experts
    order = [int(s) for s in lay.slot_table.cpu().tolist()]
    if lay.shared_slot >= 0:
        order.append(lay.shared_slot)
    assert min(order[:E]) >= 0, "every routed expert must be resident"
    idx = torch.tensor(order, dtype=torch.long, device=lay.w13.device)
    pool = {}
    for n in BANKS:
        t = getattr(lay, n)
        if t is None:
            pool[n] = None
            continue
        src = t.index_select(0, idx).contiguous()
        dst = torch.empty(src.shape, dtype=src.dtype, pin_memory=True)
        dst.copy_(src)
        pool[n] = dst
    return pool


def _desc(lay):
    E = lay.n_experts
    shared = lay.shared_slot >= 0
    return dict(lay.desc(), n_slots=E + (1 if shared else 0), shared_slot=E if shared else -1)


def _oracle(desc, pool, logits, x, tokens=None):
    banks = {n: to_np_bits(pool[n]) for n in BANKS if pool[n] is not None}
    ref, _ = oracle.moe_partial(desc, banks, to_np_bits(logits), np.arange(desc["n_experts"], dtype=np.int32),
                                to_np_bits(x), tokens=tokens)
    return ref


def _dev_bufs(desc, pool):
    return [{n: (torch.full(pool[n].shape, 0, dtype=pool[n].dtype, device="cuda") if pool[n] is not None
                 else None) for n in BANKS} for _ in range(2)]


def _run(desc, pools, lays, T, overlap):
    n = len(pools)
    bufs = _dev_bufs(desc, pools[0])
    for b in bufs:                               # garbage the loads must replace
        for t in b.values():
            if t is not None:
                t.view(torch.uint8).fill_(0x5A) if t.dtype != torch.float32 else t.fill_(7.0)
    table = torch.arange(desc["n_experts"], dtype=torch.int32, device="cuda")
    route = ftm.RouteBuffers(T, desc["top_k"], desc["n_experts"])
    ws = ftm.alloc_workspace(desc, T)
    outs = [torch.full((T, desc["hidden"]), float("nan"), device="cuda") for _ in range(n)]
    copy_stream = torch.cuda.Stream() if overlap else None
    ftm.ft_prefill_layers(desc, pools, bufs, table, [l.logits for l in lays], [l.x for l in lays], T,
                          outs, route, ws, overlap=overlap, copy_stream=copy_stream)
    torch.cuda.synchronize()
    return outs, bufs


CASES = [
    # seed, w_dtype, gating, E, k, T, H, I, shared, layers
    (0, workloads.DT_BF16, 0, 16, 4, 300, 256, 256, False, 3),     # many-token (MFMA) path
    (1, workloads.DT_FP8, 1, 12, 3, 40, 256, 384, True, 4),        # GEMV path, shared expert
    (2, workloads.DT_F32, 0, 8, 2, 20, 128, 128, False, 2),
    (3, workloads.DT_FP8, 1, 20, 4, 260, 384, 256, True, 3),       # MFMA path, fp8, shared
    (4, workloads.DT_BF16, 0, 8, 2, 17, 128, 256, False, 1),       # a single layer
    (5, workloads.DT_MXFP4, 1, 12, 3, 30, 256, 384, False, 3),     # MXFP4, GEMV path
    (6, workloads.DT_MXFP4, 0, 16, 4, 280, 256, 256, False, 2),    # MXFP4, many tokens
]


@pytest.mark.parametrize("overlap", [True, False], ids=["overlap", "serial"])
@pytest.mark.parametrize("case", CASES, ids=[str(c[0]) for c in CASES])
def test_prefill_layers_match_full_layer(case, overlap):
    seed, wdt, gating, E, k, T, H, I, shared, L = case
    lays = [workloads.random_layer(seed * 10 + l, hidden=H, inter=I, n_experts=E, top_k=k, tokens=T,
                                   gating=gating, w_dtype=wdt, n_resident=E, shared=shared).to("cuda")
            for l in range(L)]
    desc = _desc(lays[0])
    pools = [_pool_in_id_order(l) for l in lays]
    _say(f"case {seed} overlap={overlap} layers={L} T={T}")
    outs, bufs = _run(desc, pools, lays, T, overlap)
    for l in range(L):
        ref = _oracle(desc, pools[l], lays[l].logits, lays[l].x)
        err = oracle.max_rel_err(outs[l].cpu().numpy(), ref)
        assert err <= TOL[wdt], (l, err)
    # the buffers hold the last two layers, layer l in buffer l % 2
    for l in range(max(0, L - 2), L):
        for n in BANKS:
            if pools[l][n] is not None:
                assert torch.equal(bufs[l % 2][n].cpu().view(torch.uint8), pools[l][n].view(torch.uint8)), (l, n)


def test_prefill_layers_overlap_and_serial_agree():
    """Both schedules evaluate the same layers: outputs within float32 atomic-order noise of
    each other."""
    lays = [workloads.random_layer(50 + l, hidden=256, inter=256, n_experts=16, top_k=4, tokens=300,
                                   w_dtype=workloads.DT_BF16, n_resident=16).to("cuda") for l in range(3)]
    desc = _desc(lays[0])
    pools = [_pool_in_id_order(l) for l in lays]
    a, _ = _run(desc, pools, lays, 300, True)
    b, _ = _run(desc, pools, lays, 300, False)
    for x, y in zip(a, b):
        assert torch.allclose(x, y, rtol=1e-5, atol=1e-6)


def test_prefill_layers_full_size_sampled():
    """Qwen3-30B-A3B-shaped prefill chunk (T = 4096, E = 128, H = 2048, I = 768, bf16) through 3
    layers with every expert loaded per layer; the oracle evaluates sampled tokens of each."""
    T, L = 4096, 3
    lays = [workloads.make_layer("qwen3_prefill", T, layer=l, device="cuda", resident_frac=1.0)
            for l in range(L)]
    desc = _desc(lays[0])
    pools = [_pool_in_id_order(l) for l in lays]
    _say("full-size qwen3 prefill, 3 layers")
    outs, _ = _run(desc, pools, lays, T, True)
    rows = [0, 1, 777, 2048, 3001, T - 1]
    for l in range(L):
        ref = _oracle(desc, pools[l], lays[l].logits, lays[l].x, tokens=rows)
        got = outs[l].cpu().numpy()
        err = oracle.max_rel_err(got[rows], ref[rows])
        assert err <= TOL[workloads.DT_BF16], (l, err)
        assert np.isfinite(got).all()
