"""The CPU branch (ft_cpu_experts) against the oracle, on the host: no GPU involved.

The branch evaluates a list of experts from the host expert pool (indexed by expert id); its
output must equal the oracle's partial output of a cache holding exactly those experts.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_16157_amd as ftm
import workloads
from tests._util import to_np_bits

TOL = {workloads.DT_F32: 1e-3, workloads.DT_BF16: 1e-2, workloads.DT_FP8: 3e-2, workloads.DT_MXFP4: 1e-2}


def _pool_case(seed, wdt, gating, E, k, T, H, I):
    lay = workloads.random_layer(seed, hidden=H, inter=I, n_experts=E, top_k=k, tokens=T,
                                 gating=gating, w_dtype=wdt, n_resident=E)
    st = lay.slot_table.long()
    pool = {"w13": lay.w13[st].contiguous(), "w2": lay.w2[st].contiguous(),
            "s13": lay.s13[st].contiguous() if lay.s13 is not None else None,
            "s2": lay.s2[st].contiguous() if lay.s2 is not None else None}
    return lay, pool


CASES = [
    # seed, w_dtype, gating, E, k, T, H, I, pool threads (None: the calling thread alone)
    (0, workloads.DT_F32, 0, 8, 2, 5, 128, 256, None),
    (1, workloads.DT_BF16, 1, 16, 4, 9, 256, 128, 3),
    (2, workloads.DT_BF16, 0, 12, 3, 1, 384, 256, 0),
    (3, workloads.DT_FP8, 1, 10, 4, 6, 256, 384, 4),
    (4, workloads.DT_FP8, 0, 6, 6, 3, 128, 128, 2),
    (5, workloads.DT_MXFP4, 1, 10, 3, 4, 256, 384, 3),
    (6, workloads.DT_MXFP4, 0, 6, 6, 2, 128, 128, 0),
]


@pytest.mark.parametrize("case", CASES, ids=[str(c[0]) for c in CASES])
def test_cpu_experts_matches_oracle(case):
    seed, wdt, gating, E, k, T, H, I, nt = case
    lay, pool = _pool_case(seed, wdt, gating, E, k, T, H, I)
    desc = lay.desc()
    rng = np.random.default_rng(seed)
    listed = np.sort(rng.choice(E, int(rng.integers(1, E + 1)), replace=False)).astype(np.int32)
    # this step's routing (the oracle's router; the CPU branch only consumes it)
    r = oracle.route(desc, lay.logits.numpy(), lay.slot_table.numpy())
    ids = torch.tensor(r["topk_ids"], dtype=torch.int32)
    w = torch.tensor(r["topk_w"], dtype=torch.float32)
    out = torch.empty(T, H, dtype=torch.float32)
    workers = None if nt is None else ftm.ft_cpu_pool_create(nt, pin=bool(seed % 2))
    ftm.ft_cpu_experts(desc, pool, lay.x, T, ids, w, torch.tensor(listed), out, pool=workers)
    if workers is not None:
        ftm.ft_cpu_pool_destroy(workers)
    # oracle: a cache holding exactly the listed experts, bank row = expert id
    d2 = dict(desc, n_slots=E, shared_slot=-1)
    table = np.full(E, -1, np.int32)
    table[listed] = listed
    banks = {"w13": to_np_bits(pool["w13"]), "w2": to_np_bits(pool["w2"])}
    if pool["s13"] is not None:
        banks.update(s13=pool["s13"].numpy(), s2=pool["s2"].numpy())
    ref, _ = oracle.moe_partial(d2, banks, lay.logits.numpy(), table, to_np_bits(lay.x))
    assert oracle.max_rel_err(out.numpy(), ref) <= TOL[wdt]


def test_cpu_experts_is_thread_count_independent():
    """Bit-identical results on the calling thread and on pools of 1, 2 and 5 workers; one pool
    serves several calls in a row."""
    lay, pool = _pool_case(9, workloads.DT_BF16, 0, 16, 4, 7, 256, 256)
    desc = lay.desc()
    r = oracle.route(desc, lay.logits.numpy(), lay.slot_table.numpy())
    ids = torch.tensor(r["topk_ids"], dtype=torch.int32)
    w = torch.tensor(r["topk_w"], dtype=torch.float32)
    listed = torch.arange(0, 16, 2, dtype=torch.int32)
    outs = []
    for nt in (None, 1, 2, 5):
        workers = None if nt is None else ftm.ft_cpu_pool_create(nt, pin=True)
        for _ in range(3):
            out = torch.empty(7, 256, dtype=torch.float32)
            ftm.ft_cpu_experts(desc, pool, lay.x, 7, ids, w, listed, out, pool=workers)
            outs.append(out)
        if workers is not None:
            ftm.ft_cpu_pool_destroy(workers)
    assert all(torch.equal(outs[0], o) for o in outs[1:])


def test_cpu_experts_rejects_bad_lists():
    lay, pool = _pool_case(5, workloads.DT_BF16, 0, 8, 2, 3, 128, 128)
    desc = lay.desc()
    ids = torch.zeros(3, 2, dtype=torch.int32)
    w = torch.ones(3, 2, dtype=torch.float32)
    out = torch.empty(3, 128, dtype=torch.float32)
    for bad in ([1, 1], [8], [-1]):
        with pytest.raises(ftm.FtError):
            ftm.ft_cpu_experts(desc, pool, lay.x, 3, ids, w, torch.tensor(bad, dtype=torch.int32), out)
