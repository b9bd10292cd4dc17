"""GPU parity: the HIP path through the C ABI against the CPU oracle, on the same seeded inputs.

Lists, ids, slots, offsets and counts must be bit-exact; gates within 2e-6; layer outputs
within the max-relative-error bound (row-RMS floor) of 1e-3 for fp32 weights, 1e-2 for bf16,
3e-2 for fp8 and 1e-2 for MXFP4 weights (every MXFP4 weight times its scale is exact in bf16, so
that path has the bf16 path's arithmetic), and rows the oracle makes exactly zero must be exactly
zero.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_16157_amd as ftm
import workloads
from tests._util import oracle_inputs

pytestmark = pytest.mark.gpu

TOL = {workloads.DT_F32: 1e-3, workloads.DT_BF16: 1e-2, workloads.DT_FP8: 3e-2, workloads.DT_MXFP4: 1e-2}


def _say(*a):
    print(*a, flush=True)


def run_route(lay):
    T, desc = lay.tokens, lay.desc()
    ws = ftm.alloc_workspace(desc, T)
    route = ftm.RouteBuffers(T, lay.top_k, lay.n_experts)
    ftm.ft_route_only(desc, lay.logits, lay.slot_table, T, route, ws)
    torch.cuda.synchronize()
    return route


def run_forward(lay, T=None):
    T = lay.tokens if T is None else T
    desc = lay.desc()
    ws = ftm.alloc_workspace(desc, T)
    route = ftm.RouteBuffers(T, lay.top_k, lay.n_experts)
    out = torch.full((T, lay.hidden), float("nan"), dtype=torch.float32, device="cuda")
    ftm.ft_moe_forward(desc, ftm.banks_of(lay), lay.logits, lay.slot_table, lay.x, T, out, route, ws)
    torch.cuda.synchronize()
    return out, route


def check_route(route, r, T, k):
    pk = T * k
    g = lambda t: t.cpu().numpy()
    assert np.array_equal(g(route.topk_ids)[:pk].reshape(T, k), r["topk_ids"])
    assert np.array_equal(g(route.topk_slot)[:pk].reshape(T, k), r["topk_slot"])
    np.testing.assert_allclose(g(route.topk_w)[:pk].reshape(T, k), r["topk_w"], rtol=0, atol=2e-6)
    hp, mp = g(route.hit_pairs)[:pk], g(route.miss_pairs)[:pk]
    assert np.array_equal(hp[: r["n_hit"]], r["hit_pairs"])
    assert np.array_equal(mp[: r["n_miss"]], r["miss_pairs"])
    assert np.all(hp[r["n_hit"]:] == -1) and np.all(mp[r["n_miss"]:] == -1)
    assert np.array_equal(g(route.hit_off), r["hit_off"])
    assert np.array_equal(g(route.miss_off), r["miss_off"])
    assert g(route.counts).tolist() == [r["n_hit"], r["n_miss"], r["m_unique_miss"], r["status"]]


def check_output(out, ref, w_dtype, rows=None):
    got = out.cpu().numpy()
    if rows is not None:
        got, ref = got[rows], ref[rows]
    assert np.isfinite(got).all()
    zero = ~ref.any(axis=1)
    assert not got[zero].any(), "rows without hits must be exactly zero"
    err = oracle.max_rel_err(got, ref)
    _say(f"   max_rel_err={err:.3e} (tol {TOL[w_dtype]:.0e})")
    assert err <= TOL[w_dtype]


# ------------------------------------------------------------------ routing, bit-exact

ROUTE_CASES = [("tiny", 16), ("qwen3_decode", 1), ("qwen3_decode", 8), ("qwen3_decode", 32),
               ("dsv3_decode", 1), ("dsv3_decode", 16), ("dsv3_decode", 64),
               ("qwen3_prefill", 4096), ("dsv3_prefill", 8192), ("qwen3_decode", 300),
               ("dsv4flash_decode", 64)]


def _route_only_layer(name, T):
    """Logits and slot table of a config; weights are not needed for routing."""
    cfg = workloads.CONFIGS[name]
    small = workloads.LayerConfig(**{**cfg.__dict__, "hidden": 128, "inter": 128})
    return workloads.make_layer_from(small, T, device="cuda")


@pytest.mark.parametrize("name,T", ROUTE_CASES)
def test_route_bit_exact_configs(name, T):
    _say(f"route {name} T={T}")
    lay = _route_only_layer(name, T)
    route = run_route(lay)
    desc, banks, logits, st, x = oracle_inputs(lay)
    check_route(route, oracle.route(desc, logits, st), T, lay.top_k)


# Decode batches of T * E >= 4096 logits take their top-k in a kernel ahead of the fused router:
# cases on both sides of that edge, for 1, 2, 4, 8 and 16 experts per lane.
@pytest.mark.parametrize("seed,E,k,T,ties", [(0, 8, 8, 5, True), (1, 1024, 64, 3, False),
                                             (2, 1000, 7, 33, True), (3, 64, 1, 2500, False),
                                             (4, 256, 8, 257, True), (5, 130, 13, 4099, True),
                                             (6, 1024, 8, 600, False), (7, 2, 2, 1, True),
                                             (8, 128, 8, 31, True), (9, 128, 8, 32, True),
                                             (10, 256, 8, 16, False), (11, 64, 4, 64, True),
                                             (12, 512, 8, 8, True), (13, 130, 13, 40, True)])
def test_route_bit_exact_random(seed, E, k, T, ties):
    _say(f"route random seed={seed} E={E} k={k} T={T}")
    lay = workloads.random_layer(seed, hidden=128, inter=128, n_experts=E, top_k=k, tokens=T,
                                 tie_logits=ties, zipf_s=1.0 if seed % 2 else 0.0, device="cuda")
    route = run_route(lay)
    desc, banks, logits, st, x = oracle_inputs(lay)
    check_route(route, oracle.route(desc, logits, st), T, k)


# One or two tokens (at most 64 pairs) are routed by a single wave: its edges are 8 experts per
# lane, k = 64 and two tokens of 32 choices (every lane holds a pair), an expert count that is not
# a multiple of 64, sigmoid gating, and the shared expert's rows after the hit rows.
@pytest.mark.parametrize("seed,E,k,T,ties,gating,shared",
                         [(20, 512, 8, 2, True, workloads.GATE_SOFTMAX, False),
                          (21, 256, 64, 1, False, workloads.GATE_SOFTMAX, True),
                          (22, 300, 6, 2, True, workloads.GATE_SIGMOID, True),
                          (23, 64, 32, 2, False, workloads.GATE_SOFTMAX, False),
                          (24, 200, 3, 1, True, workloads.GATE_SIGMOID, True),
                          (25, 8, 2, 2, True, workloads.GATE_SOFTMAX, False)])
def test_route_bit_exact_single_wave(seed, E, k, T, ties, gating, shared):
    _say(f"route single-wave seed={seed} E={E} k={k} T={T} shared={shared}")
    lay = workloads.random_layer(seed, hidden=128, inter=128, n_experts=E, top_k=k, tokens=T,
                                 gating=gating, tie_logits=ties, shared=shared,
                                 zipf_s=1.0 if seed % 2 else 0.0, device="cuda")
    route = run_route(lay)
    desc, banks, logits, st, x = oracle_inputs(lay)
    check_route(route, oracle.route(desc, logits, st), T, k)


def test_route_deterministic():
    lay = _route_only_layer("dsv3_prefill", 8192)
    a, b = run_route(lay), run_route(lay)
    for n in ("topk_ids", "topk_w", "topk_slot", "hit_pairs", "miss_pairs", "hit_off", "miss_off",
              "counts"):
        assert torch.equal(getattr(a, n), getattr(b, n)), n


@pytest.mark.parametrize("T", [2, 5, 700])
def test_invalid_slot_tables_flagged_and_treated_as_misses(T):
    lay = workloads.random_layer(11, hidden=128, inter=128, n_experts=16, top_k=4, tokens=T,
                                 n_resident=10, shared=True, device="cuda")
    st = lay.slot_table.clone()
    res = (st >= 0).nonzero().flatten().tolist()
    st[res[0]] = st[res[1]]                  # duplicate
    st[res[2]] = lay.n_slots + 5             # out of range
    st[res[3]] = lay.shared_slot             # points at the shared expert
    lay.slot_table = st
    _say(f"invalid slot table T={T}: {st.tolist()}")
    route = run_route(lay)
    desc, banks, logits, stn, x = oracle_inputs(lay)
    r = oracle.route(desc, logits, stn)
    assert r["status"] == 7
    check_route(route, r, T, lay.top_k)


# ------------------------------------------------------------------ whole layer

@pytest.mark.parametrize("name,T", [("tiny", 16), ("qwen3_decode", 1), ("qwen3_decode", 8),
                                    ("qwen3_decode", 32), ("dsv3_decode", 1), ("dsv3_decode", 16),
                                    ("dsv3_decode", 64), ("dsv4flash_decode", 1),
                                    ("dsv4flash_decode", 16), ("dsv4flash_decode", 64),
                                    ("qwen3_prefill", 4096)])
def test_forward_configs_full(name, T):
    _say(f"forward {name} T={T}")
    lay = workloads.make_layer(name, T, device="cuda")
    out, route = run_forward(lay)
    ref, r = oracle.moe_partial(*oracle_inputs(lay))
    check_route(route, r, T, lay.top_k)
    check_output(out, ref, lay.w_dtype)


# One- and two-token calls with 65 to 256 experts are routed inside the gate/up kernel (each
# workgroup routes with one wave; workgroup 0 writes the routing's outputs).  Its edges through
# the whole layer: two and four experts per router lane, an expert count that is not a multiple
# of 64, 64 pairs (every lane holds one), the shared expert's rows after the hit rows, every
# weight dtype, sigmoid gating, no resident expert, and a faulty slot table.  The cases of three
# to eight tokens check the same shapes just past that edge, where the router kernel runs first.
@pytest.mark.parametrize("seed,E,k,T,gating,shared,wdt,n_res", [
    (40, 128, 8, 2, workloads.GATE_SOFTMAX, False, workloads.DT_BF16, None),
    (41, 200, 3, 1, workloads.GATE_SIGMOID, True, workloads.DT_FP8, None),
    (42, 65, 32, 2, workloads.GATE_SOFTMAX, True, workloads.DT_MXFP4, None),
    (43, 256, 6, 2, workloads.GATE_SIGMOID, False, workloads.DT_F32, None),
    (44, 256, 8, 1, workloads.GATE_SOFTMAX, True, workloads.DT_BF16, 256),
    (45, 129, 4, 2, workloads.GATE_SOFTMAX, True, workloads.DT_FP8, 0),
    (46, 192, 16, 2, workloads.GATE_SOFTMAX, False, workloads.DT_BF16, 0),
    (48, 128, 8, 8, workloads.GATE_SOFTMAX, True, workloads.DT_BF16, None),
    (49, 256, 8, 5, workloads.GATE_SIGMOID, False, workloads.DT_FP8, None),
    (50, 200, 16, 4, workloads.GATE_SOFTMAX, True, workloads.DT_MXFP4, None),
    (51, 130, 2, 7, workloads.GATE_SOFTMAX, False, workloads.DT_F32, 0),
    (52, 256, 6, 3, workloads.GATE_SIGMOID, True, workloads.DT_BF16, 256)])
def test_forward_self_routed(seed, E, k, T, gating, shared, wdt, n_res):
    _say(f"forward self-routed seed={seed} E={E} k={k} T={T} dtype={wdt} shared={shared} resident={n_res}")
    lay = workloads.random_layer(seed, hidden=256, inter=256, n_experts=E, top_k=k, tokens=T, gating=gating,
                                 w_dtype=wdt, n_resident=n_res, shared=shared, zipf_s=1.0, device="cuda")
    out, route = run_forward(lay)
    ref, r = oracle.moe_partial(*oracle_inputs(lay))
    check_route(route, r, T, k)
    check_output(out, ref, lay.w_dtype)


def test_forward_self_routed_invalid_slot_table():
    lay = workloads.random_layer(47, hidden=256, inter=256, n_experts=128, top_k=8, tokens=2,
                                 n_resident=40, shared=True, device="cuda")
    st = lay.slot_table.clone()
    res = (st >= 0).nonzero().flatten().tolist()
    st[res[0]] = st[res[1]]                  # duplicate
    st[res[2]] = lay.n_slots + 5             # out of range
    st[res[3]] = lay.shared_slot             # points at the shared expert
    lay.slot_table = st
    _say(f"forward self-routed, invalid slot table: {st.tolist()}")
    out, route = run_forward(lay)
    ref, r = oracle.moe_partial(*oracle_inputs(lay))
    assert r["status"] == 7
    check_route(route, r, 2, lay.top_k)
    check_output(out, ref, lay.w_dtype)


GEMM_BM = 128      # token rows of one M tile of the many-token (matrix-core) path


def tile_covering_tokens(r, T, k, shared):
    """Tokens whose rows cover the first and the last row of every M tile of every evaluation
    group: each hit expert's rows in the oracle's hit-list order, then the shared expert's T rows
    in token order.  Every tile, every band of tiles and every ragged tail then holds a checked
    row.  Derived from the oracle's routing only."""
    toks = set()
    hit_pairs, hit_off = r["hit_pairs"], r["hit_off"]
    groups = [[int(p) // k for p in hit_pairs[hit_off[e]:hit_off[e + 1]]]
              for e in range(len(hit_off) - 1) if hit_off[e + 1] > hit_off[e]]
    if shared:
        groups.append(list(range(T)))
    for g in groups:
        for m0 in range(0, len(g), GEMM_BM):
            toks.add(g[m0])
            toks.add(g[min(len(g), m0 + GEMM_BM) - 1])
    return sorted(toks)


@pytest.mark.parametrize("name,T", [("dsv3_prefill", 8192), ("dsv4flash_prefill", 8192)])
def test_forward_configs_tile_covering(name, T):
    lay = workloads.make_layer(name, T, device="cuda")
    out, route = run_forward(lay)
    inp = oracle_inputs(lay)
    r = oracle.route(*[inp[0], inp[2], inp[3]])
    rows = tile_covering_tokens(r, T, lay.top_k, lay.shared_slot >= 0)
    _say(f"forward {name} T={T}: {len(rows)} tile-covering rows")
    ref, r2 = oracle.moe_partial(*inp, tokens=rows)
    check_route(route, r2, T, lay.top_k)
    check_output(out, ref, lay.w_dtype, rows=rows)


RANDOM_FWD = [
    # seed, w_dtype, gating, E, k, T, n_res, shared, H, I, zipf
    (0, workloads.DT_BF16, 0, 8, 2, 1, 4, False, 128, 256, 0.0),
    (1, workloads.DT_BF16, 1, 16, 4, 37, 16, False, 256, 128, 0.0),
    (2, workloads.DT_BF16, 0, 16, 4, 70, 0, False, 128, 128, 0.0),
    (3, workloads.DT_BF16, 0, 16, 4, 70, 0, True, 128, 128, 0.0),
    (4, workloads.DT_FP8, 1, 32, 8, 19, 9, True, 384, 256, 0.0),
    (5, workloads.DT_FP8, 0, 12, 3, 130, 12, False, 256, 384, 0.0),
    (6, workloads.DT_F32, 0, 8, 3, 45, 5, True, 128, 384, 0.0),
    (7, workloads.DT_F32, 1, 4, 4, 3, 2, False, 640, 128, 0.0),
    (8, workloads.DT_BF16, 0, 64, 6, 700, 40, True, 256, 256, 0.0),
    # many-token chunks: MFMA GEMM path, ragged M tiles, skewed group sizes
    (9, workloads.DT_BF16, 1, 16, 4, 300, 12, True, 256, 384, 1.5),
    (10, workloads.DT_BF16, 0, 32, 8, 1000, 20, False, 384, 128, 0.8),
    (11, workloads.DT_BF16, 0, 8, 1, 256, 8, False, 128, 128, 3.0),
    (12, workloads.DT_FP8, 1, 24, 6, 400, 10, True, 256, 256, 1.0),
    (13, workloads.DT_BF16, 0, 16, 4, 700, 11, False, 512, 256, 1.0),
    (14, workloads.DT_FP8, 1, 32, 8, 520, 13, True, 512, 384, 2.0),
    (15, workloads.DT_BF16, 1, 8, 8, 260, 8, True, 768, 128, 0.0),
    # MXFP4 weights: streaming and many-token shapes, ragged groups, shared expert, no residency
    (16, workloads.DT_MXFP4, 1, 16, 4, 37, 10, True, 256, 384, 0.0),
    (17, workloads.DT_MXFP4, 0, 8, 2, 5, 8, False, 128, 128, 0.0),
    (18, workloads.DT_MXFP4, 0, 24, 6, 300, 14, True, 384, 256, 1.2),
    (19, workloads.DT_MXFP4, 1, 12, 3, 70, 0, True, 256, 256, 0.0),
    (20, workloads.DT_MXFP4, 0, 32, 8, 520, 13, False, 512, 384, 2.0),
    # every streaming-kernel variant the launcher picks: T <= 16 takes the one-M-tile kernels;
    # fp8 items are wide above 128 pairs, MXFP4 items above 12; the wide gate/up items take four M
    # tiles a pass above 32 tokens (fp8) or from 64 (MXFP4); fp8 down items are wide, two K blocks
    # a batch, above 32 tokens
    (21, workloads.DT_FP8, 1, 32, 12, 16, 20, True, 256, 256, 0.0),    # fp8, one tile, wide
    (22, workloads.DT_FP8, 0, 16, 4, 20, 10, False, 256, 384, 0.0),    # fp8, two tiles, narrow
    (23, workloads.DT_MXFP4, 1, 16, 4, 16, 12, True, 256, 256, 0.0),   # MXFP4, one tile, wide
    (24, workloads.DT_BF16, 0, 16, 4, 16, 16, True, 384, 256, 0.0),    # bf16, T = 16 exactly
    (25, workloads.DT_FP8, 1, 8, 4, 60, 8, True, 256, 256, 0.0),       # fp8 wide gate/up, 4 M tiles a pass
    (26, workloads.DT_MXFP4, 0, 16, 4, 100, 12, True, 256, 256, 0.7),  # MXFP4 wide gate/up, 4 M tiles a pass
    (30, workloads.DT_FP8, 0, 16, 4, 48, 10, True, 512, 640, 0.5),     # fp8 wide down, 5 K blocks (tail batch)
    # groups above 1024 rows (more than one band of 8 M tiles, the last band short): strong skew
    # puts most tokens on the top experts, and the shared expert's 2900 rows make 23 M tiles
    (27, workloads.DT_BF16, 0, 16, 4, 2900, 12, True, 256, 256, 3.0),
    (28, workloads.DT_FP8, 1, 16, 4, 2900, 12, True, 256, 256, 3.0),
    (29, workloads.DT_MXFP4, 0, 16, 4, 2900, 12, True, 256, 256, 3.0),
]


@pytest.mark.parametrize("case", RANDOM_FWD, ids=[str(c[0]) for c in RANDOM_FWD])
def test_forward_random_shapes(case):
    seed, wdt, gating, E, k, T, n_res, shared, H, I, zipf = case
    _say(f"forward random {case}")
    lay = workloads.random_layer(seed, hidden=H, inter=I, n_experts=E, top_k=k, tokens=T,
                                 gating=gating, w_dtype=wdt, n_resident=n_res, shared=shared,
                                 zipf_s=zipf, device="cuda")
    out, route = run_forward(lay)
    ref, r = oracle.moe_partial(*oracle_inputs(lay))
    check_route(route, r, T, k)
    check_output(out, ref, wdt)
    if n_res == 0 and not shared:
        assert not out.any()
    if T >= 2000:
        sizes = np.diff(r["hit_off"])
        assert sizes.max() > 8 * GEMM_BM, "a group must span more than one band of M tiles"


def _sweep_cases(seed, n):
    rng = np.random.default_rng(seed)
    for _ in range(n):
        wdt = int(rng.choice([workloads.DT_BF16, workloads.DT_FP8, workloads.DT_MXFP4]))
        E = int(rng.choice([8, 16, 24, 40, 64, 130]))
        k = int(rng.integers(1, min(E, 9)))
        T = int(rng.choice([int(rng.integers(3, 120)), int(rng.integers(256, 2400))]))
        yield dict(seed=int(rng.integers(0, 1 << 30)), w_dtype=wdt, n_experts=E, top_k=k, tokens=T,
                   hidden=int(rng.choice([256, 512])), inter=int(rng.choice([128, 256, 384])),
                   shared=bool(rng.integers(0, 2)), n_resident=int(rng.integers(0, E + 1)),
                   zipf_s=float(rng.choice([0.0, 1.0, 2.5])), gating=int(rng.integers(0, 2)))


@pytest.mark.parametrize("chunk", range(4))
def test_forward_random_sweep(chunk):
    """A seeded sweep of 40 random layers over every weight format, both paths (3-119 and
    256-2399 tokens), residency from none to full, skew and the shared expert, every row
    checked."""
    for i, c in enumerate(_sweep_cases(2024, 40)):
        if i % 4 != chunk:
            continue
        _say(f"sweep {i}: {c}")
        seed = c.pop("seed")
        lay = workloads.random_layer(seed, device="cuda", **c)
        out, route = run_forward(lay)
        ref, r = oracle.moe_partial(*oracle_inputs(lay))
        check_route(route, r, c["tokens"], c["top_k"])
        check_output(out, ref, c["w_dtype"])


@pytest.mark.parametrize("wdt", [workloads.DT_BF16, workloads.DT_FP8, workloads.DT_MXFP4])
def test_gemm_tile_classes(wdt):
    """Groups sized at the edges of the router's GEMM tile classes (1, 32, 33, 64, 65, 96, 97, 128,
    129 and 300 rows, one routed expert per token, plus a shared expert): every class, the class
    boundaries and groups of one and of several M tiles in one call, checked on every row."""
    sizes = [32, 33, 64, 65, 96, 97, 128, 129, 1, 300]
    E, T = 12, sum(sizes)
    lay = workloads.random_layer(77, hidden=256, inter=256, n_experts=E, top_k=1, tokens=T,
                                 w_dtype=wdt, gating=0, n_resident=E, shared=True)
    owner = np.repeat(np.arange(len(sizes)), sizes)
    np.random.default_rng(5).shuffle(owner)      # tokens of one expert scattered over the batch
    logits = np.random.default_rng(6).normal(size=(T, E)).astype(np.float32)
    logits[np.arange(T), owner] += 20.0
    lay.logits = torch.from_numpy(logits)
    lay = lay.to("cuda")
    _say(f"GEMM tile classes, dtype {wdt}")
    out, route = run_forward(lay)
    ref, r = oracle.moe_partial(*oracle_inputs(lay))
    assert sorted(np.diff(r["hit_off"])[np.diff(r["hit_off"]) > 0].tolist()) == sorted(sizes)
    check_route(route, r, T, 1)
    check_output(out, ref, wdt)


@pytest.mark.parametrize("T", [20, 300])
def test_fp8_zero_block_scales(T):
    """fp8 block scales of 0 (the weights of that block are 0) on the streaming path (T = 20) and
    the matrix-core path (T = 300): a zero first block, a run of zero blocks, a zero last block,
    and one expert whose gate/up scales are all zero."""
    lay = workloads.random_layer(50 + T, hidden=512, inter=384, n_experts=8, top_k=3, tokens=T,
                                 w_dtype=workloads.DT_FP8, gating=1, n_resident=8, shared=True,
                                 device="cuda")
    s13, s2 = lay.s13, lay.s2               # [slots][2I/128][H/128], [slots][H/128][I/128]
    s13[0, :, 0] = 0
    s13[1, 1, 1:3] = 0
    s13[2, :, -1] = 0
    s13[3] = 0
    s2[0, :, 0] = 0
    s2[4, 2, :] = 0
    s2[5, :, 1] = 0
    _say(f"fp8 zero block scales T={T}")
    out, route = run_forward(lay)
    ref, r = oracle.moe_partial(*oracle_inputs(lay))
    check_route(route, r, T, lay.top_k)
    check_output(out, ref, lay.w_dtype)


@pytest.mark.parametrize("name,T", [("qwen3_decode", 1), ("qwen3_decode", 32), ("dsv3_decode", 16),
                                    ("dsv4flash_decode", 16), ("tiny", 16)])
def test_forward_atomic_combine(name, T):
    """The atomic combine (float32 atomics from the down projection) matches the oracle too."""
    _say(f"forward atomic combine {name} T={T}")
    lay = workloads.make_layer(name, T, device="cuda")
    desc = dict(lay.desc(), combine=ftm.FT_COMBINE_ATOMIC)
    ws = ftm.alloc_workspace(desc, T)
    route = ftm.RouteBuffers(T, lay.top_k, lay.n_experts)
    out = torch.full((T, lay.hidden), float("nan"), dtype=torch.float32, device="cuda")
    ftm.ft_moe_forward(desc, ftm.banks_of(lay), lay.logits, lay.slot_table, lay.x, T, out, route, ws)
    torch.cuda.synchronize()
    ref, r = oracle.moe_partial(*oracle_inputs(lay))
    check_route(route, r, T, lay.top_k)
    check_output(out, ref, lay.w_dtype)


def test_forward_T0_is_noop():
    lay = workloads.make_layer("tiny", 16, device="cuda")
    desc = lay.desc()
    ws = ftm.alloc_workspace(desc, 16)
    route = ftm.RouteBuffers(16, lay.top_k, lay.n_experts)
    out = torch.full((16, lay.hidden), 7.0, device="cuda")
    ftm.ft_moe_forward(desc, ftm.banks_of(lay), lay.logits, lay.slot_table, lay.x, 0, out, route, ws)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())


@pytest.mark.parametrize("case", ["tiny", "random"])
def test_miss_list_to_host(case):
    """The host copies of the miss list equal the oracle's routing."""
    if case == "tiny":
        lay = workloads.make_layer("tiny", 16, device="cuda")
    else:
        lay = workloads.random_layer(31, hidden=128, inter=128, n_experts=40, top_k=6, tokens=77,
                                     n_resident=15, shared=True, tie_logits=True, device="cuda")
    T, k = lay.tokens, lay.top_k
    out, route = run_forward(lay)
    host = ftm.HostMissBuffers(T, k, lay.n_experts)
    ftm.ft_miss_list_to_host(lay.desc(), route, T, host)
    torch.cuda.synchronize()
    desc, banks, logits, st, x = oracle_inputs(lay)
    r = oracle.route(desc, logits, st)
    assert r["n_miss"] > 0
    assert host.counts.tolist() == [r["n_hit"], r["n_miss"], r["m_unique_miss"], r["status"]]
    mp = host.miss_pairs.numpy()[: T * k]
    assert np.array_equal(mp[: r["n_miss"]], r["miss_pairs"]) and np.all(mp[r["n_miss"]:] == -1)
    assert np.array_equal(host.miss_off.numpy(), r["miss_off"])
    assert np.array_equal(host.topk_ids.numpy()[: T * k].reshape(T, k), r["topk_ids"])
    np.testing.assert_allclose(host.topk_w.numpy()[: T * k].reshape(T, k), r["topk_w"], rtol=0, atol=2e-6)


def test_forward_deterministic_and_slot_table_change():
    """Same inputs twice give identical routing bits and, on the streaming path (whose combine
    sums every output element in a fixed order), bit-identical outputs; a new slot table between
    calls (the runtime cache rebuild of Section 3.3) is honoured, down to zero residency."""
    lay = workloads.random_layer(12, hidden=256, inter=256, n_experts=32, top_k=4, tokens=40,
                                 w_dtype=workloads.DT_BF16, n_resident=20, device="cuda")
    a, ra = run_forward(lay)
    b, rb = run_forward(lay)
    for n in ("topk_ids", "topk_w", "topk_slot", "hit_pairs", "miss_pairs", "hit_off", "miss_off",
              "counts"):
        assert torch.equal(getattr(ra, n), getattr(rb, n)), n
    assert torch.equal(a, b)
    st = lay.slot_table.clone()
    st[: 16] = -1
    lay.slot_table = st
    out, route = run_forward(lay)
    ref, r = oracle.moe_partial(*oracle_inputs(lay))
    check_route(route, r, 40, 4)
    check_output(out, ref, workloads.DT_BF16)
    lay.slot_table = torch.full_like(st, -1)
    out, route = run_forward(lay)
    assert not out.any() and int(route.counts[0]) == 0


def test_binding_rejects_undersized_or_mistyped_device_tensors():
    """Buffers too small for T, k or E, or of the wrong dtype, raise before the library runs."""
    lay = workloads.make_layer("tiny", 16, device="cuda")
    desc, T = lay.desc(), 16
    ws = ftm.alloc_workspace(desc, T)
    banks = ftm.banks_of(lay)
    out = torch.empty(T, lay.hidden, device="cuda")
    ok_route = ftm.RouteBuffers(T, lay.top_k, lay.n_experts)
    fwd = lambda **kw: ftm.ft_moe_forward(desc, kw.get("banks", banks), kw.get("logits", lay.logits),
                                          lay.slot_table, kw.get("x", lay.x), T, kw.get("out", out),
                                          kw.get("route", ok_route), ws)
    with pytest.raises(ValueError, match="route"):
        fwd(route=ftm.RouteBuffers(T - 1, lay.top_k, lay.n_experts))
    with pytest.raises(ValueError, match="route"):
        fwd(route=ftm.RouteBuffers(T, lay.top_k, lay.n_experts - 1))
    with pytest.raises(ValueError, match="logits"):
        fwd(logits=lay.logits.double())
    with pytest.raises(ValueError, match="x"):
        fwd(x=lay.x[: T - 1])
    with pytest.raises(ValueError, match="out_partial"):
        fwd(out=out[: T - 1])
    with pytest.raises(ValueError, match="w13"):
        fwd(banks=dict(banks, w13=lay.w13[:-1]))
    fwd()
    torch.cuda.synchronize()
