"""Host-side checks of the C ABI: the library loads, exports what include/ftmoe.h declares,
and rejects bad arguments before touching the GPU.  CPU only."""
import ctypes
import os
import re

import pytest

import paper_2608_16157_amd as ftm
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "ftmoe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ft_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = ftm.load()
    names = _declared_functions()
    assert set(names) == set(ftm.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    for s in range(6):
        assert ftm.ft_status_string(s).startswith("FT_")
    assert ftm.ft_status_string(99) == "unknown status"


def _desc(**kw):
    d = workloads.make_layer("tiny", 4).desc()
    d.update(kw)
    return d


def test_workspace_bytes():
    for name, cfg in workloads.CONFIGS.items():
        d = dict(hidden=cfg.hidden, inter=cfg.inter, n_experts=cfg.n_experts, top_k=cfg.top_k,
                 gating=cfg.gating, w_dtype=cfg.w_dtype, x_dtype=cfg.x_dtype, n_slots=200,
                 shared_slot=-1)
        for T in cfg.tokens:
            assert ftm.ft_moe_workspace_bytes(d, T) > 0
        assert ftm.ft_moe_workspace_bytes(d, 64) >= ftm.ft_moe_workspace_bytes(d, 8)
    assert ftm.ft_moe_workspace_bytes(_desc(hidden=100), 4) == 0
    assert ftm.ft_moe_workspace_bytes(_desc(top_k=9), 4) == 0       # k > E
    assert ftm.ft_moe_workspace_bytes(_desc(n_experts=2000, top_k=2), 4) == 0
    assert ftm.ft_moe_workspace_bytes(_desc(shared_slot=4), 4) == 0  # shared slot outside pool
    assert ftm.ft_moe_workspace_bytes(_desc(), -1) == 0


FAKE = 0x10000  # never dereferenced: every case below fails host validation first


def _route_call(desc, T, ws_bytes=1 << 40, logits=FAKE, null_route=False):
    lib = ftm.load()
    r = ftm.ft_route_t(*([None] * 8 if null_route else [FAKE] * 8))
    return lib.ft_route_only(ctypes.byref(ftm.make_desc(desc)), logits, FAKE, T, ctypes.byref(r),
                             FAKE, ws_bytes, None)



@pytest.mark.parametrize("desc_kw,T,kw,want", [
    ({}, 0, {}, ftm.FT_OK),                                    # T == 0 is a no-op
    ({}, 4, {"logits": None}, ftm.FT_ERR_NULL),
    ({}, 4, {"null_route": True}, ftm.FT_ERR_NULL),
    ({"hidden": 200}, 4, {}, ftm.FT_ERR_SHAPE),
    ({}, -1, {}, ftm.FT_ERR_SHAPE),
    ({"gating": 7}, 4, {}, ftm.FT_ERR_DTYPE),
    ({"w_dtype": 1, "x_dtype": 0}, 4, {}, ftm.FT_ERR_DTYPE),   # bf16 weights need bf16 x
    ({"w_dtype": 0, "x_dtype": 1}, 4, {}, ftm.FT_ERR_DTYPE),
    ({}, 4, {"ws_bytes": 64}, ftm.FT_ERR_CAPACITY),
])
def test_route_only_rejects_before_enqueue(desc_kw, T, kw, want):
    assert _route_call(_desc(**desc_kw), T, **kw) == want


def test_forward_rejects_null_banks():
    lib = ftm.load()
    d = ftm.make_desc(_desc())
    r = ftm.ft_route_t(*[FAKE] * 8)
    b = ftm.ft_banks_t(None, None, None, None)
    st = lib.ft_moe_forward(ctypes.byref(d), ctypes.byref(b), FAKE, FAKE, FAKE, 4, FAKE,
                            ctypes.byref(r), FAKE, 1 << 40, None)
    assert st == ftm.FT_ERR_NULL
    st = lib.ft_moe_forward(ctypes.byref(d), None, FAKE, FAKE, FAKE, 4, FAKE,
                            ctypes.byref(r), FAKE, 1 << 40, None)
    assert st == ftm.FT_ERR_NULL
    fp8 = ftm.make_desc(_desc(w_dtype=2, x_dtype=1))
    b = ftm.ft_banks_t(FAKE, FAKE, None, None)                  # fp8 without scales
    st = lib.ft_moe_forward(ctypes.byref(fp8), ctypes.byref(b), FAKE, FAKE, FAKE, 4, FAKE,
                            ctypes.byref(r), FAKE, 1 << 40, None)
    assert st == ftm.FT_ERR_NULL


def test_miss_list_to_host_rejects_nulls():
    lib = ftm.load()
    d = ftm.make_desc(_desc())
    r = ftm.ft_route_t(*[FAKE] * 8)
    h = ftm.ft_host_miss_t(None, FAKE, FAKE, FAKE, FAKE)
    assert lib.ft_miss_list_to_host(ctypes.byref(d), ctypes.byref(r), 4, ctypes.byref(h), None) == ftm.FT_ERR_NULL


def test_cache_plan_rejects_before_enqueue():
    """Host-side validation of ft_cache_plan (fake device pointers: nothing may be enqueued)."""
    lib = ftm.load()
    d = ftm.make_desc(_desc())
    r = ftm.ft_route_t(*[FAKE] * 8)
    st = ftm.ft_cache_state_t(FAKE, FAKE)
    pl = ftm.ft_fill_plan_t(*[FAKE] * 5)

    def call(desc=d, route=r, T=4, table=FAKE, state=st, pol=None, plan=pl):
        pol = pol or ftm.ft_cache_policy_t(1.0, 2.0, 4, 1)
        return lib.ft_cache_plan(ctypes.byref(desc), ctypes.byref(route), T, table,
                                 ctypes.byref(state), ctypes.byref(pol), ctypes.byref(plan), None)

    assert call(table=None) == ftm.FT_ERR_NULL
    assert call(state=ftm.ft_cache_state_t(None, FAKE)) == ftm.FT_ERR_NULL
    assert call(plan=ftm.ft_fill_plan_t(FAKE, FAKE, FAKE, None, FAKE)) == ftm.FT_ERR_NULL
    assert call(route=ftm.ft_route_t(*([FAKE] * 7 + [None]))) == ftm.FT_ERR_NULL
    assert call(T=-1) == ftm.FT_ERR_SHAPE
    assert call(pol=ftm.ft_cache_policy_t(1.0, 2.0, 0, 1)) == ftm.FT_ERR_SHAPE
    assert call(pol=ftm.ft_cache_policy_t(1.0, 2.0, 65, 1)) == ftm.FT_ERR_SHAPE
    assert call(pol=ftm.ft_cache_policy_t(0.0, 2.0, 4, 1)) == ftm.FT_ERR_SHAPE
    assert call(pol=ftm.ft_cache_policy_t(1.0, float("nan"), 4, 1)) == ftm.FT_ERR_SHAPE
    assert call(desc=ftm.make_desc(_desc(n_slots=5000))) == ftm.FT_ERR_SHAPE
    assert call(T=0) == ftm.FT_OK          # nothing to plan, nothing enqueued


def test_fill_and_hybrid_reject_before_enqueue():
    lib = ftm.load()
    d = ftm.make_desc(_desc(w_dtype=1, x_dtype=1, hidden=128, inter=128))
    b = ftm.ft_banks_t(FAKE, FAKE, None, None)
    pl = ftm.ft_fill_plan_t(*[FAKE] * 5)
    assert lib.ft_cache_fill(ctypes.byref(d), None, ctypes.byref(b), ctypes.byref(pl), 4, None) == ftm.FT_ERR_NULL
    assert lib.ft_cache_fill(ctypes.byref(d), ctypes.byref(b), ctypes.byref(b), ctypes.byref(pl), 0, None) == ftm.FT_ERR_SHAPE
    assert lib.ft_cache_fill(ctypes.byref(d), ctypes.byref(b), ctypes.byref(b), ctypes.byref(pl), 65, None) == ftm.FT_ERR_SHAPE
    nb = ftm.ft_banks_t(None, FAKE, None, None)
    assert lib.ft_cache_fill(ctypes.byref(d), ctypes.byref(nb), ctypes.byref(b), ctypes.byref(pl), 4, None) == ftm.FT_ERR_NULL
    st = ftm.ft_cache_state_t(FAKE, FAKE, None)
    pol = ftm.ft_cache_policy_t(1.0, 2.0, 4, 1)
    r = ftm.ft_route_t(*[FAKE] * 8)
    h = ftm.ft_hybrid_host_t(*[FAKE] * 7)
    args = [ctypes.byref(d), ctypes.byref(b), ctypes.byref(b), FAKE, FAKE, ctypes.byref(st),
            ctypes.byref(pol), FAKE, 4, FAKE, ctypes.byref(r), ctypes.byref(pl), ctypes.byref(h),
            FAKE, 1 << 20, None, FAKE]
    a = list(args)
    a[12] = ctypes.byref(ftm.ft_hybrid_host_t(FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE))
    assert lib.ft_moe_step_hybrid(*a) == ftm.FT_ERR_NULL
    a = list(args)
    a[12] = ctypes.byref(ftm.ft_hybrid_host_t(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None))   # no task
    assert lib.ft_moe_step_hybrid(*a) == ftm.FT_ERR_NULL
    a = list(args)
    a[9] = None                # no output
    assert lib.ft_moe_step_hybrid(*a) == ftm.FT_ERR_NULL
    a = list(args)
    a[12] = ctypes.byref(ftm.ft_hybrid_host_t(FAKE, FAKE, FAKE, FAKE, FAKE + 4, FAKE, FAKE))   # misaligned x staging
    assert lib.ft_moe_step_hybrid(*a) == ftm.FT_ERR_SHAPE
    a = list(args)
    a[8] = 0
    assert lib.ft_moe_step_hybrid(*a) == ftm.FT_OK


def test_cpu_pool_create_destroy():
    """Pools start, serve a no-op call and stop; unpinned and pinned, explicit and default sizes."""
    for n, pin in ((1, False), (3, True), (0, True)):
        p = ftm.ft_cpu_pool_create(n, pin)
        assert p.handle
        ftm.ft_cpu_pool_destroy(p)
        assert p.handle is None


def test_library_has_no_undefined_library_symbols():
    """Every kernel stub and internal function of libftmoe is defined in the library itself (a
    kernel whose host stub the compiler dropped would only fail when first launched)."""
    import subprocess
    out = subprocess.run(["nm", "-D", "--undefined-only", ftm.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    missing = [l for l in out.splitlines() if "ftmoe" in l]
    assert not missing, missing


def _prefill_call(desc, n_layers=2, T=4, overlap=1, copy_stream=FAKE + 8, stream=FAKE, null=None,
                  ws_bytes=1 << 40, same_buf=False):
    """ft_prefill_layers with fake device pointers; ``null`` names one argument to pass as NULL."""
    lib = ftm.load()
    n = max(n_layers, 1)
    bank = lambda base: ftm.ft_banks_t(base, base + 0x100, base + 0x200, base + 0x300)
    hl = (ftm.ft_banks_t * n)(*[bank(FAKE * (l + 3)) for l in range(n)])
    db = (ftm.ft_banks_t * 2)(bank(FAKE), bank(FAKE if same_buf else 2 * FAKE))
    arr = lambda: (ctypes.c_void_p * n)(*([FAKE] * n))
    logits, x, out = arr(), arr(), arr()
    if null == "x_layer":
        x[n - 1] = None
    if null == "dev_w2":
        db[1].w2 = None
    r = ftm.ft_route_t(*[FAKE] * 8)
    args = dict(hl=hl, db=db, logits=logits, x=x, out=out, route=ctypes.byref(r))
    if null in args:
        args[null] = None
    return lib.ft_prefill_layers(ctypes.byref(ftm.make_desc(desc)), n_layers, args["hl"], args["db"],
                                 FAKE, args["logits"], args["x"], T, args["out"], args["route"], FAKE,
                                 ws_bytes, overlap, stream, copy_stream)


@pytest.mark.parametrize("kw,want", [
    ({"n_layers": 0}, ftm.FT_OK),
    ({"T": 0}, ftm.FT_OK),
    ({"n_layers": -1}, ftm.FT_ERR_SHAPE),
    ({"overlap": 2}, ftm.FT_ERR_SHAPE),
    ({"copy_stream": None}, ftm.FT_ERR_SHAPE),           # overlap needs its own transfer stream
    ({"copy_stream": FAKE}, ftm.FT_ERR_SHAPE),           # ... distinct from the evaluation stream
    ({"same_buf": True}, ftm.FT_ERR_SHAPE),              # the two buffers must be distinct
    ({"null": "hl"}, ftm.FT_ERR_NULL),
    ({"null": "db"}, ftm.FT_ERR_NULL),
    ({"null": "route"}, ftm.FT_ERR_NULL),
    ({"null": "x_layer"}, ftm.FT_ERR_NULL),
    ({"null": "dev_w2"}, ftm.FT_ERR_NULL),
    ({"ws_bytes": 64}, ftm.FT_ERR_CAPACITY),
])
def test_prefill_layers_rejects_before_enqueue(kw, want):
    assert _prefill_call(_desc(), **kw) == want
    assert _prefill_call(_desc(hidden=100), **kw) in (ftm.FT_ERR_SHAPE, ftm.FT_ERR_NULL, want)


def test_missing_library_fails_loudly(tmp_path):
    """Without the built library every call raises; nothing falls back to another path."""
    import subprocess
    import sys
    code = ("import paper_2608_16157_amd as ftm\n"
            "try:\n"
            "    ftm.ft_moe_workspace_bytes({'hidden': 256, 'inter': 512, 'n_experts': 8, 'top_k': 2,"
            " 'gating': 0, 'w_dtype': 0, 'x_dtype': 0, 'n_slots': 4, 'shared_slot': -1}, 4)\n"
            "except RuntimeError as e:\n"
            "    print('raised:', e)\n"
            "    raise SystemExit(0)\n"
            "raise SystemExit(1)\n")
    env = dict(os.environ, FTMOE_LIBRARY=str(tmp_path / "absent.so"))
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "not built" in r.stdout


def test_binding_rejects_host_tensors_and_bad_sizes_before_the_call():
    """The binding checks device, dtype and size of every tensor it hands to the C ABI (which
    carries no capacities) and raises ValueError before entering the library."""
    import torch
    d = _desc()
    T, E, H = 4, d["n_experts"], d["hidden"]
    route = ftm.RouteBuffers.__new__(ftm.RouteBuffers)
    route.T, route.k, route.E = T, d["top_k"], E
    with pytest.raises(ValueError, match="device"):
        ftm.ft_route_only(d, torch.zeros(T, E), torch.zeros(E, dtype=torch.int32), T, route,
                          torch.zeros(16, dtype=torch.uint8))
    with pytest.raises(ValueError, match="route"):
        ftm._need_route(route, d, T + 1)
    with pytest.raises(ValueError, match="route"):
        ftm._need_route(route, dict(d, n_experts=E + 1), T)
    # host-side checks of the CPU branch run without a GPU
    ids = torch.zeros(T, d["top_k"], dtype=torch.int32)
    w = torch.zeros(T, d["top_k"])
    lst = torch.zeros(1, dtype=torch.int32)
    x = torch.zeros(T, H)
    with pytest.raises(ValueError, match="out"):
        ftm.ft_cpu_experts(d, {}, x, T, ids, w, lst, torch.zeros(T * H - 1))
    with pytest.raises(ValueError, match="dtype"):
        ftm.ft_cpu_experts(d, {}, x, T, ids.float(), w, lst, torch.zeros(T, H))
    with pytest.raises(ValueError, match="host_pool"):
        ftm.ft_cpu_experts(d, {"w13": torch.zeros(1), "w2": torch.zeros(1)}, x, T, ids, w, lst,
                           torch.zeros(T, H))
    assert ftm.expert_bank_bytes(dict(d, w_dtype=ftm.FT_DT_FP8E4M3FN_B128, hidden=256, inter=128)) == \
        (2 * 128 * 256, 256 * 128, 2 * 2 * 4, 2 * 1 * 4)


def test_act_quant_validation():
    """The fp8-activation mode: unknown values make the description invalid, non-fp8 weights
    are refused as a dtype error, the CPU branch (which evaluates exactly) refuses the mode, and
    the workspace follows the mode: the streaming path adds a bf16 copy of the quantised x, the
    matrix-core path holds x and h as codes and exponents in place of the bf16 h."""
    lib = ftm.load()
    H, I, k = 256, 256, 2
    fp8 = _desc(w_dtype=2, x_dtype=1, hidden=H, inter=I, top_k=k)
    assert lib.ft_moe_workspace_bytes(ctypes.byref(ftm.make_desc(dict(fp8, act_quant=2))), 8) == 0
    ws = lambda d, T: lib.ft_moe_workspace_bytes(ctypes.byref(ftm.make_desc(d)), T)
    T = 8   # streaming path (ordered combine)
    assert ws(dict(fp8, act_quant=1), T) - ws(fp8, T) in range(T * H * 2, T * H * 2 + 256)
    T = 300
    rows = T * (k + 1)   # evaluation rows are sized for a shared expert in every case
    codes = T * H + T * H // 128 + rows * I + rows * I // 128
    diff = ws(dict(fp8, act_quant=1), T) - ws(fp8, T)
    assert abs(diff - (codes - rows * I * 2)) < 5 * 256
    d = ftm.make_desc(dict(fp8, act_quant=1))
    pool = ftm.ft_banks_t(FAKE, FAKE, FAKE, FAKE)
    assert lib.ft_cpu_experts(ctypes.byref(d), ctypes.byref(pool), FAKE, 1, FAKE, FAKE, FAKE, 1, FAKE,
                              None) == ftm.FT_ERR_DTYPE
    # the hybrid step merges with the CPU branch's exact partial: the mode is refused there too
    fb = ftm.ft_banks_t(FAKE, FAKE, FAKE, FAKE)
    pl = ftm.ft_fill_plan_t(*[FAKE] * 5)
    st = ftm.ft_cache_state_t(FAKE, FAKE, None)
    pol = ftm.ft_cache_policy_t(1.0, 2.0, 4, 1)
    hh = ftm.ft_hybrid_host_t(*[FAKE] * 7)
    rr = ftm.ft_route_t(*[FAKE] * 8)
    hyb = lambda desc: lib.ft_moe_step_hybrid(
        ctypes.byref(desc), ctypes.byref(fb), ctypes.byref(fb), FAKE, FAKE, ctypes.byref(st), ctypes.byref(pol),
        FAKE, 4, FAKE, ctypes.byref(rr), ctypes.byref(pl), ctypes.byref(hh), FAKE, 1 << 30, None, FAKE)
    assert hyb(d) == ftm.FT_ERR_DTYPE
    assert hyb(ftm.make_desc(fp8)) == ftm.FT_ERR_SHAPE   # exact: passes to the staging lookup, which fails
    bf = ftm.make_desc(_desc(w_dtype=1, x_dtype=1, act_quant=1))
    r = ftm.ft_route_t(*[FAKE] * 8)
    assert lib.ft_route_only(ctypes.byref(bf), FAKE, FAKE, 4, ctypes.byref(r), FAKE, 1 << 30, None) == ftm.FT_ERR_DTYPE
