"""Python binding of libftmoe: the MoE layer executed against a GPU expert cache on gfx950.

Argument marshalling only.  Every step of the layer runs in the HIP kernels of
``libftmoe.so``; torch provides device memory and streams.  The entry points keep the names
of the C ABI declared in ``include/ftmoe.h``:

    ft_moe_workspace_bytes(desc, max_tokens) -> int
    ft_route_only(desc, logits, slot_table, T, route, ws, stream=None)
    ft_moe_forward(desc, banks, logits, slot_table, x, T, out_partial, route, ws, stream=None)
    ft_moe_forward_profiled(desc, banks, logits, slot_table, x, T, out_partial, route, ws,
                            events, stream=None)
    ft_moe_forward_noalloc(desc, banks, logits, slot_table, x, T, out_partial, route, stream=None)
    ft_miss_list_to_host(desc, route, T, host, stream=None)
    ft_cache_plan(desc, route, T, slot_table, state, policy, plan, stream=None)
    ft_cpu_pool_create(n_threads=0, pin=True) -> CpuPool;  ft_cpu_pool_destroy(pool)
    ft_cpu_experts(desc, host_pool, x, T, topk_ids, topk_w, experts, out, pool=None)
    ft_cache_fill(desc, host_pool, dev_banks, plan, max_fill, stream=None)
    ft_moe_step_hybrid(desc, dev_banks, host_pool, logits, slot_table, state, b_pcie, b_host,
                       max_fill, step, x, T, out, route, plan, host, ws, pool, stream=None)
    ft_prefill_layers(desc, host_layers, dev_bufs, slot_table, logits, x, T, out, route, ws,
                      overlap=True, stream=None, copy_stream=None)
    ft_status_string(status) -> str

``desc`` is a dict with the ft_moe_desc_t fields; ``route`` a RouteBuffers; ``banks`` a dict
with w13, w2 (and s13, s2 for fp8) device tensors; everything else device tensors.  A non-OK
status raises FtError.  If the library is not built, importing works but every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libftmoe.so")

FT_OK, FT_ERR_NULL, FT_ERR_SHAPE, FT_ERR_DTYPE, FT_ERR_CAPACITY, FT_ERR_HIP = range(6)
FT_GATE_SOFTMAX_TOPK_RENORM, FT_GATE_SIGMOID_TOPK_RENORM = 0, 1
FT_COMBINE_ORDERED, FT_COMBINE_ATOMIC = 0, 1
FT_ACT_EXACT, FT_ACT_FP8_1x128_POW2 = 0, 1
FT_DT_F32, FT_DT_BF16, FT_DT_FP8E4M3FN_B128, FT_DT_MXFP4 = 0, 1, 2, 3
FT_SLOT_MISS = -1
FT_DEV_SLOT_RANGE, FT_DEV_SLOT_DUP, FT_DEV_SLOT_SHARED = 1, 2, 4

EXPORTED = ("ft_moe_workspace_bytes", "ft_route_only", "ft_moe_forward", "ft_moe_forward_noalloc",
            "ft_moe_forward_profiled", "ft_miss_list_to_host", "ft_cache_plan", "ft_cpu_experts",
            "ft_cache_fill", "ft_moe_step_hybrid", "ft_prefill_layers", "ft_status_string",
            "ft_cpu_pool_create", "ft_cpu_pool_destroy")
FT_PROF_STAGES = 4
FT_NOALLOC_SCRATCH_BYTES = 64 << 20


class FtError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {_status_text(status)}")


class ft_moe_desc_t(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("hidden", "inter", "n_experts", "top_k", "gating",
                                              "w_dtype", "x_dtype", "n_slots", "shared_slot",
                                              "combine", "act_quant")]


class ft_banks_t(ctypes.Structure):
    _fields_ = [("w13", ctypes.c_void_p), ("w2", ctypes.c_void_p), ("s13", ctypes.c_void_p),
                ("s2", ctypes.c_void_p)]


class ft_route_t(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("topk_ids", "topk_w", "topk_slot", "hit_pairs",
                                               "miss_pairs", "hit_off", "miss_off", "counts")]


class ft_prof_events_t(ctypes.Structure):
    _fields_ = [("ev", ctypes.c_void_p * 5)]


class ft_host_miss_t(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("counts", "miss_pairs", "miss_off", "topk_ids",
                                               "topk_w")]


class ft_cache_state_t(ctypes.Structure):
    _fields_ = [("slot_expert", ctypes.c_void_p), ("slot_stamp", ctypes.c_void_p),
                ("clock", ctypes.c_void_p)]


class ft_cache_policy_t(ctypes.Structure):
    _fields_ = [("b_pcie", ctypes.c_double), ("b_host", ctypes.c_double),
                ("max_fill", ctypes.c_int32), ("step", ctypes.c_uint32)]


class ft_fill_plan_t(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("fill_expert", "fill_slot", "evict_expert",
                                               "cpu_expert", "counts")]


class ft_hybrid_host_t(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("plan_counts", "cpu_expert", "topk_ids", "topk_w", "x",
                                               "cpu_out", "task")]


FT_HYBRID_TASK_BYTES = 24 * 8


_lib: Optional[ctypes.CDLL] = None


def load(path: str = None) -> ctypes.CDLL:
    """Load libftmoe.so once (FTMOE_LIBRARY may name another build); raise if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or os.environ.get("FTMOE_LIBRARY") or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"libftmoe.so not built ({path}); run __graft_entry__.build() or "
                           "python paper_2608_16157_amd/build.py")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    lib.ft_moe_workspace_bytes.restype = ctypes.c_size_t
    lib.ft_moe_workspace_bytes.argtypes = [P(ft_moe_desc_t), ctypes.c_int32]
    lib.ft_route_only.restype = ctypes.c_int
    lib.ft_route_only.argtypes = [P(ft_moe_desc_t), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                  P(ft_route_t), ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    lib.ft_moe_forward.restype = ctypes.c_int
    lib.ft_moe_forward.argtypes = [P(ft_moe_desc_t), P(ft_banks_t), ctypes.c_void_p, ctypes.c_void_p,
                                   ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, P(ft_route_t),
                                   ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    lib.ft_moe_forward_noalloc.restype = ctypes.c_int
    lib.ft_moe_forward_noalloc.argtypes = [P(ft_moe_desc_t), P(ft_banks_t), ctypes.c_void_p,
                                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                           ctypes.c_void_p, P(ft_route_t), ctypes.c_void_p]
    lib.ft_moe_forward_profiled.restype = ctypes.c_int
    lib.ft_moe_forward_profiled.argtypes = lib.ft_moe_forward.argtypes + [P(ft_prof_events_t)]
    lib.ft_miss_list_to_host.restype = ctypes.c_int
    lib.ft_miss_list_to_host.argtypes = [P(ft_moe_desc_t), P(ft_route_t), ctypes.c_int32,
                                         P(ft_host_miss_t), ctypes.c_void_p]
    lib.ft_cache_plan.restype = ctypes.c_int
    lib.ft_cache_plan.argtypes = [P(ft_moe_desc_t), P(ft_route_t), ctypes.c_int32, ctypes.c_void_p,
                                  P(ft_cache_state_t), P(ft_cache_policy_t), P(ft_fill_plan_t),
                                  ctypes.c_void_p]
    lib.ft_cpu_pool_create.restype = ctypes.c_void_p
    lib.ft_cpu_pool_create.argtypes = [ctypes.c_int32, ctypes.c_int32]
    lib.ft_cpu_pool_destroy.restype = None
    lib.ft_cpu_pool_destroy.argtypes = [ctypes.c_void_p]
    lib.ft_cpu_experts.restype = ctypes.c_int
    lib.ft_cpu_experts.argtypes = [P(ft_moe_desc_t), P(ft_banks_t), ctypes.c_void_p, ctypes.c_int32,
                                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                   ctypes.c_void_p, ctypes.c_void_p]
    lib.ft_cache_fill.restype = ctypes.c_int
    lib.ft_cache_fill.argtypes = [P(ft_moe_desc_t), P(ft_banks_t), P(ft_banks_t), P(ft_fill_plan_t),
                                  ctypes.c_int32, ctypes.c_void_p]
    lib.ft_moe_step_hybrid.restype = ctypes.c_int
    lib.ft_moe_step_hybrid.argtypes = [P(ft_moe_desc_t), P(ft_banks_t), P(ft_banks_t), ctypes.c_void_p,
                                       ctypes.c_void_p, P(ft_cache_state_t), P(ft_cache_policy_t),
                                       ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                       P(ft_route_t), P(ft_fill_plan_t), P(ft_hybrid_host_t),
                                       ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p]
    lib.ft_prefill_layers.restype = ctypes.c_int
    lib.ft_prefill_layers.argtypes = [P(ft_moe_desc_t), ctypes.c_int32, P(ft_banks_t), P(ft_banks_t),
                                      ctypes.c_void_p, P(ctypes.c_void_p), P(ctypes.c_void_p),
                                      ctypes.c_int32, P(ctypes.c_void_p), P(ft_route_t), ctypes.c_void_p,
                                      ctypes.c_size_t, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    lib.ft_status_string.restype = ctypes.c_char_p
    lib.ft_status_string.argtypes = [ctypes.c_int]
    _lib = lib
    return lib


def _status_text(status: int) -> str:
    try:
        return load().ft_status_string(status).decode()
    except RuntimeError:
        return f"status {status}"


def ft_status_string(status: int) -> str:
    return load().ft_status_string(status).decode()


# ------------------------------------------------------------------------------ marshalling

def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libftmoe must be contiguous")
    return t.data_ptr()


# ------------------------------------------------------------------------------ validation
# The C ABI carries device pointers without capacities, so every wrapper checks the tensors it
# passes (device, dtype, element count) against the sizes the call will touch, and raises
# ValueError before the library is entered.

_X_DTYPES = {FT_DT_F32: torch.float32, FT_DT_BF16: torch.bfloat16}
_W_DTYPES = {FT_DT_F32: (torch.float32,), FT_DT_BF16: (torch.bfloat16, torch.int16),
             FT_DT_FP8E4M3FN_B128: (torch.uint8, torch.float8_e4m3fn), FT_DT_MXFP4: (torch.uint8,)}
_S_DTYPES = {FT_DT_FP8E4M3FN_B128: (torch.float32,), FT_DT_MXFP4: (torch.uint8,)}


def expert_bank_bytes(desc: dict) -> tuple:
    """Bytes of one expert in each bank (w13, w2, s13, s2) for the layout of ``desc``."""
    H, I, wd = int(desc["hidden"]), int(desc["inter"]), int(desc["w_dtype"])
    if wd == FT_DT_F32:
        return 8 * I * H, 4 * H * I, 0, 0
    if wd == FT_DT_BF16:
        return 4 * I * H, 2 * H * I, 0, 0
    if wd == FT_DT_FP8E4M3FN_B128:
        return 2 * I * H, H * I, (2 * I // 128) * (H // 128) * 4, (H // 128) * (I // 128) * 4
    return I * H, H * I // 2, 2 * I * (H // 32), H * (I // 32)


def _need(t, name: str, dtypes, numel: int, device: str = "cuda") -> None:
    """Raise ValueError unless ``t`` is a tensor on ``device`` of one of ``dtypes`` holding at
    least ``numel`` elements."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name}: expected a torch.Tensor, got {type(t).__name__}")
    if device == "cuda" and not t.is_cuda:
        raise ValueError(f"{name}: must be a device (cuda) tensor")
    if device == "cpu" and t.is_cuda:
        raise ValueError(f"{name}: must be a host tensor")
    if not isinstance(dtypes, tuple):
        dtypes = (dtypes,)
    if t.dtype not in dtypes:
        raise ValueError(f"{name}: dtype {t.dtype}, expected {' or '.join(map(str, dtypes))}")
    if t.numel() < numel:
        raise ValueError(f"{name}: {t.numel()} elements, the call needs {numel}")


def _need_bytes(t, name: str, dtypes, nbytes: int, device: str = "cuda") -> None:
    _need(t, name, dtypes, 0, device)
    if t.numel() * t.element_size() < nbytes:
        raise ValueError(f"{name}: {t.numel() * t.element_size()} bytes, the call needs {nbytes}")


def _need_banks(desc: dict, banks: dict, rows: int, name: str, device: str = "cuda") -> None:
    """Every bank holds ``rows`` expert rows of the layout of ``desc``."""
    if rows <= 0:
        return
    wd = int(desc["w_dtype"])
    b13, b2, bs13, bs2 = expert_bank_bytes(desc)
    _need_bytes(banks.get("w13"), f"{name}['w13']", _W_DTYPES[wd], rows * b13, device)
    _need_bytes(banks.get("w2"), f"{name}['w2']", _W_DTYPES[wd], rows * b2, device)
    if wd in _S_DTYPES:
        _need_bytes(banks.get("s13"), f"{name}['s13']", _S_DTYPES[wd], rows * bs13, device)
        _need_bytes(banks.get("s2"), f"{name}['s2']", _S_DTYPES[wd], rows * bs2, device)


def _need_route(route, desc: dict, T: int) -> None:
    if not isinstance(route, RouteBuffers):
        raise ValueError("route: expected a RouteBuffers")
    E, k = int(desc["n_experts"]), int(desc["top_k"])
    if route.E != E or route.k != k or route.T < T:
        raise ValueError(f"route: sized for T={route.T}, k={route.k}, E={route.E}; the call needs "
                         f"T={T}, k={k}, E={E}")


def _need_layer_inputs(desc: dict, logits, slot_table, T: int, x=None, out=None) -> None:
    E, H = int(desc["n_experts"]), int(desc["hidden"])
    _need(logits, "logits", torch.float32, T * E)
    _need(slot_table, "slot_table", torch.int32, E)
    if x is not None or out is not None:
        xd = _X_DTYPES.get(int(desc["x_dtype"]))
        if xd is None:
            raise ValueError(f"x_dtype {desc['x_dtype']} is not supported")
        _need(x, "x", xd, T * H)
        _need(out, "out_partial", torch.float32, T * H)


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def make_desc(d: dict) -> ft_moe_desc_t:
    """ft_moe_desc_t from a dict; ``combine`` defaults to FT_COMBINE_ORDERED and ``act_quant`` to
    FT_ACT_EXACT."""
    return ft_moe_desc_t(**{f: int(d.get(f, 0) if f in ("combine", "act_quant") else d[f])
                            for f, _ in ft_moe_desc_t._fields_})


class RouteBuffers:
    """Device tensors behind one ft_route_t, sized for T tokens."""

    def __init__(self, T: int, top_k: int, n_experts: int, device="cuda"):
        pk = max(T * top_k, 1)
        i32 = dict(dtype=torch.int32, device=device)
        self.T, self.k, self.E = T, top_k, n_experts
        self.topk_ids = torch.empty(pk, **i32)
        self.topk_w = torch.empty(pk, dtype=torch.float32, device=device)
        self.topk_slot = torch.empty(pk, **i32)
        self.hit_pairs = torch.empty(pk, **i32)
        self.miss_pairs = torch.empty(pk, **i32)
        self.hit_off = torch.empty(n_experts + 1, **i32)
        self.miss_off = torch.empty(n_experts + 1, **i32)
        self.counts = torch.empty(4, **i32)

    def c(self) -> ft_route_t:
        return ft_route_t(*[_ptr(getattr(self, n)) for n, _ in ft_route_t._fields_])


class HostMissBuffers:
    """Pinned host buffers behind one ft_host_miss_t."""

    def __init__(self, T: int, top_k: int, n_experts: int):
        pk = max(T * top_k, 1)
        kw = dict(pin_memory=True)
        self.counts = torch.empty(4, dtype=torch.int32, **kw)
        self.miss_pairs = torch.empty(pk, dtype=torch.int32, **kw)
        self.miss_off = torch.empty(n_experts + 1, dtype=torch.int32, **kw)
        self.topk_ids = torch.empty(pk, dtype=torch.int32, **kw)
        self.topk_w = torch.empty(pk, dtype=torch.float32, **kw)

    def c(self) -> ft_host_miss_t:
        return ft_host_miss_t(*[_ptr(getattr(self, n)) for n, _ in ft_host_miss_t._fields_])


def _check(status: int, where: str):
    if status != FT_OK:
        raise FtError(status, where)


def ft_moe_workspace_bytes(desc: dict, max_tokens: int) -> int:
    return int(load().ft_moe_workspace_bytes(ctypes.byref(make_desc(desc)), int(max_tokens)))


def alloc_workspace(desc: dict, max_tokens: int, device="cuda") -> torch.Tensor:
    n = ft_moe_workspace_bytes(desc, max_tokens)
    if n == 0:
        raise FtError(FT_ERR_SHAPE, "ft_moe_workspace_bytes")
    return torch.empty(n, dtype=torch.uint8, device=device)


def ft_route_only(desc: dict, logits: torch.Tensor, slot_table: torch.Tensor, T: int,
                  route: RouteBuffers, ws: torch.Tensor, stream=None) -> None:
    _need_layer_inputs(desc, logits, slot_table, T)
    _need_route(route, desc, T)
    _need(ws, "ws", torch.uint8, 0)
    st = load().ft_route_only(ctypes.byref(make_desc(desc)), _ptr(logits), _ptr(slot_table), int(T),
                              ctypes.byref(route.c()), _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "ft_route_only")


def _need_forward(desc, banks, logits, slot_table, x, T, out_partial, route, ws) -> None:
    if int(T) <= 0:
        return
    _need_layer_inputs(desc, logits, slot_table, T, x, out_partial)
    _need_route(route, desc, T)
    _need(ws, "ws", torch.uint8, 0)
    _need_banks(desc, banks, int(desc["n_slots"]), "banks")


def ft_moe_forward(desc: dict, banks: dict, logits: torch.Tensor, slot_table: torch.Tensor,
                   x: torch.Tensor, T: int, out_partial: torch.Tensor, route: RouteBuffers,
                   ws: torch.Tensor, stream=None) -> None:
    _need_forward(desc, banks, logits, slot_table, x, T, out_partial, route, ws)
    b = ft_banks_t(_ptr(banks.get("w13")), _ptr(banks.get("w2")), _ptr(banks.get("s13")),
                   _ptr(banks.get("s2")))
    st = load().ft_moe_forward(ctypes.byref(make_desc(desc)), ctypes.byref(b), _ptr(logits),
                               _ptr(slot_table), _ptr(x), int(T), _ptr(out_partial),
                               ctypes.byref(route.c()), _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "ft_moe_forward")


def ft_moe_forward_noalloc(desc: dict, banks: dict, logits: torch.Tensor, slot_table: torch.Tensor,
                           x: torch.Tensor, T: int, out_partial: torch.Tensor, route: RouteBuffers,
                           stream=None) -> None:
    """ft_moe_forward on the library's own device scratch array (no workspace argument)."""
    if int(T) > 0:
        _need_layer_inputs(desc, logits, slot_table, T, x, out_partial)
        _need_route(route, desc, T)
        _need_banks(desc, banks, int(desc["n_slots"]), "banks")
    b = ft_banks_t(_ptr(banks.get("w13")), _ptr(banks.get("w2")), _ptr(banks.get("s13")),
                   _ptr(banks.get("s2")))
    st = load().ft_moe_forward_noalloc(ctypes.byref(make_desc(desc)), ctypes.byref(b), _ptr(logits),
                                       _ptr(slot_table), _ptr(x), int(T), _ptr(out_partial),
                                       ctypes.byref(route.c()), _stream(stream))
    _check(st, "ft_moe_forward_noalloc")


def ft_moe_forward_profiled(desc: dict, banks: dict, logits: torch.Tensor, slot_table: torch.Tensor,
                            x: torch.Tensor, T: int, out_partial: torch.Tensor, route: RouteBuffers,
                            ws: torch.Tensor, events, stream=None) -> None:
    """``events``: FT_PROF_STAGES + 1 hipEvent_t handles (ints) or None entries."""
    _need_forward(desc, banks, logits, slot_table, x, T, out_partial, route, ws)
    b = ft_banks_t(_ptr(banks.get("w13")), _ptr(banks.get("w2")), _ptr(banks.get("s13")),
                   _ptr(banks.get("s2")))
    ev = ft_prof_events_t()
    for i, e in enumerate(events):
        ev.ev[i] = e
    st = load().ft_moe_forward_profiled(ctypes.byref(make_desc(desc)), ctypes.byref(b), _ptr(logits),
                                        _ptr(slot_table), _ptr(x), int(T), _ptr(out_partial),
                                        ctypes.byref(route.c()), _ptr(ws), ws.numel(),
                                        _stream(stream), ctypes.byref(ev))
    _check(st, "ft_moe_forward_profiled")


def ft_miss_list_to_host(desc: dict, route: RouteBuffers, T: int, host: HostMissBuffers,
                         stream=None) -> None:
    _need_route(route, desc, T)
    pk, E = int(T) * int(desc["top_k"]), int(desc["n_experts"])
    for n, dt, cnt in (("counts", torch.int32, 4), ("miss_pairs", torch.int32, pk),
                       ("miss_off", torch.int32, E + 1), ("topk_ids", torch.int32, pk),
                       ("topk_w", torch.float32, pk)):
        _need(getattr(host, n, None), f"host.{n}", dt, cnt, "cpu")
    st = load().ft_miss_list_to_host(ctypes.byref(make_desc(desc)), ctypes.byref(route.c()), int(T),
                                     ctypes.byref(host.c()), _stream(stream))
    _check(st, "ft_miss_list_to_host")


class CacheState:
    """Device tensors behind one ft_cache_state_t: slot -> expert (-1 empty), the slot stamps
    (uint32 in the ABI; held as int32 here, stamps stay below 2**31) and an optional one-element
    device step clock."""

    def __init__(self, slot_expert: torch.Tensor, slot_stamp: torch.Tensor,
                 clock: Optional[torch.Tensor] = None):
        self.slot_expert = slot_expert
        self.slot_stamp = slot_stamp
        self.clock = clock

    def c(self) -> ft_cache_state_t:
        return ft_cache_state_t(_ptr(self.slot_expert), _ptr(self.slot_stamp), _ptr(self.clock))


class FillPlanBuffers:
    """Device tensors behind one ft_fill_plan_t (max_fill fills, n_experts CPU entries)."""

    def __init__(self, max_fill: int, n_experts: int, device="cuda"):
        i32 = dict(dtype=torch.int32, device=device)
        self.fill_expert = torch.empty(max_fill, **i32)
        self.fill_slot = torch.empty(max_fill, **i32)
        self.evict_expert = torch.empty(max_fill, **i32)
        self.cpu_expert = torch.empty(max(n_experts, 1), **i32)
        self.counts = torch.empty(4, **i32)

    def c(self) -> ft_fill_plan_t:
        return ft_fill_plan_t(*[_ptr(getattr(self, n)) for n, _ in ft_fill_plan_t._fields_])


def _need_plan(desc: dict, slot_table, state, plan, max_fill: int) -> None:
    E, S = int(desc["n_experts"]), int(desc["n_slots"])
    _need(slot_table, "slot_table", torch.int32, E)
    _need(state.slot_expert, "state.slot_expert", torch.int32, S)
    _need(state.slot_stamp, "state.slot_stamp", (torch.int32, torch.uint32), S)
    for n in ("fill_expert", "fill_slot", "evict_expert"):
        _need(getattr(plan, n), f"plan.{n}", torch.int32, int(max_fill))
    _need(plan.cpu_expert, "plan.cpu_expert", torch.int32, E)
    _need(plan.counts, "plan.counts", torch.int32, 4)


def ft_cache_plan(desc: dict, route: RouteBuffers, T: int, slot_table: torch.Tensor,
                  state: CacheState, b_pcie: float, b_host: float, max_fill: int, step: int,
                  plan: FillPlanBuffers, stream=None) -> None:
    _need_route(route, desc, T)
    _need_plan(desc, slot_table, state, plan, max_fill)
    pol = ft_cache_policy_t(float(b_pcie), float(b_host), int(max_fill), int(step))
    st = load().ft_cache_plan(ctypes.byref(make_desc(desc)), ctypes.byref(route.c()), int(T),
                              _ptr(slot_table), ctypes.byref(state.c()), ctypes.byref(pol),
                              ctypes.byref(plan.c()), _stream(stream))
    _check(st, "ft_cache_plan")


class CpuPool:
    """A persistent CPU worker pool (ft_cpu_pool_t); destroyed with ft_cpu_pool_destroy or when
    garbage-collected."""

    def __init__(self, handle: int, n_threads: int, pin: bool):
        self.handle, self.n_threads, self.pin = handle, n_threads, pin

    def close(self) -> None:
        if self.handle:
            load().ft_cpu_pool_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def ft_cpu_pool_create(n_threads: int = 0, pin: bool = True) -> CpuPool:
    h = load().ft_cpu_pool_create(int(n_threads), 1 if pin else 0)
    if not h:
        raise RuntimeError("ft_cpu_pool_create failed")
    return CpuPool(h, n_threads, pin)


def ft_cpu_pool_destroy(pool: CpuPool) -> None:
    pool.close()


def _pool_handle(pool) -> Optional[int]:
    if pool is None:
        return None
    if not isinstance(pool, CpuPool) or not pool.handle:
        raise ValueError("pool: expected an open CpuPool or None")
    return pool.handle


def ft_cpu_experts(desc: dict, host_pool: dict, x: torch.Tensor, T: int, topk_ids: torch.Tensor,
                   topk_w: torch.Tensor, experts: torch.Tensor, out: torch.Tensor,
                   pool: Optional[CpuPool] = None) -> None:
    """CPU branch on host tensors: ``host_pool`` holds w13, w2 (s13, s2) indexed by expert id;
    runs on ``pool``'s workers, or on the calling thread without one."""
    if int(T) > 0:
        E, H, k = int(desc["n_experts"]), int(desc["hidden"]), int(desc["top_k"])
        xd = _X_DTYPES.get(int(desc["x_dtype"]))
        if xd is None:
            raise ValueError(f"x_dtype {desc['x_dtype']} is not supported")
        _need(x, "x", xd, int(T) * H, "cpu")
        _need(topk_ids, "topk_ids", torch.int32, int(T) * k, "cpu")
        _need(topk_w, "topk_w", torch.float32, int(T) * k, "cpu")
        _need(experts, "experts", torch.int32, 0, "cpu")
        _need(out, "out", torch.float32, int(T) * H, "cpu")
        if experts.numel() > 0:
            _need_banks(desc, host_pool, E, "host_pool", "cpu")
    b = ft_banks_t(_ptr(host_pool.get("w13")), _ptr(host_pool.get("w2")), _ptr(host_pool.get("s13")),
                   _ptr(host_pool.get("s2")))
    st = load().ft_cpu_experts(ctypes.byref(make_desc(desc)), ctypes.byref(b), _ptr(x), int(T),
                               _ptr(topk_ids), _ptr(topk_w), _ptr(experts), int(experts.numel()),
                               _ptr(out), _pool_handle(pool))
    _check(st, "ft_cpu_experts")


def _banks(b: dict) -> ft_banks_t:
    return ft_banks_t(_ptr(b.get("w13")), _ptr(b.get("w2")), _ptr(b.get("s13")), _ptr(b.get("s2")))


def ft_cache_fill(desc: dict, host_pool: dict, dev_banks: dict, plan: FillPlanBuffers, max_fill: int,
                  stream=None) -> None:
    _need_banks(desc, host_pool, int(desc["n_experts"]), "host_pool", "cpu")
    _need_banks(desc, dev_banks, int(desc["n_slots"]), "dev_banks")
    for n in ("fill_expert", "fill_slot"):
        _need(getattr(plan, n), f"plan.{n}", torch.int32, int(max_fill))
    _need(plan.counts, "plan.counts", torch.int32, 4)
    st = load().ft_cache_fill(ctypes.byref(make_desc(desc)), ctypes.byref(_banks(host_pool)),
                              ctypes.byref(_banks(dev_banks)), ctypes.byref(plan.c()), int(max_fill),
                              _stream(stream))
    _check(st, "ft_cache_fill")


class HybridHostBuffers:
    """Pinned host staging behind one ft_hybrid_host_t, for T tokens."""

    def __init__(self, T: int, top_k: int, n_experts: int, hidden: int, x_dtype=torch.bfloat16):
        kw = dict(pin_memory=True)
        pk = max(T * top_k, 1)
        self.plan_counts = torch.empty(4, dtype=torch.int32, **kw)
        self.cpu_expert = torch.empty(n_experts, dtype=torch.int32, **kw)
        self.topk_ids = torch.empty(pk, dtype=torch.int32, **kw)
        self.topk_w = torch.empty(pk, dtype=torch.float32, **kw)
        self.x = torch.empty(max(T, 1), hidden, dtype=x_dtype, **kw)
        self.cpu_out = torch.empty(max(T, 1), hidden, dtype=torch.float32, **kw)
        self.task = torch.zeros(FT_HYBRID_TASK_BYTES, dtype=torch.uint8)   # plain host memory
        self.T, self.k, self.E, self.H = T, top_k, n_experts, hidden

    def c(self) -> ft_hybrid_host_t:
        return ft_hybrid_host_t(*[_ptr(getattr(self, n)) for n, _ in ft_hybrid_host_t._fields_])


def ft_moe_step_hybrid(desc: dict, dev_banks: dict, host_pool: dict, logits: torch.Tensor,
                       slot_table: torch.Tensor, state: CacheState, b_pcie: float, b_host: float,
                       max_fill: int, step: int, x: torch.Tensor, T: int, out: torch.Tensor,
                       route: RouteBuffers, plan: FillPlanBuffers,
                       host: HybridHostBuffers, ws: torch.Tensor, pool: Optional[CpuPool],
                       stream=None) -> None:
    """One complete hybrid layer step, enqueued on ``stream`` without waiting for the device."""
    if int(T) > 0:
        _need_layer_inputs(desc, logits, slot_table, T, x, out)
        _need_route(route, desc, T)
        _need(ws, "ws", torch.uint8, 0)
        _need_banks(desc, dev_banks, int(desc["n_slots"]), "dev_banks")
        _need_banks(desc, host_pool, int(desc["n_experts"]), "host_pool", "cpu")
        _need_plan(desc, slot_table, state, plan, max_fill)
        if host.T < T or host.k != int(desc["top_k"]) or host.E != int(desc["n_experts"]) or \
                host.H != int(desc["hidden"]):
            raise ValueError("host: HybridHostBuffers sized for another layer or fewer tokens")
        if state.clock is not None:
            _need(state.clock, "state.clock", (torch.int32, torch.uint32), 1)
    pol = ft_cache_policy_t(float(b_pcie), float(b_host), int(max_fill), int(step))
    st = load().ft_moe_step_hybrid(ctypes.byref(make_desc(desc)), ctypes.byref(_banks(dev_banks)),
                                   ctypes.byref(_banks(host_pool)), _ptr(logits), _ptr(slot_table),
                                   ctypes.byref(state.c()), ctypes.byref(pol), _ptr(x), int(T),
                                   _ptr(out), ctypes.byref(route.c()),
                                   ctypes.byref(plan.c()), ctypes.byref(host.c()), _ptr(ws),
                                   ws.numel(), _pool_handle(pool), _stream(stream))
    _check(st, "ft_moe_step_hybrid")


def banks_of(layer) -> dict:
    """The bank tensors of a synthetic layer object (w13, w2, s13, s2 attributes)."""
    return {"w13": layer.w13, "w2": layer.w2, "s13": layer.s13, "s2": layer.s2}


def ft_prefill_layers(desc: dict, host_layers: list, dev_bufs: list, slot_table: torch.Tensor,
                      logits: list, x: list, T: int, out: list, route: RouteBuffers, ws: torch.Tensor,
                      overlap: bool = True, stream=None, copy_stream=None) -> None:
    """``host_layers``: one dict of pinned host tensors (w13, w2, s13, s2) per layer;
    ``dev_bufs``: two dicts of device tensors; ``logits``, ``x``, ``out``: one device tensor per
    layer.  ``copy_stream``: a torch stream or raw handle, required when ``overlap``."""
    n = len(host_layers)
    if not (len(logits) == len(x) == len(out) == n) or len(dev_bufs) != 2:
        raise ValueError("one logits, x and out tensor per layer and two device buffers")
    if int(T) > 0:
        for l in range(n):
            _need_banks(desc, host_layers[l], int(desc["n_slots"]), f"host_layers[{l}]", "cpu")
            _need_layer_inputs(desc, logits[l], slot_table, T, x[l], out[l])
        for b in range(2):
            _need_banks(desc, dev_bufs[b], int(desc["n_slots"]), f"dev_bufs[{b}]")
        _need_route(route, desc, T)
        _need(ws, "ws", torch.uint8, 0)
    hl = (ft_banks_t * max(n, 1))(*[_banks(h) for h in host_layers])
    db = (ft_banks_t * 2)(*[_banks(d) for d in dev_bufs])
    arr = lambda ts: (ctypes.c_void_p * max(n, 1))(*[_ptr(t) for t in ts])
    cs = None if copy_stream is None else _stream(copy_stream)
    st = load().ft_prefill_layers(ctypes.byref(make_desc(desc)), n, hl, db, _ptr(slot_table),
                                  arr(logits), arr(x), int(T), arr(out), ctypes.byref(route.c()),
                                  _ptr(ws), ws.numel(), 1 if overlap else 0, _stream(stream), cs)
    _check(st, "ft_prefill_layers")
