"""Seeded synthetic MoE-layer inputs shared by the tests, the benchmark and the oracle checks.

This module only draws inputs; it holds none of the MoE layer's arithmetic (no routing,
gating, partitioning or expert evaluation).  Everything it returns is plain data:

* router logits ``[T][E]`` float32,
* an expert -> slot table ``[E]`` int32 (``-1`` = expert not resident),
* hidden states ``[T][H]`` (bfloat16, or float32 for the tiny layer),
* the slot-pool expert banks, one bank row per slot, in the layout the C ABI documents:
  ``w13[n_slots][2I][H]`` (rows ``0..I-1`` = gate projection W1, rows ``I..2I-1`` = up
  projection W3), ``w2[n_slots][H][I]`` (down projection), and for fp8 weights the
  per-128x128-block float32 scales ``s13[n_slots][2I/128][H/128]``,
  ``s2[n_slots][H/128][I/128]``.

The paper evaluates the layer on real models and agentic traces (Section 5.1) that are not
available here; these synthetic layers stand in for them with the published layer shapes of
Qwen3-30B-A3B and DeepSeek-V3 and a Zipf expert-popularity skew standing in for the temporal
expert locality of Section 3.2.

Draw order (one ``torch.Generator`` per layer, seeded from ``(seed, T, layer)``):
  1. expert popularity rank permutation(s) (one per 1024-token segment when the hot set shifts),
  2. the slot permutation of the resident experts,
  3. router noise ``N(0,1)`` float32 ``[T][E]``,
  4. popularity bias ``-s * ln(rank)`` added in float32,
  5. hidden states ``N(0,1)`` float32, rounded to bfloat16 (round-to-nearest-even) unless fp32,
  6. weights, per resident expert in ascending expert id and then the shared expert:
     W1 ``[I][H]``, W3 ``[I][H]``, W2 ``[H][I]`` ~ ``N(0, 0.02)`` float32, then rounded to
     bfloat16, or quantised to fp8 e4m3fn per 128x128 block with scale ``amax/448``.

Generation runs on the torch device given (CPU for small layers, the GPU for full-size ones);
the two devices draw different streams for the same seed.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import torch

GATE_SOFTMAX = 0   # softmax over the experts, keep top-k, renormalise over the k
GATE_SIGMOID = 1   # sigmoid per expert, keep top-k, renormalise over the k

DT_F32 = 0
DT_BF16 = 1
DT_FP8 = 2         # fp8 e4m3fn codes with one float32 scale per 128x128 block
DT_MXFP4 = 3       # OCP MXFP4: E2M1 code pairs (even element in the low nibble), one E8M0 scale
                   # per 32 consecutive elements of a row

FP8_MAX = 448.0


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    name: str
    hidden: int
    inter: int
    n_experts: int
    top_k: int
    gating: int
    w_dtype: int
    x_dtype: int
    tokens: tuple           # the token counts this layer is exercised at
    seed: int
    resident_frac: float    # fraction of routed experts resident (floored); ignored if resident_set
    zipf_s: float           # popularity skew; 0 = uniform logits
    shared_expert: bool
    shift_every: int = 0    # re-permute the popularity ranking every this many tokens (0 = never)
    resident_set: Optional[tuple] = None
    slot_table: Optional[tuple] = None


CONFIGS = {
    # Tiny layer: fp32 everything, experts {0,2,5,7} resident.
    "tiny": LayerConfig("tiny", 256, 512, 8, 2, GATE_SOFTMAX, DT_F32, DT_F32, (16,), 0,
                        0.5, 0.0, False, resident_set=(0, 2, 5, 7),
                        slot_table=(0, -1, 1, -1, -1, 2, -1, 3)),
    # Qwen3-30B-A3B-shaped decode layer.
    "qwen3_decode": LayerConfig("qwen3_decode", 2048, 768, 128, 8, GATE_SOFTMAX, DT_BF16, DT_BF16,
                                (1, 8, 32), 1, 0.5, 1.1, False),
    # Qwen3-30B-A3B-shaped prefill chunk, uniform routing.
    "qwen3_prefill": LayerConfig("qwen3_prefill", 2048, 768, 128, 8, GATE_SOFTMAX, DT_BF16, DT_BF16,
                                 (4096,), 2, 0.75, 0.0, False),
    # DeepSeek-V3-shaped decode layer, fp8 block-scaled weights, one shared expert.
    "dsv3_decode": LayerConfig("dsv3_decode", 7168, 2048, 256, 8, GATE_SIGMOID, DT_FP8, DT_BF16,
                               (1, 16, 64), 3, 0.25, 1.2, True),
    # DeepSeek-V3-shaped prefill chunk whose hot set shifts every 1024 tokens.
    "dsv3_prefill": LayerConfig("dsv3_prefill", 7168, 2048, 256, 8, GATE_SIGMOID, DT_FP8, DT_BF16,
                                (8192,), 4, 0.40, 1.2, True, shift_every=1024),
    # DeepSeek-V4-Flash-shaped layer with MXFP4 routed experts: 256 routed experts, top-6 (the
    # paper's figures); H = 4096, I = 2048 make one expert 13.4 MB, the size its 140 GB pool of
    # 43 x 256 experts implies.  No shared expert (the paper names routed experts only).
    "dsv4flash_decode": LayerConfig("dsv4flash_decode", 4096, 2048, 256, 6, GATE_SIGMOID, DT_MXFP4,
                                    DT_BF16, (1, 16, 64), 5, 0.25, 1.2, False),
    "dsv4flash_prefill": LayerConfig("dsv4flash_prefill", 4096, 2048, 256, 6, GATE_SIGMOID, DT_MXFP4,
                                     DT_BF16, (8192,), 6, 0.40, 1.2, False, shift_every=1024),
}


@dataclasses.dataclass
class Layer:
    """One synthetic MoE layer instance; every tensor lives on ``device``."""
    hidden: int
    inter: int
    n_experts: int
    top_k: int
    gating: int
    w_dtype: int
    x_dtype: int
    n_slots: int
    shared_slot: int
    logits: torch.Tensor      # [T][E] float32
    slot_table: torch.Tensor  # [E] int32
    x: torch.Tensor           # [T][H] bfloat16 or float32
    w13: torch.Tensor         # [n_slots][2I][H] float32 / bfloat16 / uint8 (fp8 codes);
                              # MXFP4: [n_slots][2I][H/2] uint8 code pairs
    w2: torch.Tensor          # [n_slots][H][I] (MXFP4: [n_slots][H][I/2])
    s13: Optional[torch.Tensor]  # fp8: [n_slots][2I/128][H/128] float32; MXFP4: [n_slots][H/32][2I] uint8
    s2: Optional[torch.Tensor]   # fp8: [n_slots][H/128][I/128] float32; MXFP4: [n_slots][I/32][H] uint8

    @property
    def tokens(self) -> int:
        return self.logits.shape[0]

    def desc(self) -> dict:
        return dict(hidden=self.hidden, inter=self.inter, n_experts=self.n_experts,
                    top_k=self.top_k, gating=self.gating, w_dtype=self.w_dtype,
                    x_dtype=self.x_dtype, n_slots=self.n_slots, shared_slot=self.shared_slot)

    def to(self, device) -> "Layer":
        f = lambda t: None if t is None else t.to(device)
        return dataclasses.replace(self, logits=f(self.logits), slot_table=f(self.slot_table),
                                   x=f(self.x), w13=f(self.w13), w2=f(self.w2),
                                   s13=f(self.s13), s2=f(self.s2))


def layer_seed(seed: int, tokens: int, layer: int) -> int:
    return (seed * 1_000_003 + tokens * 10_007 + layer * 101) & 0x7FFF_FFFF_FFFF


def quantize_fp8_blocks(w: torch.Tensor):
    """Input preparation only: float32 ``[R][C]`` -> (e4m3fn codes as uint8, scales [R/128][C/128]).

    Scale = amax/448 of each 128x128 block; codes = round-to-nearest-even of w/scale,
    clamped to +-448 first so nothing overflows to NaN.
    """
    r, c = w.shape
    blk = w.view(r // 128, 128, c // 128, 128)
    amax = blk.abs().amax(dim=(1, 3))
    scale = torch.where(amax > 0, amax / FP8_MAX, torch.ones_like(amax)).to(torch.float32)
    q = (blk / scale[:, None, :, None]).clamp_(-FP8_MAX, FP8_MAX)
    codes = q.view(r, c).to(torch.float8_e4m3fn).view(torch.uint8)
    return codes, scale


def quantize_mxfp4(w: torch.Tensor):
    """Input preparation only: float32 ``[R][C]`` -> (E2M1 code pairs [R][C/2] uint8, E8M0 scales
    [C/32][R] uint8, run-major), following the OCP MX recipe: per 32-element block the shared exponent is
    floor(log2(amax)) - 2 (2 = the largest E2M1 exponent), and each element is rounded to the
    nearest E2M1 value, ties to even, saturating at +-6; an all-zero block takes scale 1."""
    r, c = w.shape
    blk = w.view(r, c // 32, 32)
    amax = blk.abs().amax(dim=2)
    e = torch.where(amax > 0, torch.floor(torch.log2(torch.where(amax > 0, amax, torch.ones_like(amax)))) - 2,
                    torch.zeros_like(amax))
    code_s = (e + 127).clamp_(0, 254)
    scale = torch.pow(2.0, code_s - 127)
    q = blk / scale[:, :, None]
    a = q.abs()
    idx = ((a > 0.25).to(torch.uint8) + (a >= 0.75) + (a > 1.25) + (a >= 1.75) + (a > 2.5) + (a >= 3.5)
           + (a > 5)).to(torch.uint8)
    codes = (idx | (torch.signbit(q).to(torch.uint8) << 3)).view(r, c)
    packed = (codes[:, 0::2] | (codes[:, 1::2] << 4)).contiguous()
    return packed, code_s.to(torch.uint8).t().contiguous()


def _weights(g, rows, cols, w_dtype, device):
    w = torch.randn(rows, cols, generator=g, dtype=torch.float32, device=device).mul_(0.02)
    if w_dtype == DT_F32:
        return w, None
    if w_dtype == DT_BF16:
        return w.to(torch.bfloat16), None
    if w_dtype == DT_MXFP4:
        return quantize_mxfp4(w)
    return quantize_fp8_blocks(w)


def alloc_banks(n_slots: int, hidden: int, inter: int, w_dtype: int, device="cpu"):
    """Zeroed (w13, w2, s13, s2) banks of n_slots rows in the bank layout of w_dtype."""
    H, I = hidden, inter
    if w_dtype == DT_MXFP4:
        u8 = dict(dtype=torch.uint8, device=device)
        return (torch.zeros(n_slots, 2 * I, H // 2, **u8), torch.zeros(n_slots, H, I // 2, **u8),
                torch.zeros(n_slots, H // 32, 2 * I, **u8), torch.zeros(n_slots, I // 32, H, **u8))
    wdt = {DT_F32: torch.float32, DT_BF16: torch.bfloat16, DT_FP8: torch.uint8}[w_dtype]
    w13 = torch.zeros(n_slots, 2 * I, H, dtype=wdt, device=device)
    w2 = torch.zeros(n_slots, H, I, dtype=wdt, device=device)
    if w_dtype != DT_FP8:
        return w13, w2, None, None
    return (w13, w2, torch.ones(n_slots, 2 * I // 128, H // 128, device=device),
            torch.ones(n_slots, H // 128, I // 128, device=device))


def put_expert(banks, slot: int, inter: int, w_dtype: int, w1, a1, w3, a3, wd, ad):
    """Store one expert's quantised projections (from _weights) in bank row ``slot``."""
    w13, w2, s13, s2 = banks
    I = inter
    w13[slot, :I] = w1
    w13[slot, I:] = w3
    w2[slot] = wd
    if w_dtype == DT_FP8:
        s13[slot, : I // 128] = a1
        s13[slot, I // 128:] = a3
        s2[slot] = ad
    elif w_dtype == DT_MXFP4:
        s13[slot, :, :I] = a1
        s13[slot, :, I:] = a3
        s2[slot] = ad


def make_layer_from(cfg: LayerConfig, tokens: int, layer: int = 0, device="cpu",
                    resident_frac: Optional[float] = None, seed: Optional[int] = None) -> Layer:
    device = torch.device(device)
    g = torch.Generator(device=device)
    g.manual_seed(layer_seed(cfg.seed if seed is None else seed, tokens, layer))
    E, H, I, T = cfg.n_experts, cfg.hidden, cfg.inter, tokens

    # 1. popularity rank permutations: expert perm[i] has rank i + 1
    n_seg = 1 if cfg.shift_every == 0 else max(1, -(-T // cfg.shift_every))
    perms = [torch.randperm(E, generator=g, device=device) for _ in range(n_seg)]
    ranks = []
    for p in perms:
        r = torch.empty(E, dtype=torch.float32, device=device)
        r[p] = torch.arange(1, E + 1, dtype=torch.float32, device=device)
        ranks.append(r)

    # residency: the most popular experts under the first ranking (or a fixed set)
    if cfg.resident_set is not None and resident_frac is None:
        resident = list(cfg.resident_set)
    else:
        frac = cfg.resident_frac if resident_frac is None else resident_frac
        n_res = int(math.floor(frac * E + 1e-9))
        resident = sorted(perms[0][:n_res].tolist())
    n_routed_slots = len(resident)

    # 2. slot permutation
    slot_perm = torch.randperm(max(n_routed_slots, 1), generator=g, device=device)[:n_routed_slots]
    if cfg.slot_table is not None and resident_frac is None:
        slot_table = torch.tensor(cfg.slot_table, dtype=torch.int32, device=device)
    else:
        slot_table = torch.full((E,), -1, dtype=torch.int32, device=device)
        if n_routed_slots:
            slot_table[torch.tensor(resident, device=device)] = slot_perm.to(torch.int32)
    shared_slot = n_routed_slots if cfg.shared_expert else -1
    n_slots = n_routed_slots + (1 if cfg.shared_expert else 0)

    # 3./4. router logits
    logits = torch.randn(T, E, generator=g, dtype=torch.float32, device=device)
    if cfg.zipf_s > 0:
        for s in range(n_seg):
            lo = s * cfg.shift_every if cfg.shift_every else 0
            hi = min(T, lo + cfg.shift_every) if cfg.shift_every else T
            logits[lo:hi] += (-cfg.zipf_s * torch.log(ranks[s]))[None, :]

    # 5. hidden states
    x = torch.randn(T, H, generator=g, dtype=torch.float32, device=device)
    if cfg.x_dtype == DT_BF16:
        x = x.to(torch.bfloat16)

    # 6. weights, one bank row per slot
    banks = alloc_banks(n_slots, H, I, cfg.w_dtype, device)
    w13, w2, s13, s2 = banks
    order = [(e, int(slot_table[e])) for e in resident]
    if cfg.shared_expert:
        order.append((-1, shared_slot))
    for _, slot in order:
        w1, a1 = _weights(g, I, H, cfg.w_dtype, device)
        w3, a3 = _weights(g, I, H, cfg.w_dtype, device)
        wd, ad = _weights(g, H, I, cfg.w_dtype, device)
        put_expert(banks, slot, I, cfg.w_dtype, w1, a1, w3, a3, wd, ad)
    return Layer(H, I, E, cfg.top_k, cfg.gating, cfg.w_dtype, cfg.x_dtype, n_slots, shared_slot,
                 logits, slot_table, x, w13, w2, s13, s2)


def make_layer(name: str, tokens: int, layer: int = 0, device="cpu", **kw) -> Layer:
    return make_layer_from(CONFIGS[name], tokens, layer, device, **kw)


def routing_trace(name: str, n_prefill: int, n_decode: int, layer: int = 0, n_topics: int = 8,
                  mean_segment: float = 64.0, device="cpu") -> torch.Tensor:
    """Router logits [n_prefill + n_decode][E] of one layer over a prefill and the decode that
    follows it, with short-range locality: the tokens come in segments of geometric length
    (mean ``mean_segment``), each segment drawn from one of ``n_topics`` popularity rankings
    chosen at random, and every logit is N(0, 1) - s ln(rank) with the config's Zipf s."""
    cfg = CONFIGS[name]
    g = torch.Generator(device="cpu")
    g.manual_seed(layer_seed(cfg.seed + 101, n_prefill + n_decode, layer))
    E, T = cfg.n_experts, n_prefill + n_decode
    bias = []
    for _ in range(n_topics):
        r = torch.empty(E, dtype=torch.float32)
        r[torch.randperm(E, generator=g)] = torch.arange(1, E + 1, dtype=torch.float32)
        bias.append(-cfg.zipf_s * torch.log(r))
    logits = torch.randn(T, E, generator=g, dtype=torch.float32)
    t = 0
    while t < T:
        n = int(torch.empty(1).geometric_(1.0 / mean_segment, generator=g).item())   # >= 1
        topic = int(torch.randint(n_topics, (1,), generator=g))
        logits[t:t + n] += bias[topic][None, :]
        t += n
    return logits.to(device)


def random_layer(seed: int, *, hidden: int, inter: int, n_experts: int, top_k: int, tokens: int,
                 gating: int = GATE_SOFTMAX, w_dtype: int = DT_BF16, n_resident: Optional[int] = None,
                 shared: bool = False, zipf_s: float = 0.0, device="cpu",
                 tie_logits: bool = False) -> Layer:
    """A small random layer for randomised parity cases (random residency and slot order)."""
    device = torch.device(device)
    g = torch.Generator(device="cpu")
    g.manual_seed(layer_seed(seed, tokens, 7))
    E = n_experts
    if n_resident is None:
        n_resident = int(torch.randint(0, E + 1, (1,), generator=g))
    resident = sorted(torch.randperm(E, generator=g)[:n_resident].tolist())
    pool_extra = int(torch.randint(0, 3, (1,), generator=g))  # empty slots in the pool
    n_routed_slots = n_resident + pool_extra
    slot_perm = torch.randperm(n_routed_slots, generator=g)[:n_resident]
    slot_table = torch.full((E,), -1, dtype=torch.int32)
    if n_resident:
        slot_table[torch.tensor(resident)] = slot_perm.to(torch.int32)
    shared_slot = n_routed_slots if shared else -1
    n_slots = n_routed_slots + (1 if shared else 0)
    logits = torch.randn(tokens, E, generator=g)
    if zipf_s > 0:
        r = torch.empty(E)
        r[torch.randperm(E, generator=g)] = torch.arange(1, E + 1, dtype=torch.float32)
        logits += -zipf_s * torch.log(r)[None, :]
    if tie_logits:
        # coarse values force many exact ties, including +0.0 and -0.0
        logits = torch.round(logits * 2) / 2
        logits[logits == 0] = 0.0
        zmask = torch.rand(logits.shape, generator=g) < 0.5
        logits[(logits == 0) & zmask] = -0.0
    x_dtype = DT_F32 if w_dtype == DT_F32 else DT_BF16
    x = torch.randn(tokens, hidden, generator=g)
    if x_dtype == DT_BF16:
        x = x.to(torch.bfloat16)
    banks = alloc_banks(n_slots, hidden, inter, w_dtype)
    w13, w2, s13, s2 = banks
    for slot in range(n_slots):   # every pool slot gets weights, also the empty ones
        w1, a1 = _weights(g, inter, hidden, w_dtype, "cpu")
        w3, a3 = _weights(g, inter, hidden, w_dtype, "cpu")
        wd, ad = _weights(g, hidden, inter, w_dtype, "cpu")
        put_expert(banks, slot, inter, w_dtype, w1, a1, w3, a3, wd, ad)
    lay = Layer(hidden, inter, E, top_k, gating, w_dtype, x_dtype, n_slots, shared_slot,
                logits.float(), slot_table, x, w13, w2, s13, s2)
    return lay.to(device)
