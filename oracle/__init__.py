"""CPU oracle for the MoE layer over a GPU expert cache.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg use this module; the
product library never imports or calls it.  It shares no code with the HIP path.

It is a plain, slow, obviously correct restatement of what one MoE layer computes when only
the experts resident in the GPU expert cache are evaluated (Section 3.2 and Section 4.1 of the
paper: gating and the slot lookup happen on the device, cache-resident experts are evaluated
there, the remaining experts are handled by the host, and adding the two partial sums gives the
layer output exactly).
Every floating-point step runs in float64 on exactly decoded weights; results are cast to
float32 at the end.

The paper does not print the layer's formulas (Section 2 only says a layer holds E experts and
routes each token to k of them).  The readings taken here:

* top-k: the k largest raw float32 logits of the token, ordered by (logit descending, expert id
  ascending); -0.0 counts as +0.0.  Both gating functions are strictly increasing, so selecting
  on logits equals selecting on scores.
* gates: softmax mode, g_j = exp(l_j - l_max) / sum_i exp(l_i - l_max) over the k selected
  (a softmax over all E renormalised over the k); sigmoid mode, g_j = s_j / sum_i s_i with
  s = 1/(1+exp(-l)).  No routed scaling factor, no group-limited routing, no bias correction.
* hit/miss: pair (t, j) is a hit iff its expert maps to a valid slot: 0 <= slot < n_slots, the
  slot is not the shared expert's slot, and no other expert maps to the same slot.  Anything
  else is a miss (Section 4.1 rewrites routed ids into slot ids or a CPU flag).
* permutation: hit pairs p = t*k + j sorted stably by expert id (so, within one expert, by
  ascending p); misses likewise.  Offsets are exclusive prefix sums of per-expert counts.
* expert FFN (SwiGLU): FFN(x) = W2 (silu(W1 x) * (W3 x)), silu(z) = z / (1 + exp(-z)).  For
  layers with bf16, fp8 or MXFP4 weights the activation between the two projections is a
  bfloat16 tensor, as in a model served in BF16 (Section 5.1): h = bf16(silu(W1 x) * (W3 x)),
  rounded to nearest, ties to even; float32 layers keep h exact.
* output: out[t] = sum over hit pairs of g_tj FFN_e(x_t) (+ FFN_shared(x_t), weight 1, when a
  shared expert is configured); a token without hits and without shared expert gets 0.
* fp8 activations (optional mode ACT_FP8_1X128_POW2, not the paper's exact method): the expert
  inputs x and the intermediate h are quantised per token and 128-channel block to e4m3fn with
  a power-of-two scale, the smallest 2^e with 448 * 2^e >= the block's largest magnitude, and
  rounded to nearest, ties to even; h is first rounded to bfloat16 (round half to even).  Then
  FFN(x) = W2 Q(bf16(silu(W1 Q(x)) * (W3 Q(x)))).  The exact mode (ACT_EXACT) is the default.
"""
from __future__ import annotations

import numpy as np

GATE_SOFTMAX = 0
GATE_SIGMOID = 1
DT_F32 = 0
DT_BF16 = 1
DT_FP8 = 2
DT_MXFP4 = 3

ACT_EXACT = 0
ACT_FP8_1X128_POW2 = 1

STATUS_SLOT_RANGE = 1     # a slot outside [-1, n_slots)
STATUS_SLOT_DUP = 2       # two experts share one slot
STATUS_SLOT_SHARED = 4    # a routed expert points at the shared expert's slot


# ----------------------------------------------------------------------------------------
# Weight codecs (exact decodes to float64)
# ----------------------------------------------------------------------------------------

def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bfloat16 is the top half of an IEEE float32: widen the bit pattern, then reinterpret."""
    b = np.ascontiguousarray(bits).view(np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def e4m3fn_value(code: int) -> float:
    """OCP FP8 E4M3 ("fn" variant): 1 sign, 4 exponent (bias 7), 3 mantissa bits.

    exponent 0 is subnormal (m/8 * 2^-6); S.1111.111 is NaN; there are no infinities.
    """
    s = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 0xF and m == 0x7:
        return float("nan")
    if e == 0:
        return s * (m / 8.0) * 2.0 ** (-6)
    return s * (1.0 + m / 8.0) * 2.0 ** (e - 7)


E4M3FN_TABLE = np.array([e4m3fn_value(c) for c in range(256)], dtype=np.float64)


def fp8_blocks_to_f64(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """Dequantise [R][C] e4m3fn codes with one float32 scale per 128x128 block."""
    r, c = codes.shape
    v = E4M3FN_TABLE[np.ascontiguousarray(codes).view(np.uint8)]
    s = np.repeat(np.repeat(scales.astype(np.float64), 128, axis=0), 128, axis=1)
    assert s.shape == (r, c)
    return v * s


def e2m1_value(code: int) -> float:
    """OCP FP4 E2M1: 1 sign, 2 exponent (bias 1), 1 mantissa bit; exponent 0 is subnormal
    (m/2); every code is finite."""
    s = -1.0 if code & 0x8 else 1.0
    e = (code >> 1) & 0x3
    m = code & 0x1
    if e == 0:
        return s * (m / 2.0)
    return s * (1.0 + m / 2.0) * 2.0 ** (e - 1)


E2M1_TABLE = np.array([e2m1_value(c) for c in range(16)], dtype=np.float64)


def e8m0_value(code: int) -> float:
    """OCP E8M0 scale: 2^(code - 127); code 255 is NaN."""
    return float("nan") if code == 255 else 2.0 ** (int(code) - 127)


E8M0_TABLE = np.array([e8m0_value(c) for c in range(256)], dtype=np.float64)


def mxfp4_to_f64(packed: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """Dequantise an MXFP4 matrix: packed [R][C/2] bytes holding E2M1 codes, element 2j in the
    low nibble of byte j and element 2j+1 in the high nibble, with one E8M0 scale per 32
    consecutive elements of a row, stored run-major: scales [C/32][R], element (r, c) scaled by
    scales[c // 32][r]."""
    b = np.ascontiguousarray(packed).view(np.uint8)
    r, half = b.shape
    codes = np.empty((r, 2 * half), dtype=np.uint8)
    codes[:, 0::2] = b & 0xF
    codes[:, 1::2] = b >> 4
    v = E2M1_TABLE[codes]
    s = np.repeat(E8M0_TABLE[np.ascontiguousarray(scales).view(np.uint8)].T, 32, axis=1)
    assert s.shape == v.shape
    return v * s


def decode_weight(bank: np.ndarray, w_dtype: int, scales=None) -> np.ndarray:
    if w_dtype == DT_F32:
        return bank.astype(np.float64)
    if w_dtype == DT_BF16:
        return bf16_bits_to_f64(bank)
    if w_dtype == DT_MXFP4:
        return mxfp4_to_f64(bank, scales)
    return fp8_blocks_to_f64(bank, scales)


# ----------------------------------------------------------------------------------------
# Routing: top-k selection and gates
# ----------------------------------------------------------------------------------------

def route_topk(logits: np.ndarray, k: int) -> np.ndarray:
    """[T][E] float32 -> [T][k] int32 expert ids, ordered by (logit desc, id asc)."""
    logits = np.asarray(logits, dtype=np.float32)
    T, E = logits.shape
    ids = np.zeros((T, k), dtype=np.int32)
    for t in range(T):
        row = logits[t].copy()
        row[row == 0] = 0.0                       # -0.0 -> +0.0
        order = np.argsort(-row, kind="stable")   # stable: equal logits keep ascending id
        ids[t] = order[:k]
    return ids


def gate_weights(logits: np.ndarray, ids: np.ndarray, gating: int) -> np.ndarray:
    """Renormalised gates of the selected experts, float64 [T][k]."""
    T, k = ids.shape
    g = np.zeros((T, k), dtype=np.float64)
    for t in range(T):
        l = logits[t, ids[t]].astype(np.float64)
        if gating == GATE_SOFTMAX:
            z = np.exp(l - l[0])                  # l[0] is the largest selected logit
        elif gating == GATE_SIGMOID:
            z = 1.0 / (1.0 + np.exp(-l))
        else:
            raise ValueError("unknown gating")
        g[t] = z / z.sum()
    return g


# ----------------------------------------------------------------------------------------
# Classification against the slot table and the expert-sorted permutation
# ----------------------------------------------------------------------------------------

def effective_slots(slot_table: np.ndarray, n_slots: int, shared_slot: int):
    """Valid slot per expert (-1 if the expert is not usable from the cache) and a status word."""
    st = np.asarray(slot_table, dtype=np.int64)
    E = st.shape[0]
    eff = np.full(E, -1, dtype=np.int32)
    status = 0
    for e in range(E):
        s = int(st[e])
        if s == -1:
            continue
        if s < -1 or s >= n_slots:
            status |= STATUS_SLOT_RANGE
            continue
        if shared_slot >= 0 and s == shared_slot:
            status |= STATUS_SLOT_SHARED
            continue
        if any(int(st[o]) == s for o in range(E) if o != e):
            status |= STATUS_SLOT_DUP
            continue
        eff[e] = s
    return eff, status


def partition(ids: np.ndarray, eff_slot: np.ndarray, n_experts: int):
    """Hit/miss lists of pair indices p = t*k + j, each stably sorted by expert id."""
    T, k = ids.shape
    pairs = [(int(ids[t, j]), t * k + j) for t in range(T) for j in range(k)]
    hits = [(e, p) for (e, p) in pairs if eff_slot[e] >= 0]
    misses = [(e, p) for (e, p) in pairs if eff_slot[e] < 0]
    hits.sort(key=lambda ep: ep[0])      # Python's sort is stable
    misses.sort(key=lambda ep: ep[0])
    hit_off = np.zeros(n_experts + 1, dtype=np.int32)
    miss_off = np.zeros(n_experts + 1, dtype=np.int32)
    for e, _ in hits:
        hit_off[e + 1] += 1
    for e, _ in misses:
        miss_off[e + 1] += 1
    hit_off = np.cumsum(hit_off).astype(np.int32)
    miss_off = np.cumsum(miss_off).astype(np.int32)
    hit_pairs = np.array([p for _, p in hits], dtype=np.int32)
    miss_pairs = np.array([p for _, p in misses], dtype=np.int32)
    return hit_pairs, hit_off, miss_pairs, miss_off


def route(desc: dict, logits, slot_table) -> dict:
    """Everything the routing side of the layer produces, as numpy arrays."""
    logits = np.asarray(logits, dtype=np.float32)
    k, E = desc["top_k"], desc["n_experts"]
    ids = route_topk(logits, k)
    gates = gate_weights(logits, ids, desc["gating"])
    eff, status = effective_slots(np.asarray(slot_table), desc["n_slots"], desc["shared_slot"])
    slots = eff[ids] if ids.size else np.zeros(ids.shape, np.int32)
    hit_pairs, hit_off, miss_pairs, miss_off = partition(ids, eff, E)
    m_unique = int(np.count_nonzero(miss_off[1:] > miss_off[:-1]))
    return dict(topk_ids=ids, topk_w=gates, topk_slot=slots.astype(np.int32), eff_slot=eff,
                hit_pairs=hit_pairs, hit_off=hit_off, miss_pairs=miss_pairs, miss_off=miss_off,
                n_hit=len(hit_pairs), n_miss=len(miss_pairs), m_unique_miss=m_unique,
                status=status)


# ----------------------------------------------------------------------------------------
# Expert evaluation and the partial layer output
# ----------------------------------------------------------------------------------------

def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def expert_ffn(x: np.ndarray, w1: np.ndarray, w3: np.ndarray, w2: np.ndarray,
               h_bf16: bool = False) -> np.ndarray:
    """SwiGLU expert on rows of x: [n][H] -> [n][H], float64 arithmetic; with h_bf16 the
    intermediate activation is rounded to bfloat16 before the down projection."""
    h = silu(x @ w1.T) * (x @ w3.T)
    if h_bf16:
        h = round_bf16(h)
    return h @ w2.T


# ----------------------------------------------------------------------------------------
# fp8 activations (optional mode): per-token, per-128-channel e4m3fn with power-of-two scales
# ----------------------------------------------------------------------------------------

def round_bf16(v: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 value (8 significant bits, round half to even), as float64.  Normal
    range and zero only (no value here comes near bfloat16's subnormals or its overflow)."""
    v = np.asarray(v, dtype=np.float64)
    m, p = np.frexp(v)                      # v = m 2^p, 0.5 <= |m| < 1
    return np.ldexp(np.rint(np.ldexp(m, 8)), p - 8)


def round_e4m3fn(v: np.ndarray) -> np.ndarray:
    """Nearest e4m3fn value, ties to even, for |v| <= 448 (no saturation needed), as float64.
    Normal values 2^-6 .. 448 have 3 mantissa bits (spacing 2^(p-4) in [2^(p-1), 2^p)); below
    2^-6 the subnormals are multiples of 2^-9."""
    v = np.asarray(v, dtype=np.float64)
    _, p = np.frexp(v)
    spacing = np.ldexp(1.0, np.maximum(p - 4, -9))
    return np.rint(v / spacing) * spacing


def act_quant_fp8(v: np.ndarray):
    """Quantise-dequantise rows of v [n][D] (D a multiple of 128) in 128-wide blocks: scale
    2^e with e the smallest integer such that 448 * 2^e >= the block's largest magnitude (0 for
    a block of zeros), values rounded to e4m3fn.  Returns (dequantised float64 [n][D], e [n][D/128])."""
    v = np.asarray(v, dtype=np.float64)
    n, D = v.shape
    blocks = v.reshape(n, D // 128, 128)
    amax = np.abs(blocks).max(axis=2)
    m, p = np.frexp(amax)                   # amax = m 2^p; 448 = 0.875 2^9
    e = np.where(amax > 0, p - 9 + (m > 0.875), 0).astype(np.int64)
    scale = np.ldexp(1.0, e)[..., None]
    q = round_e4m3fn(blocks / scale) * scale
    return q.reshape(n, D), e


def expert_ffn_fp8_act(x: np.ndarray, w1: np.ndarray, w3: np.ndarray, w2: np.ndarray) -> np.ndarray:
    """SwiGLU expert with fp8 activations: [n][H] -> [n][H], float64 arithmetic."""
    xq, _ = act_quant_fp8(x)
    h = silu(xq @ w1.T) * (xq @ w3.T)
    hq, _ = act_quant_fp8(round_bf16(h))
    return hq @ w2.T


def expert_weights(banks: dict, desc: dict, slot: int):
    """Decoded (W1, W3, W2) of the expert stored in bank row ``slot``."""
    I = desc["inter"]
    wd = desc["w_dtype"]
    s13 = banks.get("s13")
    s2 = banks.get("s2")
    w13 = decode_weight(banks["w13"][slot], wd, None if s13 is None else s13[slot])
    w2 = decode_weight(banks["w2"][slot], wd, None if s2 is None else s2[slot])
    return w13[:I], w13[I:], w2


def decode_x(x: np.ndarray, x_dtype: int) -> np.ndarray:
    if x_dtype == DT_F32:
        return np.asarray(x, dtype=np.float64)
    return bf16_bits_to_f64(x)


def moe_partial(desc: dict, banks: dict, logits, slot_table, x, tokens=None):
    """Partial MoE output over cache-resident experts.

    desc   : hidden, inter, n_experts, top_k, gating, w_dtype, x_dtype, n_slots, shared_slot,
             optionally act_quant (ACT_EXACT when absent)
    banks  : w13 [n_slots][2I][H], w2 [n_slots][H][I] (float32 arrays, bf16 bit patterns as
             uint16, fp8 codes as uint8, or MXFP4 code pairs as uint8 [..][K/2]) and for fp8 s13, s2
             float32 block scales, for MXFP4 uint8 E8M0 scales [..][K/32][rows]
    logits : [T][E] float32; slot_table : [E] int32; x : [T][H] (float32 or bf16 bits as uint16)
    tokens : optional list of token indices; only those rows are evaluated (others stay 0)

    Returns (out [T][H] float32, routing dict from ``route``).
    """
    r = route(desc, logits, slot_table)
    T = np.asarray(logits).shape[0]
    H, k = desc["hidden"], desc["top_k"]
    want = np.ones(T, dtype=bool) if tokens is None else np.isin(np.arange(T), tokens)
    if desc.get("act_quant", ACT_EXACT) == ACT_FP8_1X128_POW2:
        ffn = expert_ffn_fp8_act
    else:
        h_bf16 = desc["w_dtype"] != DT_F32
        ffn = lambda xr, w1, w3, w2: expert_ffn(xr, w1, w3, w2, h_bf16)
    acc = np.zeros((T, H), dtype=np.float64)
    # group the wanted hit pairs by expert and run each expert once over its tokens
    for e in range(desc["n_experts"]):
        lo, hi = r["hit_off"][e], r["hit_off"][e + 1]
        if hi == lo:
            continue
        ps = [int(p) for p in r["hit_pairs"][lo:hi] if want[int(p) // k]]
        if not ps:
            continue
        ts = [p // k for p in ps]
        w1, w3, w2 = expert_weights(banks, desc, int(r["eff_slot"][e]))
        y = ffn(decode_x(x[ts], desc["x_dtype"]), w1, w3, w2)
        for i, p in enumerate(ps):
            acc[p // k] += r["topk_w"][p // k, p % k] * y[i]
    if desc["shared_slot"] >= 0:
        ts = [t for t in range(T) if want[t]]
        if ts:
            w1, w3, w2 = expert_weights(banks, desc, desc["shared_slot"])
            acc[ts] += ffn(decode_x(x[ts], desc["x_dtype"]), w1, w3, w2)
    return acc.astype(np.float32), r


# ----------------------------------------------------------------------------------------
# Device-side cache control: the fill / CPU split of the misses and LRU victim selection
# (Section 3.2, Eq. (miss-partition) to Eq. (dynamic-split) and the LRU residency space;
# Section 4.1, device-side cache control)
# ----------------------------------------------------------------------------------------
#
# Readings taken where the paper leaves the details open:
# * q: for m >= 1 missing experts, q* = m B_P / B_H rounded half up, then at least 1, at most m,
#   at most K (the LRU candidates one pass yields) and at most the number of evictable slots.
#   When B_H <= B_P there is no residual host bandwidth and every miss is filled (q = m before
#   the caps).  m = 0 gives q = 0.
# * which misses are filled: the most demanded (routed pairs in this step) first, ties to the
#   lower expert id; the rest execute on the CPU, listed by ascending id.
# * recency: a slot's stamp is the last step its expert was demanded (hit or filled).  Victims
#   are the least recently used slots that were not hit in this step and are not the shared
#   expert's slot; empty slots count as oldest; equal stamps go to the lower slot id.  The i-th
#   filled expert takes the i-th victim.
# * a routing whose slot table was faulty (status != 0) changes nothing: every missing expert is
#   left to the CPU.


def fill_count(m: int, b_pcie: float, b_host: float, k_max: int, n_evictable: int) -> int:
    """Number of misses served by cache fills, q (Section 3.2, Eq. (dynamic-split))."""
    if m <= 0:
        return 0
    if b_host <= b_pcie:
        q = m
    else:
        q = int(np.floor(m * (b_pcie / b_host) + 0.5))
    q = max(1, q)
    return min(q, m, k_max, n_evictable)


def cache_plan(desc: dict, routing: dict, slot_table, slot_expert, slot_stamp, b_pcie: float,
               b_host: float, k_max: int, step: int) -> dict:
    """Fill / CPU split of one layer step's misses and the cache update it implies.

    routing : the dict ``route`` returns for this step's logits and ``slot_table``
    slot_expert [n_slots] int32 (-1 = empty), slot_stamp [n_slots] uint32: the cache state.
    Returns q, m, the fill list (expert, slot, evicted expert), the CPU list, and the new
    slot_table, slot_expert, slot_stamp and topk_slot.
    """
    E, k = desc["n_experts"], desc["top_k"]
    n_slots, shared = desc["n_slots"], desc["shared_slot"]
    hit_off, miss_off = routing["hit_off"], routing["miss_off"]
    table = np.array(slot_table, dtype=np.int32).copy()
    sexp = np.array(slot_expert, dtype=np.int32).copy()
    stamp = np.array(slot_stamp, dtype=np.uint32).copy()
    tslot = routing["topk_slot"].copy()
    missing = [e for e in range(E) if miss_off[e + 1] > miss_off[e]]
    m = len(missing)
    out = dict(m=m, status=int(routing["status"]), fill_expert=[], fill_slot=[], evict_expert=[])
    if routing["status"] != 0:
        out.update(q=0, cpu_expert=sorted(missing), slot_table=table, slot_expert=sexp,
                   slot_stamp=stamp, topk_slot=tslot)
        return out
    hit_slots = sorted({int(table[e]) for e in range(E) if hit_off[e + 1] > hit_off[e]})
    old_stamp = stamp.copy()
    for s in hit_slots:
        stamp[s] = step
    evictable = [s for s in range(n_slots) if s != shared and s not in hit_slots]
    age = lambda s: (0 if sexp[s] < 0 else 1 + int(old_stamp[s]), s)
    victims = sorted(evictable, key=age)
    q = fill_count(m, b_pcie, b_host, k_max, len(evictable))
    demand = {e: int(miss_off[e + 1] - miss_off[e]) for e in missing}
    by_demand = sorted(missing, key=lambda e: (-demand[e], e))
    fills, cpu = by_demand[:q], sorted(by_demand[q:])
    for i, e in enumerate(fills):
        v = victims[i]
        old = int(sexp[v])
        out["fill_expert"].append(e)
        out["fill_slot"].append(v)
        out["evict_expert"].append(old)
        if old >= 0:
            table[old] = -1
        table[e] = v
        sexp[v] = e
        stamp[v] = step
        for p in routing["miss_pairs"][miss_off[e]:miss_off[e + 1]]:
            tslot[int(p) // k, int(p) % k] = v
    out.update(q=q, cpu_expert=cpu, slot_table=table, slot_expert=sexp, slot_stamp=stamp,
               topk_slot=tslot)
    return out


# ----------------------------------------------------------------------------------------
# Placement replay over a routing trace (Section 5, "Expert locality", Figure 4b): the decode
# cache's global LRU against placements fixed before decode, at equal capacity
# ----------------------------------------------------------------------------------------
#
# Readings:
# * a trace is n_prefill prefill tokens followed by decode tokens of one layer; decode routes
#   one token per step.
# * 'prefill' placement: the C experts with the most routed pairs over the prefill tokens, ties
#   to the lower id, fixed for the whole decode (a placement chosen at prefill time).
# * 'blind' placement: experts 0 .. C-1, fixed (a routing-blind split; expert ids carry no
#   popularity in the synthetic traces).
# * 'lru': the decode cache starts from the prefill placement (the experts that survive prefill
#   seed decode) and every miss is filled (q = m), evicting the least recently demanded.
# * 'split': as 'lru', but each step's misses are split by Eq. (dynamic-split); the experts left
#   to the CPU are not cached.
# * initial recency: slot i holds the i-th placed expert with stamp C - i, so the most demanded
#   prefill expert is evicted last; decode step t (from 0) writes stamp C + 1 + t.
# * a miss is a routed (token, expert) pair whose expert is not resident when the token is
#   routed; the miss rate is misses / (decode tokens * k).


def placement(desc: dict, prefill_logits, capacity: int, policy: str) -> list:
    """Experts placed in slots 0 .. capacity-1 before decode, in slot order."""
    E, k = desc["n_experts"], desc["top_k"]
    if policy == "blind":
        return list(range(capacity))
    ids = route_topk(np.asarray(prefill_logits, dtype=np.float32), k)
    counts = np.bincount(ids.ravel(), minlength=E)
    order = sorted(range(E), key=lambda e: (-int(counts[e]), e))
    return order[:capacity]


def replay(desc: dict, logits, n_prefill: int, capacity: int, policy: str, b_pcie: float = 1.0,
           b_host: float = 1.0, k_max: int = 64) -> dict:
    """Per-step miss pairs of the decode tokens of one trace under a placement policy.

    desc: the layer (n_slots and shared_slot are replaced by capacity and -1).
    Returns misses [n_decode] int64 and the final slot_table, slot_expert, slot_stamp."""
    logits = np.asarray(logits, dtype=np.float32)
    E, k = desc["n_experts"], desc["top_k"]
    d = dict(desc, n_slots=capacity, shared_slot=-1)
    placed = placement(d, logits[:n_prefill], capacity, "blind" if policy == "blind" else "prefill")
    table = np.full(E, -1, dtype=np.int32)
    sexp = np.full(capacity, -1, dtype=np.int32)
    stamp = np.zeros(capacity, dtype=np.uint32)
    for i, e in enumerate(placed):
        table[e], sexp[i], stamp[i] = i, e, capacity - i
    if policy == "lru":
        b_pcie, b_host = 1.0, 1.0          # B_H <= B_P: every miss is filled
    misses = []
    for t in range(n_prefill, logits.shape[0]):
        r = route(d, logits[t:t + 1], table)
        misses.append(int(r["n_miss"]))
        if policy in ("lru", "split"):
            step = capacity + 1 + (t - n_prefill)
            p = cache_plan(d, r, table, sexp, stamp, b_pcie, b_host, k_max, step)
            table, sexp, stamp = p["slot_table"], p["slot_expert"], p["slot_stamp"]
    return dict(misses=np.array(misses, dtype=np.int64), slot_table=table, slot_expert=sexp,
                slot_stamp=stamp)


# ----------------------------------------------------------------------------------------
# Error metric used by the parity tests
# ----------------------------------------------------------------------------------------

def max_rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    """max |got - ref| / max(|ref|, rms of ref's row), over all elements."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if ref.size == 0:
        return 0.0
    rms = np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True))
    den = np.maximum(np.abs(ref), rms)
    num = np.abs(got - ref)
    rel = np.where(den > 0, num / np.where(den > 0, den, 1.0), np.where(num > 0, np.inf, 0.0))
    return float(rel.max())
