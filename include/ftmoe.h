/*
 * ftmoe.h -- C ABI of the MoE layer executed against a GPU expert cache (gfx950 / MI355X).
 *
 * What the library computes (FreeToken, Section 3.2 "Decode codesign" and Section 4.1
 * "CUDA-Graph-compatible LRU cache"): at one MoE layer, gating and the slot-table lookup are
 * device work.  A routed (token, expert) pair belongs to the hit set H when its expert occupies
 * a cache slot, and H is evaluated on the GPU; every other pair belongs to the miss set M, and
 * the m distinct experts of M are left to the host (CPU execution or a cache fill).  Summing the
 * GPU partial and the partial of the misses gives the layer output exactly.
 *
 * Layer definition used throughout (the paper states it only in words, Section 2):
 *   top-k      S_t = the k experts with the largest float32 logit, ordered by (logit desc,
 *              expert id asc); -0.0 compares equal to +0.0.  Inputs must be finite.
 *   gates      softmax mode: g_j = exp(l_j - l_max) / sum_{i in S_t} exp(l_i - l_max)
 *              sigmoid mode: g_j = s_j / sum_{i in S_t} s_i,  s = 1/(1+exp(-l))
 *   expert     FFN_e(x) = W2_e (silu(W1_e x) * (W3_e x)),  silu(z) = z / (1+exp(-z))
 *   output     out[t] = sum_{(t,j) in H} g_tj FFN_{e_tj}(x_t)  (+ FFN_shared(x_t) if configured)
 *
 * Conventions for every entry point:
 *   - All array arguments are DEVICE pointers owned by the caller, except where a field says
 *     host.  No call allocates or frees device memory or waits for the device: each validates
 *     its arguments on the host, then enqueues work on `stream` (a hipStream_t; NULL means the
 *     null stream) and returns.  Exceptions, all host-side: ft_cpu_experts computes on the
 *     calling thread or the pool's workers and returns when done; ft_cpu_pool_create starts
 *     threads; ft_prefill_layers creates five timing-free hipEvents per call (each released by
 *     the runtime once its work completes).
 *   - Host-checkable errors return a status before anything is enqueued.
 *   - The library keeps no state between calls and is reentrant; calls that share a
 *     workspace or output buffers must be ordered by the caller (same stream).
 *   - Device-detected problems with the slot table (see ft_route_t.counts[3]) cannot be
 *     returned synchronously; the offending experts are treated as misses instead.
 */
#ifndef FTMOE_H
#define FTMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FT_OK = 0,
    FT_ERR_NULL = 1,       /* a required pointer is NULL */
    FT_ERR_SHAPE = 2,      /* sizes out of the supported range (see ft_moe_desc_t) */
    FT_ERR_DTYPE = 3,      /* unsupported dtype / gating / mode combination */
    FT_ERR_CAPACITY = 4,   /* workspace smaller than ft_moe_workspace_bytes(desc, T) */
    FT_ERR_HIP = 5         /* a HIP runtime call failed while enqueuing */
} ft_status_t;

enum { FT_GATE_SOFTMAX_TOPK_RENORM = 0, FT_GATE_SIGMOID_TOPK_RENORM = 1 };

/* How the streaming (few-token) path sums a token's gate-weighted expert outputs (ft_moe_desc_t
 * .combine).  ORDERED: every expert output is stored by pair index and one kernel sums each
 * output element in a fixed order (routed pairs by ascending j, then the shared expert), so the
 * layer output is bit-reproducible; it costs one kernel launch and T*(k+1)*H*4 bytes of
 * workspace traffic.  ATOMIC: float32 atomic adds straight from the down projection, the order
 * of a token's k sums (and so the last bits) may differ between calls.  The matrix-core path
 * (T >= 256) always adds atomically. */
enum { FT_COMBINE_ORDERED = 0, FT_COMBINE_ATOMIC = 1 };

/* Activation precision of the expert evaluation (ft_moe_desc_t.act_quant).  EXACT: the paper's
 * weight-only dequantisation, activations in bf16.  FP8_1x128_POW2 (fp8 weights only; not the
 * paper's exact method, a mode for the fp8 matrix cores): the expert inputs x and the SwiGLU
 * activation h (first rounded to bf16) are quantised per token and 128-channel block to e4m3fn,
 * with the scale 2^e, e the smallest integer such that 448 * 2^e >= the block's largest
 * magnitude (clamped to [-127, 127]), values rounded to nearest, ties to even.  The many-token
 * path then multiplies fp8 by fp8 on the matrix cores (activation scales in the MFMA's
 * per-row scale operand, weight block scales on the float32 partial sums); the few-token path
 * widens the quantised values to bf16. */
enum { FT_ACT_EXACT = 0, FT_ACT_FP8_1x128_POW2 = 1 };

enum {
    FT_DT_F32 = 0,              /* IEEE float32 */
    FT_DT_BF16 = 1,             /* bfloat16 */
    FT_DT_FP8E4M3FN_B128 = 2,   /* OCP fp8 e4m3fn codes, one float32 scale per 128x128 block */
    FT_DT_MXFP4 = 3             /* OCP MXFP4: fp4 e2m1 codes, two per byte (element 2j in the low
                                   nibble of byte j), one e8m0 scale byte (2^(s-127)) per 32
                                   consecutive elements of a row */
};

#define FT_SLOT_MISS (-1)

/* Device status bits reported in ft_route_t.counts[3] (0 = slot table valid). */
#define FT_DEV_SLOT_RANGE  1    /* slot_table[e] < -1 or >= n_slots: expert treated as miss */
#define FT_DEV_SLOT_DUP    2    /* two experts share one slot: both treated as misses */
#define FT_DEV_SLOT_SHARED 4    /* a routed expert points at shared_slot: treated as miss */

/*
 * Layer description (host struct, read during the call only).
 *   hidden (H), inter (I): multiples of 128, 128 <= H, I <= 65536.
 *   n_experts (E): 1..1024 routed experts.   top_k (k): 1..min(E, 64).
 *   gating: FT_GATE_*.
 *   w_dtype: FT_DT_F32 with x_dtype FT_DT_F32, or FT_DT_BF16 / FT_DT_FP8E4M3FN_B128 /
 *            FT_DT_MXFP4 with x_dtype FT_DT_BF16.  Activations stay bf16 and products accumulate
 *            in float32.  MXFP4 weights times their scale are exact in bf16, so both paths
 *            widen them exactly.
 *            fp8 weights (weight-only dequantisation): each code is widened exactly to bf16 and
 *            the block scale multiplies the float32 partial sum of its 128-wide K block, on both
 *            the streaming (T < 256) and the matrix-core (T >= 256) path; a block scale of 0
 *            makes its block contribute exactly nothing.  The SwiGLU activation between the two
 *            projections is rounded to bf16 (float32 for f32).
 *   n_slots: number of bank rows (cache slots) in the banks, >= 0.
 *   shared_slot: bank row of an always-resident shared expert with gate 1 for every token,
 *                or -1 for none.
 *   combine: FT_COMBINE_* (0, the ordered combine, for a zero-initialised struct).
 *   act_quant: FT_ACT_* (0, exact, for a zero-initialised struct).  FT_ACT_FP8_1x128_POW2
 *              requires w_dtype FT_DT_FP8E4M3FN_B128 (FT_ERR_DTYPE otherwise) and is accepted by
 *              ft_moe_forward, ft_moe_forward_noalloc and ft_prefill_layers; ft_cpu_experts and
 *              ft_moe_step_hybrid, whose CPU branch evaluates exactly, return FT_ERR_DTYPE.
 */
typedef struct {
    int32_t hidden, inter, n_experts, top_k, gating, w_dtype, x_dtype, n_slots, shared_slot, combine,
        act_quant;
} ft_moe_desc_t;

/*
 * Expert banks: one row per cache slot, so bank row s holds the complete expert stored in
 * slot s (Section 3 "single elastic GPU expert cache", Section 4.2 "expert banks": all banks
 * share one expert-to-slot mapping, so one slot index addresses every tensor of an expert and
 * a cache fill is a plain row copy, never a relayout).  Device pointers, caller-owned,
 * row-major:
 *   w13 [n_slots][2I][H]  rows 0..I-1 = gate projection W1, rows I..2I-1 = up projection W3
 *   w2  [n_slots][H][I]   down projection
 *   s13 [n_slots][2I/128][H/128], s2 [n_slots][H/128][I/128]  float32 block scales (fp8,
 *       NULL for f32 and bf16): weight (r, c) = code(r, c) * scale(r/128, c/128).
 * MXFP4 packs two codes per byte along each row and keeps byte scales per 32 elements of a row,
 * stored run-major so that the scales of one 32-wide K run of consecutive rows are contiguous:
 *   w13 [n_slots][2I][H/2], w2 [n_slots][H][I/2]  uint8 code pairs
 *   s13 [n_slots][H/32][2I], s2 [n_slots][I/32][H]  uint8 e8m0 scales:
 *       weight (r, c) = e2m1(code(r, c)) * 2^(s(c/32, r) - 127)
 */
typedef struct {
    const void *w13;
    const void *w2;
    const void *s13;   /* float32 (fp8) or uint8 (MXFP4) scales; NULL for f32 and bf16 */
    const void *s2;
} ft_banks_t;

/*
 * Routing outputs (device pointers, caller-owned; T tokens, k = top_k, E = n_experts).
 * Section 4.1 keeps all routing-dependent control on the GPU as fixed-shape buffers with
 * device-resident valid counts; these are those buffers.
 *   topk_ids  [T][k] int32   selected experts, in top-k order
 *   topk_w    [T][k] float   renormalised gates
 *   topk_slot [T][k] int32   slot of the expert, or FT_SLOT_MISS
 *   hit_pairs [T*k]  int32   pair indices p = t*k + j of hits, sorted by (expert id, p);
 *                            entries past the hit count are -1
 *   miss_pairs[T*k]  int32   same for misses
 *   hit_off   [E+1]  int32   hit_pairs[hit_off[e] .. hit_off[e+1]) are expert e's hits
 *   miss_off  [E+1]  int32   same for misses
 *   counts    [4]    int32   n_hit, n_miss, m (distinct missing experts), device status bits
 */
typedef struct {
    int32_t *topk_ids;
    float *topk_w;
    int32_t *topk_slot;
    int32_t *hit_pairs;
    int32_t *miss_pairs;
    int32_t *hit_off;
    int32_t *miss_off;
    int32_t *counts;
} ft_route_t;

/*
 * Host-side destination of the miss list (pinned host memory, caller-owned, capacity for T
 * tokens): counts[4], miss_pairs[T*k], miss_off[E+1], topk_ids[T*k], topk_w[T*k].
 */
typedef struct {
    int32_t *counts;
    int32_t *miss_pairs;
    int32_t *miss_off;
    int32_t *topk_ids;
    float *topk_w;
} ft_host_miss_t;

/* Bytes of device workspace the calls need for up to max_tokens tokens; 0 if desc is invalid. */
size_t ft_moe_workspace_bytes(const ft_moe_desc_t *desc, int32_t max_tokens);

/*
 * Router, hit/miss classification and the expert-sorted permutation only (Section 3.2: gating
 * and the cache lookup are device work that separates hits from misses; Section 4.1: each routed
 * expert id is replaced by its slot id or by a flag that sends it to the CPU).
 *   logits     [T][E] float32 device
 *   slot_table [E] int32 device: slot of expert e, or -1 if not resident
 *   T >= 0 (T == 0 enqueues nothing and returns FT_OK)
 *   route      outputs as documented in ft_route_t
 *   ws, ws_bytes  device workspace of at least ft_moe_workspace_bytes(desc, T) bytes
 */
ft_status_t ft_route_only(const ft_moe_desc_t *desc, const float *logits, const int32_t *slot_table,
                          int32_t T, const ft_route_t *route, void *ws, size_t ws_bytes,
                          void *stream);

/*
 * The whole GPU side of one MoE layer: routing as in ft_route_only, then the grouped SwiGLU
 * expert FFN over the hit experts' slot-resident weights (plus the shared expert), then the
 * gate-weighted combine (Section 3.2: grouped evaluation of the GPU execution set; the GPU and
 * CPU partial sums merge exactly).
 *   x           [T][H] device, x_dtype
 *   out_partial [T][H] float32 device, fully overwritten; a token with no hit (and no shared
 *               expert) gets exact zeros.  The routing outputs are bit-reproducible; so is
 *               out_partial with desc->combine = FT_COMBINE_ORDERED below 256 tokens (else the
 *               order of a token's sum, and its last bits, may differ between calls).
 *   x, out_partial, banks->w13 and banks->w2 (and for MXFP4 banks->s13 and banks->s2) must be
 *   16-byte aligned (FT_ERR_SHAPE otherwise).
 */
ft_status_t ft_moe_forward(const ft_moe_desc_t *desc, const ft_banks_t *banks, const float *logits,
                           const int32_t *slot_table, const void *x, int32_t T,
                           float *out_partial, const ft_route_t *route, void *ws,
                           size_t ws_bytes, void *stream);

/*
 * ft_moe_forward without a workspace argument, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid allocation).  The
 * workspace is a device array inside the library of FT_NOALLOC_SCRATCH_BYTES per GPU, which that
 * GPU holds from the library's load until the process ends; the call itself allocates and frees
 * nothing.  Every argument and every result is as for ft_moe_forward.
 *   Returns FT_ERR_CAPACITY, before enqueuing anything, when ft_moe_workspace_bytes(desc, T)
 *   exceeds FT_NOALLOC_SCRATCH_BYTES (e.g. 64 MiB holds a Qwen3-30B-A3B-shaped layer up to 4804
 *   tokens, and a DeepSeek-V3-shaped one up to 1811 tokens, 2583 with FT_ACT_FP8_1x128_POW2,
 *   except 228..255, 217..255 with FT_ACT_FP8_1x128_POW2, under the ordered combine, whose
 *   per-pair outputs take T*(k+1)*H*4 bytes).  FT_ERR_HIP if the array's device address
 *   cannot be found: it is looked up on the first call on each device (make that first call, a
 *   T = 0 call will do, before capturing a graph).
 *   All calls on one GPU share its array and nothing in it is kept between calls: calls that may
 *   overlap on one GPU (different streams without ordering between them) race on it and must be
 *   serialised by the caller.
 */
#define FT_NOALLOC_SCRATCH_BYTES (64u << 20)
ft_status_t ft_moe_forward_noalloc(const ft_moe_desc_t *desc, const ft_banks_t *banks,
                                   const float *logits, const int32_t *slot_table, const void *x,
                                   int32_t T, float *out_partial, const ft_route_t *route,
                                   void *stream);

/*
 * Stage boundaries of one ft_moe_forward call, for attributing device time per stage without
 * a profiler.  ev[i] is recorded on the call's stream when stage i starts and ev[FT_PROF_STAGES]
 * when the last stage ends: stage 0 routing (top-k, classification, permutation), stage 1 the
 * grouped gate/up projection with SiLU-mul, stage 2 the grouped down projection, stage 3 the
 * combine (a stage that a fused kernel absorbs records two adjacent events).  Entries are
 * hipEvent_t handles created by the caller; NULL entries are skipped.
 */
#define FT_PROF_STAGES 4
typedef struct {
    void *ev[FT_PROF_STAGES + 1];
} ft_prof_events_t;

/* ft_moe_forward, plus hipEventRecord of the caller's stage events (may be NULL). */
ft_status_t ft_moe_forward_profiled(const ft_moe_desc_t *desc, const ft_banks_t *banks,
                                    const float *logits, const int32_t *slot_table, const void *x,
                                    int32_t T, float *out_partial, const ft_route_t *route,
                                    void *ws, size_t ws_bytes, void *stream,
                                    const ft_prof_events_t *events);

/*
 * Enqueue asynchronous device-to-host copies of the miss list (counts, miss_pairs, miss_off,
 * topk_ids, topk_w) into pinned host buffers, full fixed capacity, so no host synchronisation
 * is needed to size them (Section 3.2: the misses are executed on the CPU or filled into the
 * cache; Section 4.1: fixed-shape buffers with device-resident counts).  The host may read
 * them after synchronising with `stream`.
 */
ft_status_t ft_miss_list_to_host(const ft_moe_desc_t *desc, const ft_route_t *route, int32_t T,
                                 const ft_host_miss_t *host, void *stream);

/*
 * Device-side cache control of one layer step (Section 3.2: the m distinct missing experts
 * are split into q cache fills and m - q CPU executions with q* = m B_P / B_H, Eq.
 * (dynamic-split), rounded, at least one fill; the residency space is LRU: a hit refreshes an
 * expert's recency, a fill evicts the least recently demanded expert.  Section 4.1: one kernel
 * classifies, derives q, takes the first q of the K least-recently-used candidate slots found in
 * one pass, rewrites routed ids into slot ids and leaves a fixed-shape copy list with a valid
 * count).  Runs on the routing of this step (ft_route_only / ft_moe_forward with the same
 * slot_table) and updates the cache state in place; the copies themselves are the caller's.
 *
 * Rules (where the paper leaves them open):
 *   q = 0 if m = 0; else q = round_half_up(m * b_pcie / b_host) (q = m if b_host <= b_pcie),
 *       at least 1, at most m, max_fill and the number of evictable slots.
 *   Filled first: the missing experts with the most routed pairs in this step, ties to the
 *       lower expert id; the rest are listed for the CPU in ascending id.
 *   Evictable: slots not hit in this step, other than shared_slot.  Victim order: empty slots
 *       (slot_expert -1) first, then ascending stamp, ties to the lower slot id.  The i-th filled
 *       expert takes the i-th victim.
 *   If the routing reported slot-table faults (route counts[3] != 0) nothing changes and every
 *   missing expert is listed for the CPU.
 *
 * Cache state (device, caller-owned, updated in place):
 *   slot_table  [E] int32   expert -> slot or -1; filled experts get their slot, evicted
 *                           experts get -1
 *   slot_expert [n_slots] int32   slot -> expert or -1 (must be the inverse of slot_table)
 *   slot_stamp  [n_slots] uint32  step at which the slot's expert was last demanded; hit and
 *                           filled slots take `step`.  Stamps must grow with the steps.
 *   route->topk_slot        routed pairs of filled experts take the new slot id; pairs left to
 *                           the CPU keep FT_SLOT_MISS.  route->hit/miss lists are not changed.
 * Plan outputs (device, caller-owned):
 *   fill_expert, fill_slot, evict_expert [max_fill] int32: fill i copies expert fill_expert[i]
 *       into slot fill_slot[i], replacing evict_expert[i] (-1 if the slot was empty); entries
 *       from q on are -1
 *   cpu_expert [E] int32: missing experts left to the CPU, ascending; entries from m - q on -1
 *   counts [4] int32: q, m - q, m, route status
 * Limits: n_slots <= 4096, 1 <= max_fill <= 64, b_pcie > 0 and b_host > 0 (same unit).
 * T == 0 enqueues nothing.
 */
typedef struct {
    int32_t *slot_expert;
    uint32_t *slot_stamp;
    uint32_t *clock;   /* [1] device step counter, or NULL.  When set, the step's stamp is
                          clock + 1 (written back), and policy->step is ignored: a captured step
                          then advances on every replay */
} ft_cache_state_t;

typedef struct {
    double b_pcie;      /* B_P: pinned host-to-GPU expert transfer bandwidth */
    double b_host;      /* B_H: host expert-processing bandwidth */
    int32_t max_fill;   /* K: LRU candidates per step */
    uint32_t step;      /* current step (the stamp written to hit and filled slots) */
} ft_cache_policy_t;

typedef struct {
    int32_t *fill_expert;
    int32_t *fill_slot;
    int32_t *evict_expert;
    int32_t *cpu_expert;
    int32_t *counts;
} ft_fill_plan_t;

ft_status_t ft_cache_plan(const ft_moe_desc_t *desc, const ft_route_t *route, int32_t T,
                          int32_t *slot_table, const ft_cache_state_t *state,
                          const ft_cache_policy_t *policy, const ft_fill_plan_t *plan,
                          void *stream);

/*
 * Persistent CPU worker pool of the CPU branch (Section 4.1: a native worker pool with SIMD
 * kernels).  n_threads workers (<= 0: one per CPU of the process's affinity mask); pin != 0
 * pins each worker to one CPU of the mask, one hardware thread of every physical core first,
 * then their second hardware threads.  Returns NULL if
 * the threads cannot be started.  A pool runs one job at a time (calls that share it are
 * serialised); destroy it only when no call that uses it is running or enqueued.  A pool
 * holds a small mailbox in pinned host memory through which hybrid steps hand their CPU branch
 * to a listener thread of the pool (created without a GPU, the pool has none and serves
 * ft_cpu_experts only; hybrid steps then hand over with a host function).
 */
typedef struct ft_cpu_pool ft_cpu_pool_t;
ft_cpu_pool_t *ft_cpu_pool_create(int32_t n_threads, int32_t pin);
void ft_cpu_pool_destroy(ft_cpu_pool_t *pool);

/*
 * CPU branch of a layer step (Section 3.2: the missing experts the split leaves to the CPU
 * execute from the host expert pool, concurrently with the GPU, and the two partial sums add up
 * to the exact layer output; Section 4.1: in-kernel dequantisation).  HOST pointers,
 * caller-owned; runs synchronously on the workers of `pool` (NULL: on the calling thread).
 *   host_pool   the complete expert pool in host memory, indexed by EXPERT id, in the bank
 *               layout of ft_banks_t: w13 [E][2I][H], w2 [E][H][I], s13/s2 per expert (fp8)
 *   x           [T][H] x_dtype;  topk_ids, topk_w [T][k]: this step's routing
 *   experts     n_list distinct expert ids to evaluate (e.g. ft_fill_plan_t.cpu_expert)
 *   out         [T][H] float32, overwritten: out[t] = sum over (t, j) with topk_ids[t][j] in
 *               experts of topk_w[t][j] * FFN_e(x_t), every product accumulated in float32 and
 *               every element summed in a fixed order (independent of the pool); the SwiGLU
 *               activation between the two projections is rounded to bf16 (float32 for f32
 *               layers), as on the GPU
 * Returns FT_ERR_DTYPE if the host CPU lacks AVX2 and FMA.
 */
ft_status_t ft_cpu_experts(const ft_moe_desc_t *desc, const ft_banks_t *host_pool, const void *x,
                           int32_t T, const int32_t *topk_ids, const float *topk_w,
                           const int32_t *experts, int32_t n_list, float *out, ft_cpu_pool_t *pool);

/*
 * Cache fills of one step (Section 3.2: the q planned experts are copied into their slots over
 * PCIe, then execute on the GPU and stay resident; Section 4.1: one fixed-shape launch driven by
 * the device-resident fill list and its valid count, applied to every bank at once since all
 * banks share one expert -> slot mapping).  Copies, for every fill i < plan->counts[0], expert
 * plan->fill_expert[i]'s rows of every bank from host_pool into slot plan->fill_slot[i] of
 * dev_banks, reading the pool directly over PCIe; the host does not need to know q.
 *   host_pool  the complete expert pool, indexed by EXPERT id, in the ft_banks_t layout, in
 *              pinned host memory (hipHostMalloc; pageable memory returns FT_ERR_SHAPE)
 *   dev_banks  the device slot banks (as for ft_moe_forward), 16-byte aligned
 *   plan       the device plan ft_cache_plan wrote; max_fill as passed there
 */
ft_status_t ft_cache_fill(const ft_moe_desc_t *desc, const ft_banks_t *host_pool,
                          const ft_banks_t *dev_banks, const ft_fill_plan_t *plan, int32_t max_fill,
                          void *stream);

/*
 * Host side of ft_moe_step_hybrid, caller-owned, capacity for T tokens: pinned host buffers
 * (hipHostMalloc; x and cpu_out 16-byte aligned) that the device writes the step's routing and
 * plan into and reads the CPU partial from, over PCIe, and `task`, plain host memory the call
 * writes what its CPU branch needs into.  All of it must stay valid while the step (or any graph
 * captured from it) can run.
 */
typedef struct {
    uint64_t opaque[24];
} ft_hybrid_task_t;

typedef struct {
    int32_t *plan_counts;   /* [4] */
    int32_t *cpu_expert;    /* [E] */
    int32_t *topk_ids;      /* [T*k] */
    float *topk_w;          /* [T*k] */
    void *x;                /* [T][H] x_dtype */
    float *cpu_out;         /* [T][H] the CPU partial */
    ft_hybrid_task_t *task; /* written by the call (not pinned memory) */
} ft_hybrid_host_t;

/*
 * One complete MoE layer step over the GPU expert cache and the host (Section 3.2; Section 4.1
 * keeps the whole step in fixed-shape buffers with device-resident counts, so it can be captured
 * in a graph and replayed).  Enqueues on `stream`, without waiting for the device:
 *   1. the routing on the current slot table (ft_route_only) and the cache plan (ft_cache_plan,
 *      which updates the slot table and rewrites the routed slot ids of the experts it fills);
 *   2. one kernel that writes the plan counts, the CPU list, the routing and x into the pinned
 *      host staging, and one that posts the step to the pool's mailbox; the pool's listener
 *      thread, polling it, evaluates the experts the plan leaves to the CPU into host->cpu_out
 *      on the pool's workers (NULL pool: a host function, hipLaunchHostFunc, evaluates them on
 *      the runtime's callback thread before the stream goes on);
 *   3. the fills (ft_cache_fill) and the grouped evaluation of G = H u F straight from the
 *      rewritten slot ids (the step routes once), overlapping the CPU branch;
 *   4. a kernel that waits for the pool to report the step done (bounded: after tens of seconds
 *      without an answer it gives up, counting a timeout in the mailbox, and the output lacks the
 *      CPU partial), and the addition of the CPU partial (read over PCIe): `out` receives the
 *      exact layer output over all routed experts (+ shared expert).
 * Synchronise `stream` before using `out`, the cache state or the staging buffers.  Capturing
 * the call on `stream` gives a graph whose replays each run one step on the same buffers; give
 * `state` a device clock so that the stamps advance.  Steps that share a pool run their CPU
 * branches one at a time.
 *   slot_table, state  updated in place as by ft_cache_plan
 *   out          [T][H] float32 device: the full layer output
 *   route, plan, ws    as for the calls above
 *   Returns FT_ERR_SHAPE if a staging buffer is not pinned host memory or is misaligned.
 */
ft_status_t ft_moe_step_hybrid(const ft_moe_desc_t *desc, const ft_banks_t *dev_banks,
                               const ft_banks_t *host_pool, const float *logits, int32_t *slot_table,
                               const ft_cache_state_t *state, const ft_cache_policy_t *policy,
                               const void *x, int32_t T, float *out,
                               const ft_route_t *route, const ft_fill_plan_t *plan,
                               const ft_hybrid_host_t *host, void *ws, size_t ws_bytes,
                               ft_cpu_pool_t *pool, void *stream);

/*
 * Full-layer double-buffered prefill of one chunk of T tokens through n_layers MoE layers whose
 * complete expert sets live in host memory (Section 3.1, "Prefill Codesign": prefill routes nearly every
 * expert of a layer, so experts are not fetched on demand; two full-layer buffers from the slot
 * pool take turns, a transfer stream loading all experts of layer l + 1 into one, before that
 * layer's routing is known, while the GPU evaluates layer l from the other.  Section 5,
 * "Pipelined prefill": with the second buffer disabled the transfers serialise against the
 * evaluation).
 *   host_layers  [n_layers] HOST array of expert pools in PINNED host memory (hipHostMalloc;
 *                pageable memory returns FT_ERR_SHAPE), each n_slots rows in the ft_banks_t layout:
 *                the complete expert set of that layer, shared expert included
 *   dev_buf      [2] HOST array of device full-layer buffers (distinct, n_slots rows each,
 *                16-byte aligned); the call leaves the last two layers' experts in them
 *   slot_table   [E] device: row of expert e in a full-layer buffer, the same for every layer
 *                (the identity when the pools hold the experts in id order)
 *   logits, x, out  [n_layers] HOST arrays of device pointers: layer l's router logits [T][E],
 *                hidden states [T][H] (x_dtype) and output [T][H] float32, as for ft_moe_forward
 *   route, ws    as for ft_moe_forward, reused by every layer (route holds the last layer's routing)
 *   overlap      1: layer l + 1 loads on copy_stream while layer l is evaluated on stream
 *                   (copy_stream must be a different, non-NULL stream);
 *                0: load l, evaluate l, load l + 1, ... all on stream (copy_stream unused)
 * Layer l's output equals ft_moe_forward of layer l with every expert resident.  The loads are
 * DMA-engine copies (hipMemcpyAsync) and take no compute unit from the evaluation.  Everything
 * is enqueued without blocking the host; the loads start after the work already on `stream`,
 * and the last evaluation waits for the last load, so synchronising `stream` covers all of it.
 * Host arrays are read during the call only.
 */
ft_status_t ft_prefill_layers(const ft_moe_desc_t *desc, int32_t n_layers,
                              const ft_banks_t *host_layers, const ft_banks_t *dev_buf,
                              const int32_t *slot_table, const float *const *logits,
                              const void *const *x, int32_t T, float *const *out,
                              const ft_route_t *route, void *ws, size_t ws_bytes, int32_t overlap,
                              void *stream, void *copy_stream);

/* Static string for a status code. */
const char *ft_status_string(ft_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* FTMOE_H */
