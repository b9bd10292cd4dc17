// C ABI entry points of libftmoe: host-side validation, workspace carving, kernel enqueue.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <mutex>
#include <thread>
#include <vector>

#include "ftmoe_internal.h"
#include "route_wave.h"

using namespace ftmoe;

namespace {

bool desc_ok(const ft_moe_desc_t *d) {
    if (!d) return false;
    if (d->hidden < 128 || d->hidden > 65536 || d->hidden % 128) return false;
    if (d->inter < 128 || d->inter > 65536 || d->inter % 128) return false;
    if (d->n_experts < 1 || d->n_experts > kMaxExperts) return false;
    if (d->top_k < 1 || d->top_k > d->n_experts || d->top_k > kMaxTopK) return false;
    if (d->n_slots < 0) return false;
    if (d->shared_slot < -1 || d->shared_slot >= d->n_slots) return false;
    if (d->combine != FT_COMBINE_ORDERED && d->combine != FT_COMBINE_ATOMIC) return false;
    if (d->act_quant != FT_ACT_EXACT && d->act_quant != FT_ACT_FP8_1x128_POW2) return false;
    return true;
}

ft_status_t dtype_status(const ft_moe_desc_t *d) {
    if (d->gating != FT_GATE_SOFTMAX_TOPK_RENORM && d->gating != FT_GATE_SIGMOID_TOPK_RENORM)
        return FT_ERR_DTYPE;
    if (d->act_quant == FT_ACT_FP8_1x128_POW2)
        return d->w_dtype == FT_DT_FP8E4M3FN_B128 && d->x_dtype == FT_DT_BF16 ? FT_OK : FT_ERR_DTYPE;
    if (d->w_dtype == FT_DT_F32 && d->x_dtype == FT_DT_F32) return FT_OK;
    if ((d->w_dtype == FT_DT_BF16 || d->w_dtype == FT_DT_FP8E4M3FN_B128 || d->w_dtype == FT_DT_MXFP4) &&
        d->x_dtype == FT_DT_BF16)
        return FT_OK;
    return FT_ERR_DTYPE;
}

ft_status_t check_common(const ft_moe_desc_t *desc, const float *logits, const int32_t *slot_table,
                         int32_t T, const ft_route_t *route, void *ws, size_t ws_bytes) {
    if (!desc || !route) return FT_ERR_NULL;
    if (!desc_ok(desc)) return FT_ERR_SHAPE;
    if (ft_status_t s = dtype_status(desc); s != FT_OK) return s;
    if (T < 0 || T > 1048576) return FT_ERR_SHAPE;
    if (T == 0) return FT_OK;
    if (!logits || !slot_table || !ws) return FT_ERR_NULL;
    if (!route->topk_ids || !route->topk_w || !route->topk_slot || !route->hit_pairs ||
        !route->miss_pairs || !route->hit_off || !route->miss_off || !route->counts)
        return FT_ERR_NULL;
    if (ws_bytes < ft_moe_workspace_bytes(desc, T)) return FT_ERR_CAPACITY;
    return FT_OK;
}

WsView carve(const ft_moe_desc_t *d, int T, void *ws) {
    const WsLayout L = ws_layout(d->n_experts, d->hidden, d->inter, d->top_k, d->w_dtype, d->combine, d->act_quant, T);
    uint8_t *b = static_cast<uint8_t *>(ws);
    WsView v;
    v.eff_slot = reinterpret_cast<int32_t *>(b + L.eff_slot);
    v.blk_hist = reinterpret_cast<int32_t *>(b + L.blk_hist);
    v.grp_meta = reinterpret_cast<int32_t *>(b + L.grp_meta);
    v.grp_slot = reinterpret_cast<int32_t *>(b + L.grp_slot);
    v.grp_beg = reinterpret_cast<int32_t *>(b + L.grp_beg);
    v.grp_len = reinterpret_cast<int32_t *>(b + L.grp_len);
    v.grp_mt_off = reinterpret_cast<int32_t *>(b + L.grp_mt_off);
    v.mt_group = reinterpret_cast<int32_t *>(b + L.mt_group);
    v.row_tok = reinterpret_cast<int32_t *>(b + L.row_tok);
    v.row_gate = reinterpret_cast<float *>(b + L.row_gate);
    v.row_pair = reinterpret_cast<int32_t *>(b + L.row_pair);
    const bool aq = d->act_quant == FT_ACT_FP8_1x128_POW2;
    const bool gemm = gemm_shape(T, d->hidden, d->inter, d->w_dtype);
    v.h = aq && gemm ? nullptr : b + L.h;
    v.ypart = L.ypart_bytes ? reinterpret_cast<float *>(b + L.ypart) : nullptr;
    v.xq = aq && gemm ? b + L.xq : nullptr;
    v.xs = aq && gemm ? b + L.xs : nullptr;
    v.hq = aq && gemm ? b + L.hq : nullptr;
    v.hs = aq && gemm ? b + L.hs : nullptr;
    v.xd = aq && !gemm ? reinterpret_cast<uint16_t *>(b + L.xd) : nullptr;
    return v;
}

RouteOut route_out(const ft_route_t *r) {
    return RouteOut{r->topk_ids, r->topk_w, r->topk_slot, r->hit_pairs, r->miss_pairs,
                    r->hit_off, r->miss_off, r->counts};
}

RouteArgs route_args(const ft_moe_desc_t *d, const float *logits, const int32_t *slot_table, int T,
                     const ft_route_t *route, const WsView &wv) {
    RouteArgs a{};
    a.logits = logits;
    a.slot_table = slot_table;
    a.T = T;
    a.E = d->n_experts;
    a.k = d->top_k;
    a.gating = d->gating;
    a.n_slots = d->n_slots;
    a.shared_slot = d->shared_slot;
    int nbits = 1;
    while ((1 << nbits) < d->n_experts) ++nbits;
    a.nbits = nbits;
    a.scan_parts = 1;
    a.ro = route_out(route);
    a.wv = wv;
    return a;
}

}  // namespace

namespace ftmoe {

ft_status_t check_forward(const ft_moe_desc_t *desc, const ft_banks_t *banks, const float *logits,
                          const int32_t *slot_table, const void *x, int32_t T, const float *out_partial,
                          const ft_route_t *route, const void *ws, size_t ws_bytes) {
    if (ft_status_t s = check_common(desc, logits, slot_table, T, route, const_cast<void *>(ws), ws_bytes);
        s != FT_OK)
        return s;
    if (!banks) return FT_ERR_NULL;
    if (T == 0) return FT_OK;
    if (!x || !out_partial) return FT_ERR_NULL;
    if (desc->n_slots > 0 && (!banks->w13 || !banks->w2)) return FT_ERR_NULL;
    if (has_scales(desc->w_dtype) && desc->n_slots > 0 && (!banks->s13 || !banks->s2)) return FT_ERR_NULL;
    if (desc->w_dtype == FT_DT_MXFP4 &&
        (reinterpret_cast<uintptr_t>(banks->s13) | reinterpret_cast<uintptr_t>(banks->s2)) % 16)
        return FT_ERR_SHAPE;
    const uintptr_t al = reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(out_partial) |
                         reinterpret_cast<uintptr_t>(banks->w13) | reinterpret_cast<uintptr_t>(banks->w2);
    if (al % 16) return FT_ERR_SHAPE;
    return FT_OK;
}

}  // namespace ftmoe

extern "C" {

size_t ft_moe_workspace_bytes(const ft_moe_desc_t *desc, int32_t max_tokens) {
    if (!desc_ok(desc) || max_tokens < 0) return 0;
    const int T = max_tokens > 0 ? max_tokens : 1;
    return ws_layout(desc->n_experts, desc->hidden, desc->inter, desc->top_k, desc->w_dtype, desc->combine,
                     desc->act_quant, T)
        .total;
}

ft_status_t ft_route_only(const ft_moe_desc_t *desc, const float *logits, const int32_t *slot_table,
                          int32_t T, const ft_route_t *route, void *ws, size_t ws_bytes,
                          void *stream) {
    if (ft_status_t s = check_common(desc, logits, slot_table, T, route, ws, ws_bytes); s != FT_OK)
        return s;
    if (T == 0) return FT_OK;
    const WsView wv = carve(desc, T, ws);
    const RouteArgs ra = route_args(desc, logits, slot_table, T, route, wv);
    if (launch_route(ra, static_cast<hipStream_t>(stream)) != hipSuccess) return FT_ERR_HIP;
    return FT_OK;
}

}  // extern "C"

namespace {

hipError_t enqueue_experts(const ft_moe_desc_t *desc, const ft_banks_t *banks, const void *x, int32_t T,
                           float *out_partial, const ft_route_t *route, const WsView &wv, hipStream_t s,
                           const Prof &prof, const RouteArgs *self_route = nullptr);

ft_status_t forward_impl(const ft_moe_desc_t *desc, const ft_banks_t *banks, const float *logits,
                         const int32_t *slot_table, const void *x, int32_t T, float *out_partial,
                         const ft_route_t *route, void *ws, size_t ws_bytes, void *stream,
                         const ft_prof_events_t *events) {
    if (ft_status_t s = check_forward(desc, banks, logits, slot_table, x, T, out_partial, route, ws, ws_bytes);
        s != FT_OK)
        return s;
    if (T == 0) return FT_OK;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    Prof prof(events, s);
    const WsView wv = carve(desc, T, ws);
    const RouteArgs ra = route_args(desc, logits, slot_table, T, route, wv);
    if (!prof.mark(0)) return FT_ERR_HIP;
    // one or two tokens on the streaming path: the gate/up kernel routes the call itself (no
    // router launch); otherwise the router kernels run first
    const bool self_route = desc->n_slots > 0 && self_route_ok(T, desc->n_experts, desc->top_k, desc->n_slots);
    if (!self_route && launch_route(ra, s) != hipSuccess) return FT_ERR_HIP;
    if (enqueue_experts(desc, banks, x, T, out_partial, route, wv, s, prof, self_route ? &ra : nullptr) !=
        hipSuccess)
        return FT_ERR_HIP;
    if (!prof.mark(FT_PROF_STAGES)) return FT_ERR_HIP;
    return FT_OK;
}

}  // namespace

namespace {

// The grouped expert FFN and the combine over the groups the workspace holds.
hipError_t enqueue_experts(const ft_moe_desc_t *desc, const ft_banks_t *banks, const void *x, int32_t T,
                           float *out_partial, const ft_route_t *route, const WsView &wv, hipStream_t s,
                           const Prof &prof, const RouteArgs *self_route) {
    ExpertArgs ea{};
    if (self_route) {
        ea.logits = self_route->logits;
        ea.slot_table = self_route->slot_table;
        ea.E = self_route->E;
        ea.gating = self_route->gating;
        ea.shared_slot = self_route->shared_slot;
        ea.nbits = self_route->nbits;
    }
    ea.w13 = banks->w13;
    ea.w2 = banks->w2;
    ea.s13 = banks->s13;
    ea.s2 = banks->s2;
    ea.x = x;
    ea.out = out_partial;
    ea.T = T;
    ea.H = desc->hidden;
    ea.I = desc->inter;
    ea.k = desc->top_k;
    ea.w_dtype = desc->w_dtype;
    ea.n_slots = desc->n_slots;
    ea.shared = desc->shared_slot >= 0 ? 1 : 0;
    ea.act_quant = desc->act_quant;
    const long routed_slots = desc->n_slots - ea.shared;
    long mg = desc->n_experts;
    if (routed_slots < mg) mg = routed_slots;
    if (static_cast<long>(T) * desc->top_k < mg) mg = static_cast<long>(T) * desc->top_k;
    ea.max_groups = static_cast<int>(mg) + ea.shared;
    ea.ro = route_out(route);
    ea.wv = wv;
    return launch_experts(ea, s, prof);
}

}  // namespace

extern "C" {

ft_status_t ft_moe_forward(const ft_moe_desc_t *desc, const ft_banks_t *banks, const float *logits,
                           const int32_t *slot_table, const void *x, int32_t T,
                           float *out_partial, const ft_route_t *route, void *ws,
                           size_t ws_bytes, void *stream) {
    return forward_impl(desc, banks, logits, slot_table, x, T, out_partial, route, ws, ws_bytes,
                        stream, nullptr);
}

// ---- the allocation-free variant of ft_moe_forward
//
// Its workspace is a file-scope device array instead of a caller buffer.  In host code the
// array's name is only a host-side stand-in, so its device address is looked up once per device
// (with that device current) and only that address is ever handed to kernels.

}  // extern "C"

namespace {

static __device__ __align__(256) uint8_t scratch[FT_NOALLOC_SCRATCH_BYTES];

constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_addr[kScratchDevices] = {};

// Device address of `scratch` on the current device (looked up on its first use there).
ft_status_t scratch_address(void **addr) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices) return FT_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_addr[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return FT_ERR_HIP;
        g_scratch_addr[dev] = p;
    }
    *addr = g_scratch_addr[dev];
    return FT_OK;
}

}  // namespace

namespace {
void hybrid_cpu_task(void *p);
}  // namespace

extern "C" {

ft_status_t ft_moe_forward_noalloc(const ft_moe_desc_t *desc, const ft_banks_t *banks,
                                   const float *logits, const int32_t *slot_table, const void *x,
                                   int32_t T, float *out_partial, const ft_route_t *route,
                                   void *stream) {
    void *ws = nullptr;
    if (ft_status_t s = scratch_address(&ws); s != FT_OK) return s;
    // the workspace check inside rejects any call whose workspace exceeds the array
    return forward_impl(desc, banks, logits, slot_table, x, T, out_partial, route, ws,
                        FT_NOALLOC_SCRATCH_BYTES, stream, nullptr);
}

ft_status_t ft_moe_forward_profiled(const ft_moe_desc_t *desc, const ft_banks_t *banks,
                                    const float *logits, const int32_t *slot_table, const void *x,
                                    int32_t T, float *out_partial, const ft_route_t *route,
                                    void *ws, size_t ws_bytes, void *stream,
                                    const ft_prof_events_t *events) {
    return forward_impl(desc, banks, logits, slot_table, x, T, out_partial, route, ws, ws_bytes,
                        stream, events);
}

ft_status_t ft_cache_plan(const ft_moe_desc_t *desc, const ft_route_t *route, int32_t T,
                          int32_t *slot_table, const ft_cache_state_t *state,
                          const ft_cache_policy_t *policy, const ft_fill_plan_t *plan,
                          void *stream) {
    using namespace ftmoe;
    if (!desc || !route || !slot_table || !state || !policy || !plan) return FT_ERR_NULL;
    if (!desc_ok(desc)) return FT_ERR_SHAPE;
    if (T < 0) return FT_ERR_SHAPE;
    if (!state->slot_expert || !state->slot_stamp) return FT_ERR_NULL;
    if (!plan->fill_expert || !plan->fill_slot || !plan->evict_expert || !plan->cpu_expert ||
        !plan->counts)
        return FT_ERR_NULL;
    if (!route->hit_off || !route->miss_off || !route->miss_pairs || !route->topk_slot ||
        !route->counts)
        return FT_ERR_NULL;
    if (desc->n_slots > kPlanMaxSlots || policy->max_fill < 1 || policy->max_fill > kPlanMaxFill)
        return FT_ERR_SHAPE;
    if (!(policy->b_pcie > 0.0) || !(policy->b_host > 0.0) || policy->b_pcie > 1e300 ||
        policy->b_host > 1e300)
        return FT_ERR_SHAPE;
    if (T == 0) return FT_OK;
    PlanArgs a{};
    a.E = desc->n_experts;
    a.k = desc->top_k;
    a.n_slots = desc->n_slots;
    a.shared_slot = desc->shared_slot;
    a.K = policy->max_fill;
    a.b_pcie = policy->b_pcie;
    a.b_host = policy->b_host;
    a.step = policy->step;
    a.hit_off = route->hit_off;
    a.miss_off = route->miss_off;
    a.miss_pairs = route->miss_pairs;
    a.route_counts = route->counts;
    a.topk_slot = route->topk_slot;
    a.slot_table = slot_table;
    a.slot_expert = state->slot_expert;
    a.slot_stamp = state->slot_stamp;
    a.clock = state->clock;
    a.fill_expert = plan->fill_expert;
    a.fill_slot = plan->fill_slot;
    a.evict_expert = plan->evict_expert;
    a.cpu_expert = plan->cpu_expert;
    a.counts = plan->counts;
    return launch_cache_plan(a, static_cast<hipStream_t>(stream)) == hipSuccess ? FT_OK : FT_ERR_HIP;
}

ft_cpu_pool_t *ft_cpu_pool_create(int32_t n_threads, int32_t pin) {
    if (n_threads > 4096) return nullptr;
    return reinterpret_cast<ft_cpu_pool_t *>(CpuPool::create(n_threads, pin != 0, hybrid_cpu_task));
}

void ft_cpu_pool_destroy(ft_cpu_pool_t *pool) { delete reinterpret_cast<CpuPool *>(pool); }

}  // extern "C"

namespace {

ft_status_t check_cpu_experts(const ft_moe_desc_t *desc, const ft_banks_t *host_pool, int32_t T, int32_t n_list) {
    using namespace ftmoe;
    if (!desc || !host_pool) return FT_ERR_NULL;
    if (!desc_ok(desc)) return FT_ERR_SHAPE;
    if (ft_status_t st = dtype_status(desc); st != FT_OK) return st;
    if (desc->act_quant != FT_ACT_EXACT) return FT_ERR_DTYPE;   // the CPU branch evaluates exactly
    if (T < 0 || n_list < 0 || n_list > desc->n_experts) return FT_ERR_SHAPE;
    if (n_list > 0 && (!host_pool->w13 || !host_pool->w2)) return FT_ERR_NULL;
    if (n_list > 0 && has_scales(desc->w_dtype) && (!host_pool->s13 || !host_pool->s2)) return FT_ERR_NULL;
    if (!__builtin_cpu_supports("avx2") || !__builtin_cpu_supports("fma")) return FT_ERR_DTYPE;
    return FT_OK;
}

void run_cpu_experts(const ft_moe_desc_t *desc, const ft_banks_t *host_pool, const void *x, int32_t T,
                     const int32_t *topk_ids, const float *topk_w, const int32_t *experts, int32_t n_list,
                     float *out, ft_cpu_pool_t *pool) {
    using namespace ftmoe;
    CpuExpertArgs a{};
    a.E = desc->n_experts;
    a.H = desc->hidden;
    a.I = desc->inter;
    a.k = desc->top_k;
    a.T = T;
    a.w_dtype = desc->w_dtype;
    a.x_dtype = desc->x_dtype;
    a.n_list = n_list;
    a.pool = reinterpret_cast<CpuPool *>(pool);
    a.w13 = host_pool->w13;
    a.w2 = host_pool->w2;
    a.s13 = host_pool->s13;
    a.s2 = host_pool->s2;
    a.x = x;
    a.topk_ids = topk_ids;
    a.topk_w = topk_w;
    a.list = experts;
    a.out = out;
    cpu_experts(a);
}

}  // namespace

extern "C" {

ft_status_t ft_cpu_experts(const ft_moe_desc_t *desc, const ft_banks_t *host_pool, const void *x,
                           int32_t T, const int32_t *topk_ids, const float *topk_w,
                           const int32_t *experts, int32_t n_list, float *out, ft_cpu_pool_t *pool) {
    if (ft_status_t st = check_cpu_experts(desc, host_pool, T, n_list); st != FT_OK) return st;
    if (T == 0) return FT_OK;
    if (!x || !topk_ids || !topk_w || !out || (n_list > 0 && !experts)) return FT_ERR_NULL;
    std::vector<char> seen(desc->n_experts, 0);
    for (int i = 0; i < n_list; ++i) {
        const int e = experts[i];
        if (e < 0 || e >= desc->n_experts || seen[e]) return FT_ERR_SHAPE;
        seen[e] = 1;
    }
    run_cpu_experts(desc, host_pool, x, T, topk_ids, topk_w, experts, n_list, out, pool);
    return FT_OK;
}

ft_status_t ft_cache_fill(const ft_moe_desc_t *desc, const ft_banks_t *host_pool,
                          const ft_banks_t *dev_banks, const ft_fill_plan_t *plan, int32_t max_fill,
                          void *stream) {
    using namespace ftmoe;
    if (!desc || !host_pool || !dev_banks || !plan) return FT_ERR_NULL;
    if (!desc_ok(desc)) return FT_ERR_SHAPE;
    if (ft_status_t st = dtype_status(desc); st != FT_OK) return st;
    if (max_fill < 1 || max_fill > kPlanMaxFill) return FT_ERR_SHAPE;
    if (!plan->counts || !plan->fill_expert || !plan->fill_slot) return FT_ERR_NULL;
    const bool sc = has_scales(desc->w_dtype);
    const void *hp[4] = {host_pool->w13, host_pool->w2, sc ? host_pool->s13 : nullptr,
                         sc ? host_pool->s2 : nullptr};
    void *dp[4] = {const_cast<void *>(dev_banks->w13), const_cast<void *>(dev_banks->w2),
                   sc ? const_cast<void *>(dev_banks->s13) : nullptr,
                   sc ? const_cast<void *>(dev_banks->s2) : nullptr};
    const ExpertBytes eb = expert_bytes(desc->w_dtype, desc->hidden, desc->inter);
    const size_t rows[4] = {eb.w13, eb.w2, eb.s13, eb.s2};
    FillArgs a{};
    a.E = desc->n_experts;
    a.n_slots = desc->n_slots;
    a.plan_counts = plan->counts;
    a.fill_expert = plan->fill_expert;
    a.fill_slot = plan->fill_slot;
    for (int b = 0; b < 4; ++b) {
        a.row_bytes[b] = rows[b];
        if (!rows[b]) continue;
        if (!hp[b] || !dp[b]) return FT_ERR_NULL;
        if (reinterpret_cast<uintptr_t>(hp[b]) % 16 || reinterpret_cast<uintptr_t>(dp[b]) % 16)
            return FT_ERR_SHAPE;
        // the pool must be pinned host memory the GPU can read (pageable memory is rejected)
        void *mapped = nullptr;
        if (hipHostGetDevicePointer(&mapped, const_cast<void *>(hp[b]), 0) != hipSuccess || !mapped)
            return FT_ERR_SHAPE;
        a.host[b] = static_cast<const uint8_t *>(mapped);
        a.dev[b] = static_cast<uint8_t *>(dp[b]);
    }
    if (desc->n_slots == 0) return FT_OK;
    return launch_cache_fill(a, max_fill, static_cast<hipStream_t>(stream)) == hipSuccess ? FT_OK : FT_ERR_HIP;
}

}  // extern "C"

namespace {

// What the CPU branch of one hybrid step needs when its host function runs; written by the call
// into the caller's ft_hybrid_task_t, read at every execution of the step (also graph replays).
struct HybridTask {
    ft_moe_desc_t desc;
    ft_banks_t host_pool;
    ft_hybrid_host_t host;
    ft_cpu_pool_t *pool;
    int32_t T;
};
static_assert(sizeof(HybridTask) <= sizeof(ft_hybrid_task_t), "ft_hybrid_task_t too small");

// The step's CPU branch (on the pool's driver thread, or inline without a pool; makes no HIP
// call).
void hybrid_cpu_task(void *p) {
    const HybridTask *t = static_cast<const HybridTask *>(p);
    const int n_cpu = t->host.plan_counts[1];
    if (n_cpu > 0)
        run_cpu_experts(&t->desc, &t->host_pool, t->host.x, t->T, t->host.topk_ids, t->host.topk_w,
                        t->host.cpu_expert, n_cpu, t->host.cpu_out, t->pool);
    else
        std::memset(t->host.cpu_out, 0, sizeof(float) * static_cast<size_t>(t->T) * t->desc.hidden);
}

}  // namespace

extern "C" {

ft_status_t ft_moe_step_hybrid(const ft_moe_desc_t *desc, const ft_banks_t *dev_banks,
                               const ft_banks_t *host_pool, const float *logits, int32_t *slot_table,
                               const ft_cache_state_t *state, const ft_cache_policy_t *policy,
                               const void *x, int32_t T, float *out,
                               const ft_route_t *route, const ft_fill_plan_t *plan,
                               const ft_hybrid_host_t *host, void *ws, size_t ws_bytes,
                               ft_cpu_pool_t *pool, void *stream) {
    using namespace ftmoe;
    if (!desc || !dev_banks || !host_pool || !state || !policy || !route || !plan || !host)
        return FT_ERR_NULL;
    if (T == 0) return desc_ok(desc) ? FT_OK : FT_ERR_SHAPE;
    if (!out || !x || !host->plan_counts || !host->cpu_expert || !host->topk_ids || !host->topk_w ||
        !host->x || !host->cpu_out || !host->task)
        return FT_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(host->x) | reinterpret_cast<uintptr_t>(host->cpu_out)) % 16)
        return FT_ERR_SHAPE;
    if (ft_status_t st = check_forward(desc, dev_banks, logits, slot_table, x, T, out, route, ws, ws_bytes);
        st != FT_OK)
        return st;
    if (ft_status_t st = check_cpu_experts(desc, host_pool, T, desc->n_experts); st != FT_OK) return st;
    // device-visible addresses of the pinned host staging (pageable memory is rejected)
    void *dh[6] = {};
    const void *hh[6] = {host->plan_counts, host->cpu_expert, host->topk_ids, host->topk_w, host->x,
                         host->cpu_out};
    for (int i = 0; i < 6; ++i)
        if (hipHostGetDevicePointer(&dh[i], const_cast<void *>(hh[i]), 0) != hipSuccess || !dh[i])
            return FT_ERR_SHAPE;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    // 1. the step's only routing, then the cache plan, which rewrites the routed slot ids of the
    //    experts it fills
    if (ft_status_t st = ft_route_only(desc, logits, slot_table, T, route, ws, ws_bytes, stream); st != FT_OK)
        return st;
    if (ft_status_t st = ft_cache_plan(desc, route, T, slot_table, state, policy, plan, stream); st != FT_OK)
        return st;
    // 2. the CPU branch: one kernel writes what it needs into the pinned host staging at full
    //    fixed capacity, and a host function submits the experts the plan left to the CPU to the
    //    pool, which evaluates them into host->cpu_out
    HybridTask *task = reinterpret_cast<HybridTask *>(host->task);
    task->desc = *desc;
    task->host_pool = *host_pool;
    task->host = *host;
    task->pool = pool;
    task->T = T;
    StageArgs sa{};
    sa.counts = plan->counts;
    sa.cpu_expert = plan->cpu_expert;
    sa.topk_ids = route->topk_ids;
    sa.topk_w = route->topk_w;
    sa.x = x;
    sa.h_counts = static_cast<int32_t *>(dh[0]);
    sa.h_cpu = static_cast<int32_t *>(dh[1]);
    sa.h_ids = static_cast<int32_t *>(dh[2]);
    sa.h_w = static_cast<float *>(dh[3]);
    sa.h_x = dh[4];
    sa.E = desc->n_experts;
    sa.pk = static_cast<size_t>(T) * desc->top_k;
    sa.x16 = static_cast<size_t>(T) * desc->hidden * (desc->x_dtype == FT_DT_F32 ? 4 : 2) / 16;
    if (launch_stage_host(sa, s) != hipSuccess) return FT_ERR_HIP;
    // with a pool the hand-off is the pool's mailbox in pinned memory (device kernels and a
    // polling listener: no host function on the stream, so the fills and the GPU evaluation
    // below overlap the CPU branch); without one a host function evaluates the branch in line
    CpuPool *cp = reinterpret_cast<CpuPool *>(pool);
    if (cp && !cp->mbox_dev) cp = nullptr;   // a pool without a mailbox: the host-function hand-off
    if (cp) {
        if (launch_mailbox_post(cp->mbox_dev, reinterpret_cast<uint64_t>(task), s) != hipSuccess)
            return FT_ERR_HIP;
    } else if (hipLaunchHostFunc(s, hybrid_cpu_task, task) != hipSuccess) {
        return FT_ERR_HIP;
    }
    // 3. meanwhile the GPU fills the planned slots and evaluates G = H u F from the plan's slot
    //    ids (no second routing)
    if (ft_status_t st = ft_cache_fill(desc, host_pool, dev_banks, plan, policy->max_fill, stream); st != FT_OK)
        return st;
    const WsView wv = carve(desc, T, ws);
    RegroupArgs rg{};
    rg.E = desc->n_experts;
    rg.T = T;
    rg.k = desc->top_k;
    rg.shared_slot = desc->shared_slot;
    rg.hit_off = route->hit_off;
    rg.miss_off = route->miss_off;
    rg.hit_pairs = route->hit_pairs;
    rg.miss_pairs = route->miss_pairs;
    rg.topk_slot = route->topk_slot;
    rg.topk_w = route->topk_w;
    rg.wv = wv;
    if (launch_regroup(rg, s) != hipSuccess) return FT_ERR_HIP;
    if (enqueue_experts(desc, dev_banks, x, T, out, route, wv, s, Prof(nullptr, s)) != hipSuccess) return FT_ERR_HIP;
    // 4. exact merge once the CPU branch is done: out += CPU partial, read from pinned host
    //    memory over PCIe
    if (cp && launch_mailbox_wait(cp->mbox_dev, s) != hipSuccess) return FT_ERR_HIP;
    return launch_add_partial(out, static_cast<const float *>(dh[5]), static_cast<size_t>(T) * desc->hidden, s) ==
                   hipSuccess
               ? FT_OK
               : FT_ERR_HIP;
}

ft_status_t ft_miss_list_to_host(const ft_moe_desc_t *desc, const ft_route_t *route, int32_t T,
                                 const ft_host_miss_t *host, void *stream) {
    if (!desc || !route || !host) return FT_ERR_NULL;
    if (!desc_ok(desc)) return FT_ERR_SHAPE;
    if (T < 0) return FT_ERR_SHAPE;
    if (!host->counts || !host->miss_pairs || !host->miss_off || !host->topk_ids || !host->topk_w)
        return FT_ERR_NULL;
    if (!route->counts || !route->miss_pairs || !route->miss_off || !route->topk_ids ||
        !route->topk_w)
        return FT_ERR_NULL;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    const size_t pk = static_cast<size_t>(T) * desc->top_k;
    const hipMemcpyKind d2h = hipMemcpyDeviceToHost;
    if (hipMemcpyAsync(host->counts, route->counts, 4 * sizeof(int32_t), d2h, s) != hipSuccess)
        return FT_ERR_HIP;
    if (hipMemcpyAsync(host->miss_off, route->miss_off, (desc->n_experts + 1) * sizeof(int32_t), d2h,
                       s) != hipSuccess)
        return FT_ERR_HIP;
    if (pk) {
        if (hipMemcpyAsync(host->miss_pairs, route->miss_pairs, pk * sizeof(int32_t), d2h, s) != hipSuccess ||
            hipMemcpyAsync(host->topk_ids, route->topk_ids, pk * sizeof(int32_t), d2h, s) != hipSuccess ||
            hipMemcpyAsync(host->topk_w, route->topk_w, pk * sizeof(float), d2h, s) != hipSuccess)
            return FT_ERR_HIP;
    }
    return FT_OK;
}

const char *ft_status_string(ft_status_t status) {
    switch (status) {
        case FT_OK: return "FT_OK";
        case FT_ERR_NULL: return "FT_ERR_NULL: a required pointer is NULL";
        case FT_ERR_SHAPE: return "FT_ERR_SHAPE: sizes out of the supported range";
        case FT_ERR_DTYPE: return "FT_ERR_DTYPE: unsupported dtype or gating";
        case FT_ERR_CAPACITY: return "FT_ERR_CAPACITY: workspace too small";
        case FT_ERR_HIP: return "FT_ERR_HIP: a HIP runtime call failed";
    }
    return "unknown status";
}

}  // extern "C"
