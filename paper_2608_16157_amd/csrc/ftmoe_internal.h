// Internal host/device interface of libftmoe: argument bundles, workspace layout, launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <atomic>
#include <condition_variable>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

#include "ftmoe.h"

namespace ftmoe {

constexpr int kMaxExperts = 1024;
constexpr int kMaxTopK = 64;
constexpr int kTokPerBlk = 16;          // tokens per workgroup in the multi-block router
constexpr int kBlkPerPart = 16;         // router blocks per part of its scan (the part table)
constexpr int kFusedMaxPairs = 2048;    // T*k handled by the single-workgroup router
constexpr int kFusedMaxLds = 64 * 1024;
#ifndef FT_GEMM_BM
#define FT_GEMM_BM 128
#endif
#ifndef FT_GEMM_BN
#define FT_GEMM_BN 256
#endif
constexpr int kGemmBM = FT_GEMM_BM;     // token rows per MFMA GEMM tile (prefill path)
constexpr int kGemmBN = FT_GEMM_BN;     // weight rows per MFMA GEMM tile
#ifndef FT_GEMM_MIN_TOKENS
#define FT_GEMM_MIN_TOKENS 256
#endif
constexpr int kGemmMinTokens = FT_GEMM_MIN_TOKENS;   // token count from which the MFMA GEMM path is used

struct HostMailbox;   // a worker pool's device <-> host mailbox (defined with CpuPool)

// Routing outputs (the caller's ft_route_t, flattened).
struct RouteOut {
    int32_t *topk_ids;
    float *topk_w;
    int32_t *topk_slot;
    int32_t *hit_pairs;
    int32_t *miss_pairs;
    int32_t *hit_off;
    int32_t *miss_off;
    int32_t *counts;
};

// Views into the caller's workspace.
//  rows: the hit list positions 0..n_hit-1 followed by T rows of the shared expert; row r
//  evaluates token row_tok[r] with gate row_gate[r].  Groups: one per hit expert (ascending
//  expert id) and then the shared expert; group g covers rows [grp_beg[g], +grp_len[g]) and
//  reads the weights of bank row grp_slot[g].
struct WsView {
    int32_t *eff_slot;   // [E]
    int32_t *blk_hist;   // [nblk][E] per-block expert counts, then [ceil(nblk / kBlkPerPart)][E] part sums
    int32_t *grp_meta;   // [8]: G (groups incl. shared), U (hit groups), n_hit, T, M-tiles
    int32_t *grp_slot;   // [E+1]
    int32_t *grp_beg;    // [E+1]
    int32_t *grp_len;    // [E+1]
    int32_t *grp_mt_off; // [E+2] exclusive prefix of ceil(len / kGemmBM) over the groups
    int32_t *mt_group;   // [max M tiles] group of each GEMM M tile
    int32_t *row_tok;    // [T*k + T]
    float *row_gate;     // [T*k + T]
    int32_t *row_pair;   // [T*k + T] pair index p = t*k + j of the row (T*k + t for the shared rows)
    void *h;             // [T*k + T][I] SwiGLU activations (bf16, or f32 for f32 weights)
    float *ypart;        // streaming path: [T*k + T][H] gate-weighted expert outputs by pair
                         // index, summed per token in a fixed order by the combine (else null)
    // fp8 activations (FT_ACT_FP8_1x128_POW2), else null.  Matrix-core path: x and h as e4m3fn
    // codes with one e8m0 exponent byte (e + 127) per token (row) and 128-channel block.
    // Streaming path: x quantised and widened back to bf16 (h is quantised in place).
    uint8_t *xq;         // [T][H]
    uint8_t *xs;         // [T][H/128]
    uint8_t *hq;         // [T*k + T][I]
    uint8_t *hs;         // [T*k + T][I/128]
    uint16_t *xd;        // [T][H] bf16
};

struct RouteArgs {
    const float *logits;
    const int32_t *slot_table;
    int T, E, k, gating, n_slots, shared_slot, nbits, scan_parts;
    RouteOut ro;
    WsView wv;
};

struct ExpertArgs {
    const void *w13;
    const void *w2;
    const void *s13;   // float32 block scales (fp8) or uint8 e8m0 scales (MXFP4)
    const void *s2;
    const void *x;
    float *out;
    int T, H, I, k, w_dtype, n_slots, shared;
    int act_quant;    // FT_ACT_*
    int max_groups;   // upper bound on groups, known on the host
    // routing of a one- or two-token call done by the gate/up kernel itself (logits != nullptr;
    // otherwise the router ran before and the workspace holds its groups)
    const float *logits;
    const int32_t *slot_table;
    int E, gating, shared_slot, nbits;
    RouteOut ro;
    WsView wv;
};

struct WsLayout {
    size_t eff_slot, blk_hist, grp_meta, grp_slot, grp_beg, grp_len, grp_mt_off, mt_group, row_tok,
        row_gate, row_pair, h, ypart, ypart_bytes, xq, xs, hq, hs, xd, total;
};

// Whether a call of T tokens runs the matrix-core GEMM path (many tokens, shapes that tile);
// the launcher additionally needs at least one evaluation group.
inline bool gemm_shape(int T, int H, int I, int w_dtype) {
    if (w_dtype == FT_DT_F32) return false;
    if (w_dtype == FT_DT_MXFP4 && kGemmBN != 256) return false;   // its scale DMA assumes 256-row tiles
    return T >= kGemmMinTokens && H % kGemmBN == 0 && I % (kGemmBN / 2) == 0 && H <= 8192 && I <= 8192;
}

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Upper bound of the GEMM M tiles any routing of T tokens can produce: every row in full tiles
// plus one ragged tile per group (E routed groups and the shared expert).
inline size_t gemm_max_mtiles(int T, int k, int E) {
    const size_t rows = static_cast<size_t>(T) * k + T;
    return (rows + kGemmBM - 1) / kGemmBM + E + 1;
}

inline WsLayout ws_layout(int E, int H, int I, int k, int w_dtype, int combine, int act_quant, int T) {
    WsLayout L{};
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o = align_up(o + bytes, 256);
        return at;
    };
    const size_t nblk = (static_cast<size_t>(T) + kTokPerBlk - 1) / kTokPerBlk;
    const size_t rows = static_cast<size_t>(T) * k + T;
    L.eff_slot = take(4u * E);
    const size_t nparts = (nblk + kBlkPerPart - 1) / kBlkPerPart;
    L.blk_hist = take(4u * (nblk + nparts) * E);
    L.grp_meta = take(32);
    L.grp_slot = take(4u * (E + 1));
    L.grp_beg = take(4u * (E + 1));
    L.grp_len = take(4u * (E + 1));
    L.grp_mt_off = take(4u * (E + 2));
    L.mt_group = take(4u * gemm_max_mtiles(T, k, E));
    L.row_tok = take(4u * rows);
    L.row_gate = take(4u * rows);
    L.row_pair = take(4u * rows);
    const bool aq = act_quant == FT_ACT_FP8_1x128_POW2, gemm = gemm_shape(T, H, I, w_dtype);
    // the fp8-activation matrix-core path keeps h only as codes (hq, hs)
    L.h = take(aq && gemm ? 0 : rows * I * (w_dtype == FT_DT_F32 ? 4u : 2u));
    L.ypart_bytes = (gemm || combine != FT_COMBINE_ORDERED) ? 0 : rows * H * 4u;
    L.ypart = take(L.ypart_bytes);
    L.xq = take(aq && gemm ? static_cast<size_t>(T) * H : 0);
    L.xs = take(aq && gemm ? static_cast<size_t>(T) * (H / 128) : 0);
    L.hq = take(aq && gemm ? rows * I : 0);
    L.hs = take(aq && gemm ? rows * (I / 128) : 0);
    L.xd = take(aq && !gemm ? static_cast<size_t>(T) * H * 2 : 0);

    L.total = o;
    return L;
}


// Optional stage events of ft_moe_forward_profiled (recorded only when given).
struct Prof {
    const ft_prof_events_t *ev;
    hipStream_t s;
    Prof(const ft_prof_events_t *e, hipStream_t st) : ev(e), s(st) {}
    bool mark(int i) const {
        if (!ev || !ev->ev[i]) return true;
        return hipEventRecord(static_cast<hipEvent_t>(ev->ev[i]), s) == hipSuccess;
    }
};

// Device-side cache control of one layer step (cache.hip).
constexpr int kPlanMaxFill = 64;      // most LRU candidates (K) per step
constexpr int kPlanMaxSlots = 4096;   // most cache slots the planner handles

struct PlanArgs {
    int E, k, n_slots, shared_slot, K;
    double b_pcie, b_host;
    uint32_t step;
    uint32_t *clock;   // device step counter, or null (then `step` is the stamp)
    const int32_t *hit_off, *miss_off, *miss_pairs, *route_counts;
    int32_t *topk_slot;
    int32_t *slot_table, *slot_expert;
    uint32_t *slot_stamp;
    int32_t *fill_expert, *fill_slot, *evict_expert, *cpu_expert, *counts;
};

// Cache fills and the exact merge (fill.hip).
constexpr size_t kFillChunk = 64 * 1024;   // bytes of one bank row a fill block copies
struct FillArgs {
    int E, n_slots;
    const int32_t *plan_counts, *fill_expert, *fill_slot;
    const uint8_t *host[4];   // pinned host pool (device-visible addresses): w13, w2, s13, s2
    uint8_t *dev[4];          // device banks
    size_t row_bytes[4];      // bytes of one expert's row in each bank (0 = bank absent)
};
hipError_t launch_cache_fill(const FillArgs &a, int max_fill, hipStream_t s);
hipError_t launch_add_partial(float *out, const float *other, size_t n, hipStream_t s);
// Host staging of a hybrid step (device-visible addresses of pinned host buffers).
struct StageArgs {
    const int32_t *counts, *cpu_expert, *topk_ids;
    const float *topk_w;
    const void *x;
    int32_t *h_counts, *h_cpu, *h_ids;
    float *h_w;
    void *h_x;
    int E;
    size_t pk, x16;   // routed pairs; 16-byte chunks of x (x rows are 16-byte multiples)
};
hipError_t launch_stage_host(const StageArgs &a, hipStream_t s);
// Post a task to a pool's mailbox (device side), and wait until the pool reports it done.
hipError_t launch_mailbox_post(HostMailbox *mbox_dev, uint64_t task, hipStream_t s);
hipError_t launch_mailbox_wait(HostMailbox *mbox_dev, hipStream_t s);

// Bytes of one expert in each bank (w13, w2, s13, s2) for a weight dtype; H, I multiples of 128.
struct ExpertBytes {
    size_t w13, w2, s13, s2;
};
inline ExpertBytes expert_bytes(int w_dtype, size_t H, size_t I) {
    switch (w_dtype) {
        case FT_DT_F32: return {2 * I * H * 4, H * I * 4, 0, 0};
        case FT_DT_BF16: return {2 * I * H * 2, H * I * 2, 0, 0};
        case FT_DT_FP8E4M3FN_B128: return {2 * I * H, H * I, (2 * I / 128) * (H / 128) * 4, (H / 128) * (I / 128) * 4};
        default: return {I * H, H * I / 2, 2 * I * (H / 32), H * (I / 32)};   // MXFP4
    }
}
inline bool has_scales(int w_dtype) { return w_dtype == FT_DT_FP8E4M3FN_B128 || w_dtype == FT_DT_MXFP4; }

// Every host-checkable condition of ft_moe_forward (FT_OK when the call would be enqueued).
ft_status_t check_forward(const ft_moe_desc_t *desc, const ft_banks_t *banks, const float *logits,
                          const int32_t *slot_table, const void *x, int32_t T, const float *out_partial,
                          const ft_route_t *route, const void *ws, size_t ws_bytes);

// Mailbox of a worker pool in pinned host memory, written by the device and the pool's listener
// thread: the device posts a step (task pointer, then a new sequence number), the listener runs
// the task and echoes the number into `done`, which a device kernel waits for.
struct alignas(64) HostMailbox {
    uint64_t posted;     // last posted sequence number (device writes)
    uint64_t task;       // host address of the posted step's task (device writes)
    uint64_t done;       // last finished sequence number (listener writes)
    uint64_t timeouts;   // device waits that gave up (device writes)
};

// The CPU branch's persistent worker pool (host_experts.cpp), behind the opaque ft_cpu_pool_t.
struct CpuPool {
    struct Job {
        int n;
        const std::function<void(int, std::vector<float> &)> &fn;
    };
    std::vector<std::thread> workers;
    std::vector<int> cpus;        // CPU each worker is pinned to, -1 if not pinned
    std::mutex mu, run_mu;
    std::condition_variable cv_work, cv_done;
    const Job *current = nullptr;
    uint64_t gen = 0;             // job generation
    std::atomic<int> next{0};     // next work item of the current job
    int busy = 0;                 // workers not yet done with the current job
    bool stop = false;
    // the listener thread polls the mailbox and runs each posted task (through run())
    std::thread listener;
    std::atomic<bool> quit{false};
    HostMailbox *mbox = nullptr;       // pinned host memory
    HostMailbox *mbox_dev = nullptr;   // its device-visible address
    void (*task_fn)(void *) = nullptr; // what a posted task runs
    static CpuPool *create(int n_threads, bool pin, void (*task_fn)(void *));
    ~CpuPool();
    void run(int n_items, const std::function<void(int, std::vector<float> &)> &fn);
    void worker_loop();
    void listen_loop();
};

// CPU branch of a layer step (host_experts.cpp).
struct CpuBank {
    const void *w;       // one expert's matrix, row-major
    const void *s;       // its fp8 block scales (float32) or MXFP4 scales (uint8), or null
};
struct CpuExpertArgs {
    int E, H, I, k, T, w_dtype, x_dtype, n_list;
    CpuPool *pool;                   // workers, or null: the calling thread alone
    const void *w13, *w2;            // host expert pool, [E][2I][H] and [E][H][I]
    const void *s13, *s2;            // fp8 / MXFP4 scales per expert, or null
    const void *x;                   // [T][H]
    const int32_t *topk_ids;         // [T][k]
    const float *topk_w;             // [T][k]
    const int32_t *list;             // experts to evaluate (distinct ids)
    float *out;                      // [T][H], overwritten
};
void cpu_experts(const CpuExpertArgs &a);

// Evaluation groups of a hybrid step from its routing after the cache plan (route.hip).
struct RegroupArgs {
    int E, T, k, shared_slot;
    const int32_t *hit_off, *miss_off, *hit_pairs, *miss_pairs, *topk_slot;
    const float *topk_w;
    WsView wv;
};
hipError_t launch_regroup(const RegroupArgs &a, hipStream_t s);

hipError_t launch_route(const RouteArgs &a, hipStream_t s);
hipError_t launch_cache_plan(const PlanArgs &a, hipStream_t s);
hipError_t launch_experts(const ExpertArgs &a, hipStream_t s, const Prof &prof);
hipError_t launch_gemm(const ExpertArgs &a, hipStream_t s, const Prof &prof);
// fp8 activations (quant.hip): x into codes and exponents (matrix-core path) or into quantised
// bf16 (streaming path); h quantised in place (streaming path)
hipError_t launch_act_quant_x(const ExpertArgs &a, hipStream_t s);
hipError_t launch_act_quant_h(const ExpertArgs &a, hipStream_t s);

}  // namespace ftmoe
