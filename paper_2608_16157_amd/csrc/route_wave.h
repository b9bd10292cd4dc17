// One-wave routing of one or two tokens (Section 3.2: router and cache lookup on the GPU;
// Section 4.1: routed ids rewritten into slot ids), shared by the router kernels (route.hip) and
// by the decode gate/up kernel that routes a one- or two-token call for itself (experts.hip):
// top-k selection, slot-table checks and the single-wave body of the router.
#pragma once

#include "ftmoe_device.h"
#include "ftmoe_internal.h"

namespace ftmoe {

// ---------------------------------------------------------------------------------------
// Top-k of one token's logits by one wave.  Lane l holds experts [l*NPL, l*NPL + NPL), so among
// equal logits the lowest lane, and within a lane the lowest index, is the lowest expert id.
// topk_load fetches a token's keys (callers load several tokens before selecting, so the memory
// latency is paid once per batch); topk_select runs the k rounds: the wave maximum of the lanes'
// best keys (DPP) and the lowest lane holding it (ballot).  On return lane j < k holds
// (expert id, gate) of the j-th selected expert.
template <int NPL>
__device__ __forceinline__ void topk_load(const float *__restrict__ row, int E, uint32_t (&key)[NPL]) {
    const int lane = lane_id();
    float v[NPL];
    // unconditional loads of a clamped index: no branch, so no wait is forced between tokens
#pragma unroll
    for (int i = 0; i < NPL; ++i) v[i] = row[min(lane * NPL + i, E - 1)];
    // out-of-range entries are masked arithmetically (a select would let the compiler sink the
    // load into a branch again)
#pragma unroll
    for (int i = 0; i < NPL; ++i)
        key[i] = order_key(v[i]) & (0u - static_cast<uint32_t>(lane * NPL + i < E));
}

template <int NPL, int NB>
__device__ __forceinline__ void topk_select_n(uint32_t (&key)[NB][NPL], int k, int gating,
                                              int (&my_id)[NB], float (&my_w)[NB]) {
    // NB tokens' rounds interleaved: their reductions are independent, so the latencies of the
    // DPP and readlane chains overlap
    const int lane = lane_id();
    uint32_t mine[NB];
    int mine_e[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        mine[b] = 0u;
        mine_e[b] = -1;
    }
    for (int j = 0; j < k; ++j) {
        uint32_t best[NB], m[NB];
        int bi[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            best[b] = 0u;
            bi[b] = 0;
#pragma unroll
            for (int i = 0; i < NPL; ++i) {
                if (key[b][i] > best[b]) {
                    best[b] = key[b][i];
                    bi[b] = i;
                }
            }
        }
#pragma unroll
        for (int b = 0; b < NB; ++b) m[b] = wave_max_u32(best[b]);
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const uint64_t ball = __ballot(best[b] == m[b]);
            const int w = static_cast<int>(__builtin_ctzll(ball));
            const int wbi = __builtin_amdgcn_readlane(bi[b], w);
#pragma unroll
            for (int i = 0; i < NPL; ++i)
                key[b][i] &= ~(0u - static_cast<uint32_t>((lane == w) & (i == wbi)));
            if (lane == j) {
                mine[b] = m[b];
                mine_e[b] = w * NPL + wbi;
            }
        }
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const float top = key_to_float(readlane_u32(mine[b], 0));
        float z = 0.f;
        if (lane < k) {
            const float l = key_to_float(mine[b]);
            z = gating == FT_GATE_SOFTMAX_TOPK_RENORM ? expf(l - top) : 1.0f / (1.0f + expf(-l));
        }
        const float sum = wave_sum_f32(z);
        my_id[b] = lane < k ? mine_e[b] : -1;
        my_w[b] = lane < k ? z / sum : 0.f;
    }
}

template <int NPL>
__device__ __forceinline__ void topk_select(uint32_t (&key)[NPL], int k, int gating, int &my_id,
                                            float &my_w) {
    uint32_t kk[1][NPL];
#pragma unroll
    for (int i = 0; i < NPL; ++i) kk[0][i] = key[i];
    int id[1];
    float w[1];
    topk_select_n<NPL, 1>(kk, k, gating, id, w);
    my_id = id[0];
    my_w = w[0];
}

template <int NPL>
__device__ __forceinline__ void wave_topk(const float *__restrict__ row, int E, int k, int gating,
                                          int &my_id, float &my_w) {
    uint32_t key[NPL];
    topk_load<NPL>(row, E, key);
    topk_select<NPL>(key, k, gating, my_id, my_w);
}

// Slot-table validation.  An expert's slot is usable iff it lies in [0, n_slots), is not
// the shared expert's slot, and no other expert maps to it; unusable entries are treated as
// misses and reported in the device status bits.  Duplicates are found by counting experts per
// slot in LDS (slot counts, when n_slots <= kSlotCountCap), else by comparing against every
// other expert.
constexpr int kSlotCountCap = 4096;

__device__ __forceinline__ int slot_check(int raw, int e, int E, int n_slots, int shared_slot,
                                          const int32_t *s_cnt, const int32_t *s_raw, int &status) {
    const int s = raw;
    if (s == -1) return -1;
    if (s < -1 || s >= n_slots) {
        status |= FT_DEV_SLOT_RANGE;
        return -1;
    }
    if (shared_slot >= 0 && s == shared_slot) {
        status |= FT_DEV_SLOT_SHARED;
        return -1;
    }
    bool dup;
    if (n_slots <= kSlotCountCap) {
        dup = s_cnt[s] > 1;
    } else {
        dup = false;
        for (int o = 0; o < E; ++o) dup |= (o != e) & (s_raw[o] == s);
    }
    if (dup) {
        status |= FT_DEV_SLOT_DUP;
        return -1;
    }
    return s;
}

// ---------------------------------------------------------------------------------------
// Single-wave routing of one or two tokens (T*k <= 64 pairs).  The fused router's work, laid out
// so that no step waits on another wave: lane l holds the slot-table entries and pair totals of
// experts [l*epl, l*epl + epl) and, once the top-k is done, pair l.  All pairs lie in one 64-pair
// chunk, so a pair's list position is its expert's offset plus its ballot rank among the pairs
// of the same expert (pair order).  The outputs equal route_fused's.  One wave selects tokens
// one batch at a time, so beyond two tokens the 16 waves of route_fused are faster (measured at
// eight tokens: 15 against 9 us per call).
#ifndef FT_ROUTE_WAVE_MAX_TOKENS
#define FT_ROUTE_WAVE_MAX_TOKENS 2
#endif
constexpr int kWaveRouteMaxTokens = FT_ROUTE_WAVE_MAX_TOKENS;   // 0 disables the variant
constexpr int kWaveRouteMaxNpl = 8;
static_assert(kWaveRouteMaxTokens <= 2, "route_wave selects one batch of at most two tokens");

// LDS hand-off between the lanes of the one wave that routes: its own LDS operations complete in
// order, so waiting for them is enough (no workgroup barrier, which would also count the other
// waves of a workgroup that routes with one of its waves).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x0 << 8) | (0x3 << 14));   // lgkmcnt(0)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_wave_barrier();
    asm volatile("" ::: "memory");
}

// LDS bytes of route_wave_body: E experts, ncnt slot counters
constexpr int route_wave_lds_bytes(int E, int ncnt) { return 4 * (5 * E + 2 * kWave + 1 + ncnt); }

// Self-routing decode kernels (experts.hip): LDS of the sink below, and the calls they take:
// one or two tokens, at most 64 pairs, 65 to 256 experts (two or four per lane), and router LDS
// that keeps the kernel's occupancy (a slot table of at most 1024 slots).
constexpr int kWaveRouteSinkBytes = 4 * (1 + 3 * (kWave + 1) + kWave + kWaveRouteMaxTokens);
constexpr int kSelfRouteMaxLds = 16 * 1024;
inline bool self_route_ok(int T, int E, int k, int n_slots) {
    const int ncnt = n_slots <= kSlotCountCap ? n_slots : 0;
    return T >= 1 && T <= kWaveRouteMaxTokens && T * k <= kWave && E > kWave && E <= 4 * kWave &&
           n_slots <= 1024 && route_wave_lds_bytes(E, ncnt) + kWaveRouteSinkBytes <= kSelfRouteMaxLds;
}

// Where a workgroup that routes for itself finds the evaluation groups and the token of each
// evaluation row (LDS): group g (g < *G) is (slot[g], beg[g], len[g]) as in the workspace's group
// table, row r's token is row_tok[r].
struct WaveRouteSink {
    int32_t *G;
    int32_t *slot, *beg, *len;   // kWave + 1 entries
    int32_t *row_tok;            // kWave + kWaveRouteMaxTokens entries
};

// The routing of one or two tokens by one wave (lane l: experts [l*epl, l*epl + epl), then pair l).
// wr: write the routing's outputs (lists, records, counts, group table, rows) to global memory;
// FUSED: also put the evaluation groups and row tokens into `sink`.  Every global output of the
// call is written by one workgroup only, so wr is true in exactly one of them.
template <int NPL, bool FUSED>
__device__ __forceinline__ void route_wave_body(const RouteArgs &a, int32_t *lds, bool wr, const WaveRouteSink &sink) {
    const int E = a.E, k = a.k, T = a.T, P = T * k;
    const int ncnt = a.n_slots <= kSlotCountCap ? a.n_slots : 0;
    int32_t *s_raw = lds;                                     // E  slot-table entries
    int32_t *s_eff = s_raw + E;                               // E  usable slot (-1: miss)
    int32_t *s_tot = s_eff + E;                               // E  pairs per expert
    int32_t *s_hoff = s_tot + E;                              // E  first hit position
    int32_t *s_moff = s_hoff + E;                             // E  first miss position
    int32_t *s_ids = s_moff + E;                              // 64
    float *s_w = reinterpret_cast<float *>(s_ids + kWave);    // 64
    int *s_status = reinterpret_cast<int *>(s_w + kWave);     // 1
    int32_t *s_cnt = s_status + 1;                            // ncnt experts per slot
    const int lane = lane_id();
    const int epl = (E + kWave - 1) / kWave;
    const int e0 = min(E, lane * epl), e1 = min(E, e0 + epl);

    // both tokens' logits and this lane's slot-table entries, in flight together
    uint32_t key[2][NPL];
#pragma unroll
    for (int b = 0; b < 2; ++b)
        topk_load<NPL>(a.logits + static_cast<size_t>(min(b, T - 1)) * E, E, key[b]);
    int raw[NPL];
#pragma unroll
    for (int i = 0; i < NPL; ++i) raw[i] = a.slot_table[min(e0 + i, E - 1)];
    for (int i = lane; i < ncnt; i += kWave) s_cnt[i] = 0;
    for (int e = lane; e < E; e += kWave) s_tot[e] = 0;
    if (lane == 0) *s_status = 0;
    wave_lds_sync();

    // experts per slot, then the top-k of each token (lanes j < k hold token t's j-th choice)
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
        if (e0 + i < e1) {
            s_raw[e0 + i] = raw[i];
            if (raw[i] >= 0 && raw[i] < ncnt) atomicAdd(&s_cnt[raw[i]], 1);
        }
    }
    int id[2] = {-1, -1};
    float w[2] = {0.f, 0.f};
    if (T == 2) {
        topk_select_n<NPL, 2>(key, k, a.gating, id, w);
    } else {
        topk_select<NPL>(key[0], k, a.gating, id[0], w[0]);
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        if (t < T && lane < k) {
            s_ids[t * k + lane] = id[t];
            s_w[t * k + lane] = w[t];
        }
    }
    wave_lds_sync();

    // usable slot of this lane's experts; rank of pair `lane` among the pairs of its expert
    int st = 0, slot[NPL];
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
        const int e = e0 + i;
        slot[i] = e < e1 ? slot_check(raw[i], e, E, a.n_slots, a.shared_slot, s_cnt, s_raw, st) : -1;
        if (e < e1) s_eff[e] = slot[i];
    }
    if (st) atomicOr(s_status, st);
    const bool act = lane < P;
    const int pe = act ? s_ids[lane] : 0;
    const float pw = act ? s_w[lane] : 0.f;
    const uint64_t same = match_lanes(static_cast<uint32_t>(pe), a.nbits, __ballot(act));
    const int prank = __popcll(same & lanemask_lt());
    if (act && prank == __popcll(same) - 1) s_tot[pe] = prank + 1;
    wave_lds_sync();

    // exclusive scans over the experts: list offsets, groups, GEMM tile map, counts
    int tots[NPL];
    uint32_t h = 0, m = 0, g = 0, mx = 0, mtl = 0;
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
        const int e = e0 + i;
        tots[i] = e < e1 ? s_tot[e] : 0;
        const bool hit = slot[i] >= 0;
        h += hit ? tots[i] : 0;
        m += hit ? 0 : tots[i];
        g += (hit && tots[i] > 0) ? 1 : 0;
        mx += (!hit && tots[i] > 0) ? 1 : 0;
        mtl += hit ? (tots[i] + kGemmBM - 1) / kGemmBM : 0;
    }
    const uint32_t hi = wave_incl_scan_u32(h), mi = wave_incl_scan_u32(m);
    const uint32_t gi = wave_incl_scan_u32(g), xi = wave_incl_scan_u32(mx);
    const uint32_t ti = wave_incl_scan_u32(mtl);
    uint32_t hrun = hi - h, mrun = mi - m, grun = gi - g, trun = ti - mtl;
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
        const int e = e0 + i;
        if (e >= e1) continue;
        const int tot = tots[i];
        const bool hit = slot[i] >= 0;
        s_hoff[e] = hrun;
        s_moff[e] = mrun;
        if (wr) {
            a.ro.hit_off[e] = hrun;
            a.ro.miss_off[e] = mrun;
        }
        if (hit && tot > 0) {
            if (wr) {
                a.wv.grp_slot[grun] = slot[i];
                a.wv.grp_beg[grun] = hrun;
                a.wv.grp_len[grun] = tot;
                a.wv.grp_mt_off[grun] = trun;
                const int nmt = (tot + kGemmBM - 1) / kGemmBM;
                for (int u = 0; u < nmt; ++u) a.wv.mt_group[trun + u] = grun;
            }
            if constexpr (FUSED) {
                sink.slot[grun] = slot[i];
                sink.beg[grun] = hrun;
                sink.len[grun] = tot;
            }
        }
        hrun += hit ? tot : 0;
        mrun += hit ? 0 : tot;
        grun += (hit && tot > 0) ? 1 : 0;
        trun += hit ? (tot + kGemmBM - 1) / kGemmBM : 0;
    }
    const uint32_t nh = readlane_u32(hi, kWave - 1), nm = readlane_u32(mi, kWave - 1);
    const uint32_t U = readlane_u32(gi, kWave - 1), mexp = readlane_u32(xi, kWave - 1);
    const uint32_t MT = readlane_u32(ti, kWave - 1);
    if (lane == kWave - 1) {
        const int shared = a.shared_slot;
        const uint32_t G = U + (shared >= 0 ? 1 : 0);
        if constexpr (FUSED) {
            *sink.G = static_cast<int32_t>(G);
            if (shared >= 0) {
                sink.slot[U] = shared;
                sink.beg[U] = nh;
                sink.len[U] = T;
            }
        }
    }
    if (wr && lane == kWave - 1) {
        const int shared = a.shared_slot;
        a.ro.hit_off[E] = nh;
        a.ro.miss_off[E] = nm;
        a.ro.counts[0] = nh;
        a.ro.counts[1] = nm;
        a.ro.counts[2] = mexp;
        a.ro.counts[3] = *s_status;
        const uint32_t smt = shared >= 0 ? (T + kGemmBM - 1) / kGemmBM : 0;
        const uint32_t G = U + (shared >= 0 ? 1 : 0);
        a.wv.grp_meta[0] = G;
        a.wv.grp_meta[1] = U;
        a.wv.grp_meta[2] = nh;
        a.wv.grp_meta[3] = T;
        a.wv.grp_meta[4] = MT + smt;
        if (shared >= 0) {
            a.wv.grp_slot[U] = shared;
            a.wv.grp_beg[U] = nh;
            a.wv.grp_len[U] = T;
            a.wv.grp_mt_off[U] = MT;
            for (uint32_t i = 0; i < smt; ++i) a.wv.mt_group[MT + i] = U;
        }
        a.wv.grp_mt_off[G] = MT + smt;
    }
    wave_lds_sync();

    // pair `lane`: its list entry, its routing record, and the list tails
    if (act) {
        const int sl = s_eff[pe];
        const int pos = (sl >= 0 ? s_hoff[pe] : s_moff[pe]) + prank;
        if (wr) {
            a.ro.topk_ids[lane] = pe;
            a.ro.topk_w[lane] = pw;
            a.ro.topk_slot[lane] = sl;
            if (sl >= 0) {
                a.ro.hit_pairs[pos] = lane;
                a.wv.row_tok[pos] = lane / k;
                a.wv.row_pair[pos] = lane;
                a.wv.row_gate[pos] = pw;
            } else {
                a.ro.miss_pairs[pos] = lane;
            }
            if (lane >= static_cast<int>(nh)) a.ro.hit_pairs[lane] = -1;
            if (lane >= static_cast<int>(nm)) a.ro.miss_pairs[lane] = -1;
        }
        if constexpr (FUSED)
            if (sl >= 0) sink.row_tok[pos] = lane / k;
    }
    if (a.shared_slot >= 0 && lane < T) {
        if (wr) {
            a.wv.row_tok[nh + lane] = lane;
            a.wv.row_pair[nh + lane] = T * k + lane;
            a.wv.row_gate[nh + lane] = 1.0f;
        }
        if constexpr (FUSED) sink.row_tok[nh + lane] = lane;
    }
}

}  // namespace ftmoe
