// Router top-k, hit/miss classification against the slot table, and the expert-sorted stable
// permutation (Section 3.2: router and cache lookup on the GPU; Section 4.1: routed logical ids
// rewritten into slot ids or a CPU flag, kept as fixed-shape buffers with device counts).
//
// Three variants:
//  * route_wave: one wave does everything (one or two tokens, T*k <= 64 pairs).  A layer call of
//    one or two tokens over 65 to 256 experts runs the same body inside its gate/up kernel
//    instead (route_wave.h, experts.hip): every workgroup routes for itself, one writes the outputs.
//  * route_fused: one 1024-thread workgroup does everything in LDS (decode), for the larger
//    decode batches after route_topk has selected every token's experts on many CUs.
//  * route_tokens -> route_partscan -> route_scan -> route_scatter: many tokens (prefill chunks).
// All produce bit-identical outputs: the permutation is a counting sort whose within-expert
// order is the pair index, computed with wave ballots, never with order-dependent atomics.
#include "ftmoe_device.h"
#include "ftmoe_internal.h"
#include "route_wave.h"

// logits (T * E) from which the decode router takes its top-k in a kernel of its own: measured
// at 16 tokens x 256 experts and beyond, the launch the split adds costs less than the selection
// rounds it moves off the fused router's one CU (Qwen3 T = 64: routing 14.9 -> 9.8 us, dsv3
// T = 64: 20.3 -> 10.6 us); at 16 x 128 and below it does not
#ifndef FT_ROUTE_SPLIT_LOGITS
#define FT_ROUTE_SPLIT_LOGITS 4096
#endif

namespace ftmoe {

// Top-k selection, the slot checks and the one-wave router body are in route_wave.h.

__device__ __forceinline__ void slot_count(int raw, int E, int n_slots, int32_t *s_cnt) {
    if (threadIdx.x < E && n_slots <= kSlotCountCap && raw >= 0 && raw < n_slots)
        atomicAdd(&s_cnt[raw], 1);
}

// Validated slot of each expert (-1 if unusable) and the device status bits, by the whole
// block.  `raw` is this thread's slot_table entry (thread e of the block holds expert e;
// blockDim >= E); s_cnt holds min(n_slots, kSlotCountCap) counters.
__device__ void validate_slots(int raw, int E, int n_slots, int shared_slot, int32_t *s_raw,
                               int32_t *s_cnt, int32_t *s_eff, int *s_status) {
    if (threadIdx.x < E) s_raw[threadIdx.x] = raw;
    if (n_slots <= kSlotCountCap)
        for (int i = threadIdx.x; i < n_slots; i += blockDim.x) s_cnt[i] = 0;
    __syncthreads();
    slot_count(raw, E, n_slots, s_cnt);
    __syncthreads();
    int st = 0;
    if (threadIdx.x < E) s_eff[threadIdx.x] = slot_check(raw, threadIdx.x, E, n_slots, shared_slot, s_cnt, s_raw, st);
    if (st) atomicOr(s_status, st);
    __syncthreads();
}

// Scatter one wave's contiguous run of pairs [p0, p1) in pair order.  `run` holds, per expert,
// the next free position in the hit or miss list for this run (LDS, private to the wave).
__device__ void scatter_run(int p0, int p1, int k, int nbits, const int32_t *__restrict__ ids,
                            const float *__restrict__ w, const int32_t *__restrict__ s_eff,
                            int32_t *run, const RouteOut &ro, const WsView &wv) {
    const int lane = lane_id();
    for (int base = p0; base < p1; base += kWave) {
        const int p = base + lane;
        const bool act = p < p1;
        const int e = act ? ids[p] : 0;
        const uint64_t same = match_lanes(static_cast<uint32_t>(e), nbits, __ballot(act));
        const int rank = __popcll(same & lanemask_lt());
        const int cnt = __popcll(same);
        int pos = 0;
        if (act) pos = run[e] + rank;
        __builtin_amdgcn_wave_barrier();
        if (act && rank == cnt - 1) run[e] = pos + 1;
        __builtin_amdgcn_wave_barrier();
        if (act) {
            const int slot = s_eff[e];
            ro.topk_slot[p] = slot;
            if (slot >= 0) {
                ro.hit_pairs[pos] = p;
                wv.row_tok[pos] = p / k;
                wv.row_pair[pos] = p;
                wv.row_gate[pos] = w[p];
            } else {
                ro.miss_pairs[pos] = p;
            }
        }
    }
}

// Exclusive scans of per-expert hit and miss totals, group table and counts.  Called by the
// whole block after `s_tot` (pairs per expert) and `s_eff` are ready.  Writes hit_off/miss_off
// to LDS (s_hoff/s_moff, E+1 entries) and global memory.
__device__ void scan_experts(int E, int T, int k, int shared_slot, const int32_t *s_tot,
                             const int32_t *s_eff, int32_t *s_hoff, int32_t *s_moff,
                             int32_t *s_gidx, const int *s_status, const RouteOut &ro,
                             const WsView &wv) {
    if (threadIdx.x < kWave) {
        // lane l owns experts [l*epl, l*epl + epl)
        const int lane = lane_id();
        const int epl = (E + kWave - 1) / kWave;
        const int e0 = min(E, lane * epl), e1 = min(E, e0 + epl);
        // Evaluation groups are numbered, and their GEMM M tiles laid out, in classes: the shared
        // expert first, then the groups of several M tiles, then the one-tile groups by their
        // live 32-row sub-tiles (4 down to 1), each class in expert order.  The GEMM launches a
        // few hundred tiles at a time and skips the MFMAs of padding sub-tiles, so tiles of
        // similar cost then share a launch (measured at DeepSeek-V3 prefill: layer 4.03 ->
        // 3.90 ms together with the padding skip of the fp8 gate/up GEMM).
        auto cls = [&](int tot) {
            if (tot > kGemmBM) return 0;
            return 1 + min(3, (kGemmBM - tot) / 32);   // tot in (96, 128] -> 1, ..., (0, 32] -> 4
        };
        constexpr int NC = 5;
        uint32_t h = 0, m = 0, mx = 0, gc[NC] = {}, tc[NC] = {};
        for (int e = e0; e < e1; ++e) {
            const int tot = s_tot[e];
            const bool hit = s_eff[e] >= 0;
            h += hit ? tot : 0;
            m += hit ? 0 : tot;
            mx += (!hit && tot > 0) ? 1 : 0;
            if (hit && tot > 0) {
                const int c = cls(tot);
#pragma unroll
                for (int i = 0; i < NC; ++i) {
                    gc[i] += i == c ? 1u : 0u;
                    tc[i] += i == c ? static_cast<uint32_t>((tot + kGemmBM - 1) / kGemmBM) : 0u;
                }
            }
        }
        const uint32_t hi = wave_incl_scan_u32(h), mi = wave_incl_scan_u32(m), xi = wave_incl_scan_u32(mx);
        const uint32_t smt = shared_slot >= 0 ? (T + kGemmBM - 1) / kGemmBM : 0;
        const uint32_t sh = shared_slot >= 0 ? 1u : 0u;   // the shared expert is group 0
        uint32_t grun[NC], trun[NC], U = 0, MT = 0;
#pragma unroll
        for (int i = 0; i < NC; ++i) {
            const uint32_t gi = wave_incl_scan_u32(gc[i]), ti = wave_incl_scan_u32(tc[i]);
            grun[i] = sh + U + gi - gc[i];
            trun[i] = sh * smt + MT + ti - tc[i];
            U += readlane_u32(gi, kWave - 1);
            MT += readlane_u32(ti, kWave - 1);
        }
        uint32_t hrun = hi - h, mrun = mi - m;
        for (int e = e0; e < e1; ++e) {
            const int tot = s_tot[e];
            const bool hit = s_eff[e] >= 0;
            s_hoff[e] = hrun;
            s_moff[e] = mrun;
            s_gidx[e] = -1;
            if (hit && tot > 0) {
                const int c = cls(tot);
                uint32_t gg = 0, tt = 0;
#pragma unroll
                for (int i = 0; i < NC; ++i)
                    if (i == c) {
                        gg = grun[i]++;
                        tt = trun[i];
                        trun[i] += (tot + kGemmBM - 1) / kGemmBM;
                    }
                s_gidx[e] = static_cast<int>(gg);
                wv.grp_mt_off[gg] = tt;
                const int nmt = (tot + kGemmBM - 1) / kGemmBM;
                for (int i = 0; i < nmt; ++i) wv.mt_group[tt + i] = gg;
            }
            hrun += hit ? tot : 0;
            mrun += hit ? 0 : tot;
        }
        const uint32_t nh = readlane_u32(hi, kWave - 1), nm = readlane_u32(mi, kWave - 1);
        const uint32_t mexp = readlane_u32(xi, kWave - 1);
        if (lane == kWave - 1) {
            s_hoff[E] = nh;
            s_moff[E] = nm;
            ro.counts[0] = nh;
            ro.counts[1] = nm;
            ro.counts[2] = mexp;
            ro.counts[3] = *s_status;
            const uint32_t G = U + (shared_slot >= 0 ? 1 : 0);
            wv.grp_meta[0] = G;
            wv.grp_meta[1] = U;
            wv.grp_meta[2] = nh;
            wv.grp_meta[3] = T;
            wv.grp_meta[4] = MT + smt;
            if (shared_slot >= 0) {
                wv.grp_slot[0] = shared_slot;
                wv.grp_beg[0] = nh;
                wv.grp_len[0] = T;
                wv.grp_mt_off[0] = 0;
                for (uint32_t i = 0; i < smt; ++i) wv.mt_group[i] = 0;
            }
            wv.grp_mt_off[G] = MT + smt;
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e <= E; e += blockDim.x) {
        ro.hit_off[e] = s_hoff[e];
        ro.miss_off[e] = s_moff[e];
        if (e < E && s_gidx[e] >= 0) {
            const int g = s_gidx[e];
            wv.grp_slot[g] = s_eff[e];
            wv.grp_beg[g] = s_hoff[e];
            wv.grp_len[g] = s_tot[e];
        }
    }
    // list tails and the shared expert's rows
    // the list tails and the shared expert's rows are written by route_scatter, spread over its
    // workgroups
}

// ---------------------------------------------------------------------------------------
// Fused single-workgroup routing for T*k <= kFusedMaxPairs (few tokens: decode).  For the
// larger of these batches the top-k runs ahead in route_topk, and phase B only loads it (PRE).
// Four barriers separate five phases:
//   A  slot-table entry per thread, zeroed counters, logits of each wave's first token batch;
//   B  experts per slot counted; top-k per token (a wave per token, kTopkBatch tokens per wave
//      with their logits loaded together);
//   C  usable slot per expert; every 64-pair chunk (one wave) ranks its pairs among the pairs of
//      the same expert with ballots and records its per-expert count;
//   D  one wave scans the experts (hit/miss offsets, groups, GEMM tile map, counts) and writes
//      them out while the other waves add up, for each of their pairs, the counts of the earlier
//      chunks of the same expert;
//   E  each pair's list position = expert offset + earlier chunks + rank in chunk.
// The within-expert order is the pair index: the lists equal a stable counting sort.
// Waves of the fused router exchange data through LDS only, so its barriers wait for LDS
// operations alone: outstanding global loads and stores do not hold a barrier up (a
// __syncthreads would wait for every store of the phase to be acknowledged).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x0 << 8) | (0x3 << 14));   // lgkmcnt(0)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

constexpr int kFusedThreads = 1024;
constexpr int kFusedWaves = kFusedThreads / kWave;
constexpr int kTopkBatch = 4;
constexpr int kFusedPairsPerThread = kFusedMaxPairs / kFusedThreads;

// PRE: the top-k was computed by route_topk (topk_ids, topk_w hold it); phase B only loads it.
template <int NPL, bool PRE>
__global__ __launch_bounds__(kFusedThreads) void route_fused(RouteArgs a) {
    extern __shared__ int32_t lds[];
    // tokens per wave batch, within the 128 registers a 1024-thread workgroup leaves a lane
    constexpr int NBT = NPL >= 16 ? 1 : (NPL >= 8 ? 2 : kTopkBatch);
    const int E = a.E, k = a.k, T = a.T, P = T * k, nch = (P + kWave - 1) / kWave;
    const int ncnt = a.n_slots <= kSlotCountCap ? a.n_slots : 0;
    int32_t *s_raw = lds;                                   // E
    int32_t *s_eff = s_raw + E;                             // E
    int32_t *s_hoff = s_eff + E;                            // E+1
    int32_t *s_moff = s_hoff + E + 1;                       // E+1
    int32_t *s_ids = s_moff + E + 1;                        // P
    float *s_w = reinterpret_cast<float *>(s_ids + P);      // P
    int32_t *s_wh = reinterpret_cast<int32_t *>(s_w + P);   // [nch][E] pairs per chunk and expert
    int32_t *s_cnt = s_wh + nch * E;                        // [ncnt] experts per slot
    int *s_status = s_cnt + ncnt;                           // 1
    const int tid = threadIdx.x, wave = tid / kWave, lane = lane_id();

    // ---- A
    const int raw = tid < E ? a.slot_table[tid] : -1;
    // tokens of this wave: wave, wave + 16, ...; the first NBT are loaded here
    const int nmine = T > wave ? (T - wave + kFusedWaves - 1) / kFusedWaves : 0;
    uint32_t key0[NBT][NPL];
    int pre_id[kFusedPairsPerThread];
    float pre_w[kFusedPairsPerThread];
    if constexpr (PRE) {
#pragma unroll
        for (int i = 0; i < kFusedPairsPerThread; ++i) {
            const int p = min(tid + i * kFusedThreads, P - 1);
            pre_id[i] = a.ro.topk_ids[p];
            pre_w[i] = a.ro.topk_w[p];
        }
    } else {
#pragma unroll
        for (int b = 0; b < NBT; ++b)
            topk_load<NPL>(a.logits + static_cast<size_t>(min(wave + b * kFusedWaves, T - 1)) * E, E, key0[b]);
    }
    for (int i = tid; i < nch * E; i += kFusedThreads) s_wh[i] = 0;
    for (int i = tid; i < ncnt; i += kFusedThreads) s_cnt[i] = 0;
    if (tid == 0) *s_status = 0;
    // (the slot-table entry is stored in phase B, so this barrier does not wait for its load)
    lds_barrier();

    // ---- B
    if (tid < E) s_raw[tid] = raw;
    slot_count(raw, E, a.n_slots, s_cnt);
    auto put = [&](int t, int id, float w) {
        if (t < T && lane < k) {
            s_ids[t * k + lane] = id;
            s_w[t * k + lane] = w;
        }
    };
    auto select_batch = [&](uint32_t (&key)[NBT][NPL], int tb, int n) {
        // n (wave-uniform) of the batch's tokens are real; tokens tb + 16 b
        int id[NBT];
        float w[NBT];
        if constexpr (NBT >= 4) {
            if (n >= 3) {
                topk_select_n<NPL, 4>(key, k, a.gating, id, w);
#pragma unroll
                for (int b = 0; b < NBT; ++b)
                    if (b < n) put(tb + b * kFusedWaves, id[b], w[b]);
                return;
            }
        }
        if constexpr (NBT >= 2) {
            if (n >= 2) {
                uint32_t k2[2][NPL];
#pragma unroll
                for (int i = 0; i < NPL; ++i) {
                    k2[0][i] = key[0][i];
                    k2[1][i] = key[1][i];
                }
                int id2[2];
                float w2[2];
                topk_select_n<NPL, 2>(k2, k, a.gating, id2, w2);
                put(tb, id2[0], w2[0]);
                put(tb + kFusedWaves, id2[1], w2[1]);
                return;
            }
        }
        topk_select<NPL>(key[0], k, a.gating, id[0], w[0]);
        put(tb, id[0], w[0]);
    };
    if constexpr (PRE) {
#pragma unroll
        for (int i = 0; i < kFusedPairsPerThread; ++i) {
            const int p = tid + i * kFusedThreads;
            if (p < P) {
                s_ids[p] = pre_id[i];
                s_w[p] = pre_w[i];
            }
        }
    } else {
        if (nmine > 0) select_batch(key0, wave, min(nmine, NBT));
        for (int b0 = NBT; b0 < nmine; b0 += NBT) {
            uint32_t key[NBT][NPL];
            const int tb = wave + b0 * kFusedWaves;
#pragma unroll
            for (int b = 0; b < NBT; ++b)
                topk_load<NPL>(a.logits + static_cast<size_t>(min(tb + b * kFusedWaves, T - 1)) * E, E, key[b]);
            select_batch(key, tb, min(nmine - b0, NBT));
        }
    }
    lds_barrier();

    // ---- C
    if (tid < E) {
        int st = 0;
        s_eff[tid] = slot_check(raw, tid, E, a.n_slots, a.shared_slot, s_cnt, s_raw, st);
        if (st) atomicOr(s_status, st);
    }
    // pair p = tid + i * kFusedThreads lies in chunk p / 64, which is this wave's
    int pe[kFusedPairsPerThread], prank[kFusedPairsPerThread], pre[kFusedPairsPerThread];
#pragma unroll
    for (int i = 0; i < kFusedPairsPerThread; ++i) {
        const int p = tid + i * kFusedThreads;
        const bool act = p < P;
        const uint64_t live = __ballot(act);
        pe[i] = 0;
        prank[i] = 0;
        pre[i] = 0;
        if (live == 0) continue;
        const int e = act ? s_ids[p] : 0;
        const uint64_t same = match_lanes(static_cast<uint32_t>(e), a.nbits, live);
        const int rank = __popcll(same & lanemask_lt());
        if (act && rank == __popcll(same) - 1) s_wh[(p / kWave) * E + e] = rank + 1;
        pe[i] = e;
        prank[i] = rank;
    }
    lds_barrier();

    // ---- D
    auto chunk_prefix = [&]() {
#pragma unroll
        for (int i = 0; i < kFusedPairsPerThread; ++i) {
            const int p = tid + i * kFusedThreads;
            if (p < P) {
                int acc = 0;
                for (int c = 0; c < p / kWave; ++c) acc += s_wh[c * E + pe[i]];
                pre[i] = acc;
            }
        }
    };
    if (wave != 0) {
        chunk_prefix();
    } else {
        // lane l owns experts [l*epl, l*epl + epl), epl = NPL; up to 8 per lane, their totals
        // and slots stay in registers for the second pass (more would not fit the 128 registers
        // of a 1024-thread workgroup; those are read again from LDS)
        constexpr int kMaxEpl = NPL;
        constexpr bool kCache = NPL <= 8;
        const int epl = (E + kWave - 1) / kWave;
        const int e0 = min(E, lane * epl), e1 = min(E, e0 + epl);
        int tots[kCache ? kMaxEpl : 1], slots[kCache ? kMaxEpl : 1];
        auto total_of = [&](int e) {
            int tot = 0;
            for (int c = 0; c < nch; ++c) tot += s_wh[c * E + e];
            return tot;
        };
        uint32_t h = 0, m = 0, g = 0, mx = 0, mtl = 0;
#pragma unroll
        for (int i = 0; i < kMaxEpl; ++i) {
            const int e = e0 + i;
            const int tot = e < e1 ? total_of(e) : 0;
            const int slot = e < e1 ? s_eff[e] : -1;
            if constexpr (kCache) {
                tots[i] = tot;
                slots[i] = slot;
            }
            const bool hit = slot >= 0;
            h += hit ? tot : 0;
            m += hit ? 0 : tot;
            g += (hit && tot > 0) ? 1 : 0;
            mx += (!hit && tot > 0) ? 1 : 0;
            mtl += hit ? (tot + kGemmBM - 1) / kGemmBM : 0;
        }
        const uint32_t hi = wave_incl_scan_u32(h), mi = wave_incl_scan_u32(m);
        const uint32_t gi = wave_incl_scan_u32(g), xi = wave_incl_scan_u32(mx);
        const uint32_t ti = wave_incl_scan_u32(mtl);
        uint32_t hrun = hi - h, mrun = mi - m, grun = gi - g, trun = ti - mtl;
#pragma unroll
        for (int i = 0; i < kMaxEpl; ++i) {
            const int e = e0 + i;
            if (e >= e1) continue;
            int tot, slot;
            if constexpr (kCache) {
                tot = tots[i];
                slot = slots[i];
            } else {
                tot = total_of(e);
                slot = s_eff[e];
            }
            const bool hit = slot >= 0;
            s_hoff[e] = hrun;
            s_moff[e] = mrun;
            a.ro.hit_off[e] = hrun;
            a.ro.miss_off[e] = mrun;
            if (hit && tot > 0) {
                a.wv.grp_slot[grun] = slot;
                a.wv.grp_beg[grun] = hrun;
                a.wv.grp_len[grun] = tot;
                a.wv.grp_mt_off[grun] = trun;
                const int nmt = (tot + kGemmBM - 1) / kGemmBM;
                for (int u = 0; u < nmt; ++u) a.wv.mt_group[trun + u] = grun;
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
            s_hoff[E] = nh;
            s_moff[E] = nm;
            a.ro.hit_off[E] = nh;
            a.ro.miss_off[E] = nm;
            a.ro.counts[0] = nh;
            a.ro.counts[1] = nm;
            a.ro.counts[2] = mexp;
            a.ro.counts[3] = *s_status;
            const int shared = a.shared_slot;
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
        chunk_prefix();
    }
    lds_barrier();

    // ---- E
    const int nh = s_hoff[E], nm = s_moff[E];
#pragma unroll
    for (int i = 0; i < kFusedPairsPerThread; ++i) {
        const int p = tid + i * kFusedThreads;
        if (p < P) {
            const int e = pe[i], slot = s_eff[e];
            const int pos = (slot >= 0 ? s_hoff[e] : s_moff[e]) + pre[i] + prank[i];
            a.ro.topk_slot[p] = slot;
            if (slot >= 0) {
                a.ro.hit_pairs[pos] = p;
                a.wv.row_tok[pos] = p / k;
                a.wv.row_pair[pos] = p;
                a.wv.row_gate[pos] = s_w[p];
            } else {
                a.ro.miss_pairs[pos] = p;
            }
        }
    }
    for (int i = tid; i < P; i += kFusedThreads) {
        if (i >= nh) a.ro.hit_pairs[i] = -1;
        if (i >= nm) a.ro.miss_pairs[i] = -1;
        if constexpr (!PRE) {
            a.ro.topk_ids[i] = s_ids[i];
            a.ro.topk_w[i] = s_w[i];
        }
    }
    if (a.shared_slot >= 0) {
        for (int t = tid; t < T; t += kFusedThreads) {
            a.wv.row_tok[nh + t] = t;
            a.wv.row_pair[nh + t] = T * k + t;
            a.wv.row_gate[nh + t] = 1.0f;
        }
    }
}

// One or two tokens: one wave does all of the routing (route_wave_body).
template <int NPL>
__global__ __launch_bounds__(kWave) void route_wave(RouteArgs a) {
    extern __shared__ int32_t lds[];
    route_wave_body<NPL, false>(a, lds, true, WaveRouteSink{});
}

// ---------------------------------------------------------------------------------------
// Multi-workgroup routing.  Block b owns tokens [b*kTokPerBlk, (b+1)*kTokPerBlk).
template <int NPL>
__global__ __launch_bounds__(256) void route_tokens(RouteArgs a) {
    __shared__ int32_t s_hist[kMaxExperts];
    const int E = a.E, k = a.k, T = a.T;
    for (int e = threadIdx.x; e < E; e += blockDim.x) s_hist[e] = 0;
    __syncthreads();
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int t0 = blockIdx.x * kTokPerBlk;
    for (int t = t0 + wave; t < min(T, t0 + kTokPerBlk); t += 4) {
        int id;
        float w;
        wave_topk<NPL>(a.logits + static_cast<size_t>(t) * E, E, k, a.gating, id, w);
        if (lane < k) {
            a.ro.topk_ids[t * k + lane] = id;
            a.ro.topk_w[t * k + lane] = w;
            atomicAdd(&s_hist[id], 1);
        }
    }
    __syncthreads();
    int32_t *hist = a.wv.blk_hist + static_cast<size_t>(blockIdx.x) * E;
    for (int e = threadIdx.x; e < E; e += blockDim.x) hist[e] = s_hist[e];
}

// Per part of kBlkPerPart router blocks (grid: parts x ceil(E / 256)): each block's per-expert
// counts become the counts of the part's earlier blocks (in place), and the part's totals go to
// the part table after the nblk block rows.  Spreads the scan's memory rounds over many CUs: the
// one-workgroup route_scan then only scans the part table (measured at DeepSeek-V3 prefill,
// 8192 tokens: route_scan 35 us when it scanned all 512 block rows itself).
__global__ __launch_bounds__(256) void route_partscan(RouteArgs a, int nblk) {
    const int E = a.E, e = blockIdx.y * 256 + threadIdx.x;
    if (e >= E) return;
    const int b0 = blockIdx.x * kBlkPerPart, b1 = min(nblk, b0 + kBlkPerPart);
    int32_t *col = a.wv.blk_hist + e;
    int v[kBlkPerPart];
    // clamped, unconditional loads, all in flight together
#pragma unroll
    for (int i = 0; i < kBlkPerPart; ++i) v[i] = col[static_cast<size_t>(min(b0 + i, b1 - 1)) * E];
    int run = 0;
#pragma unroll
    for (int i = 0; i < kBlkPerPart; ++i) {
        if (b0 + i < b1) {
            col[static_cast<size_t>(b0 + i) * E] = run;
            run += v[i];
        }
    }
    col[(static_cast<size_t>(nblk) + blockIdx.x) * E] = run;
}

__global__ __launch_bounds__(1024) void route_scan(RouteArgs a, int nblk) {
    extern __shared__ int32_t lds[];
    const int E = a.E;
    // the part table (route_partscan): one row of per-expert counts per part of kBlkPerPart blocks
    const int nparts = (nblk + kBlkPerPart - 1) / kBlkPerPart;
    int32_t *ptab = a.wv.blk_hist + static_cast<size_t>(nblk) * E;
    int32_t *s_raw = lds, *s_eff = s_raw + E, *s_tot = s_eff + E, *s_hoff = s_tot + E;
    int32_t *s_moff = s_hoff + E + 1, *s_gidx = s_moff + E + 1;
    int *s_status = s_gidx + E;
    int32_t *s_part = s_status + 1;          // [parts][E] partial block sums
    int32_t *s_cnt = s_part + a.scan_parts * E;   // [min(n_slots, kSlotCountCap)]
    const int raw = threadIdx.x < E ? a.slot_table[threadIdx.x] : -1;
    if (threadIdx.x == 0) *s_status = 0;
    validate_slots(raw, E, a.n_slots, a.shared_slot, s_raw, s_cnt, s_eff, s_status);
    // `parts` threads per expert, each over a contiguous range of the part rows
    const int parts = a.scan_parts;
    const int e = threadIdx.x % E, part = threadIdx.x / E;
    const int per = (nparts + parts - 1) / parts;
    const int b0 = min(nparts, part * per), b1 = min(nparts, b0 + per);
    const bool active = part < parts;
    // each thread's column range is read kScanBatch entries at a time, all in flight together
    // (one workgroup does the whole scan, so its memory latency is the scan's cost)
    constexpr int kScanBatch = 32;
    if (active) {
        int sum = 0;
        for (int b = b0; b < b1; b += kScanBatch) {
            int buf[kScanBatch];
            // clamped, unconditional loads; entries past the range count 0
#pragma unroll
            for (int i = 0; i < kScanBatch; ++i) buf[i] = ptab[static_cast<size_t>(min(b + i, b1 - 1)) * E + e];
#pragma unroll
            for (int i = 0; i < kScanBatch; ++i) sum += b + i < b1 ? buf[i] : 0;
        }
        s_part[part * E + e] = sum;
    }
    __syncthreads();
    for (int x = threadIdx.x; x < E; x += blockDim.x) {
        int run = 0;
        for (int q = 0; q < parts; ++q) {
            const int c = s_part[q * E + x];
            s_part[q * E + x] = run;
            run += c;
        }
        s_tot[x] = run;
        a.wv.eff_slot[x] = s_eff[x];
    }
    __syncthreads();
    scan_experts(E, a.T, a.k, a.shared_slot, s_tot, s_eff, s_hoff, s_moff, s_gidx, s_status, a.ro, a.wv);
    __syncthreads();
    if (active) {
        int run = s_part[part * E + e] + (s_eff[e] >= 0 ? s_hoff[e] : s_moff[e]);
        for (int b = b0; b < b1; b += kScanBatch) {
            // all loads of the batch, then the running offsets, then all stores (a store between
            // two loads would make each wait cover the store too)
            int buf[kScanBatch];
#pragma unroll
            for (int i = 0; i < kScanBatch; ++i) buf[i] = ptab[static_cast<size_t>(min(b + i, b1 - 1)) * E + e];
            int off[kScanBatch];
#pragma unroll
            for (int i = 0; i < kScanBatch; ++i) {
                off[i] = run;
                run += b + i < b1 ? buf[i] : 0;
            }
#pragma unroll
            for (int i = 0; i < kScanBatch; ++i)
                if (b + i < b1) ptab[static_cast<size_t>(b + i) * E + e] = off[i];
        }
    }
}

// Block b's first list position per expert = its part's entry of the part table (the expert's
// offset plus the counts of the earlier parts) + its own entry of the block table (the counts of
// the part's earlier blocks).  Besides its pairs, block b writes the list tails in its pair range
// and the shared expert's rows of its tokens.
__global__ __launch_bounds__(64) void route_scatter(RouteArgs a) {
    __shared__ int32_t s_eff[kMaxExperts];
    __shared__ int32_t s_run[kMaxExperts];
    const int E = a.E, k = a.k, T = a.T, nblk = gridDim.x;
    const int32_t *off = a.wv.blk_hist + static_cast<size_t>(blockIdx.x) * E;
    const int32_t *base = a.wv.blk_hist + (static_cast<size_t>(nblk) + blockIdx.x / kBlkPerPart) * E;
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        s_eff[e] = a.wv.eff_slot[e];
        s_run[e] = base[e] + off[e];
    }
    const int nh = a.ro.hit_off[E], nm = a.ro.miss_off[E];
    __syncthreads();
    const int t0 = blockIdx.x * kTokPerBlk, t1 = min(T, t0 + kTokPerBlk);
    const int p0 = t0 * k, p1 = t1 * k;
    scatter_run(p0, p1, k, a.nbits, a.ro.topk_ids, a.ro.topk_w, s_eff, s_run, a.ro, a.wv);
    for (int i = p0 + static_cast<int>(threadIdx.x); i < p1; i += blockDim.x) {
        if (i >= nh) a.ro.hit_pairs[i] = -1;
        if (i >= nm) a.ro.miss_pairs[i] = -1;
    }
    if (a.shared_slot >= 0) {
        for (int t = t0 + static_cast<int>(threadIdx.x); t < t1; t += blockDim.x) {
            a.wv.row_tok[nh + t] = t;
            a.wv.row_pair[nh + t] = T * k + t;
            a.wv.row_gate[nh + t] = 1.0f;
        }
    }
}

// ---------------------------------------------------------------------------------------
// Top-k ahead of route_fused<NPL, true> for the larger decode batches: one wave per token, four
// tokens per workgroup, so the k selection rounds of all tokens run on many CUs at once instead
// of in turn on the 16 waves of the fused router.
template <int NPL>
__global__ __launch_bounds__(256) void route_topk(RouteArgs a) {
    const int t = blockIdx.x * 4 + threadIdx.x / kWave, lane = lane_id();
    if (t >= a.T) return;
    int id;
    float w;
    wave_topk<NPL>(a.logits + static_cast<size_t>(t) * a.E, a.E, a.k, a.gating, id, w);
    if (lane < a.k) {
        a.ro.topk_ids[t * a.k + lane] = id;
        a.ro.topk_w[t * a.k + lane] = w;
    }
}

template <int NPL>
static hipError_t launch_route_npl(RouteArgs a, hipStream_t s) {
    const int P = a.T * a.k;
    const int ncnt = a.n_slots <= kSlotCountCap ? a.n_slots : 0;
    const int fused_lds = 4 * (4 * a.E + 2 + 2 * P + ((P + kWave - 1) / kWave) * a.E + ncnt + 1);
    if constexpr (NPL <= kWaveRouteMaxNpl) {
        const int wave_lds = route_wave_lds_bytes(a.E, ncnt);
        if (a.T <= kWaveRouteMaxTokens && P <= kWave && wave_lds <= kFusedMaxLds) {
            hipLaunchKernelGGL(route_wave<NPL>, dim3(1), dim3(kWave), wave_lds, s, a);
            return hipGetLastError();
        }
    }
    if (P <= kFusedMaxPairs && fused_lds <= kFusedMaxLds) {
        if (a.T * a.E >= FT_ROUTE_SPLIT_LOGITS) {
            hipLaunchKernelGGL(route_topk<NPL>, dim3((a.T + 3) / 4), dim3(256), 0, s, a);
            hipLaunchKernelGGL((route_fused<NPL, true>), dim3(1), dim3(kFusedThreads), fused_lds, s, a);
        } else {
            hipLaunchKernelGGL((route_fused<NPL, false>), dim3(1), dim3(kFusedThreads), fused_lds, s, a);
        }
        return hipGetLastError();
    }
    const int nblk = (a.T + kTokPerBlk - 1) / kTokPerBlk;
    const int nparts = (nblk + kBlkPerPart - 1) / kBlkPerPart;
    a.scan_parts = max(1, min(1024 / a.E, nparts));
    hipLaunchKernelGGL(route_tokens<NPL>, dim3(nblk), dim3(256), 0, s, a);
    hipLaunchKernelGGL(route_partscan, dim3(nparts, (a.E + 255) / 256), dim3(256), 0, s, a, nblk);
    const int scan_lds = 4 * (6 * a.E + 3 + a.scan_parts * a.E + ncnt);
    hipLaunchKernelGGL(route_scan, dim3(1), dim3(1024), scan_lds, s, a, nblk);
    hipLaunchKernelGGL(route_scatter, dim3(nblk), dim3(64), 0, s, a);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Evaluation groups of a hybrid step, G = H u F (Section 3.2: after the planned fills the GPU
// evaluates the hits and the freshly filled experts), built from the step's single routing after
// the cache plan rewrote the routed slot ids: an expert with routed pairs forms a group iff its
// first pair now carries a slot (hits keep theirs, filled experts carry their new slot, experts
// left to the CPU keep FT_SLOT_MISS).  Its pairs are its hit list or, for a filled expert, its
// miss list (an expert's pairs are all hits or all misses).  Writes the same group table, M-tile
// map and row arrays as the router, in expert-id order, then the shared expert's rows.
// One 1024-thread workgroup, thread e = expert e.
__global__ __launch_bounds__(1024) void regroup_kernel(RegroupArgs a) {
    __shared__ int32_t s_beg[kMaxExperts + 1];   // first row of group g
    __shared__ int32_t s_src[kMaxExperts];       // list position of group g's first pair (miss list: + T*k)
    __shared__ uint32_t s_wsum[3][1024 / kWave];
    __shared__ int32_t s_tot[4];
    const int E = a.E, T = a.T, k = a.k, tid = threadIdx.x;
    const int lane = lane_id(), wv = tid / kWave;
    const int PK = T * k;
    // ---- this expert's group
    int n = 0, src = 0, slot = -1;
    if (tid < E) {
        const int h0 = a.hit_off[tid], h1 = a.hit_off[tid + 1];
        const int m0 = a.miss_off[tid], m1 = a.miss_off[tid + 1];
        if (h1 > h0) {
            n = h1 - h0;
            src = h0;
            slot = a.topk_slot[a.hit_pairs[h0]];
        } else if (m1 > m0) {
            n = m1 - m0;
            src = PK + m0;
            slot = a.topk_slot[a.miss_pairs[m0]];
        }
        if (slot < 0) n = 0;
    }
    const uint32_t in_g = n > 0 ? 1u : 0u;
    const uint32_t rows = static_cast<uint32_t>(n);
    const uint32_t mts = in_g ? static_cast<uint32_t>((n + kGemmBM - 1) / kGemmBM) : 0u;
    // ---- block-wide exclusive scans of (group flag, rows, M tiles) over the experts
    const uint32_t gi = wave_incl_scan_u32(in_g), ri = wave_incl_scan_u32(rows), ti = wave_incl_scan_u32(mts);
    if (lane == kWave - 1) {
        s_wsum[0][wv] = gi;
        s_wsum[1][wv] = ri;
        s_wsum[2][wv] = ti;
    }
    __syncthreads();
    uint32_t gb = 0, rb = 0, tb = 0;
    for (int w = 0; w < wv; ++w) {
        gb += s_wsum[0][w];
        rb += s_wsum[1][w];
        tb += s_wsum[2][w];
    }
    const int g = static_cast<int>(gb + gi - in_g), r0 = static_cast<int>(rb + ri - rows),
              t0 = static_cast<int>(tb + ti - mts);
    if (in_g) {
        a.wv.grp_slot[g] = slot;
        a.wv.grp_beg[g] = r0;
        a.wv.grp_len[g] = n;
        a.wv.grp_mt_off[g] = t0;
        for (uint32_t i = 0; i < mts; ++i) a.wv.mt_group[t0 + i] = g;
        s_beg[g] = r0;
        s_src[g] = src;
    }
    if (tid == 1023) {
        // totals over every wave: thread 1023 is the last lane of the last wave
        uint32_t U = 0, NR = 0, MT = 0;
        for (int w = 0; w < 1024 / kWave; ++w) {
            U += s_wsum[0][w];
            NR += s_wsum[1][w];
            MT += s_wsum[2][w];
        }
        s_tot[0] = static_cast<int>(U);
        s_tot[1] = static_cast<int>(NR);
        s_beg[U] = static_cast<int>(NR);
        const uint32_t smt = a.shared_slot >= 0 ? (T + kGemmBM - 1) / kGemmBM : 0;
        const uint32_t G = U + (a.shared_slot >= 0 ? 1 : 0);
        a.wv.grp_meta[0] = G;
        a.wv.grp_meta[1] = U;
        a.wv.grp_meta[2] = NR;
        a.wv.grp_meta[3] = T;
        a.wv.grp_meta[4] = MT + smt;
        if (a.shared_slot >= 0) {
            a.wv.grp_slot[U] = a.shared_slot;
            a.wv.grp_beg[U] = NR;
            a.wv.grp_len[U] = T;
            a.wv.grp_mt_off[U] = MT;
            for (uint32_t i = 0; i < smt; ++i) a.wv.mt_group[MT + i] = U;
        }
        a.wv.grp_mt_off[G] = MT + smt;
    }
    __syncthreads();
    // ---- rows: row r of group g is pair i = r - beg(g) of its list
    const int U = s_tot[0], NR = s_tot[1];
    for (int r = tid; r < NR; r += 1024) {
        int lo = 0, hi = U - 1;           // the last group whose first row is <= r
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_beg[mid] <= r) lo = mid;
            else hi = mid - 1;
        }
        const int at = s_src[lo] + (r - s_beg[lo]);
        const int p = at < PK ? a.hit_pairs[at] : a.miss_pairs[at - PK];
        a.wv.row_tok[r] = p / k;
        a.wv.row_pair[r] = p;
        a.wv.row_gate[r] = a.topk_w[p];
    }
    if (a.shared_slot >= 0) {
        for (int t = tid; t < T; t += 1024) {
            a.wv.row_tok[NR + t] = t;
            a.wv.row_pair[NR + t] = PK + t;
            a.wv.row_gate[NR + t] = 1.0f;
        }
    }
}

hipError_t launch_regroup(const RegroupArgs &a, hipStream_t s) {
    hipLaunchKernelGGL(regroup_kernel, dim3(1), dim3(1024), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_route(const RouteArgs &a, hipStream_t s) {
    const int npl = (a.E + kWave - 1) / kWave;
    if (npl <= 1) return launch_route_npl<1>(a, s);
    if (npl <= 2) return launch_route_npl<2>(a, s);
    if (npl <= 4) return launch_route_npl<4>(a, s);
    if (npl <= 8) return launch_route_npl<8>(a, s);
    return launch_route_npl<16>(a, s);
}

}  // namespace ftmoe
