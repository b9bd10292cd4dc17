// Router top-k, hit/miss classification against the slot table, and the expert-sorted stable
// permutation (Section 3.2: router and cache lookup on the GPU; Section 4.1: routed logical ids
// rewritten into slot ids or a CPU flag, kept as fixed-shape buffers with device counts).
//
// Two variants:
//  * route_fused: one 1024-thread workgroup does everything in LDS (few tokens: decode).
//  * route_tokens -> route_scan -> route_scatter: many tokens (prefill chunks).
// Both produce bit-identical outputs: the permutation is a counting sort whose within-expert
// order is the pair index, computed with wave ballots, never with order-dependent atomics.
#include "ftmoe_device.h"
#include "ftmoe_internal.h"

namespace ftmoe {

// ---------------------------------------------------------------------------------------
// Top-k of one token's logits by one wave.  Lane l holds experts [l*NPL, l*NPL + NPL), so among
// equal logits the lowest lane, and within a lane the lowest index, is the lowest expert id.
// Each round takes the wave maximum of the lanes' best keys (DPP) and the lowest lane holding
// it (ballot).  On return lane j < k holds (expert id, gate) of the j-th selected expert.
template <int NPL>
__device__ __forceinline__ void wave_topk(const float *__restrict__ row, int E, int k, int gating,
                                          int &my_id, float &my_w) {
    const int lane = lane_id();
    uint32_t key[NPL];
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
        const int e = lane * NPL + i;
        key[i] = e < E ? order_key(row[e]) : 0u;
    }
    uint32_t mine = 0u;
    int mine_e = -1;
    for (int j = 0; j < k; ++j) {
        uint32_t best = 0u;
        int bi = 0;
#pragma unroll
        for (int i = 0; i < NPL; ++i) {
            if (key[i] > best) {
                best = key[i];
                bi = i;
            }
        }
        const uint32_t m = wave_max_u32(best);
        const uint64_t ball = __ballot(best == m);
        const int w = static_cast<int>(__builtin_ctzll(ball));
        const int wbi = __builtin_amdgcn_readlane(bi, w);
        if (lane == w) {
#pragma unroll
            for (int i = 0; i < NPL; ++i)
                if (i == wbi) key[i] = 0u;
        }
        if (lane == j) {
            mine = m;
            mine_e = w * NPL + wbi;
        }
    }
    const float top = key_to_float(readlane_u32(mine, 0));
    float z = 0.f;
    if (lane < k) {
        const float l = key_to_float(mine);
        z = gating == FT_GATE_SOFTMAX_TOPK_RENORM ? expf(l - top) : 1.0f / (1.0f + expf(-l));
    }
    const float sum = wave_sum_f32(z);
    my_id = lane < k ? mine_e : -1;
    my_w = lane < k ? z / sum : 0.f;
}

// Validated slot of each expert (-1 if unusable) and the device status bits.  `raw` is this
// thread's slot_table entry (thread e of the block holds expert e; blockDim >= E).
__device__ void validate_slots(int raw, int E, int n_slots, int shared_slot, int32_t *s_raw,
                               int32_t *s_eff, int *s_status) {
    if (threadIdx.x < E) s_raw[threadIdx.x] = raw;
    __syncthreads();
    int st = 0;
    if (threadIdx.x < E) {
        const int e = threadIdx.x, s = raw;
        int eff = -1;
        if (s == -1) {
        } else if (s < -1 || s >= n_slots) {
            st |= FT_DEV_SLOT_RANGE;
        } else if (shared_slot >= 0 && s == shared_slot) {
            st |= FT_DEV_SLOT_SHARED;
        } else {
            bool dup = false;
            for (int o = 0; o < E; ++o) dup |= (o != e) & (s_raw[o] == s);
            if (dup) st |= FT_DEV_SLOT_DUP; else eff = s;
        }
        s_eff[e] = eff;
    }
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
        uint32_t h = 0, m = 0, g = 0, mx = 0, mtl = 0;
        for (int e = e0; e < e1; ++e) {
            const int tot = s_tot[e];
            const bool hit = s_eff[e] >= 0;
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
        for (int e = e0; e < e1; ++e) {
            const int tot = s_tot[e];
            const bool hit = s_eff[e] >= 0;
            s_hoff[e] = hrun;
            s_moff[e] = mrun;
            s_gidx[e] = (hit && tot > 0) ? static_cast<int>(grun) : -1;
            if (hit && tot > 0) {
                wv.grp_mt_off[grun] = trun;
                const int nmt = (tot + kGemmBM - 1) / kGemmBM;
                for (int i = 0; i < nmt; ++i) wv.mt_group[trun + i] = grun;
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
            ro.counts[0] = nh;
            ro.counts[1] = nm;
            ro.counts[2] = mexp;
            ro.counts[3] = *s_status;
            const uint32_t smt = shared_slot >= 0 ? (T + kGemmBM - 1) / kGemmBM : 0;
            const uint32_t G = U + (shared_slot >= 0 ? 1 : 0);
            wv.grp_meta[0] = G;
            wv.grp_meta[1] = U;
            wv.grp_meta[2] = nh;
            wv.grp_meta[3] = T;
            wv.grp_meta[4] = MT + smt;
            if (shared_slot >= 0) {
                wv.grp_slot[U] = shared_slot;
                wv.grp_beg[U] = nh;
                wv.grp_len[U] = T;
                wv.grp_mt_off[U] = MT;
                for (uint32_t i = 0; i < smt; ++i) wv.mt_group[MT + i] = U;
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
    const int nh = s_hoff[E], nm = s_moff[E];
    for (int i = threadIdx.x; i < T * k; i += blockDim.x) {
        if (i >= nh) ro.hit_pairs[i] = -1;
        if (i >= nm) ro.miss_pairs[i] = -1;
    }
    if (shared_slot >= 0) {
        for (int t = threadIdx.x; t < T; t += blockDim.x) {
            wv.row_tok[nh + t] = t;
            wv.row_gate[nh + t] = 1.0f;
        }
    }
}

// ---------------------------------------------------------------------------------------
// Fused single-workgroup routing for T*k <= kFusedMaxPairs.
constexpr int kFusedThreads = 1024;
constexpr int kFusedWaves = kFusedThreads / kWave;

template <int NPL>
__global__ __launch_bounds__(kFusedThreads) void route_fused(RouteArgs a) {
    extern __shared__ int32_t lds[];
    const int E = a.E, k = a.k, T = a.T, P = T * k;
    int32_t *s_raw = lds;                    // E
    int32_t *s_eff = s_raw + E;              // E
    int32_t *s_tot = s_eff + E;              // E
    int32_t *s_hoff = s_tot + E;             // E+1
    int32_t *s_moff = s_hoff + E + 1;        // E+1
    int32_t *s_gidx = s_moff + E + 1;        // E
    int32_t *s_ids = s_gidx + E;             // P
    float *s_w = reinterpret_cast<float *>(s_ids + P);   // P
    int32_t *s_wh = reinterpret_cast<int32_t *>(s_w + P);  // kFusedWaves * E
    int *s_status = s_wh + kFusedWaves * E;  // 1

    // issue the slot-table load first; its latency overlaps the top-k
    const int raw = threadIdx.x < E ? a.slot_table[threadIdx.x] : -1;
    if (threadIdx.x == 0) *s_status = 0;
    for (int i = threadIdx.x; i < kFusedWaves * E; i += blockDim.x) s_wh[i] = 0;

    const int wave = threadIdx.x / kWave, lane = lane_id();
    for (int t = wave; t < T; t += kFusedWaves) {
        int id;
        float w;
        wave_topk<NPL>(a.logits + static_cast<size_t>(t) * E, E, k, a.gating, id, w);
        if (lane < k) {
            s_ids[t * k + lane] = id;
            s_w[t * k + lane] = w;
            a.ro.topk_ids[t * k + lane] = id;
            a.ro.topk_w[t * k + lane] = w;
        }
    }
    validate_slots(raw, E, a.n_slots, a.shared_slot, s_raw, s_eff, s_status);
    // each wave owns a contiguous run of pairs; count its pairs per expert
    const int per = (P + kFusedWaves - 1) / kFusedWaves;
    const int p0 = min(P, wave * per), p1 = min(P, p0 + per);
    int32_t *wh = s_wh + wave * E;
    for (int p = p0 + lane; p < p1; p += kWave) atomicAdd(&wh[s_ids[p]], 1);
    __syncthreads();
    // per expert: exclusive offsets of each wave's run, total
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        int run = 0;
        for (int w = 0; w < kFusedWaves; ++w) {
            const int c = s_wh[w * E + e];
            s_wh[w * E + e] = run;
            run += c;
        }
        s_tot[e] = run;
    }
    __syncthreads();
    scan_experts(E, T, k, a.shared_slot, s_tot, s_eff, s_hoff, s_moff, s_gidx, s_status, a.ro, a.wv);
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        const int b = s_eff[e] >= 0 ? s_hoff[e] : s_moff[e];
        for (int w = 0; w < kFusedWaves; ++w) s_wh[w * E + e] += b;
    }
    __syncthreads();
    scatter_run(p0, p1, k, a.nbits, s_ids, s_w, s_eff, wh, a.ro, a.wv);
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

__global__ __launch_bounds__(1024) void route_scan(RouteArgs a, int nblk) {
    extern __shared__ int32_t lds[];
    const int E = a.E;
    int32_t *s_raw = lds, *s_eff = s_raw + E, *s_tot = s_eff + E, *s_hoff = s_tot + E;
    int32_t *s_moff = s_hoff + E + 1, *s_gidx = s_moff + E + 1;
    int *s_status = s_gidx + E;
    int32_t *s_part = s_status + 1;          // [parts][E] partial block sums
    const int raw = threadIdx.x < E ? a.slot_table[threadIdx.x] : -1;
    if (threadIdx.x == 0) *s_status = 0;
    validate_slots(raw, E, a.n_slots, a.shared_slot, s_raw, s_eff, s_status);
    // `parts` threads per expert, each over a contiguous range of the blocks
    const int parts = a.scan_parts;
    const int e = threadIdx.x % E, part = threadIdx.x / E;
    const int per = (nblk + parts - 1) / parts;
    const int b0 = min(nblk, part * per), b1 = min(nblk, b0 + per);
    const bool active = part < parts;
    if (active) {
        int sum = 0;
#pragma unroll 8
        for (int b = b0; b < b1; ++b) sum += a.wv.blk_hist[static_cast<size_t>(b) * E + e];
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
        int buf[8];
        for (int b = b0; b < b1; b += 8) {
            const int n = min(8, b1 - b);
#pragma unroll
            for (int i = 0; i < 8; ++i)
                buf[i] = i < n ? a.wv.blk_hist[static_cast<size_t>(b + i) * E + e] : 0;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                if (i < n) {
                    a.wv.blk_hist[static_cast<size_t>(b + i) * E + e] = run;
                    run += buf[i];
                }
            }
        }
    }
}

__global__ __launch_bounds__(64) void route_scatter(RouteArgs a) {
    __shared__ int32_t s_eff[kMaxExperts];
    __shared__ int32_t s_run[kMaxExperts];
    const int E = a.E, k = a.k, T = a.T;
    const int32_t *off = a.wv.blk_hist + static_cast<size_t>(blockIdx.x) * E;
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        s_eff[e] = a.wv.eff_slot[e];
        s_run[e] = off[e];
    }
    __syncthreads();
    const int p0 = blockIdx.x * kTokPerBlk * k;
    const int p1 = min(T, (blockIdx.x + 1) * kTokPerBlk) * k;
    scatter_run(p0, p1, k, a.nbits, a.ro.topk_ids, a.ro.topk_w, s_eff, s_run, a.ro, a.wv);
}

// ---------------------------------------------------------------------------------------

template <int NPL>
static hipError_t launch_route_npl(RouteArgs a, hipStream_t s) {
    const int P = a.T * a.k;
    const int fused_lds = fused_route_lds_bytes(a.E, P);
    if (P <= kFusedMaxPairs && fused_lds <= kFusedMaxLds) {
        hipLaunchKernelGGL(route_fused<NPL>, dim3(1), dim3(kFusedThreads), fused_lds, s, a);
        return hipGetLastError();
    }
    const int nblk = (a.T + kTokPerBlk - 1) / kTokPerBlk;
    a.scan_parts = max(1, min(1024 / a.E, nblk));
    hipLaunchKernelGGL(route_tokens<NPL>, dim3(nblk), dim3(256), 0, s, a);
    hipLaunchKernelGGL(route_scan, dim3(1), dim3(1024), scan_route_lds_bytes(a.E, a.scan_parts), s,
                       a, nblk);
    hipLaunchKernelGGL(route_scatter, dim3(nblk), dim3(64), 0, s, a);
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
