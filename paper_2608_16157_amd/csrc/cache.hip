// Device-side cache control for one MoE layer step (Section 3.2: the m missing experts split
// into q cache fills and m - q CPU executions, q* = m B_P / B_H, Eq. (dynamic-split), at least
// one fill, and a shared LRU residency space where a hit refreshes recency and a fill evicts the
// least recently demanded expert; Section 4.1: one kernel classifies the routed experts against
// the residency table, derives q, finds K least-recently-used candidate slots in a single pass,
// consumes the first q of them and rewrites routed ids into slot ids, leaving a fixed-shape copy
// list with a valid count).
//
// One workgroup, one thread per expert (E <= 1024).  Phases, separated by barriers:
//   1  cache state and per-expert demand into LDS (the routing's hit/miss offsets give, per
//      expert, the pairs that hit and the pairs that missed); every per-expert value the later
//      phases need is loaded here, in one batch, and kept in the thread's registers, so the
//      kernel waits on global memory once before its last phase;
//   2  every hit expert marks its slot as used in this step;
//   3  every evictable slot (not hit, not the shared expert's) gets its rank by
//      (age, slot id), age 0 for an empty slot and stamp + 1 otherwise; ranks below K are the
//      LRU candidates (up to 256 slots each slot counts the slots before it; larger pools sort
//      (age, slot id) keys with a bitonic network in LDS and take the first K).  Every missing
//      expert gets its rank by (demand desc, id asc);
//   4  q from m, B_P / B_H (double precision, rounded half up), K and the evictable count;
//   5  the expert of demand rank i < q takes candidate i: fill list, slot table, slot owner,
//      stamp and the routed pairs' slot ids are updated; the other missing experts are listed
//      for the CPU by ascending id; hit slots take the current step as stamp.
// The ranks are counts over all slots / experts (one pass each, no sort), so the result does not
// depend on thread timing.  A routing that flagged a faulty slot table changes nothing.
#include "ftmoe_device.h"
#include "ftmoe_internal.h"

namespace ftmoe {

constexpr int kPlanThreads = 1024;
static_assert(kMaxExperts <= kPlanThreads, "one thread per expert");
constexpr int kPlanCountSlots = 256;   // pools up to this size rank slots by counting

__host__ __device__ constexpr int pow2_at_least(int n) {
    int p = 1;
    while (p < n) p <<= 1;
    return p;
}

__global__ __launch_bounds__(kPlanThreads) void cache_plan_kernel(PlanArgs a) {
    extern __shared__ uint64_t plan_lds[];
    const int E = a.E, S = a.n_slots, K = a.K, tid = threadIdx.x;
    const bool sorted = S > kPlanCountSlots;
    const int SP = sorted ? pow2_at_least(S) : S;                    // key array length
    uint64_t *s_key = plan_lds;                                      // [SP] age key, ~0 = not evictable
    int32_t *s_owner = reinterpret_cast<int32_t *>(s_key + SP);      // [S] expert in the slot
    int32_t *s_dem = s_owner + S;                                    // [E] missed pairs, 0 = not missing
    int32_t *s_rank = s_dem + E;                                     // [E] demand rank of missing experts
    int32_t *s_cand = s_rank + E;                                    // [K] candidate slot by LRU rank
    int32_t *s_misc = s_cand + kPlanMaxFill;                         // [0] evictable count, [1] q
    constexpr uint64_t kNotEvictable = ~0ull;

    // ---- 1
    const int status = a.route_counts[3], m = a.route_counts[2];
    // the step's stamp: from the device clock when there is one (a captured step replays with
    // the same arguments), else from the call
    const uint32_t step = a.clock ? a.clock[0] + 1u : a.step;
    // this thread's expert e = tid: its missed pairs [mo0, mo1), whether it hit, its slot
    const int e_me = tid;
    const bool has_e = e_me < E;
    const int mo0 = has_e ? a.miss_off[e_me] : 0, mo1 = has_e ? a.miss_off[e_me + 1] : 0;
    const bool hit = has_e && a.hit_off[e_me + 1] > a.hit_off[e_me];
    const int slot_me = has_e ? a.slot_table[e_me] : -1;
    for (int s = tid; s < S; s += kPlanThreads) {
        s_owner[s] = a.slot_expert[s];
        s_key[s] = s == a.shared_slot ? kNotEvictable
                                      : (s_owner[s] < 0 ? 0ull : static_cast<uint64_t>(a.slot_stamp[s]) + 1ull);
    }
    if (has_e) s_dem[e_me] = mo1 - mo0;
    for (int s = S + tid; s < SP; s += kPlanThreads) s_key[s] = kNotEvictable;   // sort padding
    if (tid == 0) s_misc[0] = 0;
    __syncthreads();

    // ---- 2
    if (status == 0 && hit) s_key[slot_me] = kNotEvictable;
    __syncthreads();

    // ---- 3
    int nev = 0;
    if (!sorted) {
        for (int s = tid; s < S; s += kPlanThreads) {
            const uint64_t key = s_key[s];
            if (key == kNotEvictable) continue;
            ++nev;
            int rank = 0;
            for (int o = 0; o < S; ++o) {
                const uint64_t ko = s_key[o];
                rank += (ko < key) | ((ko == key) & (o < s));
            }
            if (rank < K) s_cand[rank] = s;
        }
    } else {
        // (age, slot id) in one key: ages are at most 2^32, slot ids below 4096
        for (int s = tid; s < S; s += kPlanThreads) {
            const uint64_t key = s_key[s];
            if (key == kNotEvictable) continue;
            ++nev;
            s_key[s] = (key << 12) | static_cast<uint64_t>(s);
        }
        __syncthreads();
        for (int size = 2; size <= SP; size <<= 1)
            for (int stride = size >> 1; stride > 0; stride >>= 1) {
                for (int i = tid; i < SP / 2; i += kPlanThreads) {
                    const int lo = 2 * i - (i & (stride - 1)), hi = lo + stride;
                    const uint64_t x = s_key[lo], y = s_key[hi];
                    if (((lo & size) == 0) == (x > y)) {
                        s_key[lo] = y;
                        s_key[hi] = x;
                    }
                }
                __syncthreads();
            }
        for (int r = tid; r < K; r += kPlanThreads)
            if (s_key[r] != kNotEvictable) s_cand[r] = static_cast<int>(s_key[r] & 0xFFF);
    }
    if (nev) atomicAdd(&s_misc[0], nev);
    for (int e = tid; e < E; e += kPlanThreads) {
        const int d = s_dem[e];
        if (d == 0) continue;
        int rank = 0;
        for (int o = 0; o < E; ++o) {
            const int dd = s_dem[o];
            rank += (dd > d) | ((dd == d) & (o < e));
        }
        s_rank[e] = rank;
    }
    __syncthreads();

    // ---- 4
    if (tid == 0) {
        if (a.clock) a.clock[0] = step;   // every thread read the clock before the first barrier
        int q = 0;
        if (status == 0 && m > 0) {
            q = a.b_host <= a.b_pcie ? m : static_cast<int>(floor(m * (a.b_pcie / a.b_host) + 0.5));
            q = max(1, q);
            q = min(min(q, m), min(K, s_misc[0]));
        }
        s_misc[1] = q;
        a.counts[0] = q;
        a.counts[1] = m - q;
        a.counts[2] = m;
        a.counts[3] = status;
    }
    __syncthreads();

    // ---- 5
    const int q = s_misc[1];
    if (has_e && mo1 > mo0) {
        const int e = e_me, i = s_rank[e];
        if (i < q) {
            const int v = s_cand[i], old = s_owner[v];
            a.fill_expert[i] = e;
            a.fill_slot[i] = v;
            a.evict_expert[i] = old;
            if (old >= 0) a.slot_table[old] = -1;
            a.slot_table[e] = v;
            a.slot_expert[v] = e;
            a.slot_stamp[v] = step;
            for (int j = mo0; j < mo1; ++j) a.topk_slot[a.miss_pairs[j]] = v;
        } else {
            // position among the missing experts left to the CPU, in id order
            int pos = 0;
            for (int o = 0; o < e; ++o) pos += (s_dem[o] > 0) & (s_rank[o] >= q);
            a.cpu_expert[pos] = e;
        }
    }
    if (status == 0 && hit) a.slot_stamp[slot_me] = step;   // hits keep their slot
    for (int i = q + tid; i < K; i += kPlanThreads) {
        a.fill_expert[i] = -1;
        a.fill_slot[i] = -1;
        a.evict_expert[i] = -1;
    }
    for (int i = m - q + tid; i < E; i += kPlanThreads) a.cpu_expert[i] = -1;
}

hipError_t launch_cache_plan(const PlanArgs &a, hipStream_t s) {
    const int sp = a.n_slots > kPlanCountSlots ? pow2_at_least(a.n_slots) : a.n_slots;
    const size_t lds = 8 * static_cast<size_t>(sp) + 4 * static_cast<size_t>(a.n_slots) +
                       8 * static_cast<size_t>(a.E) + 4 * (kPlanMaxFill + 2);
    hipLaunchKernelGGL(cache_plan_kernel, dim3(1), dim3(kPlanThreads), lds, s, a);
    return hipGetLastError();
}

}  // namespace ftmoe
