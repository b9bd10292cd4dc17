// Grouped SwiGLU expert evaluation over slot-resident weights (Section 3.2: grouped evaluation
// of the GPU execution set; Section 4.2: every bank row is one slot, so a group's weights are
// addressed as bank + slot * expert_stride with no relayout), and the gate-weighted combine.
//
// Streaming (GEMV-like) path, any token count and any weight dtype:
//   grouped_gemv<GATEUP>: h[r] = silu(W1 x_tok(r)) * (W3 x_tok(r))       per (group, 8 NB h columns)
//   grouped_gemv<DOWN>  : y[pair(r)] = gate(r) * W2 h[r]                 per (group, 16 NB columns)
//   combine             : out[t] = sum_j y[t k + j] over the pairs evaluated on the GPU, in
//                         j order, then the shared expert's row: every output element is summed
//                         in one fixed order, so the layer output is bit-reproducible
// With the atomic combine the down projection adds gate(r) * W2 h[r] into out[tok(r)] with
// float32 atomics instead (the gate/up kernel zeroes out first): one launch less.  In the
// optional fp8-activation mode x and h are quantised (quant.hip) and widened back to bf16 before
// the projections read them.
// A call of one or two tokens over 65 to 256 experts is routed inside the gate/up kernel: the
// first wave of every workgroup runs the one-wave router on the call's logits and slot table and
// the workgroup takes its group from LDS (workgroup 0 also writes the routing's outputs, which
// the down kernel and the combine read), so the layer needs no router launch (measured: Qwen3
// T = 1 layer 26.1 -> 23.5 us, DeepSeek-V4-Flash T = 1 34.8 -> 32.0 us).
// The weights stream from HBM once per (group, column tile).  Tokens of a group are the MFMA M
// dimension (16-row tiles), weight rows the N dimension; the contraction (hidden or intermediate
// dimension) is split over the 4 waves of a workgroup in contiguous runs of 128-wide blocks (the
// fp8 scale block), whose weight loads a wave issues in batches before any MFMA consumes them;
// the waves' partial sums are reduced through LDS.
#include "ftmoe_device.h"
#include "ftmoe_internal.h"
#include "route_wave.h"

#include <algorithm>
#include <type_traits>

namespace ftmoe {

// Tuning constants, chosen by sweeping them on MI355X.
// weight rows per work item = 16 * NB; fp8 and MXFP4 weights may take wider items (their bf16
// activation loads are 2 or 4 times the weight bytes per element, so one activation load should
// feed more rows once there are enough groups to fill the chip)
#ifndef FT_GEMV_NB
#define FT_GEMV_NB 2
#endif
// fp8 and MXFP4 take items of 2 or 4 blocks: the narrow ones spread few-token calls (few groups)
// over more workgroups
#ifndef FT_GEMV_NB_FP8
#define FT_GEMV_NB_FP8 4
#endif
// the fp8 down projection takes the wide items, two K blocks a batch, above this many tokens
// (measured at dsv3 T = 64: down 160 -> 152 us; at 1 and 16 tokens the narrow ones are faster)
#ifndef FT_GEMV_FP8_DN_WIDE_TOKENS
#define FT_GEMV_FP8_DN_WIDE_TOKENS 32
#endif
#ifndef FT_GEMV_NB_FP4
#define FT_GEMV_NB_FP4 4
#endif
#ifndef FT_GEMV_FP8_NARROW_PAIRS
#define FT_GEMV_FP8_NARROW_PAIRS 128   // T * k up to which fp8 gate/up items are narrow
#endif
#ifndef FT_GEMV_FP4_NARROW_PAIRS
#define FT_GEMV_FP4_NARROW_PAIRS 12    // same for MXFP4, both projections
#endif
#ifndef FT_GEMV_BF16_NARROW_TOKENS
#define FT_GEMV_BF16_NARROW_TOKENS 16  // T up to which bf16 items are one block (16 rows) wide
#endif
#ifndef FT_GEMV_MT_MAX
#define FT_GEMV_MT_MAX 2
#endif
#ifndef FT_GEMV_D_F32
#define FT_GEMV_D_F32 1
#endif
#ifndef FT_GEMV_D_BF16
#define FT_GEMV_D_BF16 1
#endif
// bf16 gate/up batch depth of the kernels with several M tiles a pass (more than 16 tokens): two
// K blocks a batch halve the workgroups per CU (LDS) and still keep more bytes in flight
// (measured +2 % on that kernel at Qwen3 T = 32; the down projection and the one-M-tile kernels
// lost with it)
#ifndef FT_GEMV_DGU_BF16
#define FT_GEMV_DGU_BF16 2
#endif
// the same for fp8 and MXFP4 stays at one K block: two measured +0.5 % and +2 % at 32 tokens,
// -7 % and -11 % in the four-M-tile kernels at 64 tokens (dsv3, dsv4flash decode)
#ifndef FT_GEMV_DGU_FP8
#define FT_GEMV_DGU_FP8 1
#endif
#ifndef FT_GEMV_DGU_FP4
#define FT_GEMV_DGU_FP4 1
#endif
#ifndef FT_GEMV_D_FP8
#define FT_GEMV_D_FP8 1
#endif
#ifndef FT_GEMV_D_FP4
#define FT_GEMV_D_FP4 1
#endif
// fp8 and MXFP4 batch depth of the one-M-tile kernels (few tokens): their smaller register and
// LDS footprint leaves room for two K blocks in flight per batch
#ifndef FT_GEMV_D1_FP8
#define FT_GEMV_D1_FP8 2
#endif
#ifndef FT_GEMV_D1_FP4
#define FT_GEMV_D1_FP4 2
#endif

constexpr int kGemvThreads = 256;
constexpr int kGemvWaves = kGemvThreads / kWave;

enum { EPI_GATEUP = 0, EPI_DOWN = 1 };

template <int WT> struct WTr;
// kLoads: 16-byte weight loads per lane per 128-wide K block; kBlock: bytes of one row's
// 128-wide K block; kBatch: K blocks in flight ahead (kBatch1 in the one-M-tile kernels, kBatchGU
// in the gate/up kernels with several M tiles a pass)
template <> struct WTr<FT_DT_F32> {
    static constexpr int kLoads = 8, kBlock = 512, kBatch = FT_GEMV_D_F32, kBatch1 = FT_GEMV_D_F32,
                         kBatchGU = FT_GEMV_D_F32;
};
template <> struct WTr<FT_DT_BF16> {
    static constexpr int kLoads = 4, kBlock = 256, kBatch = FT_GEMV_D_BF16, kBatch1 = FT_GEMV_D_BF16,
                         kBatchGU = FT_GEMV_DGU_BF16;
};
template <> struct WTr<FT_DT_FP8E4M3FN_B128> {
    static constexpr int kLoads = 2, kBlock = 128, kBatch = FT_GEMV_D_FP8, kBatch1 = FT_GEMV_D1_FP8,
                         kBatchGU = FT_GEMV_DGU_FP8;
};
template <> struct WTr<FT_DT_MXFP4> {
    static constexpr int kLoads = 1, kBlock = 64, kBatch = FT_GEMV_D_FP4, kBatch1 = FT_GEMV_D1_FP4,
                         kBatchGU = FT_GEMV_DGU_FP4;
};

__device__ __forceinline__ u32x4_t ld16(const void *p) {
    return *reinterpret_cast<const u32x4_t *>(p);
}

typedef __attribute__((address_space(3))) void gemv_lds_t;

// Weight staging through LDS: a wave copies its own K block of the item's weight
// rows into its own LDS region with global_load_lds, 16 bytes per lane and whole rows per
// instruction (a 16x16x32 MFMA operand read straight from global memory would take only 64 bytes
// of each of 16 rows per instruction), then reads the MFMA operands from there.  Within a row
// the 16-byte chunks are XOR-swizzled by the row so that the operand reads of 16 rows hit 16
// distinct bank groups: row bytes KB = 64 (MXFP4), 128 (fp8), 256 (bf16) or 512 (f32).  (Loading
// the operands into registers straight from global memory, with or without non-temporal hints,
// was measured slower.)
__device__ __forceinline__ void gemv_dma16(const void *g, uint8_t *lds) {
    __builtin_amdgcn_global_load_lds(g, (gemv_lds_t *)(lds), 16, 0, 0);
}

template <int KB>
__device__ __forceinline__ int wswz(int row, int chunk) {
    if constexpr (KB == 64) return chunk ^ ((row >> 2) & 3);
    else if constexpr (KB == 128) return chunk ^ ((row >> 1) & 7);
    else return chunk ^ (row & 15);
}


// Activation loads of one 128-wide K block for one 16-row M tile, 16 bytes each, at the K
// offsets the lane's weight operand uses (f32: 8 x 4 floats at c*16 + q*4; bf16: 4 x 8 at
// c*32 + q*8; fp8 weights widened to bf16: 4 x 8 at (c/2)*64 + q*16 + (c%2)*8; MXFP4 widened to
// bf16: 4 x 8 at q*32 + c*8).  `a_row` points
// at this lane's activation row offset to the K block; padding rows point at a real row and
// their results are never stored, so the loads need no branch.
template <int WT> struct ALd { static constexpr int n = WT == FT_DT_F32 ? 8 : 4; };

template <int WT>
__device__ __forceinline__ void aload(u32x4_t (&dst)[ALd<WT>::n], const uint8_t *a_row, int q) {
#pragma unroll
    for (int c = 0; c < ALd<WT>::n; ++c) {
        int ofs;
        if constexpr (WT == FT_DT_F32) ofs = (c * 16 + q * 4) * 4;
        else if constexpr (WT == FT_DT_BF16) ofs = (c * 32 + q * 8) * 2;
        else if constexpr (WT == FT_DT_MXFP4) ofs = (q * 32 + c * 8) * 2;
        else ofs = ((c >> 1) * 64 + q * 16 + (c & 1) * 8) * 2;
        dst[c] = ld16(a_row + ofs);
    }
}

// acc += A(rows, kblock) * B(kblock, 16 cols) for one 16-row M tile.  `av` from aload; `w` the
// lane's weight operand of the block (for fp8 already widened to 4 x 8 bf16).
template <int WT>
__device__ __forceinline__ void mfma_kblock(const u32x4_t (&av)[ALd<WT>::n], const u32x4_t *w,
                                            floatx4_t &acc) {
    if constexpr (WT == FT_DT_F32) {
#pragma unroll
        for (int c = 0; c < 8; ++c)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(av[c][i]),
                                                           __uint_as_float(w[c][i]), acc, 0, 0, 0);
    } else {
#pragma unroll
        for (int c = 0; c < 4; ++c)
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(av[c]), as_bf16x8(w[c]), acc, 0, 0, 0);
    }
}

// One work item = (group, NB x 16 weight rows).  The 4 waves of the workgroup split the item's
// K blocks into contiguous quarters and meet in LDS (KSP = 4), or, when the K blocks do not split
// evenly four ways (Qwen3's down projection: 6 blocks), pairs of waves take half of the item's
// weight blocks each and split their K blocks in halves (KSP = 2), so no wave idles; rows of the
// group are taken 16 at a time,
// up to MTX M tiles per pass (MTX = 1 when no group can hold more than 16 rows, which keeps the
// register count, and so the occupancy, of few-token calls down).  Each activation load feeds
// the NB weight blocks of the item.
// Workgroups per CU the bf16 kernels are held to (128 registers a lane, no spills): one more
// than the register count the compiler picks by itself allows; two for the gate/up kernels whose
// deeper batches fill that much LDS.  The fp8 and MXFP4 kernels would spill under the same bound
// and keep the compiler's choice.
template <int WT, int EPI, int MTX> constexpr int gemv_min_blocks() {
    return WT != FT_DT_BF16 ? 1 : (EPI == EPI_GATEUP && MTX > 1 && FT_GEMV_DGU_BF16 > 1 ? 2 : 4);
}

// RNPL > 0 (gate/up of one or two tokens): the workgroup routes the call itself first, with its
// first wave (route_wave_body, RNPL experts per lane), instead of reading the groups a router
// kernel wrote: the routing's global outputs come from workgroup 0, every workgroup takes its own
// group and rows from LDS.  This saves the router's launch and its dependent global reads.
template <int WT, int EPI, int NB, int MTX, int KSP = kGemvWaves, int RNPL = 0>
__global__ __launch_bounds__(kGemvThreads, (gemv_min_blocks<WT, EPI, MTX>())) void grouped_gemv(ExpertArgs a, int tiles) {
    static_assert(RNPL == 0 || (EPI == EPI_GATEUP && MTX == 1 && RNPL <= kWaveRouteMaxNpl), "self-routing");
    static_assert(KSP == kGemvWaves || (KSP == 2 && NB % 2 == 0), "K split: 4 waves, or 2 with an even block count");
    constexpr int NBW = NB * KSP / kGemvWaves;   // weight blocks of each wave
    // the deeper batch of the one-M-tile kernels is used where the registers allow it (not by
    // the wide fp8 items)
    constexpr int D = (MTX == 1 && (WT != FT_DT_FP8E4M3FN_B128 || NB == 2))
                          ? WTr<WT>::kBatch1
                          : (MTX > 1 && EPI == EPI_GATEUP
                                 ? WTr<WT>::kBatchGU
                                 : (WT == FT_DT_FP8E4M3FN_B128 && EPI == EPI_DOWN && NB == 4 ? 2 : WTr<WT>::kBatch));
    constexpr int NL = WTr<WT>::kLoads, NA = ALd<WT>::n;
    constexpr int COLS = NB * 16;
    constexpr int KB = WTr<WT>::kBlock;                        // bytes of one row's K block
    constexpr int STAGE = D * NBW * 16 * KB;                  // per wave
    constexpr int REDW = 16 * (COLS + 1) * 4;                  // one wave's partial sums
    constexpr int PW = ((STAGE > REDW ? STAGE : REDW) + 255) / 256 * 256;
    // A wave writes its partial sums into its own staging area once its own K range is done (its
    // staged rows have all been read into registers by then); the area stays private to the wave
    // until the barrier, while other waves may still be streaming into theirs.
    __shared__ __attribute__((aligned(1024))) uint8_t s_lds[kGemvWaves * PW];
    auto s_red = [&](int w) { return reinterpret_cast<float (*)[COLS + 1]>(s_lds + w * PW); };
    if (EPI == EPI_GATEUP && !a.wv.ypart) {
        // atomic combine: zero the output the down projection adds into
        const size_t n4 = static_cast<size_t>(a.T) * a.H / 4;
        float4 *o4 = reinterpret_cast<float4 *>(a.out);
        for (size_t i = static_cast<size_t>(blockIdx.x) * kGemvThreads + threadIdx.x; i < n4;
             i += static_cast<size_t>(gridDim.x) * kGemvThreads)
            o4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    const int g = blockIdx.x / tiles, tile = blockIdx.x % tiles;
    int slot, beg, len;
    const int32_t *s_rtok = nullptr;   // self-routing: the token of each evaluation row (LDS)
    if constexpr (RNPL > 0) {
        extern __shared__ int32_t s_route[];
        const int ncnt = a.n_slots <= kSlotCountCap ? a.n_slots : 0;
        int32_t *sk = s_route + route_wave_lds_bytes(a.E, ncnt) / 4;
        const WaveRouteSink sink{sk, sk + 1, sk + 1 + (kWave + 1), sk + 1 + 2 * (kWave + 1), sk + 1 + 3 * (kWave + 1)};
        const RouteArgs ra{a.logits, a.slot_table, a.T, a.E, a.k, a.gating, a.n_slots, a.shared_slot, a.nbits, 1,
                           a.ro, a.wv};
        if (threadIdx.x < kWave) route_wave_body<RNPL, true>(ra, s_route, blockIdx.x == 0, sink);
        __syncthreads();
        if (g >= *sink.G) return;
        slot = sink.slot[g];
        beg = sink.beg[g];
        len = sink.len[g];
        s_rtok = sink.row_tok;
    } else {
        if (g >= a.wv.grp_meta[0]) return;
        slot = a.wv.grp_slot[g];
        beg = a.wv.grp_beg[g];
        len = a.wv.grp_len[g];
    }
    const int H = a.H, I = a.I;
    const int K = EPI == EPI_GATEUP ? H : I;
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int n = lane & 15, q = lane >> 4;
    const int bw0 = (wave / KSP) * NBW, kw = wave % KSP;   // first block and K part of this wave
    const int nrows = EPI == EPI_GATEUP ? 2 * I : H;
    const int nkb = K / 128;
    // weight row of this lane's N column in block b: a gate/up block pairs 8 gate rows with the
    // 8 matching up rows, so SiLU(gate) * up of one h column stays inside the block
    const size_t row_bytes = static_cast<size_t>(nkb) * KB;
    const float *sbase[NBW];     // fp8: the row's 128 x 128 block scales
    const uint8_t *xbase[NBW];   // MXFP4: this lane's e8m0 scale of the row in K block 0
#pragma unroll
    for (int b = 0; b < NBW; ++b) {
        const int col0 = (tile * NB + bw0 + b) * (EPI == EPI_GATEUP ? 8 : 16);
        const int wrow = EPI == EPI_GATEUP ? (n < 8 ? col0 + n : I + col0 + n - 8) : col0 + n;
        sbase[b] = nullptr;
        xbase[b] = nullptr;
        if constexpr (WT == FT_DT_FP8E4M3FN_B128)
            sbase[b] = static_cast<const float *>(EPI == EPI_GATEUP ? a.s13 : a.s2) +
                       (static_cast<size_t>(slot) * (nrows / 128) + wrow / 128) * nkb;
        if constexpr (WT == FT_DT_MXFP4)   // run-major scales: run 4 kb + q of row wrow
            xbase[b] = static_cast<const uint8_t *>(EPI == EPI_GATEUP ? a.s13 : a.s2) +
                       (static_cast<size_t>(slot) * (K / 32) + q) * nrows + wrow;
    }
    // global_load_lds sources: instruction c of block b covers rows [c * RPI, c * RPI + RPI) of
    // the block's 16, LPR lanes per row; lane i fills LDS chunk i % LPR of its row, so it fetches
    // the chunk the swizzle puts there
    constexpr int LPR = KB / 16, RPI = 64 / LPR;
    static_assert(RPI * NL == 16, "one block is NL whole-row instructions");
    const uint8_t *dsrc[NBW][NL];
#pragma unroll
    for (int b = 0; b < NBW; ++b)
#pragma unroll
        for (int c = 0; c < NL; ++c) {
            const int j = c * RPI + lane / LPR;
            const int col0 = (tile * NB + bw0 + b) * (EPI == EPI_GATEUP ? 8 : 16);
            const int wr = EPI == EPI_GATEUP ? (j < 8 ? col0 + j : I + col0 + j - 8) : col0 + j;
            dsrc[b][c] = static_cast<const uint8_t *>(EPI == EPI_GATEUP ? a.w13 : a.w2) +
                         (static_cast<size_t>(slot) * nrows + wr) * row_bytes + wswz<KB>(j, lane % LPR) * 16;
        }
    uint8_t *wst = s_lds + wave * PW;
    const size_t a_elem = (WT == FT_DT_F32) ? 4 : 2;
    const int per = (nkb + KSP - 1) / KSP;
    const int kb0 = min(nkb, kw * per), kb1 = min(nkb, kb0 + per);

    // One pass over the K blocks for MT 16-row M tiles starting at row r0 (MT chosen per pass).
    auto pass = [&](auto mt_const, int r0, floatx4_t (&acc)[MTX][NBW]) {
        constexpr int MT = decltype(mt_const)::value;
        const uint8_t *arow[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            // this lane's activation row; padding rows repeat the last row (their sums are dropped)
            const int rr = min(len - 1, r0 + mt * 16 + n);
            if constexpr (EPI == EPI_GATEUP)
                arow[mt] = static_cast<const uint8_t *>(a.x) +
                           static_cast<size_t>(RNPL > 0 ? s_rtok[beg + rr] : a.wv.row_tok[beg + rr]) * H * a_elem;
            else
                arow[mt] = static_cast<const uint8_t *>(a.wv.h) + static_cast<size_t>(beg + rr) * I * a_elem;
        }
        // Each iteration issues every load of a batch of D K blocks (activations, weights, fp8
        // scales) before any MFMA consumes them, and consumes them all before the next batch:
        // no load is carried across the loop back-edge (the wait-count insertion would drain
        // such a pipeline at the loop header) and no load sits under a branch (the tail batch
        // re-reads the last block and multiplies its contribution by zero).  The scheduling
        // barrier keeps the compiler from interleaving the loads with the MFMAs that use them.
        for (int kbb = kb0; kbb < kb1; kbb += D) {
            u32x4_t av[D][MT][NA];
            u32x4_t wv[D][NBW][NL];
            float sv[D][NBW];
            uint32_t xv[D][NBW];
#pragma unroll
            for (int d = 0; d < D; ++d) {
                const int kb = min(kbb + d, kb1 - 1);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    aload<WT>(av[d][mt], arow[mt] + static_cast<size_t>(kb) * 128 * a_elem, q);
#pragma unroll
                for (int b = 0; b < NBW; ++b) {
#pragma unroll
                    for (int c = 0; c < NL; ++c)
                        gemv_dma16(dsrc[b][c] + static_cast<size_t>(kb) * KB, wst + ((d * NBW + b) * 16 * KB + c * 1024));
                    if constexpr (WT == FT_DT_FP8E4M3FN_B128) sv[d][b] = sbase[b][kb];
                    if constexpr (WT == FT_DT_MXFP4) xv[d][b] = xbase[b][static_cast<size_t>(kb) * 4 * nrows];
                }
            }
            {
                // this wave's staged rows have landed (its own DMA: no barrier needed); lane
                // (n, q)'s operand chunk c is chunk 4 c + q of row n
                __builtin_amdgcn_s_waitcnt(0x0 | (0x7 << 4) | (0xF << 8) | (0x0 << 14));   // vmcnt(0)
                asm volatile("" ::: "memory");
#pragma unroll
                for (int d = 0; d < D; ++d)
#pragma unroll
                    for (int b = 0; b < NBW; ++b)
#pragma unroll
                        for (int c = 0; c < NL; ++c)
                            wv[d][b][c] = *reinterpret_cast<const u32x4_t *>(
                                wst + (d * NBW + b) * 16 * KB + n * KB + wswz<KB>(n, 4 * c + q) * 16);
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int d = 0; d < D; ++d) {
                const float keep = kbb + d < kb1 ? 1.f : 0.f;
#pragma unroll
                for (int b = 0; b < NBW; ++b) {
                    u32x4_t wc[4];
                    if constexpr (WT == FT_DT_FP8E4M3FN_B128) {
                        wc[0] = fp8x8_to_bf16x8(wv[d][b][0][0], wv[d][b][0][1]);
                        wc[1] = fp8x8_to_bf16x8(wv[d][b][0][2], wv[d][b][0][3]);
                        wc[2] = fp8x8_to_bf16x8(wv[d][b][1][0], wv[d][b][1][1]);
                        wc[3] = fp8x8_to_bf16x8(wv[d][b][1][2], wv[d][b][1][3]);
                    }
                    if constexpr (WT == FT_DT_MXFP4) {
                        // the lane's 32 codes share the scale of its 32-value run q
                        const float xs = fp4_scale_operand(xv[d][b]);
#pragma unroll
                        for (int i = 0; i < 4; ++i) wc[i] = fp4x8_scaled_to_bf16x8(wv[d][b][0][i], xs);
                    }
                    const float sc = keep * (WT == FT_DT_FP8E4M3FN_B128 ? sv[d][b] : 1.f);
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        floatx4_t part{0.f, 0.f, 0.f, 0.f};
                        if constexpr (WT == FT_DT_FP8E4M3FN_B128 || WT == FT_DT_MXFP4) mfma_kblock<WT>(av[d][mt], wc, part);
                        else mfma_kblock<WT>(av[d][mt], wv[d][b], part);
#pragma unroll
                        for (int i = 0; i < 4; ++i) acc[mt][b][i] += sc * part[i];
                    }
                }
            }
        }
    };

    for (int r0 = 0; r0 < len; r0 += 16 * MTX) {
        floatx4_t acc[MTX][NBW];
#pragma unroll
        for (int mt = 0; mt < MTX; ++mt)
#pragma unroll
            for (int b = 0; b < NBW; ++b) acc[mt][b] = floatx4_t{0.f, 0.f, 0.f, 0.f};
        const int nmt = min(MTX, (len - r0 + 15) / 16);
        if constexpr (MTX > 1) {
            if (nmt > 1) pass(std::integral_constant<int, MTX>{}, r0, acc);
            else pass(std::integral_constant<int, 1>{}, r0, acc);
        } else {
            pass(std::integral_constant<int, 1>{}, r0, acc);
        }

        // lane (n, q) holds rows 4q + i of column n of each of the wave's blocks; the KSP K parts
        // of a block meet in LDS
        for (int mt = 0; mt < nmt; ++mt) {
            const int rt = r0 + mt * 16;
#pragma unroll
            for (int b = 0; b < NBW; ++b)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float v = acc[0][b][i];
#pragma unroll
                    for (int j = 1; j < MTX; ++j)
                        if (j == mt) v = acc[j][b][i];
                    s_red(wave)[4 * q + i][(bw0 + b) * 16 + n] = v;
                }
            __syncthreads();
            if constexpr (EPI == EPI_GATEUP) {
                // 16 rows x NB*8 h columns
                for (int idx = threadIdx.x; idx < 16 * NB * 8; idx += kGemvThreads) {
                    const int m = idx / (NB * 8), cc = idx % (NB * 8), b = cc / 8, c = cc % 8;
                    const int r = rt + m;
                    if (r < len) {
                        float gs = 0.f, us = 0.f;
                        const int w0 = (b / NBW) * KSP;   // the waves that hold block b
#pragma unroll
                        for (int w = 0; w < KSP; ++w) {
                            gs += s_red(w0 + w)[m][b * 16 + c];
                            us += s_red(w0 + w)[m][b * 16 + c + 8];
                        }
                        const float hv = silu_f32(gs) * us;
                        const size_t o = static_cast<size_t>(beg + r) * I + (tile * NB + b) * 8 + c;
                        if constexpr (WT == FT_DT_F32) static_cast<float *>(a.wv.h)[o] = hv;
                        else static_cast<uint16_t *>(a.wv.h)[o] = f32_to_bf16(hv);
                    }
                }
            } else {
                // gate-weighted outputs of 16 rows x NB*16 columns, stored by pair index
                for (int idx = threadIdx.x; idx < 16 * COLS; idx += kGemvThreads) {
                    const int m = idx / COLS, c = idx % COLS;
                    const int r = rt + m;
                    if (r < len) {
                        float sum = 0.f;
                        const int w0 = (c / 16 / NBW) * KSP;
#pragma unroll
                        for (int w = 0; w < KSP; ++w) sum += s_red(w0 + w)[m][c];
                        const float y = a.wv.row_gate[beg + r] * sum;
                        if (a.wv.ypart) {
                            const int p = a.wv.row_pair[beg + r];
                            a.wv.ypart[static_cast<size_t>(p) * H + tile * COLS + c] = y;
                        } else {
                            const int tok = a.wv.row_tok[beg + r];
                            unsafeAtomicAdd(a.out + static_cast<size_t>(tok) * H + tile * COLS + c, y);
                        }
                    }
                }
            }
            __syncthreads();
        }
    }
}

__global__ __launch_bounds__(256) void zero_out(float *out, size_t n4) {
    float4 *o4 = reinterpret_cast<float4 *>(out);
    for (size_t i = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x; i < n4;
         i += static_cast<size_t>(gridDim.x) * 256)
        o4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
}

// out[t] = sum over j of y[t k + j] for the pairs evaluated on the GPU (routed slot >= 0), in
// ascending j, then + y[T k + t] for the shared expert; tokens without any are exactly 0.
__global__ __launch_bounds__(256) void combine_kernel(float *out, const float *y, const int32_t *topk_slot,
                                                      int T, int k, int H, int shared) {
    constexpr int U = 8;   // pairs whose loads are issued together (no load waits on a branch)
    const int h4 = H / 4;
    const size_t n4 = static_cast<size_t>(T) * h4;
    const float4 *y4 = reinterpret_cast<const float4 *>(y);
    for (size_t i = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x; i < n4;
         i += static_cast<size_t>(gridDim.x) * 256) {
        const int t = static_cast<int>(i / h4), c = static_cast<int>(i % h4);
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int j0 = 0; j0 < k; j0 += U) {
            int sl[U];
            float4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) sl[u] = j0 + u < k ? topk_slot[t * k + j0 + u] : -1;
            // rows of pairs not evaluated on the GPU (or past k) are read but never added
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int p = t * k + min(j0 + u, k - 1);
                v[u] = y4[static_cast<size_t>(p) * h4 + c];
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (sl[u] >= 0) {
                    acc.x += v[u].x;
                    acc.y += v[u].y;
                    acc.z += v[u].z;
                    acc.w += v[u].w;
                }
            }
        }
        if (shared) {
            const float4 v = y4[(static_cast<size_t>(T) * k + t) * h4 + c];
            acc.x += v.x;
            acc.y += v.y;
            acc.z += v.z;
            acc.w += v.w;
        }
        reinterpret_cast<float4 *>(out)[i] = acc;
    }
}

// The self-routing gate/up kernel of a one- or two-token call (self_route_ok): two or four
// experts per router lane.
template <int WT, int NB, int KSP>
static void launch_gemv_routed(const ExpertArgs &a, hipStream_t s, int tiles) {
    const int ncnt = a.n_slots <= kSlotCountCap ? a.n_slots : 0;
    const size_t lds = static_cast<size_t>(route_wave_lds_bytes(a.E, ncnt)) + kWaveRouteSinkBytes;
    const dim3 grid(a.max_groups * tiles), blk(kGemvThreads);
    if (a.E <= 2 * kWave)
        hipLaunchKernelGGL((grouped_gemv<WT, EPI_GATEUP, NB, 1, KSP, 2>), grid, blk, lds, s, a, tiles);
    else
        hipLaunchKernelGGL((grouped_gemv<WT, EPI_GATEUP, NB, 1, KSP, 4>), grid, blk, lds, s, a, tiles);
}

template <int WT, int EPI>
static void launch_gemv(const ExpertArgs &a, hipStream_t s) {
    auto go = [&](auto nb) {
        constexpr int NB = decltype(nb)::value;
        const int tiles = EPI == EPI_GATEUP ? a.I / (8 * NB) : a.H / (16 * NB);
        const int nkb = (EPI == EPI_GATEUP ? a.H : a.I) / 128;
        const bool ksp2 = nkb % kGemvWaves != 0 && nkb % 2 == 0;
        auto run = [&](auto mtx) {
            constexpr int MTX = decltype(mtx)::value;
            if constexpr (EPI == EPI_GATEUP && MTX == 1) {
                if (a.logits) {
                    if constexpr (NB % 2 == 0)
                        if (ksp2) return launch_gemv_routed<WT, NB, 2>(a, s, tiles);
                    return launch_gemv_routed<WT, NB, kGemvWaves>(a, s, tiles);
                }
            }
            if constexpr (NB % 2 == 0) {
                if (ksp2) {
                    hipLaunchKernelGGL((grouped_gemv<WT, EPI, NB, MTX, 2>), dim3(a.max_groups * tiles),
                                       dim3(kGemvThreads), 0, s, a, tiles);
                    return;
                }
            }
            hipLaunchKernelGGL((grouped_gemv<WT, EPI, NB, MTX>), dim3(a.max_groups * tiles), dim3(kGemvThreads), 0,
                               s, a, tiles);
        };
        // a group holds at most T rows (the shared expert's group exactly T).  The wide fp8
        // gate/up items take four M tiles per pass above 32 tokens: a group of up to 64 rows
        // then streams its weights once, at no cost in occupancy (their register count allows
        // two waves per SIMD either way); measured +4 % on that kernel at dsv3 T = 64.  The wide
        // MXFP4 gate/up items do so from 64 tokens (their occupancy halves: measured -1 % at
        // T = 48, +1 % at T = 64, +4 % at T = 128).
        if (a.T <= 16) {
            run(std::integral_constant<int, 1>{});
            return;
        }
        if constexpr ((WT == FT_DT_FP8E4M3FN_B128 || WT == FT_DT_MXFP4) && EPI == EPI_GATEUP && NB == 4) {
            if (a.T >= (WT == FT_DT_MXFP4 ? 64 : 33)) {
                run(std::integral_constant<int, 4>{});
                return;
            }
        }
        run(std::integral_constant<int, FT_GEMV_MT_MAX>{});
    };
    const int pairs = a.T * a.k;
    if constexpr (WT == FT_DT_FP8E4M3FN_B128) {
        if constexpr (EPI == EPI_DOWN) {
            if (a.T > FT_GEMV_FP8_DN_WIDE_TOKENS) go(std::integral_constant<int, 4>{});
            else go(std::integral_constant<int, 2>{});
        }
        else if (pairs <= FT_GEMV_FP8_NARROW_PAIRS) go(std::integral_constant<int, 2>{});
        else go(std::integral_constant<int, FT_GEMV_NB_FP8>{});
    } else if constexpr (WT == FT_DT_MXFP4) {
        if (pairs <= FT_GEMV_FP4_NARROW_PAIRS) go(std::integral_constant<int, 2>{});
        else go(std::integral_constant<int, FT_GEMV_NB_FP4>{});
    } else if constexpr (WT == FT_DT_BF16) {
        // one-block items double the workgroups of few-token calls: measured +5 % at Qwen3 T = 2,
        // +3 % at T = 4 and 8, -1 % at T = 32
        if (a.T <= FT_GEMV_BF16_NARROW_TOKENS) go(std::integral_constant<int, 1>{});
        else go(std::integral_constant<int, FT_GEMV_NB>{});
    } else {
        go(std::integral_constant<int, FT_GEMV_NB>{});
    }
}

template <int WT>
static hipError_t launch_stream_path(const ExpertArgs &a, hipStream_t s, const Prof &prof) {
    // the combine is a kernel of its own: folding it into the down kernel's last workgroup per
    // column tile needed a device-scope fence in every workgroup, whose L2 writeback on this
    // multi-XCD part cost far more than the launch (measured: Qwen3 T = 32 down 26 -> 395 us)
    const size_t n4 = static_cast<size_t>(a.T) * a.H / 4;
    const unsigned blocks = static_cast<unsigned>(std::min<size_t>(2048, (n4 + 255) / 256));
    if (!prof.mark(1)) return hipErrorUnknown;
    // fp8 activations: the GEMVs read x and h quantised and widened back to bf16
    ExpertArgs ag = a;
    if (a.act_quant && a.max_groups > 0) {
        if (hipError_t e = launch_act_quant_x(a, s); e != hipSuccess) return e;
        ag.x = a.wv.xd;
    }
    if (a.max_groups > 0) launch_gemv<WT, EPI_GATEUP>(ag, s);
    else if (!a.wv.ypart) hipLaunchKernelGGL(zero_out, dim3(blocks), dim3(256), 0, s, a.out, n4);
    if (a.act_quant && a.max_groups > 0)
        if (hipError_t e = launch_act_quant_h(a, s); e != hipSuccess) return e;
    if (!prof.mark(2)) return hipErrorUnknown;
    if (a.max_groups > 0) launch_gemv<WT, EPI_DOWN>(a, s);
    if (!prof.mark(3)) return hipErrorUnknown;
    if (a.wv.ypart)
        hipLaunchKernelGGL(combine_kernel, dim3(blocks), dim3(256), 0, s, a.out, a.wv.ypart, a.ro.topk_slot, a.T,
                           a.k, a.H, a.shared);
    return hipGetLastError();
}

// Many-token chunks whose shapes tile evenly go to the MFMA GEMM.
static bool gemm_path(const ExpertArgs &a) { return a.max_groups > 0 && gemm_shape(a.T, a.H, a.I, a.w_dtype); }

hipError_t launch_experts(const ExpertArgs &a, hipStream_t s, const Prof &prof) {
    switch (a.w_dtype) {
        case FT_DT_F32: return launch_stream_path<FT_DT_F32>(a, s, prof);
        case FT_DT_BF16:
            if (gemm_path(a)) return launch_gemm(a, s, prof);
            return launch_stream_path<FT_DT_BF16>(a, s, prof);
        case FT_DT_MXFP4:
            if (gemm_path(a)) return launch_gemm(a, s, prof);
            return launch_stream_path<FT_DT_MXFP4>(a, s, prof);
        default:
            if (gemm_path(a)) return launch_gemm(a, s, prof);
            return launch_stream_path<FT_DT_FP8E4M3FN_B128>(a, s, prof);
    }
}

}  // namespace ftmoe
