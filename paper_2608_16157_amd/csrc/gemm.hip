// Grouped expert GEMM on MFMA tiles for many-token chunks (prefill): bf16 or fp8 weights,
// bf16 activations, float32 accumulation.
//
// The same two projections as the streaming path (Section 3.2, grouped evaluation of the GPU
// execution set; weights addressed through the slot, Section 4.2), shaped for matrix-core reuse:
//   gate/up: h[rows of g] = silu(X_g W1^T) * (X_g W3^T)       tile = BM rows x BN/2 h columns
//   down   : out[tok] += gate * (h_g W2^T)                    tile = BM rows x BN out columns
//
// Work decomposition.  One workgroup (8 waves, BM/64 x BN/64 over the tile, 64 x 64 each as
// 2 x 2 MFMA 32x32x16 tiles, the bf16 MFMA shape with the highest measured throughput on
// gfx950) per (group, BM-row M tile, N tile).  Tiles are enumerated on the device from
// the per-group M-tile prefix the router writes: group-major, then N tile, then M tile, so the
// M tiles sharing a weight tile run back to back, and the block -> tile map keeps consecutive
// tiles on one XCD (workgroups are dealt to the 8 XCDs round-robin) to share its L2.
//
// Data movement.  A (activation rows, gathered through row_tok for gate/up) and B (weight rows,
// kept in their storage format: bf16, or fp8 widened to bf16 only when read for the MFMA) go
// straight from global memory into LDS with global_load_lds (16 bytes per lane), through a ring
// of 3 stages of 64 K each, two stages in flight while one is multiplied.  Every LDS row keeps
// its 16-byte chunks XOR-swizzled by the row index, so MFMA operand reads of consecutive rows
// hit distinct banks.  The stage hand-off is an explicit vmcnt wait plus s_barrier (a
// __syncthreads would drain every in-flight stage).
//
// fp8 weights carry one float32 scale per 128 x 128 block: partial sums of each 128-wide K
// block are scaled once and added to the accumulators.  The gate/up B tile puts each wave's 32
// gate rows next to the 32 matching up rows, so SiLU(gate) * up is formed in registers.
#include "ftmoe_device.h"
#include "ftmoe_internal.h"

namespace ftmoe {

constexpr int kBM = kGemmBM;          // token rows per tile
constexpr int kBN = kGemmBN;          // weight rows per tile
constexpr int kWavesN = kBN / 64;     // waves across N, 64 columns each
constexpr int kWavesM = kBM / 64;     // waves across M, 64 rows each
constexpr int kBK = 64;               // K elements per stage
constexpr int kStages = 3;
constexpr int kGemmThreads = 512;
constexpr int kGemmWaves = kGemmThreads / kWave;
constexpr int kARowBytes = kBK * 2;   // bf16 activations: 128 bytes per row per stage
constexpr int kAStage = kBM * kARowBytes;
static_assert(kWavesN * kWavesM == kGemmThreads / 64, "8 waves of 64 x 64");

enum { GEMM_GATEUP = 0, GEMM_DOWN = 1 };

template <int WT> struct GTr;
template <> struct GTr<FT_DT_BF16> {
    static constexpr int kRowBytes = kBK * 2;          // 128
    static constexpr int kChunks = kRowBytes / 16;     // 8 chunks per row
    static constexpr int kBStage = kBN * kRowBytes;
    static constexpr int kBInstr = kBStage / 1024 / kGemmWaves;   // DMA instructions per wave
};
template <> struct GTr<FT_DT_FP8E4M3FN_B128> {
    static constexpr int kRowBytes = kBK;              // 64
    static constexpr int kChunks = kRowBytes / 16;     // 4
    static constexpr int kBStage = kBN * kRowBytes;
    static constexpr int kBInstr = kBStage / 1024 / kGemmWaves;
};
constexpr int kAInstr = kAStage / 1024 / kGemmWaves;

// Block index -> logical tile index such that logical tiles [x*q + min(x,r), ...) run on XCD x.
__device__ __forceinline__ int xcd_remap(int b, int n) {
    const int q = n / 8, r = n % 8, x = b % 8, i = b / 8;
    return x * q + min(x, r) + i;
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}
__device__ __forceinline__ void wait_lgkmcnt0() {
    __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x0 << 8) | (0x3 << 14));
}

typedef __attribute__((address_space(3))) void lds_void_t;

// Workgroup barrier between pipeline stages.  The empty asm statements are compiler-level memory
// fences: they keep LDS reads of a stage from being moved across the barrier, without the
// wait-for-everything a __syncthreads fence would add.
__device__ __forceinline__ void stage_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// 16-byte chunk position of chunk c in LDS row r.  A 128-byte row covers half of the 64 x 4-byte
// banks, so rows r and r+1 already sit in opposite halves; XOR with (r / 2) mod 8 then gives the
// 16 rows an MFMA operand read touches 16 distinct bank groups.  A 64-byte (fp8) row covers a
// quarter of the banks, hence (r / 4) mod 4.
__device__ __forceinline__ int swz128(int r, int c) { return c ^ ((r >> 1) & 7); }
__device__ __forceinline__ int swz64(int r, int c) { return c ^ ((r >> 2) & 3); }

__device__ __forceinline__ void dma16(const void *g, uint8_t *lds_block) {
    __builtin_amdgcn_global_load_lds(g, (lds_void_t *)(lds_block), 16, 0, 0);
}

template <int WT, int EPI>
__global__ __launch_bounds__(kGemmThreads, 1) void grouped_gemm(ExpertArgs a, int ntn) {
    using Tr = GTr<WT>;
    // three separately declared stage buffers: with the loop unrolled by three every LDS read and
    // every DMA target is a distinct object, so the compiler's wait-count pass can tell that the
    // stage being read does not alias the stages still being written
    __shared__ __attribute__((aligned(1024))) uint8_t sA0[kAStage], sA1[kAStage], sA2[kAStage];
    __shared__ __attribute__((aligned(1024))) uint8_t sB0[Tr::kBStage], sB1[Tr::kBStage], sB2[Tr::kBStage];
    static_assert(kStages == 3, "the stage ring is unrolled by three");
    const int t = threadIdx.x;
    if constexpr (EPI == GEMM_GATEUP) {
        // zero the output that the down projection accumulates into
        const size_t n4 = static_cast<size_t>(a.T) * a.H / 4;
        float4 *o4 = reinterpret_cast<float4 *>(a.out);
        for (size_t i = static_cast<size_t>(blockIdx.x) * kGemmThreads + t; i < n4;
             i += static_cast<size_t>(gridDim.x) * kGemmThreads)
            o4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    const int L = xcd_remap(blockIdx.x, gridDim.x);
    const int MTT = a.wv.grp_meta[4];
    if (L >= MTT * ntn) return;
    // tiles run M-tile-major with the N tile fastest: the N tiles of one M tile (sharing its
    // activation rows) and the M tiles of one group (sharing its weight tiles) sit close together
    const int mtg = L / ntn, nt = L % ntn;
    const int g = a.wv.mt_group[mtg];
    const int mt = mtg - a.wv.grp_mt_off[g];
    const int slot = a.wv.grp_slot[g], beg = a.wv.grp_beg[g], len = a.wv.grp_len[g];
    const int H = a.H, I = a.I;
    const int K = EPI == GEMM_GATEUP ? H : I;
    const int nrows = EPI == GEMM_GATEUP ? 2 * I : H;
    const int m0 = mt * kBM;
    const int wave = __builtin_amdgcn_readfirstlane(t / kWave), lane = lane_id();

    // ---- DMA sources: this lane's rows in each of its 1 KB DMA instructions
    const uint8_t *asrc[kAInstr];
#pragma unroll
    for (int ii = 0; ii < kAInstr; ++ii) {
        const int row = (wave * kAInstr + ii) * 8 + lane / 8;
        const int r = min(len - 1, m0 + row);      // padding rows repeat the last row; never stored
        const uint8_t *rowp;
        if constexpr (EPI == GEMM_GATEUP)
            rowp = static_cast<const uint8_t *>(a.x) + static_cast<size_t>(a.wv.row_tok[beg + r]) * H * 2;
        else
            rowp = static_cast<const uint8_t *>(a.wv.h) + static_cast<size_t>(beg + r) * I * 2;
        asrc[ii] = rowp + (swz128(row, lane & 7) << 4);
    }
    constexpr int kBRowsPerInstr = 1024 / Tr::kRowBytes;
    const uint8_t *bsrc[Tr::kBInstr];
#pragma unroll
    for (int ii = 0; ii < Tr::kBInstr; ++ii) {
        const int row = (wave * Tr::kBInstr + ii) * kBRowsPerInstr + lane / Tr::kChunks;
        int wrow;
        if constexpr (EPI == GEMM_GATEUP) {
            const int wn = row >> 6, q = row & 63, hc0 = nt * (kBN / 2) + wn * 32;
            wrow = q < 32 ? hc0 + q : I + hc0 + q - 32;
        } else {
            wrow = nt * kBN + row;
        }
        const size_t wb = WT == FT_DT_BF16 ? 2 : 1;
        const int chunk = WT == FT_DT_BF16 ? swz128(row, lane & 7) : swz64(row, lane & 3);
        bsrc[ii] = static_cast<const uint8_t *>(EPI == GEMM_GATEUP ? a.w13 : a.w2) +
                   (static_cast<size_t>(slot) * nrows + wrow) * K * wb + (chunk << 4);
    }
    auto issue = [&](int kt, uint8_t *dA, uint8_t *dB) {
#pragma unroll
        for (int ii = 0; ii < kAInstr; ++ii)
            dma16(asrc[ii] + static_cast<size_t>(kt) * kARowBytes, dA + (wave * kAInstr + ii) * 1024);
#pragma unroll
        for (int ii = 0; ii < Tr::kBInstr; ++ii)
            dma16(bsrc[ii] + static_cast<size_t>(kt) * Tr::kRowBytes, dB + (wave * Tr::kBInstr + ii) * 1024);
    };
    constexpr int kPerStage = kAInstr + Tr::kBInstr;

    // ---- MFMA fragments
    const int wm = wave / kWavesN, wn = wave % kWavesN;
    const int fn = lane & 31, fq = lane >> 5;
    // fp8 block scales of each wave's columns (the gate and the up rows of a gate/up tile, or
    // the down tile's rows), one per 128-wide K block, staged in LDS before the pipeline starts:
    // a vector load inside the loop would make the wait-count pass drain the DMA stages
    constexpr int kMaxKb = 64;                      // K <= 8192
    __shared__ float s_scale[kWavesN][2][kMaxKb];
    // token and gate of each row of the tile (down projection epilogue), loaded with the prologue
    __shared__ int32_t s_tok[kBM];
    __shared__ float s_gate[kBM];
    if constexpr (EPI == GEMM_DOWN) {
        for (int i = t; i < kBM; i += kGemmThreads) {
            const int r = min(len - 1, m0 + i);
            s_tok[i] = a.wv.row_tok[beg + r];
            s_gate[i] = a.wv.row_gate[beg + r];
        }
    }
    const int nkb = K / 128;
    if constexpr (WT == FT_DT_FP8E4M3FN_B128) {
        const float *s = EPI == GEMM_GATEUP ? a.s13 : a.s2;
        for (int idx = t; idx < kWavesN * 2 * nkb; idx += kGemmThreads) {
            const int w = idx / (2 * nkb), which = (idx / nkb) & 1, kb = idx % nkb;
            int r;
            if constexpr (EPI == GEMM_GATEUP) {
                const int hc0 = nt * (kBN / 2) + w * 32;
                r = which == 0 ? hc0 / 128 : (I + hc0) / 128;
            } else {
                r = (nt * kBN + w * 64) / 128;
            }
            s_scale[w][which][kb] = s[(static_cast<size_t>(slot) * (nrows / 128) + r) * nkb + kb];
        }
        __syncthreads();
    }
    // 2 x 2 tiles of 32 x 32 per wave; for a gate/up tile, column tile 0 holds the wave's 32
    // gate columns and column tile 1 the matching up columns
    floatx16_t acc[2][2], part[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            acc[i][j] = floatx16_t{};
            part[i][j] = floatx16_t{};
        }

    const int nk = K / kBK;
    // one stage: read slot (A, B) for K stage kt while the DMA for stage kt + 2 fills (dA, dB).
    // Stage kt landed once this wave's DMA count allows only stage kt+1 to be outstanding and
    // the barrier has passed (every wave's share of it landed, every wave finished reading
    // stage kt-1); only then may stage kt+2 overwrite the slot stage kt-1 used.  Past the end
    // the DMA re-reads the last stage into that free slot, keeping the counts constant.
    auto step = [&](int kt, const uint8_t *A, const uint8_t *B, uint8_t *dA, uint8_t *dB) {
        wait_vmcnt<(kStages - 2) * kPerStage>();
        wait_lgkmcnt0();
        stage_barrier();
        issue(min(kt + kStages - 1, nk - 1), dA, dB);
        if (kt < nk) {
            // all operand fragments of the stage are read before the first MFMA (distinct
            // registers, fenced by a scheduling barrier), so the MFMAs wait on them one by one
            // instead of stalling at every K step
            constexpr int KS = kBK / 16;
            u32x4_t af[KS][2], bf[KS][2];
            uint2 b8[KS][2];
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                // 32x32x16 MFMA operands: lane (r = lane % 32, kg = lane / 32) holds 8 K values
                // of row r, chunk 2 ks + kg of the stage
                const int c = ks * 2 + fq;
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const int ra = wm * 64 + i * 32 + fn;
                    af[ks][i] = *reinterpret_cast<const u32x4_t *>(A + ra * kARowBytes + (swz128(ra, c) << 4));
                    const int rb = wn * 64 + i * 32 + fn;
                    if constexpr (WT == FT_DT_BF16) {
                        bf[ks][i] = *reinterpret_cast<const u32x4_t *>(B + rb * Tr::kRowBytes + (swz128(rb, c) << 4));
                    } else {
                        const int kq = c * 8;                          // first of 8 fp8 bytes
                        const int ch = swz64(rb, kq >> 4);
                        b8[ks][i] = *reinterpret_cast<const uint2 *>(B + rb * Tr::kRowBytes + (ch << 4) + (kq & 15));
                    }
                }
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                if constexpr (WT == FT_DT_FP8E4M3FN_B128) {
#pragma unroll
                    for (int i = 0; i < 2; ++i) bf[ks][i] = fp8x8_to_bf16x8(b8[ks][i].x, b8[ks][i].y);
                }
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j) {
                        if constexpr (WT == FT_DT_BF16)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(af[ks][i]), as_bf16x8(bf[ks][j]),
                                                                                acc[i][j], 0, 0, 0);
                        else
                            part[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(af[ks][i]), as_bf16x8(bf[ks][j]),
                                                                                 part[i][j], 0, 0, 0);
                    }
            }
            if constexpr (WT == FT_DT_FP8E4M3FN_B128) {
                if ((kt & 1) == 1) {            // end of a 128-wide K block: scale and fold
                    const int kb = kt >> 1;
                    const float slo = s_scale[wn][0][kb], shi = s_scale[wn][1][kb];
#pragma unroll
                    for (int i = 0; i < 2; ++i)
#pragma unroll
                        for (int j = 0; j < 2; ++j) {
                            const float sc = (EPI == GEMM_GATEUP && j == 1) ? shi : slo;
#pragma unroll
                            for (int e = 0; e < 16; ++e) acc[i][j][e] += sc * part[i][j][e];
                            part[i][j] = floatx16_t{};
                        }
                }
            }
        }
    };

    // outstanding stores of the zeroing loop must not be counted against the DMA waits below;
    // the barrier publishes the staged token / gate / scale tables
    wait_vmcnt<0>();
    __syncthreads();
    issue(0, sA0, sB0);
    issue(min(1, nk - 1), sA1, sB1);
    for (int kt = 0; kt < nk; kt += 3) {
        step(kt + 0, sA0, sB0, sA2, sB2);
        step(kt + 1, sA1, sB1, sA0, sB0);
        step(kt + 2, sA2, sB2, sA1, sB1);
    }
    wait_vmcnt<0>();   // the redundant tail stages

    // ---- epilogue: element e of a 32 x 32 tile in lane (fn, fq) is row 8 (e / 4) + 4 fq + e % 4,
    // column fn
    if constexpr (EPI == GEMM_GATEUP) {
        uint16_t *hout = static_cast<uint16_t *>(a.wv.h);
        const int col = nt * (kBN / 2) + wn * 32 + fn;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = m0 + wm * 64 + i * 32 + (e >> 2) * 8 + 4 * fq + (e & 3);
                if (row < len) {
                    const float hv = silu_f32(acc[i][0][e]) * acc[i][1][e];
                    hout[static_cast<size_t>(beg + row) * I + col] = f32_to_bf16(hv);
                }
            }
    } else {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = m0 + wm * 64 + i * 32 + (e >> 2) * 8 + 4 * fq + (e & 3);
                if (row < len) {
                    const int tok = s_tok[row - m0];
                    const float gw = s_gate[row - m0];
                    float *orow = a.out + static_cast<size_t>(tok) * H + nt * kBN + wn * 64 + fn;
#pragma unroll
                    for (int j = 0; j < 2; ++j) unsafeAtomicAdd(orow + j * 32, gw * acc[i][j][e]);
                }
            }
    }
}

// Upper bound of the M tiles this call's routing can produce (rows / BM, plus one ragged tile
// per group); never above the workspace's table size gemm_max_mtiles(T, k, E).
static long max_mtiles(const ExpertArgs &a) {
    const long rows = static_cast<long>(a.T) * a.k + (a.shared ? a.T : 0);
    return (rows + kBM - 1) / kBM + a.max_groups;
}

template <int WT>
static hipError_t launch_gemm_wt(const ExpertArgs &a, hipStream_t s, const Prof &prof) {
    const long mtiles = max_mtiles(a);
    if (!prof.mark(1)) return hipErrorUnknown;
    const int ntn_gu = a.I / (kBN / 2);
    hipLaunchKernelGGL((grouped_gemm<WT, GEMM_GATEUP>), dim3(static_cast<unsigned>(mtiles * ntn_gu)),
                       dim3(kGemmThreads), 0, s, a, ntn_gu);
    if (!prof.mark(2)) return hipErrorUnknown;
    const int ntn_dn = a.H / kBN;
    hipLaunchKernelGGL((grouped_gemm<WT, GEMM_DOWN>), dim3(static_cast<unsigned>(mtiles * ntn_dn)),
                       dim3(kGemmThreads), 0, s, a, ntn_dn);
    if (!prof.mark(3)) return hipErrorUnknown;
    return hipGetLastError();
}

hipError_t launch_gemm(const ExpertArgs &a, hipStream_t s, const Prof &prof) {
    if (a.w_dtype == FT_DT_BF16) return launch_gemm_wt<FT_DT_BF16>(a, s, prof);
    return launch_gemm_wt<FT_DT_FP8E4M3FN_B128>(a, s, prof);
}

}  // namespace ftmoe
