// Grouped expert GEMM on MFMA tiles for many-token chunks (prefill): bf16, fp8 or MXFP4 weights,
// bf16 activations (fp8 ones in the optional FT_ACT_FP8_1x128_POW2 mode), float32 accumulation.
//
// The same two projections as the streaming path (Section 3.2, grouped evaluation of the GPU
// execution set; weights addressed through the slot, Section 4.2), shaped for matrix-core reuse:
//   gate/up: h[rows of g] = silu(X_g W1^T) * (X_g W3^T)       tile = BM rows x BN/2 h columns
//   down   : out[tok] += gate * (h_g W2^T)                    tile = BM rows x BN out columns
//
// Work decomposition.  One workgroup per (group, BM-row M tile, BN-row N tile).  Each wave
// computes 128 rows of the tile for its own 64 columns, as 4 x 2 MFMA 32x32x16 tiles (the bf16
// MFMA shape with the highest measured throughput on gfx950), so every weight element is read
// from LDS (and, for fp8 or MXFP4, widened) by exactly one wave.  The default tile is 128 x 256
// with 4 waves and two workgroups per CU, so one multiplies while the other waits at a stage
// barrier or runs its prologue or epilogue.  A build with FT_GEMM_BM = 256 uses 256 x 256 tiles
// of 8 waves, one workgroup per CU: a third fewer bytes per flop, measured faster on dense
// shapes but slower on routed prefill batches, whose expert groups of about 256 rows leave
// nearly empty tail tiles that still stream a whole weight tile.
// The kernel is bound by how fast global memory fills LDS (measured: 17 TB/s for L2-resident
// 64-byte row pieces, 7-11 TB/s once the data comes from the Infinity Cache or HBM), so the tile
// is as large as LDS and the occupancy allow: a 128 x 256 tile moves 768 bytes per K step for
// 65536 flops, a third less per flop than 128 x 128, while the 128-row M tile keeps the padding
// of the small expert groups in check.
// Tiles are enumerated per group, in bands of up to kBandM M tiles, each band N-tile-major with
// the M tile fastest, through the per-M-tile group map the router writes, so the tiles that
// share a weight tile and those that share activation rows run at the same time; the block ->
// tile map keeps consecutive tiles on one XCD (workgroups are dealt to the 8 XCDs round-robin)
// to share its L2.  The router numbers the groups in cost classes (the shared expert, groups of
// several M tiles, then one-tile groups by their live 32-row sub-tiles), and tiles skip the
// MFMAs of sub-tiles that hold only padding rows (the fp8-activation kernels in steps of two
// sub-tiles), so the tiles of one launch cost about the same.
//
// Data movement.  A (activation rows, gathered through row_tok for gate/up) and B (weight rows,
// kept in their storage format) go straight from global memory into LDS with global_load_lds
// (16 bytes per lane), through a ring of NS stages of BK K-values.  Every LDS row keeps its
// 16-byte chunks XOR-swizzled by the row index, so MFMA operand reads of consecutive rows hit
// distinct banks.  The main loop is software-pipelined: each MFMA sub-step's operands are read
// from LDS while the previous sub-step's MFMAs run, and the stage hand-off (an explicit vmcnt
// wait plus s_barrier; a __syncthreads would drain every stage in flight) sits in the last
// sub-step of a stage, so the first reads of the next stage overlap its last MFMAs.  The ring is
// unrolled, every stage buffer is an array of its own and whole turns of the ring run without
// branches, so the compiler can tell the stage being read from the stages still being written
// and adds no wait of its own.
//
// fp8 weights carry one float32 scale per 128 x 128 block, and the product is formed exactly as
// weight-only dequantisation defines it: the codes are widened to bf16 unscaled (exact), the
// MFMAs sum each 128-wide K block's products in float32, and the block's scale multiplies that
// partial sum.  A wave's 64 columns lie in at most two scale blocks (the gate and the up half of
// a gate/up tile, one block for down), so one scale per column half and K block applies to all
// of the wave's accumulators of that half.  Rather than keeping a second accumulator set for the
// running block, the accumulators carry the sum in units of the current block's scale: at the
// start of block k they are multiplied by s(k-1) / s(k), the MFMAs then add block k's unscaled
// partial sum, and after the last block one multiply by its scale gives sum_k s(k) P(k).  A block
// with scale 0 contributes nothing: its ratio is 1 (the previous scale is carried on) and, in the
// tiles that hold such a block, its widened codes are masked to zero.  The gate/up B tile puts
// each wave's 32 gate rows next to the 32 matching up rows, so SiLU(gate) * up is formed in
// registers.
#include <type_traits>

#include "ftmoe_device.h"
#include "ftmoe_internal.h"

namespace ftmoe {

#ifndef FT_GEMM_WAVE_ROWS
#define FT_GEMM_WAVE_ROWS 128
#endif
constexpr int kWaveRows = FT_GEMM_WAVE_ROWS, kWaveCols = 64;   // per-wave output tile
constexpr int kWavesM = kGemmBM / kWaveRows, kWavesN = kGemmBN / kWaveCols;
constexpr int kGemmWaves = kWavesM * kWavesN;
constexpr int kGemmThreads = kGemmWaves * kWave;
#ifndef FT_GEMM_OCC
#define FT_GEMM_OCC 2
#endif
constexpr int kGemmOcc = FT_GEMM_OCC;                   // workgroups per CU
constexpr int kMI = kWaveRows / 32, kNJ = kWaveCols / 32; // 32 x 32 MFMA tiles per wave
constexpr int kBM = kGemmBM;                            // token rows per tile
constexpr int kBN = kGemmBN;                            // weight rows per tile
static_assert(kGemmWaves == 4 || kGemmWaves == 8, "4 or 8 waves");
static_assert(kBM == kWavesM * kWaveRows && kBN == kWavesN * kWaveCols, "tile = waves x wave tile");
#ifndef FT_GEMM_BAND
#define FT_GEMM_BAND 8
#endif
constexpr int kBandM = FT_GEMM_BAND;  // M tiles that run together on each weight tile

enum { GEMM_GATEUP = 0, GEMM_DOWN = 1 };

// Per weight format: K values per stage (BK), ring slots (NS: two workgroups of the default tile
// fit one CU's LDS; after the hand-off in a stage's last sub-step up to NS - 1 later stages are
// in flight) and weight row bytes per stage (BRB).
#ifndef FT_GEMM_BF16_BK
#define FT_GEMM_BF16_BK 32
#endif
#ifndef FT_GEMM_BF16_NS
#define FT_GEMM_BF16_NS 3
#endif
#ifndef FT_GEMM_FP8_BK
#define FT_GEMM_FP8_BK 64
#endif
#ifndef FT_GEMM_FP8_NS
#define FT_GEMM_FP8_NS 2
#endif
// Internal weight-format code of fp8 weights with fp8 activations (FT_ACT_FP8_1x128_POW2): fp8 x
// fp8 products on the scaled 32x32x64 MFMA.
constexpr int kWtFp8Act = 16;
template <int WT> struct GTr;
// CHUNK_GU, CHUNK_DN: workgroups per launch of the gate/up and the down GEMM (see launch_tiles).
// SKIP_PAD_GU, SKIP_PAD_DN: tiles skip the MFMAs of 32-row sub-tiles that hold only padding
// rows.  With the router's tile order (tiles of similar cost together) this pays on the fp8
// gate/up GEMM too (DeepSeek-V3 prefill: 2.37 -> 2.26 ms).
template <> struct GTr<FT_DT_BF16> {
    static constexpr int BK = FT_GEMM_BF16_BK, NS = FT_GEMM_BF16_NS, BRB = 2 * BK;
    static constexpr int OCC_GU = kGemmOcc, OCC_DN = kGemmOcc, NS_GU = NS, NS_DN = NS;
    static constexpr long CHUNK_GU = 768, CHUNK_DN = 2048;   // down 1024 before the tile classes
    static constexpr bool SKIP_PAD_GU = true, SKIP_PAD_DN = true;
};
#ifndef FT_GEMM_FP8_CHUNK_GU
#define FT_GEMM_FP8_CHUNK_GU 512
#endif
#ifndef FT_GEMM_FP8_CHUNK_DN
#define FT_GEMM_FP8_CHUNK_DN 2560   // 1536 before the cost-class tile order; 2560 measured 1-4 % faster at 2048-8192 tokens
#endif
template <> struct GTr<FT_DT_FP8E4M3FN_B128> {
    static constexpr int BK = FT_GEMM_FP8_BK, NS = FT_GEMM_FP8_NS, BRB = BK;
    static constexpr int OCC_GU = kGemmOcc, OCC_DN = kGemmOcc, NS_GU = NS, NS_DN = NS;
    static constexpr long CHUNK_GU = FT_GEMM_FP8_CHUNK_GU, CHUNK_DN = FT_GEMM_FP8_CHUNK_DN;
    static constexpr bool SKIP_PAD_GU = true, SKIP_PAD_DN = true;
};
// fp8 weights and fp8 activations: 64 K values per stage (one 32x32x64 MFMA step).  Two
// workgroups per CU with a two-stage ring (one workgroup with four stages was slower: 5.1 ms
// against 3.4 ms for the DeepSeek-V3 prefill layer); both projections skip padding in steps of
// two 32-row sub-tiles (layer 3.32 -> 3.27 ms).
#ifndef FT_GEMM_AQ_OCC_GU
#define FT_GEMM_AQ_OCC_GU 2
#endif
#ifndef FT_GEMM_AQ_OCC_DN
#define FT_GEMM_AQ_OCC_DN 2
#endif
#ifndef FT_GEMM_AQ_CHUNK_GU
#define FT_GEMM_AQ_CHUNK_GU 512
#endif
#ifndef FT_GEMM_AQ_CHUNK_DN
#define FT_GEMM_AQ_CHUNK_DN 2560   // as for the exact fp8 down GEMM (1536: down 1.40 against 1.25 ms)
#endif
template <> struct GTr<kWtFp8Act> {
    static constexpr int BK = 64, BRB = BK;
    static constexpr int OCC_GU = FT_GEMM_AQ_OCC_GU, OCC_DN = FT_GEMM_AQ_OCC_DN;
    static constexpr int NS_GU = OCC_GU == 2 ? 2 : 4, NS_DN = OCC_DN == 2 ? 2 : 4;
    static constexpr long CHUNK_GU = FT_GEMM_AQ_CHUNK_GU, CHUNK_DN = FT_GEMM_AQ_CHUNK_DN;
    static constexpr bool SKIP_PAD_GU = true, SKIP_PAD_DN = true;
};
// MXFP4: 64 K values (32 code bytes) per weight row and stage, so that one lane's 16-byte chunk
// of a row is a whole 32-value scale run
template <> struct GTr<FT_DT_MXFP4> {
    static constexpr int BK = 64, NS = 3, BRB = BK / 2;
    static constexpr int OCC_GU = kGemmOcc, OCC_DN = kGemmOcc, NS_GU = NS, NS_DN = NS;
    static constexpr long CHUNK_GU = 512, CHUNK_DN = 1536;
    static constexpr bool SKIP_PAD_GU = true, SKIP_PAD_DN = true;
};

template <int V> using ic = std::integral_constant<int, V>;

constexpr int gcd_c(int a, int b) { return b == 0 ? a : gcd_c(b, a % b); }

// Calls f(ic<S>) for S = B .. E-1.
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (B < E) {
        f(ic<B>{});
        static_for<B + 1, E>(f);
    }
}

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
// wait-for-everything a __syncthreads fence adds.
__device__ __forceinline__ void stage_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Position of 16-byte chunk c in LDS row r.  A 16-byte-per-lane LDS read serves 16 lanes (256
// bytes, all 64 banks) per pass; the operand reads give those lanes 16 consecutive rows and one
// chunk index, so the XOR spreads the same chunk of 16 consecutive rows over all 16 chunk
// positions of a 256-byte window: a 128-byte row holds 8 chunks (XOR (r / 2) mod 8), a 64-byte
// row 4 (XOR (r / 4) mod 4), a 32-byte row 2 (XOR (r / 8) mod 2).
template <int ROW_BYTES>
__device__ __forceinline__ int swz(int r, int c) {
    static_assert(ROW_BYTES == 32 || ROW_BYTES == 64 || ROW_BYTES == 128, "row size");
    if constexpr (ROW_BYTES == 128) return c ^ ((r >> 1) & 7);
    else if constexpr (ROW_BYTES == 64) return c ^ ((r >> 2) & 3);
    else return c ^ ((r >> 3) & 1);
}

typedef int i32x8_t __attribute__((ext_vector_type(8)));
__device__ __forceinline__ i32x8_t cat_u32x8(u32x4_t lo, u32x4_t hi) {
    return i32x8_t{static_cast<int>(lo[0]), static_cast<int>(lo[1]), static_cast<int>(lo[2]), static_cast<int>(lo[3]),
                   static_cast<int>(hi[0]), static_cast<int>(hi[1]), static_cast<int>(hi[2]), static_cast<int>(hi[3])};
}

__device__ __forceinline__ void dma16(const void *g, uint8_t *lds_block) {
    __builtin_amdgcn_global_load_lds(g, (lds_void_t *)(lds_block), 16, 0, 0);
}

// 4 bytes per lane: lane i writes LDS bytes [4 i, 4 i + 4) of the 256-byte block
__device__ __forceinline__ void dma4(const void *g, uint8_t *lds_block) {
    __builtin_amdgcn_global_load_lds(g, (lds_void_t *)(lds_block), 4, 0, 0);
}

template <int WT, int EPI>
__global__ __launch_bounds__(kGemmThreads, EPI == GEMM_GATEUP ? GTr<WT>::OCC_GU : GTr<WT>::OCC_DN) void grouped_gemm(
    ExpertArgs a, int ntn, int base) {
    constexpr bool kAq = WT == kWtFp8Act;                          // fp8 activations (fp8 x fp8 MFMA)
    constexpr bool kFp8 = WT == FT_DT_FP8E4M3FN_B128 || kAq;        // fp8 weights with block scales
    constexpr bool kWiden8 = WT == FT_DT_FP8E4M3FN_B128;            // fp8 weights widened to bf16
    constexpr bool kFp4 = WT == FT_DT_MXFP4;
    constexpr int BK = GTr<WT>::BK, NS = EPI == GEMM_GATEUP ? GTr<WT>::NS_GU : GTr<WT>::NS_DN;
    constexpr int ARB = kAq ? BK : BK * 2;           // A row bytes per stage (bf16, or fp8 codes)
    constexpr int BRB = GTr<WT>::BRB;                // B row bytes per stage
    constexpr int ASTAGE = kBM * ARB, BSTAGE = kBN * BRB;
    constexpr int A_INSTR = ASTAGE / 1024 / kGemmWaves;   // 1 KB DMA instructions per wave
    constexpr int B_INSTR = BSTAGE / 1024 / kGemmWaves;
    // MXFP4: one more DMA per wave and stage brings a quarter of the stage's e8m0 scales
    constexpr int PER_STAGE = A_INSTR + B_INSTR + (kFp4 ? 1 : 0);
    constexpr int XSTAGE = kFp4 ? 1024 : 16;         // LDS per scale stage: 4 waves x 256 bytes
    static_assert(A_INSTR >= 1 && B_INSTR >= 1, "stage too small");
    static_assert(NS >= 2 && NS <= 4, "ring depth");
    static_assert(NS * PER_STAGE < 64, "vmcnt range");
    static_assert(!kFp8 || 128 % BK == 0, "an fp8 K stage lies in one scale block");
    static_assert(!kAq || (BK % 64 == 0 && kWavesM == 1), "fp8 activations: 64-K MFMA steps, 4 waves");
    // stages unrolled per main-loop turn: whole ring turns and, for fp8, whole 128-wide K blocks
    constexpr int kStagesPerKb = kFp8 ? 128 / BK : 1;
    constexpr int kUnit = NS / gcd_c(NS, kStagesPerKb) * kStagesPerKb;   // lcm
    // one array per stage (see the header comment); unused ones shrink to 16 bytes
    __shared__ __attribute__((aligned(1024))) uint8_t sA0[ASTAGE], sA1[ASTAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t sA2[NS > 2 ? ASTAGE : 16];
    __shared__ __attribute__((aligned(1024))) uint8_t sA3[NS > 3 ? ASTAGE : 16];
    __shared__ __attribute__((aligned(1024))) uint8_t sB0[BSTAGE], sB1[BSTAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t sB2[NS > 2 ? BSTAGE : 16];
    __shared__ __attribute__((aligned(1024))) uint8_t sB3[NS > 3 ? BSTAGE : 16];
    __shared__ __attribute__((aligned(512))) uint8_t sX0[XSTAGE], sX1[XSTAGE];
    __shared__ __attribute__((aligned(512))) uint8_t sX2[kFp4 && NS > 2 ? XSTAGE : 16];
    __shared__ __attribute__((aligned(512))) uint8_t sX3[kFp4 && NS > 3 ? XSTAGE : 16];
    constexpr int kMaxKb = 64;                       // K <= 8192
    // fp8: per wave and column half, the factor applied to the accumulators at the start of each
    // 128-wide K block, a mask that zeroes the widened codes of blocks with scale 0, and the scale
    // of the last block (applied after the K loop)
    __shared__ float s_ratio[kFp8 ? kWavesN : 1][2][kFp8 ? kMaxKb : 1];
    __shared__ uint32_t s_keep[kFp8 ? kWavesN : 1][2][kFp8 ? kMaxKb : 1];
    __shared__ float s_last[kWavesN][2];
    __shared__ int32_t s_zeroblk[kWavesN];   // fp8: a column group's scales hold a 0
    __shared__ int32_t s_tok[kBM];
    __shared__ float s_gate[kBM];
    // fp8 activations: e8m0 scale byte of each tile row and K block, and (gate/up epilogue) the
    // per-wave largest |h| of each row and the rows' h exponents
    __shared__ uint8_t s_ascale[kAq ? kBM * kMaxKb : 1];
    __shared__ float s_hmax[kAq ? kWavesN : 1][kAq ? kBM : 1];
    __shared__ int32_t s_hexp[kAq ? kBM : 1];
    auto stA = [&](auto s) -> uint8_t * {
        constexpr int S = decltype(s)::value;
        if constexpr (S == 0) return sA0;
        else if constexpr (S == 1) return sA1;
        else if constexpr (S == 2) return sA2;
        else return sA3;
    };
    auto stB = [&](auto s) -> uint8_t * {
        constexpr int S = decltype(s)::value;
        if constexpr (S == 0) return sB0;
        else if constexpr (S == 1) return sB1;
        else if constexpr (S == 2) return sB2;
        else return sB3;
    };
    auto stX = [&](auto s) -> uint8_t * {
        constexpr int S = decltype(s)::value;
        if constexpr (S == 0) return sX0;
        else if constexpr (S == 1) return sX1;
        else if constexpr (S == 2) return sX2;
        else return sX3;
    };

    const int t = threadIdx.x;
    if (EPI == GEMM_GATEUP && base == 0) {
        // zero the output that the down projection accumulates into (first launch only)
        const size_t n4 = static_cast<size_t>(a.T) * a.H / 4;
        float4 *o4 = reinterpret_cast<float4 *>(a.out);
        for (size_t i = static_cast<size_t>(blockIdx.x) * kGemmThreads + t; i < n4;
             i += static_cast<size_t>(gridDim.x) * kGemmThreads)
            o4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    const int L = base + xcd_remap(blockIdx.x, gridDim.x);
    const int MTT = a.wv.grp_meta[4];
    if (L >= MTT * ntn) return;
    // group g owns logical tiles [off_g * ntn, off_{g+1} * ntn), so L / ntn is one of its M tiles;
    // inside the group, bands of up to kBandM M tiles, each band N-tile-major with the M tile
    // fastest
    const int g = a.wv.mt_group[L / ntn];
    const int off = a.wv.grp_mt_off[g], mtc = a.wv.grp_mt_off[g + 1] - off;
    const int local = L - off * ntn;
    const int band = local / (kBandM * ntn), rem = local - band * (kBandM * ntn);
    const int bm = min(kBandM, mtc - band * kBandM);
    const int nt = rem / bm, mt = band * kBandM + rem % bm;
    const int slot = a.wv.grp_slot[g], beg = a.wv.grp_beg[g], len = a.wv.grp_len[g];
    const int H = a.H, I = a.I;
    const int K = EPI == GEMM_GATEUP ? H : I;
    const int nrows = EPI == GEMM_GATEUP ? 2 * I : H;
    const int m0 = mt * kBM;
    const int wave = __builtin_amdgcn_readfirstlane(t / kWave), lane = lane_id();

    // ---- DMA sources: this lane's 16 bytes in each of its 1 KB DMA instructions.  Lane i of
    // an instruction writes LDS bytes [16 i, 16 i + 16) of its 1 KB block, i.e. row i / CHUNKS of
    // the block at chunk position i % CHUNKS, so it fetches the chunk that belongs there.
    constexpr int A_ROWS = 1024 / ARB, B_ROWS = 1024 / BRB;   // rows per DMA instruction
    constexpr int A_CHUNKS = ARB / 16, B_CHUNKS = BRB / 16;
    const uint8_t *asrc[A_INSTR];
#pragma unroll
    for (int ii = 0; ii < A_INSTR; ++ii) {
        const int row = (wave * A_INSTR + ii) * A_ROWS + lane / A_CHUNKS;
        const int r = min(len - 1, m0 + row);      // padding rows repeat the last row; never stored
        const uint8_t *rowp;
        constexpr size_t EB = kAq ? 1 : 2;   // bytes per activation element
        if constexpr (EPI == GEMM_GATEUP)
            rowp = (kAq ? a.wv.xq : static_cast<const uint8_t *>(a.x)) +
                   static_cast<size_t>(a.wv.row_tok[beg + r]) * H * EB;
        else
            rowp = (kAq ? a.wv.hq : static_cast<const uint8_t *>(a.wv.h)) + static_cast<size_t>(beg + r) * I * EB;
        asrc[ii] = rowp + (swz<ARB>(row, lane % A_CHUNKS) << 4);
    }
    // B tile row -> weight row.  gate/up: wave n's 64 rows are the 32 gate rows of h columns
    // [hc0, hc0 + 32), hc0 = nt * BN/2 + 32 n, followed by the 32 matching up rows (I + hc0 ...).
    const uint8_t *bsrc[B_INSTR];
#pragma unroll
    for (int ii = 0; ii < B_INSTR; ++ii) {
        const int row = (wave * B_INSTR + ii) * B_ROWS + lane / B_CHUNKS;
        int wrow;
        if constexpr (EPI == GEMM_GATEUP) {
            const int wn = row / kWaveCols, q = row % kWaveCols;
            const int hc0 = nt * (kBN / 2) + wn * (kWaveCols / 2);
            wrow = q < kWaveCols / 2 ? hc0 + q : I + hc0 + q - kWaveCols / 2;
        } else {
            wrow = nt * kBN + row;
        }
        bsrc[ii] = static_cast<const uint8_t *>(EPI == GEMM_GATEUP ? a.w13 : a.w2) +
                   (static_cast<size_t>(slot) * nrows + wrow) * static_cast<size_t>(K / BK) * BRB +
                   (swz<BRB>(row, lane % B_CHUNKS) << 4);
    }
    const int wm = wave / kWavesN, wn = wave % kWavesN;
    const int fn = lane & 31, fq = lane >> 5;
    // MXFP4 scales (run-major in memory: the scales of one 32-wide K run of consecutive weight
    // rows are contiguous).  A stage covers runs 2 kt and 2 kt + 1 of the tile's 256 weight rows,
    // which are 4 segments of 128 contiguous bytes (gate/up: the 128 gate rows and the 128 up
    // rows of the tile; down: two halves of its 256 rows).  Wave w = 2 run + half (mod 4) moves
    // segment (run, half) with one 4-byte-per-lane DMA into bytes [256 w, 256 w + 128) of the
    // stage; lanes 32..63 fetch the same segment again into the next 128 bytes, so the instruction
    // has every lane active and stays in bounds.  With 8 waves, waves w and w + 4 write the same
    // bytes, which keeps every wave's DMA count per stage equal.
    const uint8_t *xsrc = nullptr;
    int xcol[kNJ] = {};
    if constexpr (kFp4) {
        const int xr = (wave >> 1) & 1, xh = wave & 1;
        const int row0 = EPI == GEMM_GATEUP ? (xh ? I : 0) + nt * (kBN / 2) : nt * kBN + xh * (kBN / 2);
        xsrc = static_cast<const uint8_t *>(EPI == GEMM_GATEUP ? a.s13 : a.s2) +
               (static_cast<size_t>(slot) * (K / 32) + xr) * nrows + row0 + 4 * (lane & 31);
        // this lane's scale byte for column tile j, run fq: segment (fq, half) at 256 (2 fq + half)
#pragma unroll
        for (int j = 0; j < kNJ; ++j) {
            const int half = EPI == GEMM_GATEUP ? j : (wn * kWaveCols + j * 32) / (kBN / 2);
            const int r = EPI == GEMM_GATEUP ? wn * (kWaveCols / 2) + fn : (wn * kWaveCols + j * 32 + fn) % (kBN / 2);
            xcol[j] = 256 * (2 * fq + half) + r;
        }
    }
    auto issue = [&](int kt, uint8_t *dA, uint8_t *dB, auto ws) {
#pragma unroll
        for (int ii = 0; ii < A_INSTR; ++ii)
            dma16(asrc[ii] + static_cast<size_t>(kt) * ARB, dA + (wave * A_INSTR + ii) * 1024);
#pragma unroll
        for (int ii = 0; ii < B_INSTR; ++ii)
            dma16(bsrc[ii] + static_cast<size_t>(kt) * BRB, dB + (wave * B_INSTR + ii) * 1024);
        if constexpr (kFp4) {
            dma4(xsrc + static_cast<size_t>(kt) * (BK / 32) * nrows, stX(ws) + (wave & 3) * 256);
        }
    };
    const int nkb = K / 128;
    // fp8 block-scale tables of each wave's columns (gate half and up half of a gate/up tile; one
    // block for down), staged in LDS before the pipeline starts: a vector load inside the loop
    // would make the compiler drain the DMA stages.  Lane kb of the waves of the first M row holds
    // K block kb: s'(kb) = the scale of the last block at or before kb whose scale is not 0 (1
    // before the first), found with a wave max-scan of the indices of such blocks; the ratio of
    // block kb is s'(kb-1) / s'(kb) (1 for block 0).  One load per lane instead of a walk over
    // the K blocks, whose dependent loads held every tile's start back by several microseconds.
    if constexpr (kFp8) {
        if (wm == 0) {
            const float *sp = static_cast<const float *>(EPI == GEMM_GATEUP ? a.s13 : a.s2);
            uint64_t zero = 0;
#pragma unroll
            for (int which = 0; which < 2; ++which) {
                int r;
                if constexpr (EPI == GEMM_GATEUP) {
                    const int hc0 = nt * (kBN / 2) + wn * (kWaveCols / 2);
                    r = which == 0 ? hc0 / 128 : (I + hc0) / 128;
                } else {
                    r = (nt * kBN + wn * kWaveCols) / 128;
                }
                const float *row = sp + (static_cast<size_t>(slot) * (nrows / 128) + r) * nkb;
                const float sc = lane < nkb ? row[lane] : 1.0f;
                const bool nz = sc != 0.0f;
                zero |= __ballot(lane < nkb && !nz);
                const uint32_t last = wave_incl_max_u32(nz ? static_cast<uint32_t>(lane) + 1u : 0u);
                const float cur = last ? __shfl(sc, static_cast<int>(last) - 1) : 1.0f;
                const float prev = __shfl(cur, max(lane - 1, 0));
                if (lane < nkb) {
                    s_ratio[wn][which][lane] = lane == 0 ? 1.0f : prev / cur;
                    s_keep[wn][which][lane] = nz ? 0xFFFFFFFFu : 0u;
                }
                if (lane == nkb - 1) s_last[wn][which] = cur;
            }
            if (lane == 0) s_zeroblk[wn] = zero != 0;
        }
    }
    // fp8 activations: each tile row's exponent byte of every K block (rows of x by token, rows
    // of h by position), staged like the weight scales before the pipeline starts
    if constexpr (kAq) {
        const uint8_t *src = EPI == GEMM_GATEUP ? a.wv.xs : a.wv.hs;
        for (int idx = t; idx < kBM * nkb; idx += kGemmThreads) {
            const int r = idx / nkb, kb = idx - r * nkb;
            const int rr = min(len - 1, m0 + r);
            const size_t srow = EPI == GEMM_GATEUP ? static_cast<size_t>(a.wv.row_tok[beg + rr]) : static_cast<size_t>(beg + rr);
            s_ascale[r * kMaxKb + kb] = src[srow * nkb + kb];
        }
    }
    // token and gate of each row of the tile (down projection epilogue)
    if constexpr (EPI == GEMM_DOWN) {
        for (int i = t; i < kBM; i += kGemmThreads) {
            const int r = min(len - 1, m0 + i);
            s_tok[i] = a.wv.row_tok[beg + r];
            s_gate[i] = a.wv.row_gate[beg + r];
        }
    }

    // kMI x kNJ tiles of 32 x 32 per wave; for a gate/up tile, column tiles [0, kNJ/2) are the
    // wave's gate columns and [kNJ/2, kNJ) the matching up columns
    floatx16_t acc[kMI][kNJ];
#pragma unroll
    for (int i = 0; i < kMI; ++i)
#pragma unroll
        for (int j = 0; j < kNJ; ++j) acc[i][j] = floatx16_t{};

    const int nk = K / BK;
    constexpr int KS = kAq ? BK / 64 : BK / 16;   // MFMA sub-steps per K stage
    // Operands of one 32x32x16 MFMA sub-step.  The lane (r = lane % 32, kg = lane / 32) holds 8 K
    // values of row r for each operand; which 8 is free as long as A and B agree.  bf16 weights:
    // sub-step ks takes K [16 ks + 8 kg, +8), i.e. 16-byte chunk 2 ks + kg of both rows.  fp8
    // weights: a lane reads one 16-byte chunk of its weight row, 16 K values, for two sub-steps,
    // so sub-step ks = 2 p + s takes K [32 p + 16 kg + 8 s, +8): weight chunk 2 p + kg (bytes
    // 8 s ..), activation chunk 4 p + 2 kg + s.  MXFP4 weights: a lane reads weight chunk kg, 32
    // K values under one scale, for all four sub-steps, so sub-step ks takes K [32 kg + 8 ks, +8):
    // word ks of the chunk, activation chunk 4 kg + ks.  Weight chunks and scales are carried
    // over from the sub-step that read them.
    // fp8 activations: lane (r, kg) holds bytes [32 kg, 32 kg + 32) of the stage's 64-byte row r
    // for both operands (chunks 2 kg and 2 kg + 1; the MFMA pairs the same byte slots of A and
    // B), and its row's exponent byte for the K block.
    struct Frag {
        u32x4_t a[kMI];
        u32x4_t b[kNJ];
        u32x4_t a2[kAq ? kMI : 1];   // fp8 activations: second 16 bytes of each operand
        u32x4_t b2[kAq ? kNJ : 1];
        uint32_t as[kAq ? kMI : 1];  // fp8 activations: e8m0 scale byte of the lane's row
        uint32_t xb[kNJ];   // MXFP4 e8m0 scale byte of each column tile
        float sc[2];        // fp8: accumulator factor of this K block, gate (or down) and up half
        uint32_t keep[2];   // fp8: code mask of this K block (0 for a block with scale 0)
    };
    // zs: the tile holds an fp8 K block with scale 0 (codes of such blocks are masked)
    auto load_frag = [&](auto rs, auto ks, auto ml, auto zs, Frag &f, const Frag &prev, int kt) {
        constexpr int KSI = decltype(ks)::value, ML = decltype(ml)::value;
        constexpr bool ZS = decltype(zs)::value;
        const uint8_t *A = stA(rs);
        const uint8_t *B = stB(rs);
        const int ca = kWiden8 ? 4 * (KSI / 2) + 2 * fq + (KSI % 2) : (kFp4 ? 4 * fq + KSI : 2 * KSI + fq);
        if constexpr (kFp8) {
            if constexpr (KSI == 0) {
                const int kb = (kt * BK) / 128;
                f.sc[0] = s_ratio[wn][0][kb];
                f.sc[1] = s_ratio[wn][1][kb];
                if constexpr (ZS) {
                    f.keep[0] = s_keep[wn][0][kb];
                    f.keep[1] = s_keep[wn][1][kb];
                }
            } else {
                f.sc[0] = prev.sc[0];
                f.sc[1] = prev.sc[1];
                if constexpr (ZS) {
                    f.keep[0] = prev.keep[0];
                    f.keep[1] = prev.keep[1];
                }
            }
        }
#pragma unroll
        for (int i = 0; i < ML; ++i) {
            const int ra = wm * kWaveRows + i * 32 + fn;
            if constexpr (kAq) {
                f.a[i] = *reinterpret_cast<const u32x4_t *>(A + ra * ARB + (swz<ARB>(ra, 4 * KSI + 2 * fq) << 4));
                f.a2[i] = *reinterpret_cast<const u32x4_t *>(A + ra * ARB + (swz<ARB>(ra, 4 * KSI + 2 * fq + 1) << 4));
                if constexpr (KSI == 0) f.as[i] = s_ascale[ra * kMaxKb + (kt * BK) / 128];
                else f.as[i] = prev.as[i];
            } else {
                f.a[i] = *reinterpret_cast<const u32x4_t *>(A + ra * ARB + (swz<ARB>(ra, ca) << 4));
            }
        }
#pragma unroll
        for (int j = 0; j < kNJ; ++j) {
            const int rb = wn * kWaveCols + j * 32 + fn;
            if constexpr (kFp4) {
                if constexpr (KSI == 0) {
                    f.b[j] = *reinterpret_cast<const u32x4_t *>(B + rb * BRB + (swz<BRB>(rb, fq) << 4));
                    f.xb[j] = stX(rs)[xcol[j]];
                } else {
                    f.b[j] = prev.b[j];
                    f.xb[j] = prev.xb[j];
                }
            } else if constexpr (kAq) {
                f.b[j] = *reinterpret_cast<const u32x4_t *>(B + rb * BRB + (swz<BRB>(rb, 4 * KSI + 2 * fq) << 4));
                f.b2[j] = *reinterpret_cast<const u32x4_t *>(B + rb * BRB + (swz<BRB>(rb, 4 * KSI + 2 * fq + 1) << 4));
                if constexpr (ZS) {
                    const uint32_t keep = (EPI == GEMM_GATEUP && j >= kNJ / 2) ? f.keep[1] : f.keep[0];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        f.b[j][q] &= keep;
                        f.b2[j][q] &= keep;
                    }
                }
            } else if constexpr (kFp8) {
                if constexpr (KSI % 2 == 0) {
                    f.b[j] = *reinterpret_cast<const u32x4_t *>(B + rb * BRB + (swz<BRB>(rb, 2 * (KSI / 2) + fq) << 4));
                    if constexpr (ZS) {
                        // codes of a block with scale 0 become +0
                        const uint32_t keep = (EPI == GEMM_GATEUP && j >= kNJ / 2) ? f.keep[1] : f.keep[0];
#pragma unroll
                        for (int q = 0; q < 4; ++q) f.b[j][q] &= keep;
                    }
                } else {
                    f.b[j] = prev.b[j];
                }
            } else {
                f.b[j] = *reinterpret_cast<const u32x4_t *>(B + rb * BRB + (swz<BRB>(rb, ca) << 4));
            }
        }
    };
    // rs: this sub-step opens a 128-wide K block (fp8: the accumulators take the block's factor)
    auto mma = [&](const Frag &f, auto ks, auto ml, auto zs, auto rs) {
        constexpr int KSI = decltype(ks)::value, ML = decltype(ml)::value;
        constexpr bool ZS = decltype(zs)::value, RS = decltype(rs)::value;
        u32x4_t bf[kNJ];
#pragma unroll
        for (int j = 0; j < kNJ; ++j) {
            if constexpr (kFp4) {
                bf[j] = fp4x8_scaled_to_bf16x8(f.b[j][KSI], fp4_scale_operand(f.xb[j]));
            } else if constexpr (kWiden8) {
                bf[j] = KSI % 2 == 0 ? fp8x8_to_bf16x8(f.b[j][0], f.b[j][1]) : fp8x8_to_bf16x8(f.b[j][2], f.b[j][3]);
            } else {
                bf[j] = f.b[j];
            }
        }
        // a tile's accumulators take the block factor just before its MFMA, so the multiplies of one
        // tile can run while the previous tile's MFMA executes (see interleave)
#pragma unroll
        for (int i = 0; i < ML; ++i)
#pragma unroll
            for (int j = 0; j < kNJ; ++j) {
                if constexpr (kFp8 && RS) acc[i][j] *= (EPI == GEMM_GATEUP && j >= kNJ / 2) ? f.sc[1] : f.sc[0];
                if constexpr (kAq)   // formats 0 (fp8 e4m3) for both; B's scale byte 127 (1.0)
                    acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                        cat_u32x8(f.a[i], f.a2[i]), cat_u32x8(f.b[j], f.b2[j]), acc[i][j], 0, 0, 0,
                        static_cast<int>(f.as[i]), 0, 127);
                else
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(f.a[i]), as_bf16x8(bf[j]),
                                                                         acc[i][j], 0, 0, 0);
            }
    };

    // Software pipeline.  The ring holds NS stages; the DMA of stage kt + NS goes into the slot of
    // stage kt once every wave has read all of stage kt.  Each sub-step's operands are read from
    // LDS while the previous sub-step's MFMAs run, and the hand-off sits in the last sub-step of
    // a stage: wait for this wave's share of stage kt + 1 (stages kt + 2 .. kt + NS - 1 may stay
    // outstanding) and for its LDS reads of stage kt, barrier, refill the slot of stage kt, read
    // the first operands of stage kt + 1, then run the last MFMAs of stage kt.  Past the end the
    // DMA re-reads the last stage, which keeps the counts constant.
    // ML: the 32-row MFMA sub-tiles of the M tile that hold at least one real row; the others
    // hold padding only, so their operand reads and MFMAs are skipped.
    // Order of one sub-step's instructions: its MFMAs with the next sub-step's operand reads
    // (sub-step ks2 of the same or the next stage) threaded between them, one read after each
    // MFMA.  Measured 2-4 % faster than issuing all the reads first behind an explicit wait.
    // In a sub-step that opens an fp8 K block (rsv) each MFMA is preceded by the 16 multiplies of
    // its tile's block factor (the first also by the widening of the sub-step's weight operands).
    auto interleave = [&](auto ks2, auto ml, auto zs, auto rsv) {
        constexpr int K2 = decltype(ks2)::value, ML = decltype(ml)::value;
        constexpr bool ZS = decltype(zs)::value, RSV = decltype(rsv)::value;
        constexpr bool kReadsB = kFp4 ? K2 == 0 : (kWiden8 ? K2 % 2 == 0 : true);
        constexpr int kReads = (kAq ? (K2 == 0 ? 3 : 2) * ML : ML) + (kReadsB ? (kAq ? 2 : 1) * kNJ : 0) +
                               (kFp4 && K2 == 0 ? kNJ : 0) + (kFp8 && K2 == 0 ? (ZS ? 4 : 2) : 0);
        constexpr int kMfma = ML * kNJ;
        constexpr int kPairs = kReads < kMfma ? kReads : kMfma;
        if constexpr (RSV) {
            static_for<0, kMfma>([&](auto q) {
                constexpr int Q = decltype(q)::value;
                __builtin_amdgcn_sched_group_barrier(0x002, Q == 0 && kWiden8 ? 16 + 4 * kNJ : 16, 0);   // VALU
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                           // one MFMA
                if constexpr (Q < kReads) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
            });
            if constexpr (kReads > kMfma) __builtin_amdgcn_sched_group_barrier(0x100, kReads - kMfma, 0);
        } else {
            static_for<0, kPairs>([&](auto) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
            });
            if constexpr (kMfma > kPairs) __builtin_amdgcn_sched_group_barrier(0x008, kMfma - kPairs, 0);
            if constexpr (kReads > kPairs) __builtin_amdgcn_sched_group_barrier(0x100, kReads - kPairs, 0);
        }
    };
    auto mainloop = [&](auto ml, auto zs) {
        Frag cur, nxt;
        // stage kt, the I-th stage of an unrolled unit of U stages (U a multiple of the ring depth
        // and, for fp8, of the stages per 128-wide K block), in ring slot S = I mod NS; fp8 K
        // blocks open at the stages with I * BK = 0 mod 128
        auto stage = [&](auto i, int kt) {
            constexpr int I = decltype(i)::value, S = I % NS;
            constexpr bool kOpens = kFp8 && (I * BK) % 128 == 0;
            const auto s = ic<S>{};
            static_for<0, KS>([&](auto ks) {
                constexpr int KSI = decltype(ks)::value;
                if constexpr (KSI + 1 == KS) {
                    wait_vmcnt<(NS - 2) * PER_STAGE>();
                    wait_lgkmcnt0();
                    stage_barrier();
                    issue(min(kt + NS, nk - 1), stA(s), stB(s), s);
                }
                __builtin_amdgcn_sched_barrier(0);
                constexpr int kRescale = (kOpens && KSI == 0) ? 1 : 0;
                mma(cur, ks, ml, zs, ic<kRescale>{});
                if constexpr (KSI + 1 < KS)
                    load_frag(s, ic<KSI + 1>{}, ml, zs, nxt, cur, kt);
                else
                    load_frag(ic<(S + 1) % NS>{}, ic<0>{}, ml, zs, nxt, cur, min(kt + 1, nk - 1));
                interleave(ic<(KSI + 1) % KS>{}, ml, zs, ic<kRescale>{});
                __builtin_amdgcn_sched_barrier(0);
                cur = nxt;
            });
        };
        wait_vmcnt<(NS - 1) * PER_STAGE>();
        wait_lgkmcnt0();
        stage_barrier();
        load_frag(ic<0>{}, ic<0>{}, ml, zs, cur, cur, 0);
        // whole turns of the ring without branches (a branch around a stage would make the
        // compiler lose track of which slot each DMA writes, and drain them all), then the rest
        int kt0 = 0;
        for (; kt0 + kUnit <= nk; kt0 += kUnit)
            static_for<0, kUnit>([&](auto i) { stage(i, kt0 + decltype(i)::value); });
        static_for<0, kUnit - 1>([&](auto i) {
            if (kt0 + decltype(i)::value < nk) stage(i, kt0 + decltype(i)::value);
        });
    };

    // outstanding stores of the zeroing loop must not count against the DMA waits below; the
    // barrier publishes the staged scale / token / gate tables
    wait_vmcnt<0>();
    __syncthreads();
    static_for<0, NS>([&](auto s) { issue(min(decltype(s)::value, nk - 1), stA(s), stB(s), s); });
    bool any_zero_scale = false;
    if constexpr (kFp8)
        for (int w = 0; w < kWavesN; ++w) any_zero_scale |= s_zeroblk[w] != 0;
    // one main loop per live sub-tile count, in steps of MLQ sub-tiles for tall tiles and for the
    // fp8-activation kernels (with steps of one their registers spilled in the common main loop;
    // with steps of two only the loop for zero block scales, which real weights rarely take,
    // spills)
    constexpr int MLQ = kMI > 4 || kAq ? 2 : 1;
    const int wrows = min(max(len - m0 - wm * kWaveRows, 0), kWaveRows);   // real rows of this wave
    constexpr bool kSkipPad = EPI == GEMM_DOWN ? GTr<WT>::SKIP_PAD_DN : GTr<WT>::SKIP_PAD_GU;
    const int mlive = kSkipPad ? __builtin_amdgcn_readfirstlane((wrows + 32 * MLQ - 1) / (32 * MLQ) * MLQ)
                               : (wrows > 0 || kWavesM == 1 ? kMI : 0);
    // (a wave of a tall tile may hold no real rows; it still moves its share of the stages)
    static_for<(kWavesM > 1 ? 0 : 1), kMI / MLQ + 1>([&](auto q) {
        constexpr int ML = decltype(q)::value * MLQ;
        if (mlive == ML) {
            if constexpr (kFp8) {
                if (any_zero_scale) mainloop(ic<ML>{}, ic<1>{});
                else mainloop(ic<ML>{}, ic<0>{});
            } else {
                mainloop(ic<ML>{}, ic<0>{});
            }
        }
    });
    wait_vmcnt<0>();   // the redundant tail stages
    if constexpr (kFp8) {
        // the accumulators hold the sum in units of the last block's scale
        const float sg = s_last[wn][0], su = s_last[wn][1];
#pragma unroll
        for (int i = 0; i < kMI; ++i)
#pragma unroll
            for (int j = 0; j < kNJ; ++j) acc[i][j] *= (EPI == GEMM_GATEUP && j >= kNJ / 2) ? su : sg;
    }

    // ---- epilogue: element e of a 32 x 32 tile in lane (fn, fq) is row 8 (e / 4) + 4 fq + e % 4,
    // column fn
    if constexpr (EPI == GEMM_GATEUP && kAq) {
        // fp8 activations: h = silu(gate) * up rounded to bf16, then quantised per row over the
        // tile's 128 h columns (one 128-channel block): the row's largest |h| over the 4 waves'
        // 32 columns each, its exponent, e4m3fn codes into hq and the exponent byte into hs.
        // A lane holds column fn of rows 8 (e / 4) + 4 fq + e % 4 of each 32-row sub-tile i.
        const int nbh = I / 128;
#pragma unroll
        for (int i = 0; i < kMI; ++i)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const float hv = bf16_to_f32(f32_to_bf16(silu_f32(acc[i][0][e]) * acc[i][1][e]));
                acc[i][0][e] = hv;
                // largest |h| of the row over the 32 lanes of this half-wave
                uint32_t m = __float_as_uint(fabsf(hv));
                m = max(m, dpp_u32<kDppRowRor1>(m));
                m = max(m, dpp_u32<kDppRowRor2>(m));
                m = max(m, dpp_u32<kDppRowRor4>(m));
                m = max(m, dpp_u32<kDppRowRor8>(m));
                m = max(m, static_cast<uint32_t>(__shfl_xor(static_cast<int>(m), 16)));
                if (fn == 0) s_hmax[wn][i * 32 + (e >> 2) * 8 + 4 * fq + (e & 3)] = __uint_as_float(m);
            }
        __syncthreads();
        if (t < kBM) {
            float m = s_hmax[0][t];
#pragma unroll
            for (int w = 1; w < kWavesN; ++w) m = fmaxf(m, s_hmax[w][t]);
            const int ex = act_scale_exp(m);
            s_hexp[t] = ex;
            if (m0 + t < len) a.wv.hs[static_cast<size_t>(beg + m0 + t) * nbh + nt] = static_cast<uint8_t>(ex + 127);
        }
        __syncthreads();
        const int col0 = nt * (kBN / 2) + wn * (kWaveCols / 2) + fn;
#pragma unroll
        for (int i = 0; i < kMI; ++i)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int rl = i * 32 + (e >> 2) * 8 + 4 * fq + (e & 3);
                if (m0 + rl < len)
                    a.wv.hq[static_cast<size_t>(beg + m0 + rl) * I + col0] =
                        static_cast<uint8_t>(e4m3_rne(ldexpf(acc[i][0][e], -s_hexp[rl])));
            }
    } else if constexpr (EPI == GEMM_GATEUP) {
        uint16_t *hout = static_cast<uint16_t *>(a.wv.h);
        const int col0 = nt * (kBN / 2) + wn * (kWaveCols / 2) + fn;
#pragma unroll
        for (int i = 0; i < kMI; ++i)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = m0 + wm * kWaveRows + i * 32 + (e >> 2) * 8 + 4 * fq + (e & 3);
                if (row < len) {
                    uint16_t *hrow = hout + static_cast<size_t>(beg + row) * I + col0;
#pragma unroll
                    for (int j = 0; j < kNJ / 2; ++j)
                        hrow[j * 32] = f32_to_bf16(silu_f32(acc[i][j][e]) * acc[i][j + kNJ / 2][e]);
                }
            }
    } else {
#pragma unroll
        for (int i = 0; i < kMI; ++i)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int rl = wm * kWaveRows + i * 32 + (e >> 2) * 8 + 4 * fq + (e & 3);
                if (m0 + rl < len) {
                    float *orow = a.out + static_cast<size_t>(s_tok[rl]) * H + nt * kBN + wn * kWaveCols + fn;
                    const float gw = s_gate[rl];
#pragma unroll
                    for (int j = 0; j < kNJ; ++j) unsafeAtomicAdd(orow + j * 32, gw * acc[i][j][e]);
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

// The grid is cut into launches of a few hundred to a thousand workgroups (GTr::CHUNK_GU,
// CHUNK_DN): the tiles of one launch start together and stay in step, so the tiles that share an
// activation tile (the N tiles of an M tile) or a weight tile (the M tiles of a band) read it
// while it is still in their XCD's L2.  Launched all at once, tiles drift apart in K as slots free
// up at different times, and the 4 MB L2 loses the shared rows before their last reader: the fp8
// gate/up GEMM of the DeepSeek-V3 prefill then fetched 10.8 GB per launch against 3.3 GB
// algorithmic.  Measured per dtype (gate/up, down; ms at DeepSeek-V3 / Qwen3 / DeepSeek-V4-Flash
// prefill): one launch 4.25 / 0.300 / 1.36 and 2.17 / 0.224 / 0.77; launches of 512 workgroups
// (one per slot of the chip) 2.70 / 0.265 / 0.944 and, for down, 1536: 1.64 / 0.257 / 0.578, 1024:
// 1.69 / 0.222 / 0.61; Qwen3's bf16 gate/up is best at 768 (0.252).
template <int WT, int EPI>
static void launch_tiles(const ExpertArgs &a, hipStream_t s, long tiles, int ntn) {
    const long chunk = EPI == GEMM_GATEUP ? GTr<WT>::CHUNK_GU : GTr<WT>::CHUNK_DN;
    for (long b = 0; b < tiles; b += chunk)
        hipLaunchKernelGGL((grouped_gemm<WT, EPI>), dim3(static_cast<unsigned>(std::min(chunk, tiles - b))),
                           dim3(kGemmThreads), 0, s, a, ntn, static_cast<int>(b));
}

template <int WT>
static hipError_t launch_gemm_wt(const ExpertArgs &a, hipStream_t s, const Prof &prof) {
    const long mtiles = max_mtiles(a);
    if (!prof.mark(1)) return hipErrorUnknown;
    if constexpr (WT == kWtFp8Act)   // x into e4m3fn codes and exponents
        if (hipError_t e = launch_act_quant_x(a, s); e != hipSuccess) return e;
    const int ntn_gu = a.I / (kBN / 2);
    launch_tiles<WT, GEMM_GATEUP>(a, s, mtiles * ntn_gu, ntn_gu);
    if (!prof.mark(2)) return hipErrorUnknown;
    const int ntn_dn = a.H / kBN;
    launch_tiles<WT, GEMM_DOWN>(a, s, mtiles * ntn_dn, ntn_dn);
    if (!prof.mark(3)) return hipErrorUnknown;
    return hipGetLastError();
}

hipError_t launch_gemm(const ExpertArgs &a, hipStream_t s, const Prof &prof) {
    if (a.act_quant) return launch_gemm_wt<kWtFp8Act>(a, s, prof);
    if (a.w_dtype == FT_DT_BF16) return launch_gemm_wt<FT_DT_BF16>(a, s, prof);
    if (a.w_dtype == FT_DT_MXFP4) return launch_gemm_wt<FT_DT_MXFP4>(a, s, prof);
    return launch_gemm_wt<FT_DT_FP8E4M3FN_B128>(a, s, prof);
}

}  // namespace ftmoe
