// Grouped SwiGLU expert evaluation over slot-resident weights (Section 3.2: grouped evaluation
// of the GPU execution set; Section 4.2: every bank row is one slot, so a group's weights are
// addressed as bank + slot * expert_stride with no relayout), then the gate-weighted combine.
//
// General path, any token count and any weight dtype:
//   grouped_gemv<GATEUP>: h[r] = silu(W1 x_tok(r)) * (W3 x_tok(r))        per group, 8 h-columns/WG
//   grouped_gemv<DOWN>  : y[r] = gate(r) * W2 h[r]                         per group, 16 y-columns/WG
//   combine             : out[t] = sum_j y[row(t,j)] (+ y[shared row of t]) in fixed j order
// The weights stream from HBM once per (group, column tile); tokens of a group are the MFMA M
// dimension (16-row tiles), weight rows the N dimension, and the hidden/intermediate dimension
// is the contraction, split over the 4 waves of a workgroup in 128-wide blocks (the fp8 scale
// block size) and reduced through LDS.
#include "ftmoe_device.h"
#include "ftmoe_internal.h"

namespace ftmoe {

constexpr int kGemvThreads = 256;
constexpr int kGemvWaves = kGemvThreads / kWave;
constexpr int kMTiles = 4;                 // 16-row M tiles per pass (64 rows)
constexpr int kPassRows = 16 * kMTiles;

enum { EPI_GATEUP = 0, EPI_DOWN = 1 };

template <int WT> struct WTr;
template <> struct WTr<FT_DT_F32> { static constexpr int kLoads = 8, kElem = 4; };
template <> struct WTr<FT_DT_BF16> { static constexpr int kLoads = 4, kElem = 2; };
template <> struct WTr<FT_DT_FP8E4M3FN_B128> { static constexpr int kLoads = 2, kElem = 1; };

__device__ __forceinline__ u32x4_t ld16(const void *p) {
    return *reinterpret_cast<const u32x4_t *>(p);
}

// Element offset (within a 128-wide K block) of a lane's 16-byte weight load number c.
template <int WT> __device__ __forceinline__ int wofs(int c, int q) {
    if constexpr (WT == FT_DT_F32) return c * 16 + q * 4;
    else if constexpr (WT == FT_DT_BF16) return c * 32 + q * 8;
    else return c * 64 + q * 16;
}

// One 128-wide K block for one 16-row M tile: acc += A(rows, kblock) * B(kblock, 16 cols).
// `a_row` points at the activation row of this lane's M row (nullptr = padding row) already
// offset to the K block; activations are f32 for f32 weights, bf16 otherwise.
template <int WT>
__device__ __forceinline__ void mfma_kblock(const void *a_row, const u32x4_t (&w)[WTr<WT>::kLoads],
                                            const u32x4_t (&wcvt)[4], int q, floatx4_t &acc) {
    if constexpr (WT == FT_DT_F32) {
        const float *a = static_cast<const float *>(a_row);
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            u32x4_t av = a ? ld16(a + c * 16 + q * 4) : u32x4_t{0, 0, 0, 0};
#pragma unroll
            for (int i = 0; i < 4; ++i)
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(av[i]),
                                                           __uint_as_float(w[c][i]), acc, 0, 0, 0);
        }
    } else if constexpr (WT == FT_DT_BF16) {
        const uint16_t *a = static_cast<const uint16_t *>(a_row);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            u32x4_t av = a ? ld16(a + c * 32 + q * 8) : u32x4_t{0, 0, 0, 0};
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(av), as_bf16x8(w[c]), acc, 0, 0, 0);
        }
    } else {
        const uint16_t *a = static_cast<const uint16_t *>(a_row);
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            u32x4_t a0 = a ? ld16(a + c * 64 + q * 16) : u32x4_t{0, 0, 0, 0};
            u32x4_t a1 = a ? ld16(a + c * 64 + q * 16 + 8) : u32x4_t{0, 0, 0, 0};
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a0), as_bf16x8(wcvt[2 * c]), acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a1), as_bf16x8(wcvt[2 * c + 1]), acc, 0, 0, 0);
        }
    }
}

template <int WT, int EPI>
__global__ __launch_bounds__(kGemvThreads) void grouped_gemv(ExpertArgs a, int tiles) {
    __shared__ float s_red[kGemvWaves][kPassRows][16];
    const int g = blockIdx.x / tiles, tile = blockIdx.x % tiles;
    if (g >= a.wv.grp_meta[0]) return;
    const int slot = a.wv.grp_slot[g], beg = a.wv.grp_beg[g], len = a.wv.grp_len[g];
    const int H = a.H, I = a.I;
    const int K = EPI == EPI_GATEUP ? H : I;
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int n = lane & 15, q = lane >> 4;
    // weight row of this lane's N column
    const int wrow = EPI == EPI_GATEUP ? (n < 8 ? tile * 8 + n : I + tile * 8 + n - 8) : tile * 16 + n;
    const size_t wstride = static_cast<size_t>(EPI == EPI_GATEUP ? 2 * I : H) * K;  // per slot
    const uint8_t *wbase = static_cast<const uint8_t *>(EPI == EPI_GATEUP ? a.w13 : a.w2) +
                           (static_cast<size_t>(slot) * wstride + static_cast<size_t>(wrow) * K) *
                               WTr<WT>::kElem;
    const float *sbase = nullptr;
    if constexpr (WT == FT_DT_FP8E4M3FN_B128) {
        const float *s = EPI == EPI_GATEUP ? a.s13 : a.s2;
        const int nkb = K / 128, nrb = (EPI == EPI_GATEUP ? 2 * I : H) / 128;
        sbase = s + (static_cast<size_t>(slot) * nrb + wrow / 128) * nkb;
    }
    const int nkb = K / 128;
    const size_t a_elem = (WT == FT_DT_F32) ? 4 : 2;

    for (int r0 = 0; r0 < len; r0 += kPassRows) {
        // activation row pointers of this lane's M row in each M tile
        const uint8_t *arow[kMTiles];
#pragma unroll
        for (int mt = 0; mt < kMTiles; ++mt) {
            const int r = r0 + mt * 16 + n;
            arow[mt] = nullptr;
            if (r < len) {
                if constexpr (EPI == EPI_GATEUP) {
                    const int tok = a.wv.row_tok[beg + r];
                    arow[mt] = static_cast<const uint8_t *>(a.x) + static_cast<size_t>(tok) * H * a_elem;
                } else {
                    arow[mt] = static_cast<const uint8_t *>(a.wv.h) + static_cast<size_t>(beg + r) * I * a_elem;
                }
            }
        }
        const int nmt = min(kMTiles, (len - r0 + 15) / 16);
        floatx4_t acc[kMTiles];
#pragma unroll
        for (int mt = 0; mt < kMTiles; ++mt) acc[mt] = floatx4_t{0.f, 0.f, 0.f, 0.f};

        for (int kb = wave; kb < nkb; kb += kGemvWaves) {
            u32x4_t w[WTr<WT>::kLoads];
#pragma unroll
            for (int c = 0; c < WTr<WT>::kLoads; ++c)
                w[c] = ld16(wbase + static_cast<size_t>(kb * 128 + wofs<WT>(c, q)) * WTr<WT>::kElem);
            u32x4_t wcvt[4];
            if constexpr (WT == FT_DT_FP8E4M3FN_B128) {
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    wcvt[2 * c] = fp8x8_to_bf16x8(w[c][0], w[c][1]);
                    wcvt[2 * c + 1] = fp8x8_to_bf16x8(w[c][2], w[c][3]);
                }
            }
            const size_t koff = static_cast<size_t>(kb) * 128 * a_elem;
#pragma unroll
            for (int mt = 0; mt < kMTiles; ++mt) {
                if (mt < nmt) {
                    const void *ap = arow[mt] ? arow[mt] + koff : nullptr;
                    if constexpr (WT == FT_DT_FP8E4M3FN_B128) {
                        floatx4_t part{0.f, 0.f, 0.f, 0.f};
                        mfma_kblock<WT>(ap, w, wcvt, q, part);
                        const float sc = sbase[kb];
#pragma unroll
                        for (int i = 0; i < 4; ++i) acc[mt][i] += sc * part[i];
                    } else {
                        mfma_kblock<WT>(ap, w, wcvt, q, acc[mt]);
                    }
                }
            }
        }
        // cross-wave reduction: lane holds D[m = 4q + i][n] of each M tile
#pragma unroll
        for (int mt = 0; mt < kMTiles; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) s_red[wave][mt * 16 + 4 * q + i][n] = acc[mt][i];
        __syncthreads();
        if constexpr (EPI == EPI_GATEUP) {
            // 64 rows x 8 columns of h per pass
            for (int idx = threadIdx.x; idx < kPassRows * 8; idx += kGemvThreads) {
                const int m = idx / 8, c = idx % 8;
                const int r = r0 + m;
                if (r < len) {
                    float gsum = 0.f, usum = 0.f;
#pragma unroll
                    for (int w = 0; w < kGemvWaves; ++w) {
                        gsum += s_red[w][m][c];
                        usum += s_red[w][m][c + 8];
                    }
                    const float hv = silu_f32(gsum) * usum;
                    const size_t o = static_cast<size_t>(beg + r) * I + tile * 8 + c;
                    if constexpr (WT == FT_DT_F32) static_cast<float *>(a.wv.h)[o] = hv;
                    else static_cast<uint16_t *>(a.wv.h)[o] = f32_to_bf16(hv);
                }
            }
        } else {
            for (int idx = threadIdx.x; idx < kPassRows * 16; idx += kGemvThreads) {
                const int m = idx / 16, c = idx % 16;
                const int r = r0 + m;
                if (r < len) {
                    float s = 0.f;
#pragma unroll
                    for (int w = 0; w < kGemvWaves; ++w) s += s_red[w][m][c];
                    a.wv.y[static_cast<size_t>(beg + r) * H + tile * 16 + c] = a.wv.row_gate[beg + r] * s;
                }
            }
        }
        __syncthreads();
    }
}

// out[t][c] = sum_j y[row(t, j)][c] over hit pairs in j order, then the shared expert's row.
__global__ __launch_bounds__(256) void combine(ExpertArgs a) {
    const int c = (blockIdx.x * 256 + threadIdx.x) * 4;
    if (c >= a.H) return;
    const int nh = a.wv.grp_meta[2];
    for (int t = blockIdx.y; t < a.T; t += gridDim.y) {
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int j = 0; j < a.k; ++j) {
            const int r = a.wv.pair_row[t * a.k + j];
            if (r >= 0) {
                const float4 v = *reinterpret_cast<const float4 *>(a.wv.y + static_cast<size_t>(r) * a.H + c);
                acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
            }
        }
        if (a.shared) {
            const float4 v = *reinterpret_cast<const float4 *>(a.wv.y + static_cast<size_t>(nh + t) * a.H + c);
            acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
        }
        *reinterpret_cast<float4 *>(a.out + static_cast<size_t>(t) * a.H + c) = acc;
    }
}

template <int WT>
static hipError_t launch_general(const ExpertArgs &a, hipStream_t s) {
    const int tiles_gu = a.I / 8, tiles_dn = a.H / 16;
    if (a.max_groups > 0) {
        hipLaunchKernelGGL((grouped_gemv<WT, EPI_GATEUP>), dim3(a.max_groups * tiles_gu),
                           dim3(kGemvThreads), 0, s, a, tiles_gu);
        hipLaunchKernelGGL((grouped_gemv<WT, EPI_DOWN>), dim3(a.max_groups * tiles_dn),
                           dim3(kGemvThreads), 0, s, a, tiles_dn);
    }
    hipLaunchKernelGGL(combine, dim3((a.H / 4 + 255) / 256, min(a.T, 65535)), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_experts(const ExpertArgs &a, hipStream_t s) {
    switch (a.w_dtype) {
        case FT_DT_F32: return launch_general<FT_DT_F32>(a, s);
        case FT_DT_BF16: return launch_general<FT_DT_BF16>(a, s);
        default: return launch_general<FT_DT_FP8E4M3FN_B128>(a, s);
    }
}

}  // namespace ftmoe
