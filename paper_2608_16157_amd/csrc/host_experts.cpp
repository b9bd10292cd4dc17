// CPU branch of a layer step: the missing experts the cache plan leaves to the host execute
// there, straight from the host expert pool, and their gate-weighted outputs form the CPU
// partial sum that merges exactly with the GPU's (Section 3.2: the CPU consumes the host
// bandwidth a saturated PCIe fill leaves over; the two partial sums add up to the layer output.
// Section 4.1: the CPU workers are a native thread pool with SIMD kernels and in-kernel
// dequantisation, so the branch stays bandwidth-bound).
//
// Two phases over the listed experts, each split into independent work items that threads take
// from a shared counter:
//   gate/up: items of 32 intermediate rows of one expert: h = silu(W1 x) * (W3 x) for the
//            expert's tokens (every weight row is decoded to float once and used for all of them);
//   down   : items of 32 output columns: out[t][c] += gate * (W2[c] . h), experts in list order,
//            so every output element is summed in a fixed order (the result does not depend on
//            the thread count or timing).
// Weights are decoded exactly (bf16 by widening, fp8 e4m3fn and MXFP4 e2m1 from the format
// definitions times their scales) and every product accumulates in float32.  All code in this file is
// compiled for AVX2 + FMA; the entry point checks the CPU supports them before calling in.
#include <atomic>
#include <cmath>
#include <cstring>
#include <thread>
#include <vector>

#include "ftmoe_internal.h"

#pragma clang attribute push(__attribute__((target("avx2,fma"))), apply_to = function)

namespace ftmoe {
namespace {

constexpr int kRowsPerItem = 32;

// e4m3fn: 1 sign bit, 4 exponent bits (bias 7), 3 mantissa bits; exponent field 0 encodes
// subnormals m/8 * 2^-6; exponent 15 with mantissa 7 is NaN; there are no infinities.
float e4m3fn_to_float(uint8_t code) {
    const int s = code >> 7, e = (code >> 3) & 15, m = code & 7;
    float v;
    if (e == 15 && m == 7) v = NAN;
    else if (e == 0) v = std::ldexp(static_cast<float>(m) / 8.0f, -6);
    else v = std::ldexp(1.0f + static_cast<float>(m) / 8.0f, e - 7);
    return s ? -v : v;
}

struct Fp8Table {
    float v[256];
    Fp8Table() {
        for (int i = 0; i < 256; ++i) v[i] = e4m3fn_to_float(static_cast<uint8_t>(i));
    }
};

// e2m1: 1 sign bit, 2 exponent bits (bias 1), 1 mantissa bit; exponent field 0 encodes m/2.
float e2m1_to_float(uint8_t code) {
    const int e = (code >> 1) & 3, m = code & 1;
    const float v = e == 0 ? 0.5f * m : std::ldexp(1.0f + 0.5f * m, e - 1);
    return code & 8 ? -v : v;
}

// Both codes of every byte decoded at once: entry b = (element of the low nibble, of the high).
struct Fp4PairTable {
    float v[256][2];
    Fp4PairTable() {
        for (int b = 0; b < 256; ++b) {
            v[b][0] = e2m1_to_float(static_cast<uint8_t>(b & 15));
            v[b][1] = e2m1_to_float(static_cast<uint8_t>(b >> 4));
        }
    }
};

// e8m0 scale: 2^(s - 127), 255 is NaN.
float e8m0_to_float(uint8_t s) { return s == 255 ? NAN : std::ldexp(1.0f, static_cast<int>(s) - 127); }

float bf16_to_float(uint16_t b) {
    const uint32_t u = static_cast<uint32_t>(b) << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

// Row r (of nrows) of one expert's matrix with K columns, decoded to float.
void decode_row(const CpuBank &bank, int w_dtype, int nrows, int K, int r, float *dst) {
    if (w_dtype == FT_DT_F32) {
        std::memcpy(dst, static_cast<const float *>(bank.w) + static_cast<size_t>(r) * K, 4 * static_cast<size_t>(K));
    } else if (w_dtype == FT_DT_BF16) {
        const uint16_t *src = static_cast<const uint16_t *>(bank.w) + static_cast<size_t>(r) * K;
        for (int c = 0; c < K; ++c) dst[c] = bf16_to_float(src[c]);
    } else if (w_dtype == FT_DT_MXFP4) {
        static const Fp4PairTable pairs;
        const uint8_t *src = static_cast<const uint8_t *>(bank.w) + static_cast<size_t>(r) * (K / 2);
        // scales are run-major: run cb of row r at [cb][r]
        const uint8_t *sc = static_cast<const uint8_t *>(bank.s) + r;
        for (int cb = 0; cb < K / 32; ++cb) {
            const float s = e8m0_to_float(sc[static_cast<size_t>(cb) * nrows]);
            for (int j = cb * 16; j < cb * 16 + 16; ++j) {
                dst[2 * j] = pairs.v[src[j]][0] * s;
                dst[2 * j + 1] = pairs.v[src[j]][1] * s;
            }
        }
    } else {
        static const Fp8Table table;
        const uint8_t *src = static_cast<const uint8_t *>(bank.w) + static_cast<size_t>(r) * K;
        const float *sc = static_cast<const float *>(bank.s) + static_cast<size_t>(r / 128) * (K / 128);
        for (int cb = 0; cb < K / 128; ++cb) {
            const float s = sc[cb];
            for (int c = cb * 128; c < cb * 128 + 128; ++c) dst[c] = table.v[src[c]] * s;
        }
    }
}

// Dot product of two float vectors (n a multiple of 128) with 8 independent partial sums.
float dot(const float *a, const float *b, int n) {
    float s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int i = 0; i < n; i += 8)
#pragma clang loop vectorize(enable)
        for (int l = 0; l < 8; ++l) s[l] += a[i + l] * b[i + l];
    return ((s[0] + s[1]) + (s[2] + s[3])) + ((s[4] + s[5]) + (s[6] + s[7]));
}

template <class F>
void run_items(int n_items, int n_threads, F &&fn) {
    std::atomic<int> next{0};
    auto worker = [&]() {
        std::vector<float> scratch;
        for (int it = next.fetch_add(1); it < n_items; it = next.fetch_add(1)) fn(it, scratch);
    };
    const int nt = std::max(1, std::min(n_threads, n_items));
    std::vector<std::thread> pool;
    pool.reserve(nt - 1);
    for (int i = 1; i < nt; ++i) pool.emplace_back(worker);
    worker();
    for (auto &t : pool) t.join();
}

}  // namespace

void cpu_experts(const CpuExpertArgs &a) {
    const int H = a.H, I = a.I, k = a.k, T = a.T;
    const ExpertBytes eb = expert_bytes(a.w_dtype, H, I);
    // tokens and gates of every listed expert, in token order
    std::vector<std::vector<int>> toks(a.n_list);
    std::vector<std::vector<float>> gates(a.n_list);
    std::vector<int> pos_of(a.E, -1);
    for (int i = 0; i < a.n_list; ++i) pos_of[a.list[i]] = i;
    for (int t = 0; t < T; ++t)
        for (int j = 0; j < k; ++j) {
            const int e = a.topk_ids[static_cast<size_t>(t) * k + j];
            if (e >= 0 && e < a.E && pos_of[e] >= 0) {
                toks[pos_of[e]].push_back(t);
                gates[pos_of[e]].push_back(a.topk_w[static_cast<size_t>(t) * k + j]);
            }
        }
    // activations as float
    std::vector<float> xf(static_cast<size_t>(T) * H);
    for (size_t i = 0; i < xf.size(); ++i)
        xf[i] = a.x_dtype == FT_DT_F32 ? static_cast<const float *>(a.x)[i]
                                       : bf16_to_float(static_cast<const uint16_t *>(a.x)[i]);
    std::memset(a.out, 0, sizeof(float) * static_cast<size_t>(T) * H);

    auto bank13 = [&](int e) {
        CpuBank b;
        b.w = static_cast<const uint8_t *>(a.w13) + static_cast<size_t>(e) * eb.w13;
        b.s = a.s13 ? static_cast<const uint8_t *>(a.s13) + static_cast<size_t>(e) * eb.s13 : nullptr;
        return b;
    };
    auto bank2 = [&](int e) {
        CpuBank b;
        b.w = static_cast<const uint8_t *>(a.w2) + static_cast<size_t>(e) * eb.w2;
        b.s = a.s2 ? static_cast<const uint8_t *>(a.s2) + static_cast<size_t>(e) * eb.s2 : nullptr;
        return b;
    };

    // ---- gate/up
    std::vector<std::vector<float>> h(a.n_list);
    for (int i = 0; i < a.n_list; ++i) h[i].assign(toks[i].size() * static_cast<size_t>(I), 0.f);
    const int blocks_i = (I + kRowsPerItem - 1) / kRowsPerItem;
    std::vector<int> gu_items;
    for (int i = 0; i < a.n_list; ++i)
        if (!toks[i].empty())
            for (int b = 0; b < blocks_i; ++b) gu_items.push_back(i * blocks_i + b);
    run_items(static_cast<int>(gu_items.size()), a.n_threads, [&](int it, std::vector<float> &scr) {
        const int li = gu_items[it] / blocks_i, b = gu_items[it] % blocks_i;
        const int e = a.list[li];
        const CpuBank bk = bank13(e);
        scr.resize(2 * static_cast<size_t>(H));
        float *g = scr.data(), *u = scr.data() + H;
        for (int r = b * kRowsPerItem; r < std::min(I, (b + 1) * kRowsPerItem); ++r) {
            decode_row(bk, a.w_dtype, 2 * I, H, r, g);
            decode_row(bk, a.w_dtype, 2 * I, H, I + r, u);
            for (size_t n = 0; n < toks[li].size(); ++n) {
                const float *xv = xf.data() + static_cast<size_t>(toks[li][n]) * H;
                const float gs = dot(g, xv, H), us = dot(u, xv, H);
                h[li][n * I + r] = gs / (1.0f + std::exp(-gs)) * us;
            }
        }
    });

    // ---- down + gate-weighted combine
    const int blocks_c = (H + kRowsPerItem - 1) / kRowsPerItem;
    run_items(blocks_c, a.n_threads, [&](int b, std::vector<float> &scr) {
        scr.resize(I);
        float *w = scr.data();
        for (int li = 0; li < a.n_list; ++li) {
            if (toks[li].empty()) continue;
            const CpuBank bk = bank2(a.list[li]);
            for (int c = b * kRowsPerItem; c < std::min(H, (b + 1) * kRowsPerItem); ++c) {
                decode_row(bk, a.w_dtype, H, I, c, w);
                for (size_t n = 0; n < toks[li].size(); ++n)
                    a.out[static_cast<size_t>(toks[li][n]) * H + c] +=
                        gates[li][n] * dot(w, h[li].data() + n * I, I);
            }
        }
    });
}

}  // namespace ftmoe

#pragma clang attribute pop
