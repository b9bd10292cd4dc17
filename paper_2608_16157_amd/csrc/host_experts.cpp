// CPU branch of a layer step: the missing experts the cache plan leaves to the host execute
// there, straight from the host expert pool, and their gate-weighted outputs form the CPU
// partial sum that merges exactly with the GPU's (Section 3.2: the CPU consumes the host
// bandwidth a saturated PCIe fill leaves over; the two partial sums add up to the layer output.
// Section 4.1: the CPU workers are a native thread pool with SIMD kernels and in-kernel
// dequantisation, so the branch stays bandwidth-bound).
//
// Two phases over the listed experts, each split into independent work items that the threads of
// a persistent worker pool (created once, optionally pinned one per physical core) take from a
// shared counter:
//   gate/up: items of 32 intermediate rows of one expert: h = silu(W1 x) * (W3 x) for the
//            expert's tokens (every weight row is decoded to float once and used for all of them);
//   down   : items of 32 output columns: out[t][c] += gate * (W2[c] . h), experts in list order,
//            so every output element is summed in a fixed order (the result does not depend on
//            the thread count or timing).
// Weights are decoded exactly (bf16 by widening, fp8 e4m3fn and MXFP4 e2m1 from the format
// definitions times their scales) and every product accumulates in float32.  As on the GPU, h is
// held as bfloat16 values (rounded to nearest even) for all but float32 layers.  All code in this file is
// compiled for AVX2 + FMA; the entry point checks the CPU supports them before calling in.
#include <pthread.h>
#include <sched.h>

#include <atomic>
#include <chrono>
#include <cmath>
#include <condition_variable>
#include <cstdio>
#include <cstring>
#include <functional>
#include <mutex>
#include <set>
#include <thread>
#include <utility>
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

// Nearest bfloat16 value of a finite float (round half to even on the dropped 16 bits).
float round_to_bf16(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    u += 0x7FFFu + ((u >> 16) & 1u);
    u &= 0xFFFF0000u;
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

}  // namespace

#pragma clang attribute pop

// ---- the worker pool (plain x86-64 code: created and driven without the AVX2 check)

CpuPool::~CpuPool() {
    quit.store(true);
    if (listener.joinable()) listener.join();
    {
        std::lock_guard<std::mutex> lk(mu);
        stop = true;
    }
    cv_work.notify_all();
    for (auto &t : workers) t.join();
    if (mbox) (void)hipHostFree(mbox);
}

// Polls the mailbox: a new posted number means the device has staged a step's inputs in host
// memory; run its task, then report the number as done.  Spins with a pause while work arrives,
// and backs off to short sleeps after a millisecond without any.
void CpuPool::listen_loop() {
    uint64_t seen = __atomic_load_n(&mbox->posted, __ATOMIC_ACQUIRE);
    auto idle_since = std::chrono::steady_clock::now();
    while (!quit.load(std::memory_order_relaxed)) {
        const uint64_t v = __atomic_load_n(&mbox->posted, __ATOMIC_ACQUIRE);
        if (v != seen) {
            void *task = reinterpret_cast<void *>(__atomic_load_n(&mbox->task, __ATOMIC_ACQUIRE));
            if (task) task_fn(task);
            seen = v;
            __atomic_store_n(&mbox->done, v, __ATOMIC_RELEASE);
            idle_since = std::chrono::steady_clock::now();
            continue;
        }
        if (std::chrono::steady_clock::now() - idle_since < std::chrono::milliseconds(1))
            __builtin_ia32_pause();
        else
            std::this_thread::sleep_for(std::chrono::microseconds(20));
    }
}

void CpuPool::worker_loop() {
    std::vector<float> scratch;
    uint64_t seen = 0;
    for (;;) {
        std::unique_lock<std::mutex> lk(mu);
        cv_work.wait(lk, [&] { return stop || gen != seen; });
        if (stop) return;
        seen = gen;
        const Job *job = current;
        lk.unlock();
        for (int it = next.fetch_add(1); it < job->n; it = next.fetch_add(1)) job->fn(it, scratch);
        lk.lock();
        if (--busy == 0) cv_done.notify_all();
    }
}

void CpuPool::run(int n_items, const std::function<void(int, std::vector<float> &)> &fn) {
    if (n_items <= 0) return;
    std::lock_guard<std::mutex> one(run_mu);   // one job at a time
    Job job{n_items, fn};
    std::unique_lock<std::mutex> lk(mu);
    current = &job;
    next.store(0);
    busy = static_cast<int>(workers.size());
    ++gen;
    cv_work.notify_all();
    cv_done.wait(lk, [&] { return busy == 0; });
    current = nullptr;
}

// The CPUs of this process's affinity mask, one hardware thread of every physical core first
// (the first seen of each (package, core) pair, in CPU order), then the other hardware threads.
static std::vector<int> physical_cores() {
    cpu_set_t set;
    CPU_ZERO(&set);
    std::vector<int> out;
    if (sched_getaffinity(0, sizeof(set), &set) != 0) return out;
    std::set<std::pair<int, int>> seen;
    std::vector<int> rest;
    for (int c = 0; c < CPU_SETSIZE; ++c) {
        if (!CPU_ISSET(c, &set)) continue;
        int pkg = 0, core = c;
        char path[128];
        std::snprintf(path, sizeof(path), "/sys/devices/system/cpu/cpu%d/topology/core_id", c);
        if (FILE *f = std::fopen(path, "r")) {
            if (std::fscanf(f, "%d", &core) != 1) core = c;
            std::fclose(f);
        }
        std::snprintf(path, sizeof(path), "/sys/devices/system/cpu/cpu%d/topology/physical_package_id", c);
        if (FILE *f = std::fopen(path, "r")) {
            if (std::fscanf(f, "%d", &pkg) != 1) pkg = 0;
            std::fclose(f);
        }
        (seen.insert({pkg, core}).second ? out : rest).push_back(c);
    }
    out.insert(out.end(), rest.begin(), rest.end());
    return out;
}

CpuPool *CpuPool::create(int n_threads, bool pin, void (*task_fn)(void *)) {
    const std::vector<int> cores = physical_cores();
    if (n_threads <= 0) n_threads = cores.empty() ? 1 : static_cast<int>(cores.size());
    CpuPool *p = new (std::nothrow) CpuPool();
    if (!p) return nullptr;
    p->task_fn = task_fn;
    // the mailbox needs pinned host memory the device can reach; without a device the pool
    // still serves ft_cpu_experts (and hybrid steps hand it over with a host function)
    void *mb = nullptr, *mbd = nullptr;
    if (hipHostMalloc(&mb, sizeof(HostMailbox), hipHostMallocDefault) == hipSuccess && mb) {
        p->mbox = static_cast<HostMailbox *>(mb);
        std::memset(p->mbox, 0, sizeof(HostMailbox));
        if (hipHostGetDevicePointer(&mbd, mb, 0) == hipSuccess && mbd)
            p->mbox_dev = static_cast<HostMailbox *>(mbd);
    } else {
        (void)hipGetLastError();   // leave no sticky error for the caller's next HIP call
    }
    try {
        if (p->mbox_dev) p->listener = std::thread([p] { p->listen_loop(); });
        for (int i = 0; i < n_threads; ++i) {
            p->workers.emplace_back([p] { p->worker_loop(); });
            if (pin && !cores.empty()) {
                cpu_set_t one;
                CPU_ZERO(&one);
                CPU_SET(cores[i % cores.size()], &one);
                (void)pthread_setaffinity_np(p->workers.back().native_handle(), sizeof(one), &one);
                p->cpus.push_back(cores[i % cores.size()]);
            } else {
                p->cpus.push_back(-1);
            }
        }
    } catch (...) {
        delete p;
        return nullptr;
    }
    return p;
}

#pragma clang attribute push(__attribute__((target("avx2,fma"))), apply_to = function)

namespace {

// Runs fn(item, scratch) for every item, on the pool's workers (the caller waits) or, without a
// pool, on the calling thread.
template <class F>
void run_items(CpuPool *pool, int n_items, F &&fn) {
    if (!pool || pool->workers.empty()) {
        std::vector<float> scratch;
        for (int it = 0; it < n_items; ++it) fn(it, scratch);
        return;
    }
    pool->run(n_items, std::function<void(int, std::vector<float> &)>(fn));
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
    run_items(a.pool, static_cast<int>(gu_items.size()), [&](int it, std::vector<float> &scr) {
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
                const float hv = gs / (1.0f + std::exp(-gs)) * us;
                h[li][n * I + r] = a.w_dtype == FT_DT_F32 ? hv : round_to_bf16(hv);
            }
        }
    });

    // ---- down + gate-weighted combine
    const int blocks_c = (H + kRowsPerItem - 1) / kRowsPerItem;
    run_items(a.pool, blocks_c, [&](int b, std::vector<float> &scr) {
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
