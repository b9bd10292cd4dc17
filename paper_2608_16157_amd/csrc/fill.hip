// Cache fills and the exact merge of a layer step.
//
// cache_fill_kernel: the fills the cache plan decided (Section 3.2: the q filled experts are
// copied into cache slots over PCIe and then execute on the GPU; Section 4.1: the copy work
// list lives on the device with a valid count, every expert bank shares one expert -> slot
// mapping, so one fixed-shape launch serves every bank).  The grid is sized for the largest
// possible plan (max_fill experts x chunks of the largest bank row); blocks past the device-side
// fill count return at once, so the host never needs to know q.  Every block copies one chunk
// of each bank row (gate/up, down, and for fp8 the two scale tables) of one filled expert from
// the pinned host expert pool, read directly over PCIe, into the slot's row of the device banks.
// A slot row is a complete expert, so a fill is a plain row copy, never a relayout (Section 4.2).
//
// add_partial_kernel: out += other, the exact additive merge of the GPU and CPU partial sums
// (Section 3.2); `other` may be pinned host memory read over PCIe.
//
// stage_host_kernel: what the CPU branch of a hybrid step needs (plan counts, CPU expert list,
// routing, hidden states) written straight into pinned host staging over PCIe by one kernel,
// instead of one copy-engine command per buffer.
#include <algorithm>

#include "ftmoe_device.h"
#include "ftmoe_internal.h"

namespace ftmoe {

constexpr int kFillThreads = 256;

__device__ __forceinline__ void copy_chunk(const uint8_t *src, uint8_t *dst, size_t bytes, size_t lo,
                                           size_t hi) {
    if (lo >= bytes) return;
    hi = hi < bytes ? hi : bytes;
    if ((bytes & 15) == 0) {
        // 16-byte elements, 4 in flight per thread
        const size_t n = (hi - lo) / 16;
        const u32x4_t *s = reinterpret_cast<const u32x4_t *>(src + lo);
        u32x4_t *d = reinterpret_cast<u32x4_t *>(dst + lo);
        size_t i = threadIdx.x;
        for (; i + 3 * kFillThreads < n; i += 4 * kFillThreads) {
            const u32x4_t a = s[i], b = s[i + kFillThreads], c = s[i + 2 * kFillThreads],
                          e = s[i + 3 * kFillThreads];
            d[i] = a;
            d[i + kFillThreads] = b;
            d[i + 2 * kFillThreads] = c;
            d[i + 3 * kFillThreads] = e;
        }
        for (; i < n; i += kFillThreads) d[i] = s[i];
    } else {
        // scale tables: 4-byte elements
        const size_t n = (hi - lo) / 4;
        const uint32_t *s = reinterpret_cast<const uint32_t *>(src + lo);
        uint32_t *d = reinterpret_cast<uint32_t *>(dst + lo);
        for (size_t i = threadIdx.x; i < n; i += kFillThreads) d[i] = s[i];
    }
}

__global__ __launch_bounds__(kFillThreads) void cache_fill_kernel(FillArgs a) {
    const int i = blockIdx.y;
    if (i >= a.plan_counts[0]) return;
    const int e = a.fill_expert[i], v = a.fill_slot[i];
    if (e < 0 || e >= a.E || v < 0 || v >= a.n_slots) return;
    const size_t lo = static_cast<size_t>(blockIdx.x) * kFillChunk, hi = lo + kFillChunk;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        const size_t row = a.row_bytes[b];
        if (row == 0) continue;
        copy_chunk(a.host[b] + static_cast<size_t>(e) * row, a.dev[b] + static_cast<size_t>(v) * row, row,
                   lo, hi);
    }
}

__global__ __launch_bounds__(256) void add_partial_kernel(float *out, const float *other, size_t n4) {
    float4 *o = reinterpret_cast<float4 *>(out);
    const float4 *p = reinterpret_cast<const float4 *>(other);
    for (size_t i = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x; i < n4;
         i += static_cast<size_t>(gridDim.x) * 256) {
        float4 x = o[i];
        const float4 y = p[i];
        x.x += y.x;
        x.y += y.y;
        x.z += y.z;
        x.w += y.w;
        o[i] = x;
    }
}

__global__ __launch_bounds__(256) void stage_host_kernel(StageArgs a) {
    const size_t tid = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
    const size_t nth = static_cast<size_t>(gridDim.x) * 256;
    if (tid < 4) a.h_counts[tid] = a.counts[tid];
    for (size_t i = tid; i < static_cast<size_t>(a.E); i += nth) a.h_cpu[i] = a.cpu_expert[i];
    for (size_t i = tid; i < static_cast<size_t>(a.pk); i += nth) {
        a.h_ids[i] = a.topk_ids[i];
        a.h_w[i] = a.topk_w[i];
    }
    const u32x4_t *xs = reinterpret_cast<const u32x4_t *>(a.x);
    u32x4_t *xd = reinterpret_cast<u32x4_t *>(a.h_x);
    for (size_t i = tid; i < a.x16; i += nth) xd[i] = xs[i];
    __threadfence_system();
}

// Post: the step's task address, then the next sequence number (after the staging kernel, whose
// host writes are complete and fenced at system scope before this kernel starts).
__global__ void mailbox_post_kernel(HostMailbox *mb, uint64_t task) {
    if (threadIdx.x != 0) return;
    const uint64_t seq = __hip_atomic_load(&mb->posted, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_SYSTEM) + 1;
    __hip_atomic_store(&mb->task, task, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    __hip_atomic_store(&mb->posted, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Wait until the pool reports the last posted number as done.  Bounded: after 2^24 polls (tens
// of seconds) without an answer (the listener gone) it counts a timeout in the mailbox and
// returns, so the stream never hangs; the step's output is then incomplete.
constexpr uint64_t kMailboxSpins = 1ull << 24;
__global__ void mailbox_wait_kernel(HostMailbox *mb) {
    if (threadIdx.x != 0) return;
    const uint64_t seq = __hip_atomic_load(&mb->posted, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_SYSTEM);
    for (uint64_t i = 0; i < kMailboxSpins; ++i) {
        if (__hip_atomic_load(&mb->done, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_SYSTEM) == seq) return;
        __builtin_amdgcn_s_sleep(8);
    }
    const uint64_t n = __hip_atomic_load(&mb->timeouts, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    __hip_atomic_store(&mb->timeouts, n + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

hipError_t launch_mailbox_post(HostMailbox *mbox_dev, uint64_t task, hipStream_t s) {
    hipLaunchKernelGGL(mailbox_post_kernel, dim3(1), dim3(64), 0, s, mbox_dev, task);
    return hipGetLastError();
}

hipError_t launch_mailbox_wait(HostMailbox *mbox_dev, hipStream_t s) {
    hipLaunchKernelGGL(mailbox_wait_kernel, dim3(1), dim3(64), 0, s, mbox_dev);
    return hipGetLastError();
}

hipError_t launch_stage_host(const StageArgs &a, hipStream_t s) {
    const size_t work = std::max<size_t>(a.x16, std::max<size_t>(a.pk, a.E));
    const unsigned blocks = static_cast<unsigned>(std::min<size_t>(256, (work + 255) / 256));
    hipLaunchKernelGGL(stage_host_kernel, dim3(blocks ? blocks : 1), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_cache_fill(const FillArgs &a, int max_fill, hipStream_t s) {
    size_t longest = 0;
    for (int b = 0; b < 4; ++b) longest = a.row_bytes[b] > longest ? a.row_bytes[b] : longest;
    const unsigned chunks = static_cast<unsigned>((longest + kFillChunk - 1) / kFillChunk);
    hipLaunchKernelGGL(cache_fill_kernel, dim3(chunks, max_fill), dim3(kFillThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_add_partial(float *out, const float *other, size_t n, hipStream_t s) {
    const size_t n4 = n / 4;
    const unsigned blocks = static_cast<unsigned>(std::min<size_t>(4096, (n4 + 255) / 256));
    hipLaunchKernelGGL(add_partial_kernel, dim3(blocks ? blocks : 1), dim3(256), 0, s, out, other, n4);
    return hipGetLastError();
}

}  // namespace ftmoe
