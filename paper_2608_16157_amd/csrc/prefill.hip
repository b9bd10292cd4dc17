// Full-layer double-buffered prefill (Section 3.1, "Prefill Codesign"; Section 5, "Pipelined
// prefill").  Prefill routes nearly every expert of every layer, so no expert is fetched on
// demand: two device buffers, each able to hold the complete expert set of one layer, take
// turns.  While the GPU evaluates layer l from one buffer, a transfer stream loads all experts
// of layer l + 1 into the other, before that layer's routing is known; then the roles swap.
// With overlap off the load of layer l + 1 starts only after layer l is evaluated (the
// serialised schedule the paper's ablation compares against).
//
// Host-side orchestration only: the loads are DMA-engine copies (hipMemcpyAsync from pinned
// memory, so no compute unit is taken from the evaluation), the evaluation is ft_moe_forward,
// and the two streams are ordered with events.  Nothing here blocks the host.
#include <hip/hip_runtime.h>

#include "ftmoe_internal.h"

namespace {

struct EventSet {
    // [0] start, [1..2] buffer b loaded, [3..4] buffer b released by the evaluation
    hipEvent_t ev[5] = {};
    bool create() {
        for (auto &e : ev)
            if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return false;
        return true;
    }
    ~EventSet() {
        // a pending event may be destroyed: its resources are released once it completes
        for (auto e : ev)
            if (e) (void)hipEventDestroy(e);
    }
};

bool pinned(const void *p) {
    void *mapped = nullptr;
    return hipHostGetDevicePointer(&mapped, const_cast<void *>(p), 0) == hipSuccess && mapped;
}

}  // namespace

extern "C" ft_status_t ft_prefill_layers(const ft_moe_desc_t *desc, int32_t n_layers,
                                         const ft_banks_t *host_layers, const ft_banks_t *dev_buf,
                                         const int32_t *slot_table, const float *const *logits,
                                         const void *const *x, int32_t T, float *const *out,
                                         const ft_route_t *route, void *ws, size_t ws_bytes,
                                         int32_t overlap, void *stream, void *copy_stream) {
    if (!desc || !host_layers || !dev_buf || !logits || !x || !out || !route) return FT_ERR_NULL;
    if (n_layers < 0 || T < 0 || (overlap != 0 && overlap != 1)) return FT_ERR_SHAPE;
    if (overlap && (!copy_stream || copy_stream == stream)) return FT_ERR_SHAPE;
    if (ft_moe_workspace_bytes(desc, 1) == 0) return FT_ERR_SHAPE;
    if (n_layers == 0 || T == 0) return FT_OK;
    const size_t S = desc->n_slots > 0 ? desc->n_slots : 0;
    // bytes of one complete bank (all n_slots rows) of each tensor
    const ftmoe::ExpertBytes eb = ftmoe::expert_bytes(desc->w_dtype, desc->hidden, desc->inter);
    const size_t bank[4] = {S * eb.w13, S * eb.w2, S * eb.s13, S * eb.s2};
    auto ptrs = [](const ft_banks_t &b, int i) -> const void * {
        return i == 0 ? b.w13 : i == 1 ? b.w2 : i == 2 ? b.s13 : b.s2;
    };
    for (int i = 0; i < 4; ++i) {
        if (!bank[i]) continue;
        if (!ptrs(dev_buf[0], i) || !ptrs(dev_buf[1], i)) return FT_ERR_NULL;
        if (ptrs(dev_buf[0], i) == ptrs(dev_buf[1], i)) return FT_ERR_SHAPE;
        for (int l = 0; l < n_layers; ++l)
            if (!ptrs(host_layers[l], i)) return FT_ERR_NULL;
    }
    // every layer's evaluation is checked before anything is enqueued
    for (int l = 0; l < n_layers; ++l)
        for (int b = 0; b < 2; ++b)
            if (ft_status_t st = ftmoe::check_forward(desc, &dev_buf[b], logits[l], slot_table, x[l], T, out[l],
                                                      route, ws, ws_bytes);
                st != FT_OK)
                return st;
    // the loads must be asynchronous DMA from pinned memory (pageable memory is rejected)
    for (int l = 0; l < n_layers; ++l)
        for (int i = 0; i < 4; ++i)
            if (bank[i] && !pinned(ptrs(host_layers[l], i))) return FT_ERR_SHAPE;

    const hipStream_t s = static_cast<hipStream_t>(stream);
    const hipStream_t cs = overlap ? static_cast<hipStream_t>(copy_stream) : s;
    EventSet E;
    if (!E.create()) return FT_ERR_HIP;
    hipEvent_t *loaded = E.ev + 1, *released = E.ev + 3;

    auto load = [&](int l, int b) -> bool {
        for (int i = 0; i < 4; ++i)
            if (bank[i] && hipMemcpyAsync(const_cast<void *>(ptrs(dev_buf[b], i)), ptrs(host_layers[l], i),
                                          bank[i], hipMemcpyHostToDevice, cs) != hipSuccess)
                return false;
        return hipEventRecord(loaded[b], cs) == hipSuccess;
    };
    // the transfer stream starts after everything the caller enqueued on `stream`
    if (hipEventRecord(E.ev[0], s) != hipSuccess || hipStreamWaitEvent(cs, E.ev[0], 0) != hipSuccess)
        return FT_ERR_HIP;
    if (!load(0, 0)) return FT_ERR_HIP;
    for (int l = 0; l < n_layers; ++l) {
        const int b = l & 1;
        if (overlap && l + 1 < n_layers) {
            // the other buffer is free once layer l - 1 is evaluated
            if (l >= 1 && hipStreamWaitEvent(cs, released[b ^ 1], 0) != hipSuccess) return FT_ERR_HIP;
            if (!load(l + 1, b ^ 1)) return FT_ERR_HIP;
        }
        if (hipStreamWaitEvent(s, loaded[b], 0) != hipSuccess) return FT_ERR_HIP;
        if (ft_status_t st = ft_moe_forward(desc, &dev_buf[b], logits[l], slot_table, x[l], T, out[l], route,
                                            ws, ws_bytes, stream);
            st != FT_OK)
            return st;
        if (hipEventRecord(released[b], s) != hipSuccess) return FT_ERR_HIP;
        if (!overlap && l + 1 < n_layers && !load(l + 1, b ^ 1)) return FT_ERR_HIP;
    }
    return FT_OK;
}
