// fp8 activations (FT_ACT_FP8_1x128_POW2, an optional mode beside the paper's exact
// weight-only dequantisation): quantisation of the expert inputs x and, on the streaming path,
// of the SwiGLU activation h, per token (row) and 128-channel block to e4m3fn with a
// power-of-two scale.  One wave per (row, block), two values per lane.
#include "ftmoe_device.h"
#include "ftmoe_internal.h"

namespace ftmoe {

// MODE 0: e4m3fn codes into q [rows][ld] and the block's e8m0 byte (e + 127) into qs
// [rows][ld / 128].  MODE 1: the quantised values widened back to bf16 into deq (which may
// alias in).  Rows past min(nrows, the routed row count in meta) are skipped.
template <int MODE>
__global__ __launch_bounds__(256) void act_quant_kernel(const uint16_t *in, uint16_t *deq, uint8_t *q, uint8_t *qs,
                                                        int ld, int nrows, const int32_t *meta, int shared) {
    const int nb = ld / 128;
    const long gid = static_cast<long>(blockIdx.x) * 4 + threadIdx.x / kWave;
    int rows = nrows;
    if (meta) rows = min(rows, meta[2] + (shared ? meta[3] : 0));   // hit rows, then the shared rows
    const long row = gid / nb;
    const int b = static_cast<int>(gid % nb);
    if (row >= rows) return;
    const int lane = lane_id();
    const size_t o = static_cast<size_t>(row) * ld + b * 128 + 2 * lane;
    const uint32_t two = *reinterpret_cast<const uint32_t *>(in + o);
    const float v0 = bf16_to_f32(static_cast<uint16_t>(two & 0xFFFFu));
    const float v1 = bf16_to_f32(static_cast<uint16_t>(two >> 16));
    // largest magnitude of the block: float bits of non-negative values order as integers
    const uint32_t mb = wave_max_u32(max(__float_as_uint(fabsf(v0)), __float_as_uint(fabsf(v1))));
    const int e = act_scale_exp(__uint_as_float(mb));
    const uint32_t c0 = e4m3_rne(ldexpf(v0, -e)), c1 = e4m3_rne(ldexpf(v1, -e));
    if constexpr (MODE == 0) {
        *reinterpret_cast<uint16_t *>(q + o) = static_cast<uint16_t>(c0 | (c1 << 8));
        if (lane == 0) qs[static_cast<size_t>(row) * nb + b] = static_cast<uint8_t>(e + 127);
    } else {
        // a code times 2^e has at most 4 significant bits: exact in bf16
        const uint32_t d0 = f32_to_bf16(ldexpf(e4m3_value(c0), e)), d1 = f32_to_bf16(ldexpf(e4m3_value(c1), e));
        *reinterpret_cast<uint32_t *>(deq + o) = d0 | (d1 << 16);
    }
}

static unsigned quant_blocks(long rows, int ld) {
    return static_cast<unsigned>((rows * (ld / 128) + 3) / 4);
}

hipError_t launch_act_quant_x(const ExpertArgs &a, hipStream_t s) {
    const uint16_t *x = static_cast<const uint16_t *>(a.x);
    if (a.wv.xq)
        hipLaunchKernelGGL(act_quant_kernel<0>, dim3(quant_blocks(a.T, a.H)), dim3(256), 0, s, x, nullptr, a.wv.xq,
                           a.wv.xs, a.H, a.T, nullptr, 0);
    else
        hipLaunchKernelGGL(act_quant_kernel<1>, dim3(quant_blocks(a.T, a.H)), dim3(256), 0, s, x, a.wv.xd, nullptr,
                           nullptr, a.H, a.T, nullptr, 0);
    return hipGetLastError();
}

hipError_t launch_act_quant_h(const ExpertArgs &a, hipStream_t s) {
    uint16_t *h = static_cast<uint16_t *>(a.wv.h);
    const long rows = static_cast<long>(a.T) * a.k + a.T;
    hipLaunchKernelGGL(act_quant_kernel<1>, dim3(quant_blocks(rows, a.I)), dim3(256), 0, s, h, h, nullptr, nullptr,
                       a.I, static_cast<int>(rows), a.wv.grp_meta, a.shared);
    return hipGetLastError();
}

}  // namespace ftmoe
