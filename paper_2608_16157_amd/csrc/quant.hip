// fp8 activations (FT_ACT_FP8_1x128_POW2, an optional mode beside the paper's exact
// weight-only dequantisation): quantisation of the expert inputs x and, on the streaming path,
// of the SwiGLU activation h, per token (row) and 128-channel block to e4m3fn with a
// power-of-two scale.
#include "ftmoe_device.h"
#include "ftmoe_internal.h"

namespace ftmoe {

// MODE 0: e4m3fn codes into q [rows][ld] and the block's e8m0 byte (e + 127) into qs
// [rows][ld / 128].  MODE 1: the quantised values widened back to bf16 into deq (which may
// alias in).  Rows past min(nrows, the routed row count in meta) are skipped.  One 16-lane row
// of a wave per (row, block), 8 values (16 bytes) per lane: the block's maximum needs only
// rotations within the lane row, and each wave moves 1 KB per load.
template <int MODE>
__global__ __launch_bounds__(256) void act_quant_kernel(const uint16_t *in, uint16_t *deq, uint8_t *q, uint8_t *qs,
                                                        int ld, int nrows, const int32_t *meta, int shared) {
    const int nb = ld / 128;
    const long gid = (static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x) / 16;
    int rows = nrows;
    if (meta) rows = min(rows, meta[2] + (shared ? meta[3] : 0));   // hit rows, then the shared rows
    const long row = gid / nb;
    const int b = static_cast<int>(gid % nb);
    if (row >= rows) return;   // all 16 lanes of a (row, block) leave together
    const int sub = lane_id() & 15;
    const size_t o = static_cast<size_t>(row) * ld + b * 128 + 8 * sub;
    const uint4 raw = *reinterpret_cast<const uint4 *>(in + o);
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
    float v[8];
    uint32_t mb = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[2 * i] = bf16_to_f32(static_cast<uint16_t>(w[i] & 0xFFFFu));
        v[2 * i + 1] = bf16_to_f32(static_cast<uint16_t>(w[i] >> 16));
        // float bits of non-negative values order as integers
        mb = max(mb, max(__float_as_uint(fabsf(v[2 * i])), __float_as_uint(fabsf(v[2 * i + 1]))));
    }
    const int e = act_scale_exp(__uint_as_float(row_max_u32(mb)));
    uint32_t c[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = e4m3_rne(ldexpf(v[i], -e));
    if constexpr (MODE == 0) {
        const uint2 packed = {c[0] | (c[1] << 8) | (c[2] << 16) | (c[3] << 24),
                              c[4] | (c[5] << 8) | (c[6] << 16) | (c[7] << 24)};
        *reinterpret_cast<uint2 *>(q + o) = packed;
        if (sub == 0) qs[static_cast<size_t>(row) * nb + b] = static_cast<uint8_t>(e + 127);
    } else {
        // a code times 2^e has at most 4 significant bits: exact in bf16
        uint32_t d[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) d[i] = f32_to_bf16(ldexpf(e4m3_value(c[i]), e));
        *reinterpret_cast<uint4 *>(deq + o) = uint4{d[0] | (d[1] << 16), d[2] | (d[3] << 16), d[4] | (d[5] << 16),
                                                    d[6] | (d[7] << 16)};
    }
}

static unsigned quant_blocks(long rows, int ld) {
    return static_cast<unsigned>((rows * (ld / 128) + 15) / 16);   // 16 (row, block) pairs per workgroup
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
