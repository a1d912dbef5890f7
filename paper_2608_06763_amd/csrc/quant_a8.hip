// Dynamic-A8 activation quantizer (Sec. 5.4, eq. a8-activation-scale and
// eq. a8-activation-quantization): per row
//   xbar = max(max_j |x_j|, eps),  d_x = xbar / 127,
//   x8_j = clip(round_half_away(x_j / d_x), -127, 127),
// both quotients IEEE binary32 divisions, eps = 1e-10 rounded to binary32.
//
// One workgroup per row.  Rows of up to 8 vectors per thread stay in registers
// between the maximum and the quantization pass (one read of the row); longer
// rows are read twice, the second time mostly from L2.  Loads and stores are
// 16-byte and 8-byte vectors.
#include "cq_device.h"
#include "cq_internal.h"
#include "a8_quant.h"

namespace cq {

// NV > 0: every thread holds its (at most NV) 16-byte vectors of the row in
// registers between the two passes; NV == 0: the second pass re-reads the row.
// T threads per row: 256 when there are enough rows to fill the chip, up to
// 1024 for a few long rows (a single-row call is one workgroup, so its time is
// that workgroup's latency).  Quotients use the reciprocal product with the
// exact division near rounding boundaries (a8_quant.h), bit-equal to x / d.
template <int XDT, int NV, int T>
__global__ void __launch_bounds__(T) quant_a8_kernel(const uint16_t *__restrict__ x, int64_t k,
                                                     int8_t *__restrict__ x8, float *__restrict__ dx) {
    constexpr int W = T / 64;
    __shared__ float red[W];
    const int64_t row = blockIdx.x;
    const uint16_t *xr = x + row * k;
    int8_t *qr = x8 + row * k;
    const int tid = threadIdx.x;
    const int64_t vecs = k >> 3;  // 8 activations per 16-byte vector (k % 32 == 0)

    float mx = 0.f;
    uint4 keep[NV > 0 ? NV : 1];
    if constexpr (NV > 0) {
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int64_t v = tid + int64_t(i) * T;
            keep[i] = v < vecs ? reinterpret_cast<const uint4 *>(xr)[v] : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < NV; ++i) mx = absmax8<XDT>(keep[i], mx);
    } else {
        for (int64_t v = tid; v < vecs; v += T) mx = absmax8<XDT>(reinterpret_cast<const uint4 *>(xr)[v], mx);
    }
    mx = wave_max(mx);
    if ((tid & 63) == 0) red[tid >> 6] = mx;
    __syncthreads();
    mx = red[0];
#pragma unroll
    for (int w = 1; w < W; ++w) mx = fmaxf(mx, red[w]);
    const float d = a8_row_scale(mx);
    const float rcp = __fdiv_rn(1.0f, d);
    if (tid == 0) dx[row] = d;

    if constexpr (NV > 0) {
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int64_t v = tid + int64_t(i) * T;
            if (v < vecs) reinterpret_cast<uint2 *>(qr)[v] = quantize8_rcp<XDT>(keep[i], d, rcp);
        }
    } else {
        for (int64_t v = tid; v < vecs; v += T)
            reinterpret_cast<uint2 *>(qr)[v] = quantize8_rcp<XDT>(reinterpret_cast<const uint4 *>(xr)[v], d, rcp);
    }
}

template <int XDT, int T>
static hipError_t quant_launch_t(const void *x, int64_t m, int64_t k, int8_t *x8, float *dx, hipStream_t stream) {
    const int64_t per_thread = ((k >> 3) + T - 1) / T;
    const uint16_t *xp = static_cast<const uint16_t *>(x);
    const dim3 grid(static_cast<uint32_t>(m)), block(T);
    if (per_thread <= 1) hipLaunchKernelGGL((quant_a8_kernel<XDT, 1, T>), grid, block, 0, stream, xp, k, x8, dx);
    else if (per_thread <= 2) hipLaunchKernelGGL((quant_a8_kernel<XDT, 2, T>), grid, block, 0, stream, xp, k, x8, dx);
    else if (per_thread <= 4) hipLaunchKernelGGL((quant_a8_kernel<XDT, 4, T>), grid, block, 0, stream, xp, k, x8, dx);
    else if (per_thread <= 8) hipLaunchKernelGGL((quant_a8_kernel<XDT, 8, T>), grid, block, 0, stream, xp, k, x8, dx);
    else hipLaunchKernelGGL((quant_a8_kernel<XDT, 0, T>), grid, block, 0, stream, xp, k, x8, dx);
    return hipGetLastError();
}

template <int XDT>
static hipError_t quant_launch(const void *x, int64_t m, int64_t k, int8_t *x8, float *dx, hipStream_t stream) {
    const int64_t vecs = k >> 3;
    if (m >= 2 * int64_t(device_cu_count()) || vecs <= 256) return quant_launch_t<XDT, 256>(x, m, k, x8, dx, stream);
    if (vecs <= 512) return quant_launch_t<XDT, 512>(x, m, k, x8, dx, stream);
    return quant_launch_t<XDT, 1024>(x, m, k, x8, dx, stream);
}

hipError_t launch_quant_a8(const void *x, int x_dt, int64_t m, int64_t k, int8_t *x8, float *dx,
                           hipStream_t stream) {
    if (m > 0x7fffffff) return hipErrorInvalidValue;
    if (x_dt == 0) return quant_launch<0>(x, m, k, x8, dx, stream);
    return quant_launch<1>(x, m, k, x8, dx, stream);
}

}  // namespace cq
