// Dynamic-A8 activation quantizer (Sec. 5.4, eq. a8-activation-scale and
// eq. a8-activation-quantization): per row
//   xbar = max(max_j |x_j|, eps),  d_x = xbar / 127,
//   x8_j = clip(round_half_away(x_j / d_x), -127, 127),
// both quotients IEEE binary32 divisions, eps = 1e-10 rounded to binary32.
//
// One workgroup per row.  Rows of up to 16384 activations stay in registers
// between the maximum and the quantization pass (one read of the row); longer
// rows are read twice, the second time mostly from L2.  Loads and stores are
// 16-byte and 8-byte vectors.
#include "cq_device.h"
#include "cq_internal.h"
#include "a8_quant.h"

namespace cq {

// NV > 0: every thread holds its (at most NV) 16-byte vectors of the row in
// registers between the two passes; NV == 0: the second pass re-reads the row.
template <int XDT, int NV>
__global__ void __launch_bounds__(256) quant_a8_kernel(const uint16_t *__restrict__ x, int64_t k,
                                                       int8_t *__restrict__ x8, float *__restrict__ dx) {
    __shared__ float red[4];
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
            const int64_t v = tid + int64_t(i) * 256;
            keep[i] = v < vecs ? reinterpret_cast<const uint4 *>(xr)[v] : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < NV; ++i) mx = absmax8<XDT>(keep[i], mx);
    } else {
        for (int64_t v = tid; v < vecs; v += 256) mx = absmax8<XDT>(reinterpret_cast<const uint4 *>(xr)[v], mx);
    }
    mx = wave_max(mx);
    if ((tid & 63) == 0) red[tid >> 6] = mx;
    __syncthreads();
    mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    const float d = a8_row_scale(mx);
    if (tid == 0) dx[row] = d;

    if constexpr (NV > 0) {
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int64_t v = tid + int64_t(i) * 256;
            if (v < vecs) reinterpret_cast<uint2 *>(qr)[v] = quantize8<XDT>(keep[i], d);
        }
    } else {
        for (int64_t v = tid; v < vecs; v += 256)
            reinterpret_cast<uint2 *>(qr)[v] = quantize8<XDT>(reinterpret_cast<const uint4 *>(xr)[v], d);
    }
}

template <int XDT>
static hipError_t quant_launch(const void *x, int64_t m, int64_t k, int8_t *x8, float *dx, hipStream_t stream) {
    const int64_t per_thread = ((k >> 3) + 255) / 256;
    const uint16_t *xp = static_cast<const uint16_t *>(x);
    const dim3 grid(static_cast<uint32_t>(m)), block(256);
    if (per_thread <= 1) hipLaunchKernelGGL((quant_a8_kernel<XDT, 1>), grid, block, 0, stream, xp, k, x8, dx);
    else if (per_thread <= 2) hipLaunchKernelGGL((quant_a8_kernel<XDT, 2>), grid, block, 0, stream, xp, k, x8, dx);
    else if (per_thread <= 4) hipLaunchKernelGGL((quant_a8_kernel<XDT, 4>), grid, block, 0, stream, xp, k, x8, dx);
    else if (per_thread <= 8) hipLaunchKernelGGL((quant_a8_kernel<XDT, 8>), grid, block, 0, stream, xp, k, x8, dx);
    else hipLaunchKernelGGL((quant_a8_kernel<XDT, 0>), grid, block, 0, stream, xp, k, x8, dx);
    return hipGetLastError();
}

hipError_t launch_quant_a8(const void *x, int x_dt, int64_t m, int64_t k, int8_t *x8, float *dx,
                           hipStream_t stream) {
    if (m > 0x7fffffff) return hipErrorInvalidValue;
    if (x_dt == 0) return quant_launch<0>(x, m, k, x8, dx, stream);
    return quant_launch<1>(x, m, k, x8, dx, stream);
}

}  // namespace cq
