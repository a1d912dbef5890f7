// Dynamic-A8 activation quantizer (Sec. 5.4, eq. a8-activation-scale and
// eq. a8-activation-quantization): per row
//   xbar = max(max_j |x_j|, eps),  d_x = xbar / 127,
//   x8_j = clip(round_half_away(x_j / d_x), -127, 127),
// both quotients IEEE binary32 divisions, eps = 1e-10 rounded to binary32.
//
// One workgroup per row.  The row is read twice (max, then quantize); the second
// pass usually hits L2.  Loads and stores are 16-byte vectors.
#include "cq_device.h"
#include "cq_internal.h"

namespace cq {

constexpr float kEps = 1e-10f;

template <int XDT>
__global__ void __launch_bounds__(256) quant_a8_kernel(const uint16_t *__restrict__ x, int64_t k,
                                                       int8_t *__restrict__ x8, float *__restrict__ dx) {
    __shared__ float red[4];
    const int64_t row = blockIdx.x;
    const uint16_t *xr = x + row * k;
    int8_t *qr = x8 + row * k;
    const int tid = threadIdx.x;
    const int64_t vecs = k >> 3;  // 8 activations per 16-byte vector (k % 32 == 0)

    float mx = 0.f;
    for (int64_t v = tid; v < vecs; v += 256) {
        const uint4 p = reinterpret_cast<const uint4 *>(xr)[v];
        const uint32_t pw[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            mx = fmaxf(mx, fabsf(act_to_f32<XDT>(uint16_t(pw[e] & 0xffffu))));
            mx = fmaxf(mx, fabsf(act_to_f32<XDT>(uint16_t(pw[e] >> 16))));
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, kWave));
    if ((tid & 63) == 0) red[tid >> 6] = mx;
    __syncthreads();
    mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    const float xbar = fmaxf(mx, kEps);
    const float d = __fdiv_rn(xbar, 127.0f);
    if (tid == 0) dx[row] = d;

    for (int64_t v = tid; v < vecs; v += 256) {
        const uint4 p = reinterpret_cast<const uint4 *>(xr)[v];
        const uint32_t pw[4] = {p.x, p.y, p.z, p.w};
        uint32_t out[2] = {0u, 0u};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const uint16_t h = (e & 1) ? uint16_t(pw[e >> 1] >> 16) : uint16_t(pw[e >> 1] & 0xffffu);
            const float q = __fdiv_rn(act_to_f32<XDT>(h), d);
            float r = roundf(q);  // nearest, halfway cases away from zero
            r = fminf(fmaxf(r, -127.f), 127.f);
            out[e >> 2] |= (uint32_t(int(r)) & 0xffu) << (8 * (e & 3));
        }
        reinterpret_cast<uint2 *>(qr)[v] = make_uint2(out[0], out[1]);
    }
}

hipError_t launch_quant_a8(const void *x, int x_dt, int64_t m, int64_t k, int8_t *x8, float *dx,
                           hipStream_t stream) {
    if (m > 0x7fffffff) return hipErrorInvalidValue;
    if (x_dt == 0)
        hipLaunchKernelGGL(quant_a8_kernel<0>, dim3(unsigned(m)), dim3(256), 0, stream,
                           static_cast<const uint16_t *>(x), k, x8, dx);
    else
        hipLaunchKernelGGL(quant_a8_kernel<1>, dim3(unsigned(m)), dim3(256), 0, stream,
                           static_cast<const uint16_t *>(x), k, x8, dx);
    return hipGetLastError();
}

}  // namespace cq
