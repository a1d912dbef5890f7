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

namespace cq {

constexpr float kEps = 1e-10f;

// Maximum over the 64 lanes of a wavefront (every lane active), DPP moves
// within rows of 16 lanes, then readlane across the four rows.
__device__ __forceinline__ float wave_max(float v) {
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xb1, 0xf, 0xf, false)));
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4e, 0xf, 0xf, false)));
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xf, 0xf, false)));
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xf, 0xf, false)));
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

template <int XDT>
__device__ __forceinline__ uint2 quantize8(const uint4 &p, float d) {
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
    return make_uint2(out[0], out[1]);
}

template <int XDT>
__device__ __forceinline__ float absmax8(const uint4 &p, float mx) {
    const uint32_t pw[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        mx = fmaxf(mx, fabsf(act_to_f32<XDT>(uint16_t(pw[e] & 0xffffu))));
        mx = fmaxf(mx, fabsf(act_to_f32<XDT>(uint16_t(pw[e] >> 16))));
    }
    return mx;
}

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
    const float xbar = fmaxf(mx, kEps);
    const float d = __fdiv_rn(xbar, 127.0f);
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
