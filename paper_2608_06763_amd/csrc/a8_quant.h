// Dynamic-A8 activation quantization arithmetic (Sec. 5.4, eq.
// a8-activation-scale and eq. a8-activation-quantization), shared by the
// standalone quantizer and the GEMV that quantizes its own activations, so
// that both produce the same carriers and d_x bit for bit.
#pragma once

#include "cq_device.h"

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

// The same carriers as quantize8 for the same d, cheaper: with rcp = 1/d
// (IEEE division), v = x * rcp differs from the IEEE quotient fl(x / d) by at
// most 2^-23 |q| + 2^-24 |q| < 2.3e-5 (|q| <= 127.1), so when v lies farther
// than 2^-15 from every half-integer both round half away to the same integer.
// The few values inside that band (|v - round(v)| within 2^-15 of 1/2, an
// exact test) take the division.
template <int XDT>
__device__ __forceinline__ uint2 quantize8_rcp(const uint4 &p, float d, float rcp) {
    const uint32_t pw[4] = {p.x, p.y, p.z, p.w};
    uint32_t out[2] = {0u, 0u};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const uint16_t h = (e & 1) ? uint16_t(pw[e >> 1] >> 16) : uint16_t(pw[e >> 1] & 0xffffu);
        const float xv = act_to_f32<XDT>(h);
        const float v = xv * rcp;
        float r = roundf(v);
        if (__builtin_expect(fabsf(fabsf(v - r) - 0.5f) < 0x1p-15f, 0)) r = roundf(__fdiv_rn(xv, d));
        r = fminf(fmaxf(r, -127.f), 127.f);
        out[e >> 2] |= (uint32_t(int(r)) & 0xffu) << (8 * (e & 3));
    }
    return make_uint2(out[0], out[1]);
}

// d_x of a row from its maximum magnitude: xbar = max(amax, eps), d_x = xbar / 127.
__device__ __forceinline__ float a8_row_scale(float amax) { return __fdiv_rn(fmaxf(amax, kEps), 127.0f); }

}  // namespace cq
