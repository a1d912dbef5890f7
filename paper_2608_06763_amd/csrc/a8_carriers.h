// Dynamic-A8 weight carriers in registers (gfx950): exact INT8 carriers
// r(i) = RNE(127 q(i/M)) (eq. carrier, Appendix A item 7) and the byte-permute
// lookup of W4 fields.
//
// Exactness: 127 q(i/M) is first evaluated in FP32 (Horner, eq. gpu-horner);
// its rounding error is below 127 * 2^-20 * (|a| + |b| + |c| + 1).  Only when
// the estimate lies closer than that to a half-integer is the carrier
// recomputed with the exact FP64 residual test, so every carrier equals the
// RNE of the exact rational value.
//
// W4 lookup: a field n (two's complement, 8 reserved) selects from two 8-byte
// tables, TA[i] = r(i) for n = i < 8 and TB[i] = -r(8 - i) for n = 8 + i
// (TB[0] = 0 is the reserved pattern).  One v_perm_b32 looks up four fields
// in a table; a byte mask from bit 3 of each field picks TA or TB per byte.
#pragma once

#include "cq_device.h"

namespace cq {

__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel) {
    return __builtin_amdgcn_perm(hi, lo, sel);
}

// Error bound margin of the FP32 carrier estimate for one (a, b).
__device__ __forceinline__ float carrier_margin(float a, float b, float c) {
    return (__builtin_fabsf(a) + __builtin_fabsf(b) + __builtin_fabsf(c) + 1.f) * (127.0f / 1048576.0f);
}

// INT8 carrier of magnitude i with t = i / M (exact when close to a tie).
template <int M>
__device__ __forceinline__ uint32_t carrier_u8(int i, float t, float a, float b, float c, float margin) {
    const float f = 127.0f * (t * __builtin_fmaf(t, __builtin_fmaf(t, c, b), a));
    float r = __builtin_rintf(f);
    if (__builtin_expect(__builtin_fabsf(f - r) > 0.5f - margin, 0)) {
        // the exact path's double arithmetic stays inside this rarely taken
        // branch (the compiler would otherwise hoist it for every carrier)
        float ea = a, eb = b;
        __asm__ volatile("" : "+v"(ea), "+v"(eb));
        r = float(exact_carrier(i, M, double(ea), double(eb)));
    }
    r = r < 0.f ? 0.f : (r > 127.f ? 127.f : r);
    return uint32_t(int(r));
}

// DPP quad_perm move: every lane reads the lane of its quad named by CTRL.
template <int CTRL>
__device__ __forceinline__ uint32_t quad_bcast(uint32_t v) {
    return uint32_t(__builtin_amdgcn_mov_dpp(int(v), CTRL, 0xf, 0xf, true));
}

// TB from TA = [r0 r1 r2 r3 | r4 r5 r6 r7]: TB = [0, -r7, -r6, -r5 | -r4, -r3,
// -r2, -r1]; bytewise negation of values in [0, 127] without borrows is
// (0x80 - v) ^ 0x80.
__device__ __forceinline__ void w4_negative_table(uint32_t ta0, uint32_t ta1, uint32_t &tb0, uint32_t &tb1) {
    const uint32_t tbp0 = perm(ta1, ta0, 0x0506070cu);
    const uint32_t tbp1 = perm(ta1, ta0, 0x01020304u);
    tb0 = (0x80808080u - tbp0) ^ 0x80808080u;
    tb1 = (0x80808080u - tbp1) ^ 0x80808080u;
}

// Carriers of four W4 fields held one per byte (values 0..15).
__device__ __forceinline__ uint32_t w4_lookup(uint32_t f4, uint32_t ta0, uint32_t ta1, uint32_t tb0, uint32_t tb1) {
    const uint32_t idx = f4 & 0x07070707u;
    // 0xff in the bytes whose field has bit 3 set (selector 8 = sign of byte 1)
    const uint32_t msk = perm(0u, 0x00008000u, f4 & 0x08080808u);
    const uint32_t pa = perm(ta1, ta0, idx);
    const uint32_t pb = perm(tb1, tb0, idx);
    return (msk & pb) | (~msk & pa);
}

// Carriers of the eight W4 fields of one code word, in field order:
// out0 = fields 0..3, out1 = fields 4..7 (one byte each).
__device__ __forceinline__ void w4_word_carriers(uint32_t wd, uint32_t ta0, uint32_t ta1, uint32_t tb0, uint32_t tb1,
                                                 uint32_t &out0, uint32_t &out1) {
    const uint32_t ev = w4_lookup(wd & 0x0f0f0f0fu, ta0, ta1, tb0, tb1);         // fields 0 2 4 6
    const uint32_t od = w4_lookup((wd >> 4) & 0x0f0f0f0fu, ta0, ta1, tb0, tb1);  // fields 1 3 5 7
    out0 = perm(od, ev, 0x05010400u);
    out1 = perm(od, ev, 0x07030602u);
}

}  // namespace cq
