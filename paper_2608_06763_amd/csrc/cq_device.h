// Device-side building blocks shared by the CubicQuant kernels (gfx950).
//
// Field extraction follows eq. gpu-packed-extraction (Sec. 5.2): a row is one
// little-endian bitstream, field j occupies bits [jB, jB+B).  Because every
// supported group holds G = 32*u codes and G*B is a multiple of 8, a run of 32
// consecutive codes starting at a multiple of 32 is exactly B aligned 32-bit
// words ("a unit").  Kernels load whole units and extract fields with
// compile-time shifts.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

namespace cq {

constexpr int kWave = 64;

__host__ __device__ constexpr int max_code(int bits) { return bits == 1 ? 1 : (1 << (bits - 1)) - 1; }

// ---------------------------------------------------------------- dtype helpers

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

__device__ __forceinline__ float f16_to_f32(uint16_t h) {
    return static_cast<float>(__builtin_bit_cast(_Float16, h));
}

// round-to-nearest-even FP32 -> BF16 (NaN stays NaN)
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return uint16_t((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

__device__ __forceinline__ uint16_t f32_to_f16(float f) {
    return __builtin_bit_cast(uint16_t, static_cast<_Float16>(f));
}

template <int DT>  // 0 = bf16, 1 = fp16
__device__ __forceinline__ float act_to_f32(uint16_t h) {
    if constexpr (DT == 0) return bf16_to_f32(h); else return f16_to_f32(h);
}

template <int DT>  // 0 = bf16, 1 = fp16, 2 = fp32
__device__ __forceinline__ void store_out(void *y, int64_t idx, float v) {
    if constexpr (DT == 0) static_cast<uint16_t *>(y)[idx] = f32_to_bf16(v);
    else if constexpr (DT == 1) static_cast<uint16_t *>(y)[idx] = f32_to_f16(v);
    else static_cast<float *>(y)[idx] = v;
}

// ---------------------------------------------------------------- code extraction

// Field i (0..31) of a unit of B words w[0..B-1]: the signed code, with the
// reserved pattern -2^(B-1) mapped to 0 and W1 mapped to {-1, +1}.
template <int B>
__device__ __forceinline__ int unit_code(const uint32_t *w, int i) {
    const int bit = i * B;
    const int wd = bit >> 5;
    const int sh = bit & 31;
    uint32_t v;
    if (sh + B <= 32) {
        v = w[wd] >> sh;
    } else {
        v = __builtin_amdgcn_alignbit(w[wd + 1], w[wd], sh);
    }
    if constexpr (B == 1) {
        return int(v & 1u) * 2 - 1;
    } else {
        int k = __builtin_amdgcn_sbfe(int(v), 0, B);  // sign-extending field extract
        return k == -(1 << (B - 1)) ? 0 : k;
    }
}

// Generic field extraction straight from a byte row (eq. gpu-packed-extraction),
// used by the reference decode: p = jB/8, d = jB%8, second byte only when the
// field crosses a byte boundary.
__device__ __forceinline__ uint32_t extract_field(const uint8_t *row, int64_t j, int bits) {
    const int64_t bit = j * bits;
    const int64_t p = bit >> 3;
    const int d = int(bit & 7);
    uint32_t v = uint32_t(row[p]) >> d;
    if (d + bits > 8) v |= uint32_t(row[p + 1]) << (8 - d);
    return v & ((1u << bits) - 1u);
}

__device__ __forceinline__ int field_to_code(uint32_t u, int bits) {
    if (bits == 1) return int(u) * 2 - 1;
    const int half = 1 << (bits - 1);
    int k = int(u) >= half ? int(u) - (1 << bits) : int(u);
    return int(u) == half ? 0 : k;
}

// ---------------------------------------------------------------- level function

// sign(k) q(|k|/M) in FP32 with the Horner form of eq. gpu-horner:
// q(t) = t * fma(t, fma(t, c, b), a).
__device__ __forceinline__ float signed_level(int k, int m, float a, float b, float c) {
    const float t = float(k < 0 ? -k : k) / float(m);
    const float q = t * __builtin_fmaf(t, __builtin_fmaf(t, c, b), a);
    return k < 0 ? -q : q;
}

// ---------------------------------------------------------------- exact INT8 carrier

// r(i) = RNE(127 q(i/M)) for magnitude i in [0, M], exact (Sec. 4.3, eq. carrier;
// Appendix A item 7).  With a, b widened from FP16 every term below is exact in
// float64: S = a M^2 + b i M + c i^2 has at most ~40 significant bits,
// T = i S at most ~47, and the residual e = 127 T - r M^3 is formed by one fused
// multiply-add and is exact.  127 q(i/M) = 127 T / M^3.
__device__ __forceinline__ int exact_carrier(int i, int m, double a, double b) {
    if (i == 0) return 0;
    if (i == m) return 127;
    const double c = 1.0 - a - b;
    const double dm = double(m), di = double(i);
    const double s = a * dm * dm + b * di * dm + c * di * di;
    const double t = di * s;
    const double m3 = dm * dm * dm;
    double r = __builtin_rint(127.0 * t / m3);
    double e = __builtin_fma(127.0, t, -r * m3);
    const double half = 0.5 * m3;
    // bring |e| into [0, M^3/2]; a fresh rint above is within one step
    if (e > half) { r += 1.0; e -= m3; }
    else if (e < -half) { r -= 1.0; e += m3; }
    if (e == half || e == -half) {
        // exact tie between r and r +- 1: keep the even one (r is a small
        // integer, so its parity is that of its int conversion; a double
        // fmod would expand to a loop)
        const double other = (e == half) ? r + 1.0 : r - 1.0;
        if (int(r) & 1) r = other;
    }
    return int(r);
}

// Compute units of the current device, cached per device id.  Host threads
// may race to fill an entry; they store the same value through an atomic, so
// the cache is free of data races.
inline int device_cu_count() {
    static std::atomic<int> cus[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int v = cus[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
        cus[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

}  // namespace cq
