// Model-dtype narrow-row GEMV (Sec. 5.3, narrow-row tactic): y = x W_hat^T for
// m <= 16 activation rows, W streamed once from its packed form.
//
// Activations and normalised levels are multiplied in FP32, and the group
// scale is applied in FP32 to each 32-code partial reduction (a sub-reduction
// of the group reduction, which leaves the sum unchanged up to rounding order).
//
// Conservative family: one wavefront per output row, lanes stride over 32-code
// units of the row (B aligned words each), per-weight Horner decode in FP32,
// butterfly reduction across the wavefront.  Covers every B in 1..8 and every
// supported G.
#include "cq_device.h"
#include "cq_internal.h"
#include "stream_common.h"

namespace cq {

template <int B, int MR, int XDT, int YDT>
__global__ void __launch_bounds__(256) gemv_a16_generic(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int group, int64_t n, int64_t k, const uint16_t *__restrict__ x, int m_rows, void *__restrict__ y) {
    constexpr int M = max_code(B);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t units = k >> 5;
    const int64_t row_words = (k * B) >> 5;
    const int64_t ng = k / group;
    const int upg = group >> 5;  // units per group
    for (int64_t row = int64_t(blockIdx.x) * 4 + wave; row < n; row += int64_t(gridDim.x) * 4) {
        const uint32_t *wrow = reinterpret_cast<const uint32_t *>(codes) + row * row_words;
        float acc[MR];
#pragma unroll
        for (int r = 0; r < MR; ++r) acc[r] = 0.f;
        for (int64_t u = lane; u < units; u += kWave) {
            uint32_t w[B];
#pragma unroll
            for (int i = 0; i < B; ++i) w[i] = wrow[u * B + i];
            const int64_t gi = row * ng + u / upg;
            const float s = scale[gi];
            float a = 1.f, b = 0.f;
            if constexpr (B > 1) {
                a = f16_to_f32(a16[gi]);
                b = f16_to_f32(b16[gi]);
            }
            const float c = 1.f - a - b;
            float lev[32];
#pragma unroll
            for (int i = 0; i < 32; ++i) {
                const int code = unit_code<B>(w, i);
                lev[i] = (B == 1) ? float(code) : signed_level(code, M, a, b, c);
            }
#pragma unroll
            for (int r = 0; r < MR; ++r) {
                if (r < m_rows) {
                    const uint4 *xp = reinterpret_cast<const uint4 *>(x + int64_t(r) * k + u * 32);
                    float part = 0.f;
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const uint4 v = xp[q];
                        const uint32_t vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            part = __builtin_fmaf(act_to_f32<XDT>(uint16_t(vv[e] & 0xffffu)), lev[q * 8 + 2 * e], part);
                            part = __builtin_fmaf(act_to_f32<XDT>(uint16_t(vv[e] >> 16)), lev[q * 8 + 2 * e + 1], part);
                        }
                    }
                    acc[r] = __builtin_fmaf(s, part, acc[r]);
                }
            }
        }
#pragma unroll
        for (int r = 0; r < MR; ++r) {
            float v = acc[r];
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
            if (lane == 0 && r < m_rows) store_out<YDT>(y, int64_t(r) * n + row, v);
        }
    }
}

template <int B, int MR, int XDT, int YDT>
static hipError_t run_generic(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    int64_t blocks = (w.n + 3) / 4;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL((gemv_a16_generic<B, MR, XDT, YDT>), dim3(unsigned(blocks)), dim3(256), 0, stream, w.codes,
                       w.scale, w.a, w.b, w.group, w.n, w.k, static_cast<const uint16_t *>(x), int(m), y);
    return hipGetLastError();
}

template <int B, int XDT, int YDT>
static hipError_t dispatch_rows(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    if (m <= 1) return run_generic<B, 1, XDT, YDT>(w, x, m, y, stream);
    if (m <= 2) return run_generic<B, 2, XDT, YDT>(w, x, m, y, stream);
    if (m <= 4) return run_generic<B, 4, XDT, YDT>(w, x, m, y, stream);
    if (m <= 8) return run_generic<B, 8, XDT, YDT>(w, x, m, y, stream);
    return run_generic<B, 16, XDT, YDT>(w, x, m, y, stream);
}

template <int XDT, int YDT>
static hipError_t dispatch_bits(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    switch (w.bits) {
        case 1: return dispatch_rows<1, XDT, YDT>(w, x, m, y, stream);
        case 2: return dispatch_rows<2, XDT, YDT>(w, x, m, y, stream);
        case 3: return dispatch_rows<3, XDT, YDT>(w, x, m, y, stream);
        case 4: return dispatch_rows<4, XDT, YDT>(w, x, m, y, stream);
        case 5: return dispatch_rows<5, XDT, YDT>(w, x, m, y, stream);
        case 6: return dispatch_rows<6, XDT, YDT>(w, x, m, y, stream);
        case 7: return dispatch_rows<7, XDT, YDT>(w, x, m, y, stream);
        case 8: return dispatch_rows<8, XDT, YDT>(w, x, m, y, stream);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gemv_a16_generic(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                   hipStream_t stream) {
    if (x_dt == 0) {
        if (y_dt == 0) return dispatch_bits<0, 0>(w, x, m, y, stream);
        return dispatch_bits<0, 2>(w, x, m, y, stream);
    }
    if (y_dt == 1) return dispatch_bits<1, 1>(w, x, m, y, stream);
    return dispatch_bits<1, 2>(w, x, m, y, stream);
}

}  // namespace cq
