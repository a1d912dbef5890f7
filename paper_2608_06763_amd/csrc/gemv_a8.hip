// Dynamic-A8 narrow-row GEMV (Sec. 5.4) for m <= 16 rows of INT8 carriers.
//
// Each weight maps to its INT8 carrier r(k) = sign(k) RNE(127 q(|k|/M)),
// computed exactly (eq. carrier, Appendix A item 7: an FP32 estimate, and the
// exact evaluation when the estimate lies near a tie); a packed 4 x int8 dot
// product accumulates exact INT32 partials over 32-code units, which are
// K-tile partials of the group partial P_g (Sec. 5.4 allows smaller K-tile
// partials); each is converted to FP32 and multiplied by s_g, and the row
// factor d_x / 127 is applied to the FP32 sum.
//
// Conservative family: one wavefront per output row, lanes stride over units.
// When the caller asks for the group partials, the unit partials of a group
// (held by adjacent lanes) are summed exactly with lane shuffles first.
#include "cq_device.h"
#include "cq_internal.h"
#include "a8_carriers.h"

namespace cq {

template <int B, int MR, int YDT>
__global__ void __launch_bounds__(256) gemv_a8_generic(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int group, int64_t n, int64_t k, const int8_t *__restrict__ x8, const float *__restrict__ dx, int m_rows,
    void *__restrict__ y, int32_t *__restrict__ partials, const int8_t *__restrict__ ctab) {
    // ctab: optional load-time carrier table, 2^(B-1) bytes per (row, group)
    constexpr int M = max_code(B);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t units = k >> 5;
    const int64_t row_words = (k * B) >> 5;
    const int64_t ng = k / group;
    const int upg = group >> 5;
    for (int64_t row = int64_t(blockIdx.x) * 4 + wave; row < n; row += int64_t(gridDim.x) * 4) {
        const uint32_t *wrow = reinterpret_cast<const uint32_t *>(codes) + row * row_words;
        float acc[MR];
#pragma unroll
        for (int r = 0; r < MR; ++r) acc[r] = 0.f;
        // every lane runs the same number of iterations so that shuffles below
        // always see a full wavefront; lanes past the end contribute zero
        const int64_t iters = (units + kWave - 1) / kWave;
        for (int64_t it = 0; it < iters; ++it) {
            const int64_t u = it * kWave + lane;
            const bool live = u < units;
            uint32_t rq[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            float s = 0.f;
            int64_t gidx = 0;
            if (live) {
                uint32_t w[B];
#pragma unroll
                for (int i = 0; i < B; ++i) w[i] = wrow[u * B + i];
                gidx = row * ng + u / upg;
                s = scale[gidx];
                float a = 1.f, b = 0.f;
                if (B > 2 && !ctab) {
                    a = f16_to_f32(a16[gidx]);
                    b = f16_to_f32(b16[gidx]);
                }
                const float c3 = 1.f - a - b;
                const float margin = carrier_margin(a, b, c3);
#pragma unroll
                for (int i = 0; i < 32; ++i) {
                    const int code = unit_code<B>(w, i);
                    int r;
                    if constexpr (B == 1) {
                        r = code * 127;
                    } else {
                        const int mag = code < 0 ? -code : code;
                        int c;
                        if constexpr (B == 2) c = mag ? 127 : 0;
                        else if (ctab) c = int(ctab[gidx * (M + 1) + mag]);
                        // FP32 estimate of 127 q, exact fallback near a tie
                        else c = int(carrier_u8<M>(mag, float(mag) / float(M), a, b, c3, margin));
                        c = c > 127 ? 127 : (c < -127 ? -127 : c);
                        r = code < 0 ? -c : c;
                    }
                    rq[i >> 2] |= (uint32_t(r) & 0xffu) << (8 * (i & 3));
                }
            }
#pragma unroll
            for (int r = 0; r < MR; ++r) {
                if (r < m_rows) {
                    int p = 0;
                    if (live) {
                        const uint4 *xp = reinterpret_cast<const uint4 *>(x8 + int64_t(r) * k + u * 32);
                        const uint4 v0 = xp[0], v1 = xp[1];
                        const uint32_t xv[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
                        for (int q = 0; q < 8; ++q) p = __builtin_amdgcn_sdot4(int(xv[q]), int(rq[q]), p, false);
                    }
                    if (partials) {
                        // exact sum of the unit partials of one group (adjacent lanes)
                        int pg = p;
                        for (int off = 1; off < upg; off <<= 1) pg += __shfl_xor(pg, off, kWave);
                        if (live && (u % upg) == 0)
                            partials[(int64_t(r) * n + row) * ng + u / upg] = pg;
                    }
                    acc[r] = __builtin_fmaf(s, float(p), acc[r]);
                }
            }
        }
#pragma unroll
        for (int r = 0; r < MR; ++r) {
            float v = acc[r];
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
            if (lane == 0 && r < m_rows) store_out<YDT>(y, int64_t(r) * n + row, v * (dx[r] / 127.0f));
        }
    }
}

template <int B, int MR, int YDT>
static hipError_t run_generic(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                              int32_t *partials, const int8_t *ctab, hipStream_t stream) {
    int64_t blocks = (w.n + 3) / 4;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL((gemv_a8_generic<B, MR, YDT>), dim3(unsigned(blocks)), dim3(256), 0, stream, w.codes,
                       w.scale, w.a, w.b, w.group, w.n, w.k, x8, dx, int(m), y, partials, ctab);
    return hipGetLastError();
}

template <int B, int YDT>
static hipError_t dispatch_rows(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                                int32_t *partials, const int8_t *ctab, hipStream_t stream) {
    if (m <= 1) return run_generic<B, 1, YDT>(w, x8, dx, m, y, partials, ctab, stream);
    if (m <= 2) return run_generic<B, 2, YDT>(w, x8, dx, m, y, partials, ctab, stream);
    if (m <= 4) return run_generic<B, 4, YDT>(w, x8, dx, m, y, partials, ctab, stream);
    if (m <= 8) return run_generic<B, 8, YDT>(w, x8, dx, m, y, partials, ctab, stream);
    return run_generic<B, 16, YDT>(w, x8, dx, m, y, partials, ctab, stream);
}

template <int YDT>
static hipError_t dispatch_bits(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                                int32_t *partials, const int8_t *ctab, hipStream_t stream) {
    switch (w.bits) {
        case 1: return dispatch_rows<1, YDT>(w, x8, dx, m, y, partials, ctab, stream);
        case 2: return dispatch_rows<2, YDT>(w, x8, dx, m, y, partials, ctab, stream);
        case 3: return dispatch_rows<3, YDT>(w, x8, dx, m, y, partials, ctab, stream);
        case 4: return dispatch_rows<4, YDT>(w, x8, dx, m, y, partials, ctab, stream);
        case 5: return dispatch_rows<5, YDT>(w, x8, dx, m, y, partials, ctab, stream);
        case 6: return dispatch_rows<6, YDT>(w, x8, dx, m, y, partials, ctab, stream);
        case 7: return dispatch_rows<7, YDT>(w, x8, dx, m, y, partials, ctab, stream);
        case 8: return dispatch_rows<8, YDT>(w, x8, dx, m, y, partials, ctab, stream);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gemv_a8_generic(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y, int y_dt,
                                  int32_t *partials, hipStream_t stream) {
    if (y_dt == 0) return dispatch_bits<0>(w, x8, dx, m, y, partials, nullptr, stream);
    if (y_dt == 1) return dispatch_bits<1>(w, x8, dx, m, y, partials, nullptr, stream);
    return dispatch_bits<2>(w, x8, dx, m, y, partials, nullptr, stream);
}

hipError_t launch_gemv_a8_tab(const cq_weight &w, const int8_t *ctab, const int8_t *x8, const float *dx, int64_t m,
                              void *y, int y_dt, hipStream_t stream) {
    // the single-row (B <= 4) and W4 narrow-row kernels form their carriers
    // in registers (the same values); the generic kernel reads the table
    if (gemv_a8_stream_supported(w, m)) return launch_gemv_a8_stream(w, x8, dx, y, y_dt, stream);
    if (gemv_a8_narrow_supported(w, m)) return launch_gemv_a8_narrow(w, x8, dx, m, y, y_dt, stream);
    if (y_dt == 0) return dispatch_bits<0>(w, x8, dx, m, y, nullptr, ctab, stream);
    if (y_dt == 1) return dispatch_bits<1>(w, x8, dx, m, y, nullptr, ctab, stream);
    return dispatch_bits<2>(w, x8, dx, m, y, nullptr, ctab, stream);
}

}  // namespace cq
