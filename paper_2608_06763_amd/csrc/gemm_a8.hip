// Dynamic-A8 tiled GEMM (Sec. 5.4) on gfx950 int8 matrix cores.
//
// A workgroup owns a BM x BN tile of y.  At the start of every group it builds,
// for each of its BN weight rows, the exact INT8 carrier table
// r(i) = RNE(127 q(i/M)), i = 0..M (eq. carrier, Appendix A item 7) in LDS.
// Each K step decodes the packed codes of the tile to signed carriers, stages
// them with the activation carriers in LDS, and the int8 MFMA accumulates the
// exact INT32 group partials P_g (|P_g| <= G 127^2, eq. a8-int32-bound).  At the
// end of a group every partial is converted to FP32 and multiplied by s_g
// (the FP32 rescale of eq. a8-output); the row factor d_x / 127 is applied to
// the FP32 sum at the end.
//
// MFMA operand layout (v_mfma_i32_16x16x64_i8): lane l supplies row l % 16 of
// A and column l % 16 of B with the 16 consecutive K slots 16*(l/16)..+15; the
// 16x16 INT32 result has lane l holding rows 4*(l/16)+i of column l % 16.
// For G = 32 the K step is 32 (v_mfma_i32_16x16x32_i8, 8 slots per lane).
#include "cq_device.h"
#include "cq_internal.h"

namespace cq {

typedef int i32x4 __attribute__((ext_vector_type(4)));

namespace {
constexpr int BM = 64, BN = 64;
constexpr int TAB = 128;  // carrier table entries per row (M + 1 <= 128)
}  // namespace

template <int B, int KS, int YDT>
__global__ void __launch_bounds__(256) gemm_a8_tiled(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int group, int64_t n, int64_t k, const int8_t *__restrict__ x8, const float *__restrict__ dx, int64_t m,
    void *__restrict__ y, int32_t *__restrict__ partials, const int8_t *__restrict__ ctab) {
    // ctab: optional load-time carrier table, 2^(B-1) bytes per (row, group)
    constexpr int M = max_code(B);
    constexpr int STRIDE = KS + 16;  // bytes per LDS row, padded
    __shared__ __attribute__((aligned(16))) int8_t As[BM * STRIDE];
    __shared__ __attribute__((aligned(16))) int8_t Bs[BN * STRIDE];
    __shared__ int8_t tab[BN * TAB];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t n0 = int64_t(blockIdx.x) * BN;
    const int64_t m0 = int64_t(blockIdx.y) * BM;
    const int64_t row_words = (k * B) >> 5;
    const int64_t ng = k / group;
    const int wm = (wave >> 1) * 32, wn = (wave & 1) * 32;

    float accf[2][2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) accf[i][j][e] = 0.f;

    constexpr int CPT = KS / 4;  // codes per thread per step (16 or 8)
    const int br = tid >> 2, bc = (tid & 3) * CPT;
    const int ar = tid >> 2, ac = (tid & 3) * CPT;

    for (int64_t g = 0; g < ng; ++g) {
        // ---- carrier tables for this group
        if constexpr (B >= 3) {
            for (int e = tid; e < BN * (M + 1); e += 256) {
                const int r = e / (M + 1), i = e - r * (M + 1);
                const int64_t row = n0 + r;
                int c = 0;
                if (row < n) {
                    const int64_t gi = row * ng + g;
                    c = ctab ? int(ctab[gi * (M + 1) + i])
                             : exact_carrier(i, M, double(f16_to_f32(a16[gi])), double(f16_to_f32(b16[gi])));
                    c = c > 127 ? 127 : (c < -127 ? -127 : c);
                }
                tab[r * TAB + i] = int8_t(c);
            }
        }
        i32x4 acc[2][2];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[i][j] = i32x4{0, 0, 0, 0};

        for (int64_t k0 = g * group; k0 < (g + 1) * group; k0 += KS) {
            __syncthreads();  // tables ready / previous step consumed
            {
                // activation carriers
                if constexpr (CPT == 16) {
                    uint4 v = make_uint4(0, 0, 0, 0);
                    if (m0 + ar < m) v = *reinterpret_cast<const uint4 *>(x8 + (m0 + ar) * k + k0 + ac);
                    *reinterpret_cast<uint4 *>(&As[ar * STRIDE + ac]) = v;
                } else {
                    uint2 v = make_uint2(0, 0);
                    if (m0 + ar < m) v = *reinterpret_cast<const uint2 *>(x8 + (m0 + ar) * k + k0 + ac);
                    *reinterpret_cast<uint2 *>(&As[ar * STRIDE + ac]) = v;
                }
            }
            {
                uint32_t packed[CPT / 4];
#pragma unroll
                for (int i = 0; i < CPT / 4; ++i) packed[i] = 0;
                const int64_t row = n0 + br;
                if (row < n) {
                    const int cpos = int(k0 & 31) + bc;  // position inside its 32-code unit
                    const uint32_t *wp = reinterpret_cast<const uint32_t *>(codes) + row * row_words +
                                         ((k0 + bc) >> 5) * B;
                    uint32_t w[B];
#pragma unroll
                    for (int i = 0; i < B; ++i) w[i] = wp[i];
#pragma unroll
                    for (int e = 0; e < CPT; ++e) {
                        const int code = unit_code<B>(w, (cpos & 31) + e);
                        int r;
                        if constexpr (B == 1) r = code * 127;
                        else if constexpr (B == 2) r = code * 127;
                        else {
                            const int mag = code < 0 ? -code : code;
                            const int c = tab[br * TAB + mag];
                            r = code < 0 ? -c : c;
                        }
                        packed[e >> 2] |= (uint32_t(r) & 0xffu) << (8 * (e & 3));
                    }
                }
                if constexpr (CPT == 16)
                    *reinterpret_cast<uint4 *>(&Bs[br * STRIDE + bc]) =
                        make_uint4(packed[0], packed[1], packed[2], packed[3]);
                else
                    *reinterpret_cast<uint2 *>(&Bs[br * STRIDE + bc]) = make_uint2(packed[0], packed[1]);
            }
            __syncthreads();
            if constexpr (KS == 64) {
                i32x4 af[2], bfr[2];
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    af[i] = *reinterpret_cast<const i32x4 *>(&As[(wm + i * 16 + (lane & 15)) * STRIDE + 16 * (lane >> 4)]);
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    bfr[j] = *reinterpret_cast<const i32x4 *>(&Bs[(wn + j * 16 + (lane & 15)) * STRIDE + 16 * (lane >> 4)]);
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[i], bfr[j], acc[i][j], 0, 0, 0);
            } else {
                long af[2], bfr[2];
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    af[i] = *reinterpret_cast<const long *>(&As[(wm + i * 16 + (lane & 15)) * STRIDE + 8 * (lane >> 4)]);
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    bfr[j] = *reinterpret_cast<const long *>(&Bs[(wn + j * 16 + (lane & 15)) * STRIDE + 8 * (lane >> 4)]);
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x32_i8(af[i], bfr[j], acc[i][j], 0, 0, 0);
            }
        }
        // ---- FP32 group rescale (and optional partial dump)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t col = n0 + wn + j * 16 + (lane & 15);
            const float s = col < n ? scale[col * ng + g] : 0.f;
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    accf[i][j][e] = __builtin_fmaf(s, float(acc[i][j][e]), accf[i][j][e]);
                    if (partials) {
                        const int64_t row = m0 + wm + i * 16 + 4 * (lane >> 4) + e;
                        if (row < m && col < n) partials[(row * n + col) * ng + g] = acc[i][j][e];
                    }
                }
        }
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int64_t row = m0 + wm + i * 16 + 4 * (lane >> 4) + e;
            if (row >= m) continue;
            const float f = dx[row] / 127.0f;
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int64_t col = n0 + wn + j * 16 + (lane & 15);
                if (col < n) store_out<YDT>(y, row * n + col, accf[i][j][e] * f);
            }
        }
}

template <int B, int YDT>
static hipError_t run_tiled(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                            int32_t *partials, const int8_t *ctab, hipStream_t stream) {
    const int64_t gx = (w.n + BN - 1) / BN, gy = (m + BM - 1) / BM;
    if (gx > 0x7fffffff || gy > 65535) return hipErrorInvalidValue;
    if (w.group % 64 == 0)
        hipLaunchKernelGGL((gemm_a8_tiled<B, 64, YDT>), dim3(unsigned(gx), unsigned(gy)), dim3(256), 0, stream,
                           w.codes, w.scale, w.a, w.b, w.group, w.n, w.k, x8, dx, m, y, partials, ctab);
    else
        hipLaunchKernelGGL((gemm_a8_tiled<B, 32, YDT>), dim3(unsigned(gx), unsigned(gy)), dim3(256), 0, stream,
                           w.codes, w.scale, w.a, w.b, w.group, w.n, w.k, x8, dx, m, y, partials, ctab);
    return hipGetLastError();
}

template <int YDT>
static hipError_t dispatch_bits(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                                int32_t *partials, const int8_t *ctab, hipStream_t stream) {
    switch (w.bits) {
        case 1: return run_tiled<1, YDT>(w, x8, dx, m, y, partials, ctab, stream);
        case 2: return run_tiled<2, YDT>(w, x8, dx, m, y, partials, ctab, stream);
        case 3: return run_tiled<3, YDT>(w, x8, dx, m, y, partials, ctab, stream);
        case 4: return run_tiled<4, YDT>(w, x8, dx, m, y, partials, ctab, stream);
        case 5: return run_tiled<5, YDT>(w, x8, dx, m, y, partials, ctab, stream);
        case 6: return run_tiled<6, YDT>(w, x8, dx, m, y, partials, ctab, stream);
        case 7: return run_tiled<7, YDT>(w, x8, dx, m, y, partials, ctab, stream);
        case 8: return run_tiled<8, YDT>(w, x8, dx, m, y, partials, ctab, stream);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gemm_a8_tiled(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y, int y_dt,
                                int32_t *partials, hipStream_t stream) {
    if (y_dt == 0) return dispatch_bits<0>(w, x8, dx, m, y, partials, nullptr, stream);
    if (y_dt == 1) return dispatch_bits<1>(w, x8, dx, m, y, partials, nullptr, stream);
    return dispatch_bits<2>(w, x8, dx, m, y, partials, nullptr, stream);
}

hipError_t launch_gemm_a8_tab(const cq_weight &w, const int8_t *ctab, const int8_t *x8, const float *dx, int64_t m,
                              void *y, int y_dt, hipStream_t stream) {
    if (gemm_a8_mfma_supported(w, m)) return launch_gemm_a8_mfma_tab(w, ctab, x8, dx, m, y, y_dt, stream);
    if (y_dt == 0) return dispatch_bits<0>(w, x8, dx, m, y, nullptr, ctab, stream);
    if (y_dt == 1) return dispatch_bits<1>(w, x8, dx, m, y, nullptr, ctab, stream);
    return dispatch_bits<2>(w, x8, dx, m, y, nullptr, ctab, stream);
}

}  // namespace cq
