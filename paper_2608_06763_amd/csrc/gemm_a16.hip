// Model-dtype tiled GEMM (Sec. 5.3, dense tactic) on gfx950 matrix cores.
//
// A workgroup owns a BM x BN tile of y.  For every K step it decodes the packed
// weight tile once: s_g q(t_k) is formed in FP32 from the FP32 scale and the
// FP16 shapes and converted to the activation dtype (the dense-path rounding
// point of Sec. 5.3), then staged in LDS next to the activation tile; the MFMA
// accumulates in FP32.  Decoded weights never leave the workgroup.
//
// With BF16 activations a single BF16 operand (8 significant bits) costs up to
// about 2e-3 of max|y| in the worst output, so the FP32 value is carried as an
// unevaluated sum hi + lo of two BF16 numbers (hi = bf16(v), lo = bf16(v - hi),
// 16 significant bits) and both halves go through the MFMA into the same FP32
// accumulator.  FP16 activations use one FP16 operand (11 significant bits).
//
// MFMA operand layout (v_mfma_f32_16x16x32_{bf16,f16}): lane l supplies row
// (l % 16) of A and column (l % 16) of B, each with the 8 consecutive K slots
// 8*(l/16)..+7; the 16x16 FP32 result has lane l holding rows 4*(l/16)+i,
// i = 0..3, of column l % 16.
#include "cq_device.h"
#include "cq_internal.h"

namespace cq {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int BM = 64, BN = 64, BK = 32;
constexpr int LDS_STRIDE = BK + 8;  // halves; padding breaks bank conflicts

template <int XDT>
__device__ __forceinline__ f32x4 mfma16(const uint4 &a, const uint4 &b, f32x4 c) {
    if constexpr (XDT == 0)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                       c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c,
                                                      0, 0, 0);
}

template <int XDT>
__device__ __forceinline__ uint16_t to_act(float v) {
    if constexpr (XDT == 0) return f32_to_bf16(v); else return f32_to_f16(v);
}

}  // namespace

template <int B, int XDT, int YDT>
__global__ void __launch_bounds__(256) gemm_a16_tiled(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int group, int64_t n, int64_t k, const uint16_t *__restrict__ x, int64_t m, void *__restrict__ y) {
    constexpr int M = max_code(B);
    __shared__ __attribute__((aligned(16))) uint16_t As[BM * LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[BN * LDS_STRIDE];
    constexpr bool kSplit = (XDT == 0);
    __shared__ __attribute__((aligned(16))) uint16_t Bl[kSplit ? BN * LDS_STRIDE : 8];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t n0 = int64_t(blockIdx.x) * BN;
    const int64_t m0 = int64_t(blockIdx.y) * BM;
    const int64_t row_words = (k * B) >> 5;
    const int64_t ng = k / group;
    const int wm = (wave >> 1) * 32, wn = (wave & 1) * 32;

    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // activation staging: thread -> (row, 8-element chunk)
    const int ar = tid >> 2, ac = (tid & 3) * 8;
    // weight decode: thread -> (row, 8-code chunk of the 32-code unit)
    const int br = tid >> 2, bc = (tid & 3) * 8;

    for (int64_t k0 = 0; k0 < k; k0 += BK) {
        {
            uint4 v = make_uint4(0, 0, 0, 0);
            if (m0 + ar < m) v = *reinterpret_cast<const uint4 *>(x + (m0 + ar) * k + k0 + ac);
            *reinterpret_cast<uint4 *>(&As[ar * LDS_STRIDE + ac]) = v;
        }
        {
            uint32_t packed[4] = {0, 0, 0, 0};
            uint32_t packed_lo[4] = {0, 0, 0, 0};
            const int64_t row = n0 + br;
            if (row < n) {
                const uint32_t *wp = reinterpret_cast<const uint32_t *>(codes) + row * row_words + (k0 >> 5) * B;
                uint32_t w[B];
#pragma unroll
                for (int i = 0; i < B; ++i) w[i] = wp[i];
                const int64_t gi = row * ng + k0 / group;
                const float s = scale[gi];
                float a = 1.f, b = 0.f;
                if constexpr (B > 1) {
                    a = f16_to_f32(a16[gi]);
                    b = f16_to_f32(b16[gi]);
                }
                const float c = 1.f - a - b;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int code = unit_code<B>(w, bc + e);
                    const float lv = (B == 1) ? float(code) : signed_level(code, M, a, b, c);
                    const float v = s * lv;
                    const uint16_t hi = to_act<XDT>(v);
                    packed[e >> 1] |= uint32_t(hi) << (16 * (e & 1));
                    if constexpr (kSplit) packed_lo[e >> 1] |= uint32_t(f32_to_bf16(v - bf16_to_f32(hi))) << (16 * (e & 1));
                }
            }
            *reinterpret_cast<uint4 *>(&Bs[br * LDS_STRIDE + bc]) = make_uint4(packed[0], packed[1], packed[2], packed[3]);
            if constexpr (kSplit)
                *reinterpret_cast<uint4 *>(&Bl[br * LDS_STRIDE + bc]) =
                    make_uint4(packed_lo[0], packed_lo[1], packed_lo[2], packed_lo[3]);
        }
        __syncthreads();
        uint4 af[2], bfr[2];
#pragma unroll
        for (int i = 0; i < 2; ++i)
            af[i] = *reinterpret_cast<const uint4 *>(&As[(wm + i * 16 + (lane & 15)) * LDS_STRIDE + 8 * (lane >> 4)]);
#pragma unroll
        for (int j = 0; j < 2; ++j)
            bfr[j] = *reinterpret_cast<const uint4 *>(&Bs[(wn + j * 16 + (lane & 15)) * LDS_STRIDE + 8 * (lane >> 4)]);
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[i][j] = mfma16<XDT>(af[i], bfr[j], acc[i][j]);
        if constexpr (kSplit) {
#pragma unroll
            for (int j = 0; j < 2; ++j)
                bfr[j] = *reinterpret_cast<const uint4 *>(&Bl[(wn + j * 16 + (lane & 15)) * LDS_STRIDE + 8 * (lane >> 4)]);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = mfma16<XDT>(af[i], bfr[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int64_t row = m0 + wm + i * 16 + 4 * (lane >> 4) + e;
                const int64_t col = n0 + wn + j * 16 + (lane & 15);
                if (row < m && col < n) store_out<YDT>(y, row * n + col, acc[i][j][e]);
            }
}

template <int B, int XDT, int YDT>
static hipError_t run_tiled(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    const int64_t gx = (w.n + BN - 1) / BN, gy = (m + BM - 1) / BM;
    if (gx > 0x7fffffff || gy > 65535) return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemm_a16_tiled<B, XDT, YDT>), dim3(unsigned(gx), unsigned(gy)), dim3(256), 0, stream,
                       w.codes, w.scale, w.a, w.b, w.group, w.n, w.k, static_cast<const uint16_t *>(x), m, y);
    return hipGetLastError();
}

template <int XDT, int YDT>
static hipError_t dispatch_bits(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    switch (w.bits) {
        case 1: return run_tiled<1, XDT, YDT>(w, x, m, y, stream);
        case 2: return run_tiled<2, XDT, YDT>(w, x, m, y, stream);
        case 3: return run_tiled<3, XDT, YDT>(w, x, m, y, stream);
        case 4: return run_tiled<4, XDT, YDT>(w, x, m, y, stream);
        case 5: return run_tiled<5, XDT, YDT>(w, x, m, y, stream);
        case 6: return run_tiled<6, XDT, YDT>(w, x, m, y, stream);
        case 7: return run_tiled<7, XDT, YDT>(w, x, m, y, stream);
        case 8: return run_tiled<8, XDT, YDT>(w, x, m, y, stream);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gemm_a16_tiled(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                 hipStream_t stream) {
    if (x_dt == 0) {
        if (y_dt == 0) return dispatch_bits<0, 0>(w, x, m, y, stream);
        return dispatch_bits<0, 2>(w, x, m, y, stream);
    }
    if (y_dt == 1) return dispatch_bits<1, 1>(w, x, m, y, stream);
    return dispatch_bits<1, 2>(w, x, m, y, stream);
}

}  // namespace cq
