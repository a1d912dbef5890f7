// Dynamic-A8 many-row GEMM (Sec. 5.4) for W4 on gfx950 int8 matrix cores.
//
// Numerics are eq. a8-output: INT8 activations times exact INT8 weight
// carriers (eq. carrier) accumulate into exact INT32 group partials P_g
// (|P_g| <= G 127^2, eq. a8-int32-bound); at the end of every group each
// partial is converted to FP32 and multiplied by s_g, and the row factor
// d_x / 127 multiplies the FP32 sum.
//
// Tiling.  A workgroup of 2 x WN waves owns a 128 x (64 WN) tile of y (rows of
// x by rows of W); each wave owns 64 x 64 and issues v_mfma_i32_16x16x64_i8
// on 16 x 16 blocks.  K advances in steps of 64 through two LDS buffers: while
// the matrix cores work on one buffer, every thread loads the next step's
// codes and activations, decodes its 32 codes to carriers and writes them to
// the other buffer, so one barrier per step suffices.
//
// Decode.  Thread t serves weight row t / 2 and the 32-code half t % 2 of each
// step.  At the start of a group the two threads of a row each evaluate three
// carriers (exact, see a8_carriers.h) and swap them with a DPP move, which
// gives both the two 8-byte W4 carrier tables of that (row, group); every
// code word then costs two byte-permute lookups and two permutes that restore
// field order.
//
// MFMA operand layout (16x16x64 int8): lane l supplies row l % 16 of A and
// column l % 16 of B with K slots 16 (l / 16) .. +15; the INT32 result of a
// block has lane l holding rows 4 (l / 16) + i of column l % 16.
//
// Tile order: workgroups are first spread so that those on one XCD (blockIdx
// modulo 8) take consecutive tile indices, then tiles are walked in bands of
// 8 row tiles so that neighbouring workgroups share weight tiles in cache.
#include "cq_device.h"
#include "cq_internal.h"
#include "stream_common.h"
#include "a8_carriers.h"

namespace cq {

namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kTM = 128;               // rows of x per workgroup tile
constexpr int kKS = 64;                // K step
constexpr int kStride = kKS + 16;      // LDS bytes per tile row (padded)
constexpr int kBand = 8;               // row tiles per raster band

__device__ __forceinline__ void lds_store16(int8_t *p, const uint32_t *v) {
    *reinterpret_cast<u32x4 *>(p) = u32x4{v[0], v[1], v[2], v[3]};
}

}  // namespace

template <int WN, int UPG, int YDT, bool DUMP>
__global__ void __launch_bounds__(128 * WN) gemm_a8_w4_mfma(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int n, int k, const int8_t *__restrict__ x8, const float *__restrict__ dx, int m,
    void *__restrict__ y, int32_t *__restrict__ partials, int tiles_m, int tiles_n) {
    constexpr int M = 7;
    constexpr int TN = 64 * WN;
    constexpr int NT = 128 * WN;            // threads
    constexpr int G = 32 * UPG;
    constexpr int SPG = G / kKS;            // K steps per group
    constexpr int XB = kTM * kKS / NT;      // activation bytes per thread per step (32 or 16)
    static_assert(SPG >= 1 && G % kKS == 0, "group must be a multiple of the K step");
    __shared__ __attribute__((aligned(16))) int8_t As[2][kTM * kStride];
    __shared__ __attribute__((aligned(16))) int8_t Bs[2][TN * kStride];

    // ---- tile of this workgroup
    const int nwg = tiles_m * tiles_n;
    int wg = blockIdx.x;
    if (nwg % 8 == 0) wg = (wg % 8) * (nwg / 8) + wg / 8;
    const int band = wg / (kBand * tiles_n);
    const int first_m = band * kBand;
    const int band_rows = min(kBand, tiles_m - first_m);
    const int in_band = wg - band * kBand * tiles_n;
    const int m0 = (first_m + in_band % band_rows) * kTM;
    const int n0 = (in_band / band_rows) * TN;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = (wave / WN) * 64;
    const int wn = (wave % WN) * 64;

    const int ng = k / G;
    const uint32_t row_bytes = uint32_t(k) / 2u;
    const auto rc = make_rsrc(codes, uint32_t(n) * row_bytes);
    const auto rs = make_rsrc(scale, uint32_t(n) * ng * 4u);
    const auto ra = make_rsrc(a16, uint32_t(n) * ng * 2u);
    const auto rb = make_rsrc(b16, uint32_t(n) * ng * 2u);
    const auto rx = make_rsrc(x8, uint32_t(m) * uint32_t(k));

    // loader roles
    const int lr = tid >> 1;                 // weight row of the tile
    const int lh = tid & 1;                  // 32-code half of the step
    const int wrow = n0 + lr;
    const bool wok = wrow < n;
    const int xr = tid / (kKS / XB);         // activation row of the tile
    const int xc = (tid % (kKS / XB)) * XB;  // byte offset inside the step
    const int xrow = m0 + xr;
    const bool xok = xrow < m;

    // carriers this thread evaluates: magnitudes 1..3 (first thread of the row)
    // or 4..6 (second); r(0) = 0 and r(7) = 127 are fixed
    const int i0 = 1 + 3 * lh;
    const float t0 = float(i0) / float(M), t1 = float(i0 + 1) / float(M), t2 = float(i0 + 2) / float(M);

    uint32_t cw[4];        // codes of the next step
    uint32_t xw[XB / 4];   // activations of the next step
    uint32_t av = 0, bv = 0;
    float sj[4], sjn[4];   // group scales of this lane's four output columns

    auto load_step = [&](int st) {
        const uint32_t kk = uint32_t(st) * kKS;
        load_words<4>(rc, wok ? uint32_t(wrow) * row_bytes + (kk + 32u * lh) / 2u : kOobOffset, cw);
        load_words<XB / 4>(rx, xok ? uint32_t(xrow) * uint32_t(k) + kk + uint32_t(xc) : kOobOffset, xw);
        if (st % SPG == 0) {
            const int g = st / SPG;
            const uint32_t gi = uint32_t(wrow) * ng + g;
            av = load_u16(ra, wok ? gi * 2u : kOobOffset);
            bv = load_u16(rb, wok ? gi * 2u : kOobOffset);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int col = n0 + wn + 16 * j + (lane & 15);
                sjn[j] = load_f32(rs, col < n ? (uint32_t(col) * ng + g) * 4u : kOobOffset);
            }
        }
    };

    uint32_t ta0 = 0, ta1 = 0, tb0 = 0, tb1 = 0;
    auto build_tables = [&]() {
        const float a = f16_to_f32(uint16_t(av));
        const float b = f16_to_f32(uint16_t(bv));
        const float c = 1.f - a - b;
        const float mg = carrier_margin(a, b, c);
        const uint32_t c0 = carrier_u8<M>(i0, t0, a, b, c, mg);
        const uint32_t c1 = carrier_u8<M>(i0 + 1, t1, a, b, c, mg);
        const uint32_t c2 = carrier_u8<M>(i0 + 2, t2, a, b, c, mg);
        const uint32_t own = lh == 0 ? ((c0 << 8) | (c1 << 16) | (c2 << 24))   // r0 r1 r2 r3
                                     : (c0 | (c1 << 8) | (c2 << 16) | (127u << 24));  // r4 r5 r6 r7
        const uint32_t other = quad_bcast<0xb1>(own);  // the row's other thread (lane ^ 1)
        ta0 = lh == 0 ? own : other;
        ta1 = lh == 0 ? other : own;
        w4_negative_table(ta0, ta1, tb0, tb1);
    };

    auto store_step = [&](int buf) {
        uint32_t cr[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) w4_word_carriers(cw[i], ta0, ta1, tb0, tb1, cr[2 * i], cr[2 * i + 1]);
        int8_t *bp = &Bs[buf][lr * kStride + 32 * lh];
        lds_store16(bp, cr);
        lds_store16(bp + 16, cr + 4);
        int8_t *ap = &As[buf][xr * kStride + xc];
#pragma unroll
        for (int q = 0; q < XB / 16; ++q) lds_store16(ap + 16 * q, xw + 4 * q);
    };

    i32x4 acc[4][4];
    float accf[4][4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            acc[i][j] = i32x4{0, 0, 0, 0};
#pragma unroll
            for (int e = 0; e < 4; ++e) accf[i][j][e] = 0.f;
        }

    const int nsteps = k / kKS;
    load_step(0);
    build_tables();
#pragma unroll
    for (int j = 0; j < 4; ++j) sj[j] = sjn[j];
    store_step(0);
    __syncthreads();

    for (int st = 0; st < nsteps; ++st) {
        const int buf = st & 1;
        const bool more = st + 1 < nsteps;
        if (more) load_step(st + 1);

        i32x4 af[4], bf[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            af[i] = *reinterpret_cast<const i32x4 *>(&As[buf][(wm + 16 * i + (lane & 15)) * kStride + 16 * (lane >> 4)]);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            bf[j] = *reinterpret_cast<const i32x4 *>(&Bs[buf][(wn + 16 * j + (lane & 15)) * kStride + 16 * (lane >> 4)]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[i], bf[j], acc[i][j], 0, 0, 0);

        if (st % SPG == SPG - 1) {
            // group complete: FP32 rescale of the exact partials
            const int g = st / SPG;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) accf[i][j][e] = __builtin_fmaf(sj[j], float(acc[i][j][e]), accf[i][j][e]);
                }
            }
            if constexpr (DUMP) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int row = m0 + wm + 16 * i + 4 * (lane >> 4) + e;
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            const int col = n0 + wn + 16 * j + (lane & 15);
                            if (row < m && col < n) partials[(int64_t(row) * n + col) * ng + g] = acc[i][j][e];
                        }
                    }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = i32x4{0, 0, 0, 0};
#pragma unroll
            for (int j = 0; j < 4; ++j) sj[j] = sjn[j];
        }
        if (more) {
            if ((st + 1) % SPG == 0) build_tables();
            store_step(buf ^ 1);
        }
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int row = m0 + wm + 16 * i + 4 * (lane >> 4) + e;
            if (row >= m) continue;
            const float f = dx[row] / 127.0f;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int col = n0 + wn + 16 * j + (lane & 15);
                if (col < n) store_out<YDT>(y, int64_t(row) * n + col, accf[i][j][e] * f);
            }
        }
}

template <int WN, int UPG, int YDT, bool DUMP>
static hipError_t a8_mfma_launch(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                                 int32_t *partials, hipStream_t stream) {
    const int tiles_m = int((m + kTM - 1) / kTM);
    const int tiles_n = int((w.n + 64 * WN - 1) / (64 * WN));
    const int64_t nwg = int64_t(tiles_m) * tiles_n;
    if (nwg > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemm_a8_w4_mfma<WN, UPG, YDT, DUMP>), dim3(unsigned(nwg)), dim3(128 * WN), 0, stream, w.codes,
                       w.scale, w.a, w.b, int(w.n), int(w.k), x8, dx, int(m), y, partials, tiles_m, tiles_n);
    return hipGetLastError();
}

template <int YDT>
static hipError_t a8_mfma_group(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                                int32_t *partials, hipStream_t stream) {
    // The partials dump (a test path) runs four waves per workgroup, which
    // leaves room for its extra registers; the fast path runs eight.
    if (partials) {
        switch (w.group) {
            case 64: return a8_mfma_launch<2, 2, YDT, true>(w, x8, dx, m, y, partials, stream);
            case 128: return a8_mfma_launch<2, 4, YDT, true>(w, x8, dx, m, y, partials, stream);
            case 256: return a8_mfma_launch<2, 8, YDT, true>(w, x8, dx, m, y, partials, stream);
            case 512: return a8_mfma_launch<2, 16, YDT, true>(w, x8, dx, m, y, partials, stream);
        }
        return hipErrorNotSupported;
    }
    switch (w.group) {
        case 64: return a8_mfma_launch<4, 2, YDT, false>(w, x8, dx, m, y, partials, stream);
        case 128: return a8_mfma_launch<4, 4, YDT, false>(w, x8, dx, m, y, partials, stream);
        case 256: return a8_mfma_launch<4, 8, YDT, false>(w, x8, dx, m, y, partials, stream);
        case 512: return a8_mfma_launch<4, 16, YDT, false>(w, x8, dx, m, y, partials, stream);
    }
    return hipErrorNotSupported;
}

bool gemm_a8_mfma_supported(const cq_weight &w, int64_t m) {
    const int64_t lim = int64_t(1) << 31;
    return w.bits == 4 && w.group >= 64 && m * w.k < lim && stream_fits(w.n, w.k, w.bits, w.group) &&
           w.n < lim && m < lim;
}

hipError_t launch_gemm_a8_mfma(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y, int y_dt,
                               int32_t *partials, hipStream_t stream) {
    if (y_dt == 0) return a8_mfma_group<0>(w, x8, dx, m, y, partials, stream);
    if (y_dt == 1) return a8_mfma_group<1>(w, x8, dx, m, y, partials, stream);
    return a8_mfma_group<2>(w, x8, dx, m, y, partials, stream);
}

}  // namespace cq
