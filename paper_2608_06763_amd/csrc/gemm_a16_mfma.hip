// Model-dtype many-row GEMM (Sec. 5.3, dense tactic) for B <= 5 on gfx950
// matrix cores.
//
// Numerics: every weight is reconstructed in FP32 as s_g sign(k) q(|k|/M)
// (eq. cubic, Horner form of eq. gpu-horner) and rounded to the MFMA operand
// dtype before the dot (the dense-path rounding point of Sec. 5.3); products
// accumulate in FP32.  With BF16 activations the default carries the FP32
// weight as the unevaluated sum hi + lo of two BF16 numbers (hi = RNE(v),
// lo = RNE(v - hi), 16 significant bits) and both halves go through the
// matrix core into the same FP32 accumulator, because a single BF16 operand
// costs 0.7e-3 to 2.1e-3 of max|y| on the benchmark layers, above the 2e-3
// budget on some.  The ROUNDED instantiation (ONE) is the single rounded
// BF16 operand itself, one MFMA per product, for callers whose error budget
// allows it.  FP16
// activations always use one FP16 operand.  Folding s_g into
// the reconstructed operand is a regrouping of the group sum: no per-group
// rescale is needed and accumulation runs across groups in the MFMA.
//
// Tiling.  A workgroup of 4 x 2 waves owns a 256 x 128 tile of y (rows of x
// by rows of W); each wave owns 64 x 64 and issues v_mfma_f32_16x16x32_{bf16,
// f16} on 16 x 16 blocks.  K advances one 32-code unit per step through two
// LDS buffers; while the matrix cores work on one, every thread decodes 8 codes
// of the next step into the other, so one barrier per step suffices.  Codes
// are requested two steps ahead into two register slots, activations (which
// stay in cache) one step ahead.
//
// Decode.  The four adjacent threads of a quad serve one weight row.  At the
// start of each group they build that row's table of the 2^B signed levels
// s_g sign(k) q(|k|/M), packed as (hi | lo << 16) (or the FP16 value), in LDS;
// the table belongs to one wavefront, so program order orders its writes and
// reads.  Each code then costs one LDS read, and two byte permutes turn two
// table entries into the hi and lo operand pairs.
//
// MFMA operand layout (16x16x32 bf16/f16): lane l supplies row l % 16 of A and
// column l % 16 of B with K slots 8 (l / 16) .. +7; the FP32 result of a block
// has lane l holding rows 4 (l / 16) + i of column l % 16.
#include "cq_device.h"
#include "cq_internal.h"
#include "stream_common.h"

#include <type_traits>

namespace cq {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kKS = 32;                 // K step: one 32-code unit
constexpr int kRowB = kKS * 2 + 16;     // LDS bytes per operand row (padded)

template <int XDT>
__device__ __forceinline__ f32x4_t mma(const u32x4 &a, const u32x4 &b, f32x4_t c) {
    if constexpr (XDT == 0)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                       c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b),
                                                      c, 0, 0, 0);
}

__device__ __forceinline__ void lds_fence_wave() {
    // LDS operations of one wavefront complete in issue order; keeping the
    // compiler from reordering them is enough for the quad that shares a table.
    __asm__ __volatile__("" ::: "memory");
    __builtin_amdgcn_wave_barrier();
}

}  // namespace

template <int B, int UPG, int XDT, int YDT, bool ONE>
__global__ void __launch_bounds__(512) gemm_a16_mfma(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int n, int k, const uint16_t *__restrict__ x, int m, void *__restrict__ y, int tiles_m, int tiles_n) {
    constexpr int M = max_code(B);
    constexpr int WM = 4, WN = 2;
    constexpr int TM = 64 * WM, TN = 64 * WN;
    constexpr int SPG = UPG;                  // steps (units) per group
    constexpr int NE = 1 << B;                // table entries (fields)
    constexpr int EPT = NE >= 4 ? NE / 4 : 1; // entries built per thread
    constexpr int TSTR = NE + 1;              // table words per row (padded)
    constexpr bool SPLIT = (XDT == 0) && !ONE;
    __shared__ __attribute__((aligned(16))) uint8_t As[2][TM * kRowB];
    __shared__ __attribute__((aligned(16))) uint8_t Bh[2][TN * kRowB];
    __shared__ __attribute__((aligned(16))) uint8_t Bl[SPLIT ? 2 : 1][SPLIT ? TN * kRowB : 16];
    __shared__ uint32_t tab[TN * TSTR];

    // ---- tile of this workgroup: the workgroups of one XCD take consecutive
    // indices, which walk the weight tiles of one activation tile
    const int nwg = tiles_m * tiles_n;
    int wg = blockIdx.x;
    if (nwg % 8 == 0) wg = (wg % 8) * (nwg / 8) + wg / 8;
    const int m0 = (wg / tiles_n) * TM;
    const int n0 = (wg % tiles_n) * TN;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = (wave / WN) * 64;
    const int wn = (wave % WN) * 64;

    const int ng = k / (32 * UPG);
    const uint32_t row_bytes = uint32_t(k) * B / 8u;
    const auto rc = make_rsrc(codes, uint32_t(n) * row_bytes);
    const auto rs = make_rsrc(scale, uint32_t(n) * ng * 4u);
    const auto ra = make_rsrc(a16, uint32_t(n) * ng * 2u);
    const auto rb = make_rsrc(b16, uint32_t(n) * ng * 2u);
    const auto rx = make_rsrc(x, uint32_t(m) * uint32_t(k) * 2u);

    // loader roles
    const int lr = tid >> 2;                 // weight row of the tile
    const int lq = tid & 3;                  // 8-code quarter of the unit
    const int wrow = n0 + lr;
    const bool wok = wrow < n;
    const int xr = tid >> 1;                 // activation row of the tile
    const int xc = (tid & 1) * 16;           // first K element of this thread
    const int xrow = m0 + xr;
    const bool xok = xrow < m;

    uint32_t cw[2][B];                       // the row's unit of the step, two slots
    float sv[2];
    uint32_t av[2], bv[2];
    uint32_t xw[8];                          // 16 activations of the next step

    auto load_step = [&](int st, auto slot_c) {
        constexpr int SL = decltype(slot_c)::value;
        load_words<B>(rc, wok ? uint32_t(wrow) * row_bytes + uint32_t(st) * (4u * B) : kOobOffset, cw[SL]);
        if (st % SPG == 0) {
            const uint32_t gi = uint32_t(wrow) * ng + st / SPG;
            sv[SL] = load_f32(rs, wok ? gi * 4u : kOobOffset);
            av[SL] = load_u16(ra, wok ? gi * 2u : kOobOffset);
            bv[SL] = load_u16(rb, wok ? gi * 2u : kOobOffset);
        }
    };
    auto load_act = [&](int st) {
        const uint32_t off = xok ? (uint32_t(xrow) * uint32_t(k) + uint32_t(st) * kKS + xc) * 2u : kOobOffset;
        load_words<8>(rx, off, xw);
    };

    // table of the row for the group starting at the step in slot SL
    const uint32_t tbase = uint32_t(lr) * TSTR;
    auto build_table = [&](auto slot_c) {
        constexpr int SL = decltype(slot_c)::value;
        float a = 1.f, b = 0.f;
        if constexpr (B >= 3) {
            a = f16_to_f32(uint16_t(av[SL]));
            b = f16_to_f32(uint16_t(bv[SL]));
        }
        const float c = 1.f - a - b;
        const float s = sv[SL];
        lds_fence_wave();  // the previous group's reads are issued
#pragma unroll
        for (int e = 0; e < EPT; ++e) {
            const int f = lq + 4 * e;
            if (f < NE) {
                const int kc = field_to_code(uint32_t(f), B);
                const float lev = (B == 1) ? float(kc) : signed_level(kc, M, a, b, c);
                const float v = s * lev;
                uint32_t ent;
                if constexpr (SPLIT) {
                    const __bf16 hi = __bf16(v);
                    const __bf16 lo = __bf16(v - float(hi));
                    ent = uint32_t(__builtin_bit_cast(uint16_t, hi)) | (uint32_t(__builtin_bit_cast(uint16_t, lo)) << 16);
                } else if constexpr (XDT == 0) {
                    ent = uint32_t(f32_to_bf16(v));
                } else {
                    ent = uint32_t(f32_to_f16(v));
                }
                tab[tbase + f] = ent;
            }
        }
        lds_fence_wave();
    };

    auto store_step = [&](auto buf_c, auto slot_c) {
        constexpr int buf = decltype(buf_c)::value;
        constexpr int SL = decltype(slot_c)::value;
        uint32_t ent[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int i = 8 * lq + e;
            const int bit = i * B;
            const int wd = bit >> 5, sh = bit & 31;
            uint32_t v;
            if (sh + B <= 32) v = cw[SL][wd] >> sh;
            else v = __builtin_amdgcn_alignbit(cw[SL][wd + 1], cw[SL][wd], sh);
            ent[e] = tab[tbase + (v & uint32_t(NE - 1))];
        }
        uint32_t hi[4], lo[4];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            hi[p] = __builtin_amdgcn_perm(ent[2 * p + 1], ent[2 * p], 0x05040100u);
            lo[p] = __builtin_amdgcn_perm(ent[2 * p + 1], ent[2 * p], 0x07060302u);
        }
        *reinterpret_cast<u32x4 *>(&Bh[buf][lr * kRowB + 16 * lq]) = u32x4{hi[0], hi[1], hi[2], hi[3]};
        if constexpr (SPLIT)
            *reinterpret_cast<u32x4 *>(&Bl[buf][lr * kRowB + 16 * lq]) = u32x4{lo[0], lo[1], lo[2], lo[3]};
        uint8_t *ap = &As[buf][xr * kRowB + 2 * xc];
        *reinterpret_cast<u32x4 *>(ap) = u32x4{xw[0], xw[1], xw[2], xw[3]};
        *reinterpret_cast<u32x4 *>(ap + 16) = u32x4{xw[4], xw[5], xw[6], xw[7]};
    };

    f32x4_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    const int nsteps = k / kKS;
    load_step(0, S0{});
    load_act(0);
    if (nsteps > 1) load_step(1, S1{});
    build_table(S0{});
    store_step(S0{}, S0{});
    if (nsteps > 1) load_act(1);
    __syncthreads();

    auto do_step = [&](int st, auto par_c) {
        constexpr int PAR = decltype(par_c)::value;  // st % 2
        constexpr int buf = PAR;
        constexpr int SN = 1 - PAR;                   // slot and buffer of step st + 1
        if (st + 2 < nsteps) load_step(st + 2, std::integral_constant<int, PAR>{});
        u32x4 af[4], bh[4], bl[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            af[i] = *reinterpret_cast<const u32x4 *>(&As[buf][(wm + 16 * i + (lane & 15)) * kRowB + 16 * (lane >> 4)]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            bh[j] = *reinterpret_cast<const u32x4 *>(&Bh[buf][(wn + 16 * j + (lane & 15)) * kRowB + 16 * (lane >> 4)]);
            if constexpr (SPLIT)
                bl[j] = *reinterpret_cast<const u32x4 *>(&Bl[buf][(wn + 16 * j + (lane & 15)) * kRowB + 16 * (lane >> 4)]);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                acc[i][j] = mma<XDT>(af[i], bh[j], acc[i][j]);
                if constexpr (SPLIT) acc[i][j] = mma<XDT>(af[i], bl[j], acc[i][j]);
            }
        if (st + 1 < nsteps) {
            if ((st + 1) % SPG == 0) build_table(std::integral_constant<int, SN>{});
            store_step(std::integral_constant<int, SN>{}, std::integral_constant<int, SN>{});
            if (st + 2 < nsteps) load_act(st + 2);
        }
        __syncthreads();
    };

    for (int st = 0; st < nsteps; st += 2) {
        do_step(st, S0{});
        if (st + 1 < nsteps) do_step(st + 1, S1{});
    }

#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int row = m0 + wm + 16 * i + 4 * (lane >> 4) + e;
            if (row >= m) continue;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int col = n0 + wn + 16 * j + (lane & 15);
                if (col < n) store_out<YDT>(y, int64_t(row) * n + col, acc[i][j][e]);
            }
        }
}

template <int B, int UPG, int XDT, int YDT, bool ONE>
static hipError_t a16_mfma_launch(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    const int tiles_m = int((m + 255) / 256);
    const int tiles_n = int((w.n + 127) / 128);
    const int64_t nwg = int64_t(tiles_m) * tiles_n;
    if (nwg > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemm_a16_mfma<B, UPG, XDT, YDT, ONE>), dim3(unsigned(nwg)), dim3(512), 0, stream, w.codes, w.scale,
                       w.a, w.b, int(w.n), int(w.k), static_cast<const uint16_t *>(x), int(m), y, tiles_m, tiles_n);
    return hipGetLastError();
}

template <int B, int XDT, int YDT, bool ONE>
static hipError_t a16_mfma_group(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    switch (w.group) {
        case 32: return a16_mfma_launch<B, 1, XDT, YDT, ONE>(w, x, m, y, stream);
        case 64: return a16_mfma_launch<B, 2, XDT, YDT, ONE>(w, x, m, y, stream);
        case 128: return a16_mfma_launch<B, 4, XDT, YDT, ONE>(w, x, m, y, stream);
        case 256: return a16_mfma_launch<B, 8, XDT, YDT, ONE>(w, x, m, y, stream);
        case 512: return a16_mfma_launch<B, 16, XDT, YDT, ONE>(w, x, m, y, stream);
    }
    return hipErrorNotSupported;
}

template <int XDT, int YDT, bool ONE>
static hipError_t a16_mfma_bits(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    switch (w.bits) {
        case 1: return a16_mfma_group<1, XDT, YDT, ONE>(w, x, m, y, stream);
        case 2: return a16_mfma_group<2, XDT, YDT, ONE>(w, x, m, y, stream);
        case 3: return a16_mfma_group<3, XDT, YDT, ONE>(w, x, m, y, stream);
        case 4: return a16_mfma_group<4, XDT, YDT, ONE>(w, x, m, y, stream);
        case 5: return a16_mfma_group<5, XDT, YDT, ONE>(w, x, m, y, stream);
    }
    return hipErrorNotSupported;
}

bool gemm_a16_mfma_supported(const cq_weight &w, int64_t m) {
    const int64_t lim = int64_t(1) << 31;
    return w.bits <= 5 && m * w.k * 2 < lim && stream_fits(w.n, w.k, w.bits, w.group) && m < lim;
}

hipError_t launch_gemm_a16_mfma(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                hipStream_t stream) {
    if (x_dt == 0) {
        if (y_dt == 0) return a16_mfma_bits<0, 0, false>(w, x, m, y, stream);
        return a16_mfma_bits<0, 2, false>(w, x, m, y, stream);
    }
    if (y_dt == 1) return a16_mfma_bits<1, 1, false>(w, x, m, y, stream);
    return a16_mfma_bits<1, 2, false>(w, x, m, y, stream);
}

hipError_t launch_gemm_a16_mfma_rounded(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                        hipStream_t stream) {
    if (x_dt == 0) {
        if (y_dt == 0) return a16_mfma_bits<0, 0, true>(w, x, m, y, stream);
        return a16_mfma_bits<0, 2, true>(w, x, m, y, stream);
    }
    // FP16 activations: the default kernel already takes one FP16 operand
    if (y_dt == 1) return a16_mfma_bits<1, 1, false>(w, x, m, y, stream);
    return a16_mfma_bits<1, 2, false>(w, x, m, y, stream);
}

}  // namespace cq
