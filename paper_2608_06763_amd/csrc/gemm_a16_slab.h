// Model-dtype GEMM for few rows of x (Sec. 5.3 dense tactic, in the regime of
// Sec. 5.5 between the single-row GEMV and the tiled GEMM) for B <= 5 on gfx950
// matrix cores, with every weight decoded straight into the matrix-core
// operand of the lane that decoded it: no decoded tile goes through LDS and
// the K loop has no barrier.
//
// Numerics: every weight is reconstructed in FP32 as s_g sign(k) q(|k|/M)
// (eq. cubic in the Horner form of eq. gpu-horner, q(1) = 1) and carried as
// the unevaluated sum hi + lo of two numbers in the activation dtype (hi =
// RNE(v), lo = RNE(v - hi)); both halves go through the matrix core into one
// FP32 accumulator (v_mfma_f32_16x16x32_{bf16,f16}), as in the tiled GEMM's
// BF16 default.
//
// Mapping.  A wave owns BJ blocks of 16 weight rows and 16 BI rows of x.  In
// the 16x16x32 MFMA, lane l supplies column l % 16 of B and row l % 16 of A,
// each with the K slots 8 (l / 16) .. +7.  K is visited in sweeps of four
// groups: during sweep j the lanes 16 q .. 16 q + 15 feed the slots 8 q .. +7
// of each MFMA from group 4 j + q of their rows, 8 consecutive codes per
// MFMA, so a sweep takes G / 8 MFMAs and each lane stays inside one group of
// one weight row for the whole sweep.  A sum does not depend on the order of
// its terms, and the activations are read in the same order.  Each lane thus
// builds one table of the 2^B signed levels (hi | lo << 16) per group, in
// its own LDS column (byte field * 256 + lane * 4 of its wave's slot: every
// lane reads its own bank), and a code costs one address permute, one LDS
// read and one of the two byte permutes that form the hi and lo operands.
//
// Split-K.  The S waves of a workgroup share its weight rows and take the
// sweeps w, w + S, w + 2S, ...; their accumulators meet in LDS once at the
// end.  Each wave requests the codes, activations and group metadata of a
// chunk (four MFMAs) R chunks before it decodes it; every load is issued
// unconditionally and in program order, so each wait is for the oldest slot.
#pragma once

#include "cq_device.h"
#include "cq_internal.h"
#include "stream_common.h"

#include <type_traits>

namespace cq {

namespace a16_slab {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) uint32_t lds_u32;
typedef __attribute__((address_space(3))) f32x4_t lds_f32x4;

__device__ __forceinline__ uint32_t lds_ld(uint32_t a) { return *reinterpret_cast<const lds_u32 *>(uintptr_t(a)); }
__device__ __forceinline__ void lds_st(uint32_t a, uint32_t v) { *reinterpret_cast<lds_u32 *>(uintptr_t(a)) = v; }

template <int XDT>
__device__ __forceinline__ f32x4_t mma(const u32x4 &a, const u32x4 &b, f32x4_t c) {
    if constexpr (XDT == 0)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                       c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b),
                                                      c, 0, 0, 0);
}

template <int P0, int PN, typename F>
__device__ __forceinline__ void unroll_for(F &&f) {
    if constexpr (P0 < PN) {
        f(std::integral_constant<int, P0>{});
        unroll_for<P0 + 1, PN>(f);
    }
}

// vector-memory reads stay in program order (the wait before a ring slot is
// used counts the loads issued after it)
__device__ __forceinline__ void vmem_order() { __builtin_amdgcn_sched_barrier(0x78f); }

__device__ __forceinline__ void wave_lds_fence() {
    // one wavefront's LDS operations complete in issue order; only the
    // compiler must not move them across this point
    __asm__ __volatile__("" ::: "memory");
    __builtin_amdgcn_wave_barrier();
}

// table entry of the FP32 weight v: (hi | lo << 16) in the activation dtype,
// hi = RNE(v), lo = RNE(v - hi)
template <int XDT>
__device__ __forceinline__ uint32_t operand_entry(float v) {
    if constexpr (XDT == 0) {
        const __bf16 hi = __bf16(v);
        const __bf16 lo = __bf16(v - float(hi));
        return uint32_t(__builtin_bit_cast(uint16_t, hi)) | (uint32_t(__builtin_bit_cast(uint16_t, lo)) << 16);
    } else {
        const _Float16 hi = _Float16(v);
        const _Float16 lo = _Float16(v - float(hi));
        return uint32_t(__builtin_bit_cast(uint16_t, hi)) | (uint32_t(__builtin_bit_cast(uint16_t, lo)) << 16);
    }
}

}  // namespace a16_slab

template <int B, int UPG, int XDT, int YDT, int BI, int BJ, int R>
__global__ void __launch_bounds__(1024) gemm_a16_slab(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int n, int k, const uint16_t *__restrict__ x, int m, void *__restrict__ y, int tiles_n) {
    using namespace a16_slab;
    constexpr int M = max_code(B);
    constexpr int NE = 1 << B;                // table fields
    constexpr int G = 32 * UPG;
    constexpr bool SPLIT = true;
    constexpr uint32_t kTab = NE * 256u;      // bytes of one lane-column table set
    constexpr uint32_t kNeg = 0x80008000u;
    constexpr int PER = R > UPG ? R : UPG;    // chunks per unrolled period
    static_assert(PER % R == 0 && PER % UPG == 0, "ring depth and chunks per group nest");
    extern __shared__ __attribute__((aligned(16))) uint32_t lds[];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
    const int nw = blockDim.x >> 6;
    const int nl = lane & 15, q = lane >> 4;
    const int tm = blockIdx.x / tiles_n, tn = blockIdx.x - tm * tiles_n;
    const int m0 = tm * 16 * BI, n0 = tn * 16 * BJ;

    const int ng = k / G;
    const int nsw = (ng + 3) >> 2;            // sweeps of four groups
    const int mysw = wave < nsw ? (nsw - 1 - wave) / nw + 1 : 0;
    const int nch = mysw * UPG;               // chunks of this wave
    const uint32_t row_bytes = uint32_t(k) * B / 8u;
    const auto rc = make_rsrc(codes, uint32_t(n) * row_bytes);
    const auto rs = make_rsrc(scale, uint32_t(n) * ng * 4u);
    const auto ra = make_rsrc(a16, uint32_t(n) * ng * 2u);
    const auto rb = make_rsrc(b16, uint32_t(n) * ng * 2u);
    const auto rx = make_rsrc(x, uint32_t(m) * uint32_t(k) * 2u);

    // this lane's table columns (one per weight-row block)
    const uint32_t tbase = uint32_t(uintptr_t((lds_u32 *)lds));
    const uint32_t col0 = tbase + uint32_t(wave * BJ) * kTab + uint32_t(lane) * 4u;

    // ring of R chunk slots
    uint32_t cw[R][BJ][B];
    uint32_t xw[R][BI][16];
    // group metadata of a sweep, loaded by lane l for row l / 4 of the block
    // and group l % 4 of the sweep (each quad of lanes reads one run of a
    // row), then handed to lane (row, group slot) by ds_bpermute
    float sv[R][BJ];
    uint32_t abv[R][BJ];

    // chunk c of this wave: sweep wave + nw (c / UPG), unit c % UPG of the group
    auto load_slot = [&](int c, auto slot_c, auto meta_c) {
        constexpr int SL = decltype(slot_c)::value;
        constexpr bool META = decltype(meta_c)::value;
        const int sw = wave + nw * (c / UPG);
        const int u = c % UPG;
        const int g = 4 * sw + q;
        const bool gok = g < ng;
#pragma unroll
        for (int j = 0; j < BJ; ++j) {
            const int row = n0 + 16 * j + nl;
            const bool ok = gok && row < n;
            const uint32_t gi = uint32_t(row) * uint32_t(ng) + uint32_t(g);
            load_words<B>(rc, ok ? uint32_t(row) * row_bytes + (uint32_t(g) * UPG + uint32_t(u)) * (4u * B) : kOobOffset,
                          cw[SL][j]);
            if constexpr (META) {
                const int mrow = n0 + 16 * j + (lane >> 2);
                const int mg = 4 * sw + (lane & 3);
                const bool mok = mrow < n && mg < ng;
                const uint32_t mi = uint32_t(mrow) * uint32_t(ng) + uint32_t(mg);
                sv[SL][j] = load_f32(rs, mok ? mi * 4u : kOobOffset);
                abv[SL][j] = load_u16(ra, mok ? mi * 2u : kOobOffset) | (load_u16(rb, mok ? mi * 2u : kOobOffset) << 16);
            }
        }
#pragma unroll
        for (int i = 0; i < BI; ++i) {
            const int row = m0 + 16 * i + nl;
            const bool ok = gok && row < m;
            load_words<16>(rx, ok ? (uint32_t(row) * uint32_t(k) + uint32_t(g) * G + uint32_t(u) * 32u) * 2u : kOobOffset,
                           xw[SL][i]);
        }
    };

    // fields that no group rewrites: the zero code and the reserved pattern
    if constexpr (B >= 2) {
#pragma unroll
        for (int j = 0; j < BJ; ++j) {
            lds_st(col0 + j * kTab, 0u);
            lds_st(col0 + j * kTab + uint32_t(NE / 2) * 256u, 0u);
        }
    }

    // the lane's tables for the group whose metadata sit in slot SL
    auto build_tables = [&](auto slot_c) {
        constexpr int SL = decltype(slot_c)::value;
        wave_lds_fence();  // the previous group's reads are issued
#pragma unroll
        for (int j = 0; j < BJ; ++j) {
            const uint32_t cj = col0 + j * kTab;
            const int src = (4 * nl + q) << 2;
            const float s = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(sv[SL][j])));
            const uint32_t es = operand_entry<XDT>(s);  // q(1) = 1
            if constexpr (B == 1) {
                lds_st(cj, es ^ kNeg);
                lds_st(cj + 256u, es);
            } else {
                lds_st(cj + uint32_t(M) * 256u, es);
                lds_st(cj + uint32_t(NE - M) * 256u, es ^ kNeg);
                if constexpr (B >= 3) {
                    const uint32_t ab = uint32_t(__builtin_amdgcn_ds_bpermute(src, int(abv[SL][j])));
                    const float a = f16_to_f32(uint16_t(ab & 0xffffu));
                    const float b = f16_to_f32(uint16_t(ab >> 16));
                    const float cc = 1.f - a - b;
#pragma unroll
                    for (int i = 1; i < M; ++i) {
                        const float t = float(i) / float(M);
                        const float qv = t * __builtin_fmaf(t, __builtin_fmaf(t, cc, b), a);
                        const uint32_t e = operand_entry<XDT>(s * qv);
                        lds_st(cj + uint32_t(i) * 256u, e);
                        lds_st(cj + uint32_t(NE - i) * 256u, e ^ kNeg);
                    }
                }
            }
        }
        wave_lds_fence();
    };

    f32x4_t acc[BI][BJ];
#pragma unroll
    for (int i = 0; i < BI; ++i)
#pragma unroll
        for (int j = 0; j < BJ; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // the nibble mask sits in a vector register so that mask and slot tag
    // fold into one v_and_or_b32
    uint32_t nmask;
    __asm__("v_mov_b32 %0, 0x0f0f0f0f" : "=v"(nmask));

    // decode and multiply the chunk in slot SL
    auto compute = [&](auto slot_c) {
        constexpr int SL = decltype(slot_c)::value;
#pragma unroll
        for (int j = 0; j < BJ; ++j) {
            const uint32_t cj = col0 + j * kTab;
            uint32_t ent[32];
            if constexpr (B == 4) {
                // byte 1 of the address is (slot << 4) | field; bytes 0, 2, 3 come
                // from the column (the tables end below 64 KB)
                const uint32_t tag = uint32_t(wave * BJ + j) * 0x10101010u;
#pragma unroll
                for (int st = 0; st < 4; ++st) {
                    const uint32_t wd = cw[SL][j][st];
                    const uint32_t lo4 = (wd & nmask) | tag;
                    const uint32_t hi4 = ((wd >> 4) & nmask) | tag;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const uint32_t sel = 0x03020000u | (uint32_t(4 + e / 2) << 8);
                        ent[8 * st + e] = lds_ld(__builtin_amdgcn_perm((e & 1) ? hi4 : lo4, cj, sel));
                    }
                }
            } else {
#pragma unroll
                for (int e = 0; e < 32; ++e) {
                    const int bit = e * B;
                    const int wd = bit >> 5, sh = bit & 31;
                    uint32_t v;
                    if (sh + B <= 32) v = cw[SL][j][wd] >> sh;
                    else v = __builtin_amdgcn_alignbit(cw[SL][j][wd + 1], cw[SL][j][wd], sh);
                    ent[e] = lds_ld(((v & uint32_t(NE - 1)) << 8) + cj);
                }
            }
#pragma unroll
            for (int st = 0; st < 4; ++st) {
                u32x4 bh, bl;
#pragma unroll
                for (int p = 0; p < 4; ++p) {
                    bh[p] = __builtin_amdgcn_perm(ent[8 * st + 2 * p + 1], ent[8 * st + 2 * p], 0x05040100u);
                    if constexpr (SPLIT)
                        bl[p] = __builtin_amdgcn_perm(ent[8 * st + 2 * p + 1], ent[8 * st + 2 * p], 0x07060302u);
                }
#pragma unroll
                for (int i = 0; i < BI; ++i) {
                    const u32x4 af = u32x4{xw[SL][i][4 * st], xw[SL][i][4 * st + 1], xw[SL][i][4 * st + 2],
                                           xw[SL][i][4 * st + 3]};
                    acc[i][j] = mma<XDT>(af, bh, acc[i][j]);
                    if constexpr (SPLIT) acc[i][j] = mma<XDT>(af, bl, acc[i][j]);
                }
            }
        }
    };

    if (nch > 0) {
        // prologue: chunks 0 .. R - 1 requested into their slots
        unroll_for<0, R>([&](auto p_c) {
            constexpr int P = decltype(p_c)::value;
            load_slot(min(P, nch - 1), p_c, std::integral_constant<bool, P % UPG == 0>{});
            vmem_order();
        });
        for (int c0 = 0; c0 < nch; c0 += PER) {
            unroll_for<0, PER>([&](auto p_c) {
                constexpr int P = decltype(p_c)::value;
                constexpr int SL = P % R;
                const int c = c0 + P;
                if (c < nch) {
                    if constexpr (P % UPG == 0) build_tables(std::integral_constant<int, SL>{});
                    compute(std::integral_constant<int, SL>{});
                }
                // the slot just used receives chunk c + R
                load_slot(min(c + R, nch - 1), std::integral_constant<int, SL>{},
                          std::integral_constant<bool, (P + R) % UPG == 0>{});
                vmem_order();
            });
        }
    }

    // ---- cross-wave sum and store
    auto store_block = [&](int i, int j, const f32x4_t &v) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int row = m0 + 16 * i + 4 * q + e;
            const int col = n0 + 16 * j + nl;
            if (row < m && col < n) store_out<YDT>(y, int64_t(row) * n + col, v[e]);
        }
    };
    if (nw == 1) {
#pragma unroll
        for (int i = 0; i < BI; ++i)
#pragma unroll
            for (int j = 0; j < BJ; ++j) store_block(i, j, acc[i][j]);
        return;
    }
    __syncthreads();  // every wave is done with its tables
    lds_f32x4 *red = reinterpret_cast<lds_f32x4 *>(uintptr_t(tbase));
#pragma unroll
    for (int i = 0; i < BI; ++i)
#pragma unroll
        for (int j = 0; j < BJ; ++j) red[((wave * BI + i) * BJ + j) * 64 + lane] = acc[i][j];
    __syncthreads();
    for (int blk = wave; blk < BI * BJ; blk += nw) {
        f32x4_t v = f32x4_t{0.f, 0.f, 0.f, 0.f};
        for (int w = 0; w < nw; ++w) v += red[(w * BI * BJ + blk) * 64 + lane];
        store_block(blk / BJ, blk % BJ, v);
    }
}

// Staged variant for up to 16 rows of x and 16 weight rows per wave.  The
// mapping of lanes to MFMA slots, the K order and the tables are those above;
// what changes is how codes and group metadata reach a lane.  A lane's own
// slice of the weights (16 B of one group of one row per chunk) lies apart
// from its neighbours', so loading it directly touches many cache lines per
// wave load.  Here each wave takes a contiguous range of sweeps and, per
// sweep, loads the 16 rows' code bytes of the sweep's four groups as runs of
// whole cache lines (a row's bytes of one sweep are contiguous), writes them
// to its own LDS staging area and reads each lane's slice back from there;
// the group metadata of four sweeps (16 groups per row) are loaded the same
// way once per four sweeps.  Only the wave itself touches its staging area,
// so program order orders the writes and reads.  Requires a multiple of four
// groups per row and at most 512 code bytes per row and sweep.
//
// ROUTED: a bank of experts of n weight rows each, stacked; workgroup
// (e, 16 weight rows) serves every route of expert e that the grouping pass
// listed (rorder[roff[e] .. roff[e + 1])), 16 routes at a time: a route's x
// row is its token and its output is row `route` of y.
template <int B, int UPG, int XDT, int YDT, bool ROUTED, bool XT, int XB>
__global__ void __launch_bounds__((ROUTED || XT) ? 512 : 1024) gemm_a16_slab_st(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int n, int k, const uint16_t *__restrict__ x, int m, void *__restrict__ y, int tiles_n,
    const int32_t *__restrict__ rtok, const int32_t *__restrict__ rorder, const int32_t *__restrict__ roff) {
    using namespace a16_slab;
    typedef __attribute__((address_space(3))) u32x4 lds_u32x4;
    typedef __attribute__((address_space(3))) float lds_f32;
    constexpr int M = max_code(B);
    constexpr int NE = 1 << B;
    constexpr int G = 32 * UPG;
    constexpr int GB = G * B / 8;             // code bytes of one group of a row
    constexpr int SEG = 4 * GB;               // ... of one sweep
    constexpr int P = SEG / 16;               // 16-byte pieces of a row per sweep
    constexpr int T = (16 * P + 63) / 64;     // wave loads per sweep
    constexpr uint32_t CS = SEG + 16;         // staged row stride (bytes)
    constexpr int NB = 4;                     // sweeps per metadata batch
    constexpr uint32_t kTab = NE * 256u;
    constexpr uint32_t kMeta = 16u * NB * 16u;  // one metadata array of a batch (bytes)
    static_assert(XB == 1 || (XB == 2 && XT && !ROUTED), "two x-row blocks take the transposed activations");
    constexpr uint32_t kX = XT ? XB * 64u * 80u : 0u;  // transposed activations of a chunk
    constexpr uint32_t kStage = 16u * CS + 2u * kMeta + kX;
    constexpr uint32_t kNeg = 0x80008000u;
    static_assert(SEG % 16 == 0 && SEG <= 512, "staged sweep size");
    extern __shared__ __attribute__((aligned(16))) uint32_t lds[];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
    const int nw = blockDim.x >> 6;
    const int nl = lane & 15, q = lane >> 4;
    const int tm = blockIdx.x / tiles_n, tn = blockIdx.x - tm * tiles_n;
    const int n0 = tn * 16;
    const int ng = k / G;                     // a multiple of 4
    const uint32_t row_bytes = uint32_t(k) * B / 8u;
    // rows of x served by this workgroup, 16 XB at a time: rows tm * 16 XB ..,
    // or (routed: tm is the expert) the expert's routes, whose x rows are their
    // tokens and whose outputs are rows of y in route order
    int c_begin, c_end;
    if constexpr (ROUTED) {
        c_begin = roff[tm];
        c_end = roff[tm + 1];
        codes += size_t(tm) * n * row_bytes;
        scale += size_t(tm) * n * ng;
        a16 += size_t(tm) * n * ng;
        b16 += size_t(tm) * n * ng;
    } else {
        c_begin = tm * 16 * XB;
        c_end = min(c_begin + 16 * XB, m);
    }
    const int nsw = ng >> 2;
    const int per = (nsw + nw - 1) / nw;      // contiguous sweeps per wave
    const int sa = min(wave * per, nsw);
    const int sb = min(sa + per, nsw);
    const int nmy = sb - sa;
    const int nch = nmy * UPG;
    const auto rc = make_rsrc(codes, uint32_t(n) * row_bytes);
    const auto rs = make_rsrc(scale, uint32_t(n) * ng * 4u);
    const auto ra = make_rsrc(a16, uint32_t(n) * ng * 2u);
    const auto rb = make_rsrc(b16, uint32_t(n) * ng * 2u);
    const auto rx = make_rsrc(x, uint32_t(m) * uint32_t(k) * 2u);

    // LDS: the tables of all waves (below 64 KB, for the W4 address build),
    // then one staging area per wave
    const uint32_t tbase = uint32_t(uintptr_t((lds_u32 *)lds));
    const uint32_t col = tbase + uint32_t(wave) * kTab + uint32_t(lane) * 4u;
    const uint32_t stg = tbase + uint32_t(nw) * kTab + uint32_t(wave) * kStage;
    const uint32_t mst = stg + 16u * CS;      // batch scales [row][sweep][group]
    const uint32_t mab = mst + kMeta;         // batch a | b << 16, same layout
    const uint32_t xst = mab + kMeta;         // XT: activation pieces [block][q * 16 + row][80 bytes]

    uint32_t cr[T][4];                        // codes of one sweep as loaded
    uint32_t ms4[4], ma2[2], mb2[2];          // metadata of one batch as loaded
    uint32_t xw[2][XB][16];                   // activations of two chunks

    // codes of sweep sw (out-of-range sweeps and rows read zeros)
    auto load_codes = [&](int sw) {
        const bool ok = sw < sb;
#pragma unroll
        for (int t = 0; t < T; ++t) {
            const int f = 64 * t + lane;
            const int r = f / P, p = f - r * P;
            const bool okr = ok && r < 16 && n0 + r < n;
            load_words<4>(rc, okr ? uint32_t(n0 + r) * row_bytes + uint32_t(sw) * SEG + uint32_t(p) * 16u : kOobOffset,
                          cr[t]);
        }
    };
    auto store_codes = [&]() {
#pragma unroll
        for (int t = 0; t < T; ++t) {
            const int f = 64 * t + lane;
            const int r = f / P, p = f - r * P;
            if ((16 * P) % 64 == 0 || r < 16)
                *reinterpret_cast<lds_u32x4 *>(uintptr_t(stg + uint32_t(r) * CS + uint32_t(p) * 16u)) =
                    u32x4{cr[t][0], cr[t][1], cr[t][2], cr[t][3]};
        }
    };
    // batch bi (sweeps sa + 4 bi .. + 3): lane L holds the four groups of
    // sweep sa + 4 bi + L % 4 of row L / 4
    auto load_meta = [&](int bi) {
        const int r = lane >> 2;
        const int sw = sa + NB * bi + (lane & 3);
        const bool ok = sw < sb && n0 + r < n;
        const uint32_t gi = uint32_t(n0 + r) * uint32_t(ng) + 4u * uint32_t(sw);
        load_words<4>(rs, ok ? gi * 4u : kOobOffset, ms4);
        load_words<2>(ra, ok ? gi * 2u : kOobOffset, ma2);
        load_words<2>(rb, ok ? gi * 2u : kOobOffset, mb2);
    };
    auto store_meta = [&]() {
        const uint32_t o = uint32_t(lane) * 16u;  // [row][sweep of batch][group]
        *reinterpret_cast<lds_u32x4 *>(uintptr_t(mst + o)) = u32x4{ms4[0], ms4[1], ms4[2], ms4[3]};
        *reinterpret_cast<lds_u32x4 *>(uintptr_t(mab + o)) =
            u32x4{__builtin_amdgcn_perm(mb2[0], ma2[0], 0x05040100u), __builtin_amdgcn_perm(mb2[0], ma2[0], 0x07060302u),
                  __builtin_amdgcn_perm(mb2[1], ma2[1], 0x05040100u), __builtin_amdgcn_perm(mb2[1], ma2[1], 0x07060302u)};
    };
    // x row of this lane's MFMA row in the current 16 rows (-1: none); with
    // XT, the rows of the four pieces this lane loads (row 4 i + lane / 16)
    int xr = -1;
    int xrl[XB][4];
    // activations of chunk c (sweep sa + c / UPG, unit c % UPG of each lane's
    // group).  XT: a wave load brings 64-byte pieces (row r, group q) as four
    // lanes' 16-byte parts, the parts of one row's four groups lying 2G bytes
    // apart, instead of one 16-byte part per lane and cache line; the pieces
    // are handed to their lanes through LDS in compute().
    auto load_x = [&](int c, auto slot_c) {
        constexpr int SL = decltype(slot_c)::value;
        const int sw = sa + c / UPG, u = c % UPG;
        if constexpr (XT) {
            const int gq = (lane >> 2) & 3, sub = lane & 3;
#pragma unroll
            for (int b = 0; b < XB; ++b)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int row = xrl[b][i];
                    const bool ok = row >= 0 && sw < sb;
                    load_words<4>(rx,
                                  ok ? (uint32_t(row) * uint32_t(k) + uint32_t(4 * sw + gq) * G + uint32_t(u) * 32u) * 2u +
                                           16u * uint32_t(sub)
                                     : kOobOffset,
                                  &xw[SL][b][4 * i]);
                }
        } else {
            const int row = xr;
            const bool ok = row >= 0 && sw < sb;
            load_words<16>(rx, ok ? (uint32_t(row) * uint32_t(k) + uint32_t(4 * sw + q) * G + uint32_t(u) * 32u) * 2u
                                  : kOobOffset,
                           xw[SL][0]);
        }
    };

    // the lane's table for its group of sweep i of the wave (batch slot i % NB)
    auto build_table = [&](int j) {
        wave_lds_fence();  // staged metadata written, previous group's reads issued
        const uint32_t o = (uint32_t(nl) * NB + uint32_t(j)) * 16u + uint32_t(q) * 4u;
        const float s = *reinterpret_cast<const lds_f32 *>(uintptr_t(mst + o));
        const uint32_t ab = lds_ld(mab + o);
        const uint32_t es = operand_entry<XDT>(s);
        if constexpr (B == 1) {
            lds_st(col, es ^ kNeg);
            lds_st(col + 256u, es);
        } else {
            lds_st(col + uint32_t(M) * 256u, es);
            lds_st(col + uint32_t(NE - M) * 256u, es ^ kNeg);
            if constexpr (B >= 3) {
                const float a = f16_to_f32(uint16_t(ab & 0xffffu));
                const float b = f16_to_f32(uint16_t(ab >> 16));
                const float cc = 1.f - a - b;
#pragma unroll
                for (int i = 1; i < M; ++i) {
                    const float t = float(i) / float(M);
                    const float qv = t * __builtin_fmaf(t, __builtin_fmaf(t, cc, b), a);
                    const uint32_t e = operand_entry<XDT>(s * qv);
                    lds_st(col + uint32_t(i) * 256u, e);
                    lds_st(col + uint32_t(NE - i) * 256u, e ^ kNeg);
                }
            }
        }
        wave_lds_fence();
    };

    uint32_t nmask;
    __asm__("v_mov_b32 %0, 0x0f0f0f0f" : "=v"(nmask));
    const uint32_t tag = uint32_t(wave) * 0x10101010u;
    f32x4_t acc[XB];

    // decode unit u of the staged sweep and multiply with activation slot SL
    auto compute = [&](int u, auto slot_c) {
        constexpr int SL = decltype(slot_c)::value;
        u32x4 xa[XB][4];  // this lane's activations of the chunk's four MFMAs, per x-row block
        if constexpr (XT) {
            // pieces to their slots q * 16 + row (80-byte slots: the 16 lanes
            // of one block read 16 disjoint 4-bank ranges), then this lane's
            const int gq = (lane >> 2) & 3, sub = lane & 3;
#pragma unroll
            for (int b = 0; b < XB; ++b)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint32_t slot = uint32_t(64 * b) + uint32_t(gq) * 16u + uint32_t(4 * i + (lane >> 4));
                    *reinterpret_cast<lds_u32x4 *>(uintptr_t(xst + slot * 80u + 16u * uint32_t(sub))) =
                        u32x4{xw[SL][b][4 * i], xw[SL][b][4 * i + 1], xw[SL][b][4 * i + 2], xw[SL][b][4 * i + 3]};
                }
            wave_lds_fence();
#pragma unroll
            for (int b = 0; b < XB; ++b) {
                const uint32_t mine = xst + (uint32_t(64 * b) + uint32_t(q) * 16u + uint32_t(nl)) * 80u;
#pragma unroll
                for (int st = 0; st < 4; ++st)
                    xa[b][st] = *reinterpret_cast<const lds_u32x4 *>(uintptr_t(mine + 16u * st));
            }
        } else {
#pragma unroll
            for (int st = 0; st < 4; ++st)
                xa[0][st] = u32x4{xw[SL][0][4 * st], xw[SL][0][4 * st + 1], xw[SL][0][4 * st + 2], xw[SL][0][4 * st + 3]};
        }
        const uint32_t ca = stg + uint32_t(nl) * CS + uint32_t(q) * GB + uint32_t(u) * (4u * B);
        uint32_t cw[B];
        if constexpr (B == 4) {
            const u32x4 v = *reinterpret_cast<const lds_u32x4 *>(uintptr_t(ca));
            cw[0] = v[0]; cw[1] = v[1]; cw[2] = v[2]; cw[3] = v[3];
        } else {
#pragma unroll
            for (int e = 0; e < B; ++e) cw[e] = lds_ld(ca + 4u * e);
        }
        uint32_t ent[32];
        if constexpr (B == 4) {
#pragma unroll
            for (int st = 0; st < 4; ++st) {
                const uint32_t lo4 = (cw[st] & nmask) | tag;
                const uint32_t hi4 = ((cw[st] >> 4) & nmask) | tag;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint32_t sel = 0x03020000u | (uint32_t(4 + e / 2) << 8);
                    ent[8 * st + e] = lds_ld(__builtin_amdgcn_perm((e & 1) ? hi4 : lo4, col, sel));
                }
            }
        } else {
#pragma unroll
            for (int e = 0; e < 32; ++e) {
                const int bit = e * B;
                const int wd = bit >> 5, sh = bit & 31;
                uint32_t v;
                if (sh + B <= 32) v = cw[wd] >> sh;
                else v = __builtin_amdgcn_alignbit(cw[wd + 1], cw[wd], sh);
                ent[e] = lds_ld(((v & uint32_t(NE - 1)) << 8) + col);
            }
        }
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            u32x4 bh, bl;
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                bh[p] = __builtin_amdgcn_perm(ent[8 * st + 2 * p + 1], ent[8 * st + 2 * p], 0x05040100u);
                bl[p] = __builtin_amdgcn_perm(ent[8 * st + 2 * p + 1], ent[8 * st + 2 * p], 0x07060302u);
            }
#pragma unroll
            for (int b = 0; b < XB; ++b) {
                acc[b] = mma<XDT>(xa[b][st], bh, acc[b]);
                acc[b] = mma<XDT>(xa[b][st], bl, acc[b]);
            }
        }
        if constexpr (XT) wave_lds_fence();  // the pieces are read before the next chunk's are written
    };

  for (int c0 = c_begin; c0 < c_end; c0 += 16 * XB) {
    if constexpr (XT) {
#pragma unroll
        for (int b = 0; b < XB; ++b)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = c0 + 16 * b + 4 * i + (lane >> 4);
                if constexpr (ROUTED) xrl[b][i] = r < c_end ? rtok[rorder[r]] : -1;
                else xrl[b][i] = r < c_end ? r : -1;
            }
    } else {
        if constexpr (ROUTED) xr = c0 + nl < c_end ? rtok[rorder[c0 + nl]] : -1;
        else xr = c0 + nl < c_end ? c0 + nl : -1;
    }
#pragma unroll
    for (int b = 0; b < XB; ++b) acc[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (nmy > 0) {
        if constexpr (B >= 2) {
            lds_st(col, 0u);
            lds_st(col + uint32_t(NE / 2) * 256u, 0u);
        }
        // prologue: metadata of batch 0, codes of the first sweep, activations of chunks 0 and 1
        load_meta(0);
        vmem_order();
        load_codes(sa);
        vmem_order();
        load_x(0, std::integral_constant<int, 0>{});
        load_x(min(1, nch - 1), std::integral_constant<int, 1>{});
        vmem_order();
        // one period: a metadata batch of NB sweeps of UPG chunks each
        for (int i0 = 0; i0 < nmy; i0 += NB) {
            unroll_for<0, NB>([&](auto j_c) {
                constexpr int J = decltype(j_c)::value;
                const int i = i0 + J;
                const bool active = i < nmy;
                if constexpr (J == 0) {
                    store_meta();
                    load_meta(i0 / NB + 1);
                    vmem_order();
                }
                if (active) {
                    store_codes();
                    build_table(J);
                }
                unroll_for<0, UPG>([&](auto u_c) {
                    constexpr int U = decltype(u_c)::value;
                    constexpr int SL = (J * UPG + U) % 2;
                    const int c = i * UPG + U;
                    if (active) compute(U, std::integral_constant<int, SL>{});
                    load_x(min(c + 2, nch - 1), std::integral_constant<int, SL>{});
                    vmem_order();
                    if constexpr (U == 0) {
                        load_codes(sa + i + 1);
                        vmem_order();
                    }
                });
            });
        }
    }

    // ---- cross-wave sum and store
    auto store_block = [&](int b, const f32x4_t &v) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int rr = c0 + 16 * b + 4 * q + e;
            const int cl = n0 + nl;
            if (rr < c_end && cl < n) {
                const int row = ROUTED ? rorder[rr] : rr;
                store_out<YDT>(y, int64_t(row) * n + cl, v[e]);
            }
        }
    };
    if (nw == 1) {
#pragma unroll
        for (int b = 0; b < XB; ++b) store_block(b, acc[b]);
        continue;
    }
    __syncthreads();
    lds_f32x4 *red = reinterpret_cast<lds_f32x4 *>(uintptr_t(tbase));
#pragma unroll
    for (int b = 0; b < XB; ++b) red[(wave * XB + b) * 64 + lane] = acc[b];
    __syncthreads();
    for (int b = wave; b < XB; b += nw) {
        f32x4_t v = f32x4_t{0.f, 0.f, 0.f, 0.f};
        for (int w = 0; w < nw; ++w) v += red[(w * XB + b) * 64 + lane];
        store_block(b, v);
    }
    __syncthreads();  // the sums are read before the next rows' tables reuse the space
  }
}

namespace a16_slab {

template <int B, int UPG, int XDT, int YDT, int BI, int BJ>
hipError_t slab_launch(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    constexpr int R = 2;  // chunks in flight per wave
    constexpr int NE = 1 << B;
    const int64_t tiles_m = (m + 16 * BI - 1) / (16 * BI);
    const int64_t tiles_n = (w.n + 16 * BJ - 1) / (16 * BJ);
    const int64_t tiles = tiles_m * tiles_n;
    if (tiles > 0x7fffffff) return hipErrorInvalidValue;
    const int64_t ng = w.k / w.group;
    const int64_t nsw = (ng + 3) / 4;
    // waves per workgroup: enough for about four waves per SIMD over the
    // chip (one per SIMD from 9 rows in one x block, rounded down to a power
    // of two: 4096 x 4096 at 12 and 16 rows 9.2 -> 8.4 and 10.3 -> 9.2 us,
    // 4096 x 6144 at 16 rows 12.7 -> 12.3, at 12 rows 11.7 -> 12.2), no more
    // than there are sweeps, and table slots within 64 KB
    int64_t s = int64_t(device_cu_count()) * (BI == 1 && m > 8 ? 4 : 16) / tiles;
    if (BI == 1 && m > 8)
        while (s & (s - 1)) s &= s - 1;
    const int64_t smax = 65536 / (int64_t(BJ) * NE * 256);
    if (s > smax) s = smax;
    if (s > 16) s = 16;
    if (s > nsw) s = nsw;
    if (s < 1) s = 1;
    const size_t tab = size_t(s) * BJ * NE * 256;
    const size_t red = size_t(s) * BI * BJ * 1024;
    const size_t lds = tab > red ? tab : red;
    hipLaunchKernelGGL((gemm_a16_slab<B, UPG, XDT, YDT, BI, BJ, R>), dim3(unsigned(tiles)), dim3(unsigned(64 * s)),
                       lds, stream, w.codes, w.scale, w.a, w.b, int(w.n), int(w.k), static_cast<const uint16_t *>(x),
                       int(m), y, int(tiles_n));
    return hipGetLastError();
}

template <int B, int XDT, int YDT, int BI, int BJ>
hipError_t slab_group(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    switch (w.group) {
        case 32: return slab_launch<B, 1, XDT, YDT, BI, BJ>(w, x, m, y, stream);
        case 64: return slab_launch<B, 2, XDT, YDT, BI, BJ>(w, x, m, y, stream);
        case 128: return slab_launch<B, 4, XDT, YDT, BI, BJ>(w, x, m, y, stream);
        case 256: return slab_launch<B, 8, XDT, YDT, BI, BJ>(w, x, m, y, stream);
        case 512: return slab_launch<B, 16, XDT, YDT, BI, BJ>(w, x, m, y, stream);
    }
    return hipErrorNotSupported;
}

template <int XDT, int YDT, int BI, int BJ>
hipError_t slab_bits(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    switch (w.bits) {
        case 1: return slab_group<1, XDT, YDT, BI, BJ>(w, x, m, y, stream);
        case 2: return slab_group<2, XDT, YDT, BI, BJ>(w, x, m, y, stream);
        case 3: return slab_group<3, XDT, YDT, BI, BJ>(w, x, m, y, stream);
        case 4: return slab_group<4, XDT, YDT, BI, BJ>(w, x, m, y, stream);
        case 5: return slab_group<5, XDT, YDT, BI, BJ>(w, x, m, y, stream);
    }
    return hipErrorNotSupported;
}


// staged variant: groups of at most 128 codes with at most 256 code bytes per
// row and sweep (larger ones spill registers in the unrolled sweep loop)
template <int B, int UPG, int XDT, int YDT, bool XT, int XB = 1>
hipError_t slab_st_launch_x(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    constexpr int NE = 1 << B;
    constexpr uint32_t kTab = NE * 256u;
    constexpr uint32_t CS = 4 * (32 * UPG) * B / 8 + 16;
    constexpr uint32_t kStage = 16u * CS + 2u * 16u * 4u * 16u + (XT ? XB * 64u * 80u : 0u);
    const int64_t tiles_n = (w.n + 15) / 16;
    const int64_t tiles = (m + 16 * XB - 1) / (16 * XB) * tiles_n;
    if (tiles > 0x7fffffff) return hipErrorInvalidValue;
    const int64_t nsw = w.k / w.group / 4;
    // waves per workgroup: about 8 waves per compute unit over the grid,
    // rounded up with up to 4 rows and down above (two x-row blocks: about
    // 4), then down to a power of two, so that each wave walks a longer run
    // of sweeps than with 16 per compute unit (measured, W4 G128, K x N:
    // 4096 x 28672 and 8192 x 28672 at 8-16 rows 7-15% faster with one wave
    // instead of two, at 2-4 rows keeping two; 14336 x 4096 at 2-8 rows 8-18%
    // faster with 8 instead of 16; 8192 x 8192 at 2-4 rows 25-30% faster
    // with 4 instead of 8; 4096 x 14336 at 2-4 rows 2 better than 3 or 4;
    // two blocks at 24-32 rows: 8192 x 28672 and 4096 x 28672 16-17% faster
    // with one wave instead of two, 14336 x 4096 10-16% with 4 instead of 8,
    // 4096 x 6144 21-26% with 2 instead of 7, 8192 x 8192 5-9% with 2
    // instead of 7)
    const int64_t cus = device_cu_count();
    int64_t s = XB == 2 ? cus * 4 / tiles : m <= 4 ? (cus * 8 + tiles - 1) / tiles : cus * 8 / tiles;
    while (s & (s - 1)) s &= s - 1;
    if (s > (XT ? 8 : 16)) s = XT ? 8 : 16;  // the kernel's launch bound
    if (s > nsw) s = nsw;
    // LDS: tables below 64 KB, whole workgroup within 128 KB
    while (s > 1 && (s * kTab > 65536 || s * (kTab + kStage) > 131072)) --s;
    if (s < 1) s = 1;
    const size_t lds = size_t(s) * (kTab + kStage) > size_t(s) * 1024 * XB ? size_t(s) * (kTab + kStage)
                                                                           : size_t(s) * 1024 * XB;
    hipLaunchKernelGGL((gemm_a16_slab_st<B, UPG, XDT, YDT, false, XT, XB>), dim3(unsigned(tiles)),
                       dim3(unsigned(64 * s)), lds, stream, w.codes, w.scale, w.a, w.b, int(w.n), int(w.k),
                       static_cast<const uint16_t *>(x), int(m), y, int(tiles_n), nullptr, nullptr, nullptr);
    return hipGetLastError();
}

// more than 8 rows: activations through the transposing LDS pieces (they
// cost a wave per SIMD of occupancy, which 5..8 rows do not win back); more
// than 16: two x-row blocks per wave share every decoded weight operand
template <int B, int UPG, int XDT, int YDT>
hipError_t slab_st_launch(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    if (m > 16) return slab_st_launch_x<B, UPG, XDT, YDT, true, 2>(w, x, m, y, stream);
    if (m > 8) return slab_st_launch_x<B, UPG, XDT, YDT, true>(w, x, m, y, stream);
    return slab_st_launch_x<B, UPG, XDT, YDT, false>(w, x, m, y, stream);
}

// routed: one workgroup per (expert, 16 weight rows); route chunks of 16
template <int B, int UPG, int XDT, int YDT, bool XT>
hipError_t slab_st_routed_launch_x(const cq_weight &w, int n_experts, const void *x, int64_t tokens,
                                   const int32_t *token, const int32_t *order, const int32_t *offsets, void *y,
                                   hipStream_t stream) {
    constexpr int NE = 1 << B;
    constexpr uint32_t kTab = NE * 256u;
    constexpr uint32_t CS = 4 * (32 * UPG) * B / 8 + 16;
    constexpr uint32_t kStage = 16u * CS + 2u * 16u * 4u * 16u + (XT ? 64u * 80u : 0u);
    const int64_t tiles_n = (w.n + 15) / 16;
    const int64_t blocks = tiles_n * n_experts;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    const int64_t nsw = w.k / w.group / 4;
    int64_t s = int64_t(device_cu_count()) * 16 / blocks;
    if (s > 8) s = 8;  // the routed kernel's launch bound
    if (s > nsw) s = nsw;
    while (s > 1 && (s * kTab > 65536 || s * (kTab + kStage) > 131072)) --s;
    if (s < 1) s = 1;
    const size_t lds = size_t(s) * (kTab + kStage) > size_t(s) * 1024 ? size_t(s) * (kTab + kStage) : size_t(s) * 1024;
    hipLaunchKernelGGL((gemm_a16_slab_st<B, UPG, XDT, YDT, true, XT, 1>), dim3(unsigned(blocks)),
                       dim3(unsigned(64 * s)), lds, stream, w.codes, w.scale, w.a, w.b, int(w.n), int(w.k),
                       static_cast<const uint16_t *>(x), int(tokens), y, int(tiles_n), token, order, offsets);
    return hipGetLastError();
}

// more than 8 routes per expert on average: the transposing activation pieces
template <int B, int UPG, int XDT, int YDT>
hipError_t slab_st_routed_launch(const cq_weight &w, int n_experts, const void *x, int64_t tokens, int64_t routes,
                                 const int32_t *token, const int32_t *order, const int32_t *offsets, void *y,
                                 hipStream_t stream) {
    if (routes > 8 * int64_t(n_experts))
        return slab_st_routed_launch_x<B, UPG, XDT, YDT, true>(w, n_experts, x, tokens, token, order, offsets, y, stream);
    return slab_st_routed_launch_x<B, UPG, XDT, YDT, false>(w, n_experts, x, tokens, token, order, offsets, y, stream);
}

template <int B, int XDT, int YDT>
hipError_t slab_st_group(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    switch (w.group) {
        case 32: return slab_st_launch<B, 1, XDT, YDT>(w, x, m, y, stream);
        case 64: return slab_st_launch<B, 2, XDT, YDT>(w, x, m, y, stream);
        case 128:
            if constexpr (B <= 4) return slab_st_launch<B, 4, XDT, YDT>(w, x, m, y, stream);
            break;
    }
    return hipErrorNotSupported;
}

template <int B, int XDT, int YDT>
hipError_t slab_st_routed_group(const cq_weight &w, int n_experts, const void *x, int64_t tokens, int64_t routes,
                                const int32_t *token, const int32_t *order, const int32_t *offsets, void *y,
                                hipStream_t stream) {
    switch (w.group) {
        case 32: return slab_st_routed_launch<B, 1, XDT, YDT>(w, n_experts, x, tokens, routes, token, order, offsets, y, stream);
        case 64: return slab_st_routed_launch<B, 2, XDT, YDT>(w, n_experts, x, tokens, routes, token, order, offsets, y, stream);
        case 128:
            if constexpr (B <= 4)
                return slab_st_routed_launch<B, 4, XDT, YDT>(w, n_experts, x, tokens, routes, token, order, offsets, y, stream);
            break;
    }
    return hipErrorNotSupported;
}

template <int XDT, int YDT>
hipError_t slab_st_routed_bits(const cq_weight &w, int n_experts, const void *x, int64_t tokens, int64_t routes,
                               const int32_t *token, const int32_t *order, const int32_t *offsets, void *y,
                               hipStream_t stream) {
    switch (w.bits) {
        case 1: return slab_st_routed_group<1, XDT, YDT>(w, n_experts, x, tokens, routes, token, order, offsets, y, stream);
        case 2: return slab_st_routed_group<2, XDT, YDT>(w, n_experts, x, tokens, routes, token, order, offsets, y, stream);
        case 3: return slab_st_routed_group<3, XDT, YDT>(w, n_experts, x, tokens, routes, token, order, offsets, y, stream);
        case 4: return slab_st_routed_group<4, XDT, YDT>(w, n_experts, x, tokens, routes, token, order, offsets, y, stream);
        case 5: return slab_st_routed_group<5, XDT, YDT>(w, n_experts, x, tokens, routes, token, order, offsets, y, stream);
    }
    return hipErrorNotSupported;
}

template <int XDT, int YDT>
hipError_t slab_st_bits(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    switch (w.bits) {
        case 1: return slab_st_group<1, XDT, YDT>(w, x, m, y, stream);
        case 2: return slab_st_group<2, XDT, YDT>(w, x, m, y, stream);
        case 3: return slab_st_group<3, XDT, YDT>(w, x, m, y, stream);
        case 4: return slab_st_group<4, XDT, YDT>(w, x, m, y, stream);
        case 5: return slab_st_group<5, XDT, YDT>(w, x, m, y, stream);
    }
    return hipErrorNotSupported;
}

// every width, group and dtype pair of one (x-row blocks, weight-row blocks) shape
template <int BI, int BJ>
hipError_t slab_dtypes(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                       hipStream_t stream) {
    if (x_dt == 0) {
        if (y_dt == 0) return slab_bits<0, 0, BI, BJ>(w, x, m, y, stream);
        return slab_bits<0, 2, BI, BJ>(w, x, m, y, stream);
    }
    if (y_dt == 1) return slab_bits<1, 1, BI, BJ>(w, x, m, y, stream);
    return slab_bits<1, 2, BI, BJ>(w, x, m, y, stream);
}

}  // namespace a16_slab

// one file per shape: 16 rows of x with 16 or 32 weight rows per wave, and
// 32 rows of x with 16
hipError_t launch_a16_slab_1x1(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                               hipStream_t stream);
hipError_t launch_a16_slab_1x2(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                               hipStream_t stream);
hipError_t launch_a16_slab_2x1(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                               hipStream_t stream);
// the staged variant (m <= 32, G <= 128, G B <= 512, a multiple of four groups per row)
bool a16_slab_st_fits(const cq_weight &w, int64_t m);
hipError_t launch_a16_slab_st(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                              hipStream_t stream);

}  // namespace cq
