// Dynamic-A8 many-row GEMM (Sec. 5.4) for W4 on gfx950 int8 matrix cores.
//
// Numerics are eq. a8-output: INT8 activations times exact INT8 weight
// carriers (eq. carrier) accumulate into exact INT32 group partials P_g
// (|P_g| <= G 127^2, eq. a8-int32-bound); at the end of every group each
// partial is converted to FP32 and multiplied by s_g, and the row factor
// d_x / 127 multiplies the FP32 sum.
//
// Tiling.  A workgroup of WM x WN waves owns a (64 WM) x (64 WN) tile of y
// (rows of x by rows of W; 256 x 128 on the fast path, so that every decoded
// carrier feeds 256 activation rows); each wave owns 64 x 64 and issues v_mfma_i32_16x16x64_i8
// on 16 x 16 blocks.  K advances in steps of 64 through two LDS buffers: while
// the matrix cores work on one buffer, every thread loads the next step's
// codes and activations, decodes its 32 codes to carriers and writes them to
// the other buffer, so one barrier per step suffices.  Codes and activations are
// requested two steps ahead into two register slots; a group's (a, b) and
// scales are requested a whole group ahead, right after the registers that
// hold them are consumed.  The step loop is unrolled over the positions of a
// group, so that slots, buffers and group boundaries are compile-time and
// each step is one basic block, in which scheduling hints spread the
// decode and rescale VALU work between the 16 MFMAs (the kernel is bound
// by VALU issue, not by the matrix cores).
//
// Decode.  The WM adjacent threads t of a quad (or half quad) serve weight row
// t / WM, each one 64 / WM codes of every step.  At the start of a group they
// each evaluate 8 / WM of the row's carriers (exact, see a8_carriers.h) and
// share them with DPP quad moves, which gives every one of them the two
// 8-byte W4 carrier tables of that (row, group); every code word then costs
// two byte-permute lookups and two permutes that restore field order.  The
// first MFMA of a group takes a zero accumulator, so partials need no clearing.
//
// MFMA operand layout (16x16x64 int8): lane l supplies row l % 16 of A and
// column l % 16 of B with K slots 16 (l / 16) .. +15; the INT32 result of a
// block has lane l holding rows 4 (l / 16) + i of column l % 16.
//
// Tile order: workgroups are first spread so that those on one XCD (blockIdx
// modulo 8) take consecutive tile indices; consecutive indices then walk the
// weight tiles of one activation tile, which stays in that XCD's L2 while the
// packed weights stream past it.
#include "cq_device.h"
#include "cq_internal.h"
#include "stream_common.h"
#include "a8_carriers.h"

#include <type_traits>

// the step bodies are large; every lambda of the kernel must be inlined so
// that register slots stay registers
#define CQ_INLINE __attribute__((always_inline))

namespace cq {

namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kKS = 64;                // K step
constexpr int kStride = kKS + 16;      // LDS bytes per tile row (padded)
constexpr int kBand = 1;               // row tiles per raster band

__device__ __forceinline__ void lds_store16(int8_t *p, const uint32_t *v) {
    *reinterpret_cast<u32x4 *>(p) = u32x4{v[0], v[1], v[2], v[3]};
}

// f(integral_constant<P>) for P = P0 .. PN - 1, in order
template <int P0, int PN, typename F>
__device__ __forceinline__ void unroll_positions(F &&f) {
    if constexpr (P0 < PN) {
        f(std::integral_constant<int, P0>{});
        unroll_positions<P0 + 1, PN>(f);
    }
}

// Scheduling hints for one step: the LDS fragment reads first, then each of
// the 16 MFMAs followed by R VALU instructions; the first VM of them also
// take one global load each.
template <int R, int VM>
__device__ __forceinline__ void interleave_step() {
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);  // DS reads
#pragma unroll
    for (int q = 0; q < 16; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, R, 0);  // VALU
        if (q < VM) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read
    }
}

}  // namespace

// B = 4 or 3.  TB: the carriers come from a load-time table (2^(B-1) bytes per
// (row, group), r(0) .. r(2^(B-1) - 1), which is the table TA itself) instead
// of being evaluated from (a, b); the schedule is unchanged.
//
// W3: a 3-bit field f indexes the 8-byte pair TA = [r0 r1 r2 r3], TB = [0 -r3
// -r2 -r1] (f = 4 is the reserved pattern, f = 5..7 are -3..-1) directly, so
// one byte permute serves four fields once they are spread into bytes.  The
// 16 codes of a thread per step are 6 bytes, read from an aligned 8-byte
// window; every thread evaluates the two interior carriers itself.
template <int B, int WM, int WN, int UPG, int YDT, bool DUMP, bool TB>
__global__ void __launch_bounds__(64 * WM * WN) gemm_a8_mfma(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int n, int k, const int8_t *__restrict__ x8, const float *__restrict__ dx, int m,
    void *__restrict__ y, int32_t *__restrict__ partials, int tiles_m, int tiles_n,
    const int8_t *__restrict__ ctab) {
    constexpr int M = max_code(B);
    constexpr int TM = 64 * WM;             // rows of x per tile
    constexpr int TN = 64 * WN;             // rows of W per tile
    constexpr int NT = 64 * WM * WN;        // threads
    constexpr int G = 32 * UPG;
    constexpr int SPG = G / kKS;            // K steps per group
    constexpr int CPT = kKS / WM;           // codes per thread per step (16 or 32)
    constexpr int XB = kKS / WN * 1;        // activation bytes per thread per step (32 or 16)
    constexpr int Q = WM;                   // threads sharing a weight row (2 or 4)
    constexpr int NP = 4 / Q;               // carrier pairs evaluated per thread
    static_assert(SPG >= 1 && G % kKS == 0, "group must be a multiple of the K step");
    static_assert(Q == 2 || Q == 4, "two or four threads per weight row");
    static_assert(B == 4 || (B == 3 && Q == 4), "W3 takes four threads per weight row");
    // code words of step s are requested kCodeSlots steps ahead into slot
    // s % kCodeSlots (they stream from HBM); with G < 256 the deeper ring
    // would need a longer unrolled period than the registers allow
    constexpr int kCodeSlots = SPG >= 4 ? 4 : 2;
    __shared__ __attribute__((aligned(16))) int8_t As[2][TM * kStride];
    __shared__ __attribute__((aligned(16))) int8_t Bs[2][TN * kStride];

    // ---- tile of this workgroup
    const int nwg = tiles_m * tiles_n;
    int wg = blockIdx.x;
    if (nwg % 8 == 0) wg = (wg % 8) * (nwg / 8) + wg / 8;
    const int band = wg / (kBand * tiles_n);
    const int first_m = band * kBand;
    const int band_rows = min(kBand, tiles_m - first_m);
    const int in_band = wg - band * kBand * tiles_n;
    const int m0 = (first_m + in_band % band_rows) * TM;
    const int n0 = (in_band / band_rows) * TN;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = (wave / WN) * 64;
    const int wn = (wave % WN) * 64;

    const int ng = k / G;
    const uint32_t row_bytes = uint32_t(k) * B / 8u;
    const auto rc = make_rsrc(codes, uint32_t(n) * row_bytes);
    const auto rs = make_rsrc(scale, uint32_t(n) * ng * 4u);
    const auto ra = make_rsrc(a16, uint32_t(n) * ng * 2u);
    const auto rb = make_rsrc(b16, uint32_t(n) * ng * 2u);
    const auto rt = make_rsrc(ctab, TB ? uint32_t(n) * ng * (1u << (B - 1)) : 0u);
    const auto rx = make_rsrc(x8, uint32_t(m) * uint32_t(k));

    // loader roles: Q adjacent threads (one quad or half quad) share a weight row
    const int lr = tid / Q;                  // weight row of the tile
    const int lq = tid % Q;                  // which CPT-code part of the step
    const int wrow = n0 + lr;
    const bool wok = wrow < n;
    const int xr = tid / (kKS / XB);         // activation row of the tile
    const int xc = (tid % (kKS / XB)) * XB;  // byte offset inside the step
    const int xrow = m0 + xr;
    const bool xok = xrow < m;

    // carrier pairs this thread evaluates: pair p covers magnitudes 2p, 2p + 1
    float tp0[NP], tp1[NP];
    int ip0[NP];
#pragma unroll
    for (int j = 0; j < NP; ++j) {
        ip0[j] = 2 * (lq + Q * j);
        tp0[j] = float(ip0[j]) / float(M);
        tp1[j] = float(ip0[j] + 1) / float(M);
    }

    // Register slots: the code words of step s go to slot s % kCodeSlots and
    // its activation bytes to slot s % 2, requested kCodeSlots or two steps
    // before step s - 1 writes them to LDS.
    uint32_t cw[kCodeSlots][CPT / 8];
    uint32_t xw[2][XB / 4];
    uint32_t av = 0, bv = 0;  // (a, b) of the next group's row (FP16 bits)
    float sj[4];              // group scales of this lane's four output columns

    auto load_codes = [&](int st, auto slot_c) CQ_INLINE {
        constexpr int SL = decltype(slot_c)::value;
        const uint32_t kk = uint32_t(st) * kKS;
        if constexpr (B == 4) {
            load_words<CPT / 8>(rc, wok ? uint32_t(wrow) * row_bytes + (kk + uint32_t(CPT * lq)) / 2u : kOobOffset,
                                cw[SL]);
        } else {
            // the 6 code bytes of this thread inside an aligned 8-byte window
            const uint32_t off = uint32_t(st) * (kKS * 3 / 8) + ((6u * uint32_t(lq)) & ~3u);
            load_words<2>(rc, wok ? uint32_t(wrow) * row_bytes + off : kOobOffset, cw[SL]);
        }
    };
    auto load_acts = [&](int st, auto slot_c) CQ_INLINE {
        constexpr int SL = decltype(slot_c)::value;
        const uint32_t kk = uint32_t(st) * kKS;
        load_words<XB / 4>(rx, xok ? uint32_t(xrow) * uint32_t(k) + kk + uint32_t(xc) : kOobOffset, xw[SL]);
    };
    auto load_ab = [&](int g) CQ_INLINE {
        const uint32_t gi = uint32_t(wrow) * ng + g;
        if constexpr (TB && B == 4) {
            uint32_t t[2];
            load_words<2>(rt, wok ? gi * 8u : kOobOffset, t);
            av = t[0];  // r0 r1 r2 r3
            bv = t[1];  // r4 r5 r6 r7
        } else if constexpr (TB) {
            av = __builtin_amdgcn_raw_buffer_load_b32(rt, wok ? gi * 4u : kOobOffset, 0, 0);  // r0 r1 r2 r3
        } else {
            av = load_u16(ra, wok ? gi * 2u : kOobOffset);
            bv = load_u16(rb, wok ? gi * 2u : kOobOffset);
        }
    };
    auto load_scales = [&](int g) CQ_INLINE {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = n0 + wn + 16 * j + (lane & 15);
            sj[j] = load_f32(rs, col < n && g < ng ? (uint32_t(col) * ng + g) * 4u : kOobOffset);
        }
    };

    // Carriers of a group: each thread evaluates NP pairs (exact; the rare
    // near-tie fallback is a branch, kept at the end of a step); the tables
    // are assembled from them by DPP quad moves, branch-free, when needed.
    uint32_t pr[NP];
    uint32_t tw0 = 0, tw1 = 0;  // TB: the table words of the group whose tables come next
    auto eval_carriers = [&]() CQ_INLINE {
        if constexpr (TB) {
            tw0 = av;
            tw1 = bv;
            return;
        }
        const float a = f16_to_f32(uint16_t(av));
        const float b = f16_to_f32(uint16_t(bv));
        const float c = 1.f - a - b;
        const float mg = carrier_margin(a, b, c);
        if constexpr (B == 3) {
            // r1, r2 (r0 = 0, r3 = 127)
            pr[0] = carrier_u8<M>(1, 1.f / 3.f, a, b, c, mg) | (carrier_u8<M>(2, 2.f / 3.f, a, b, c, mg) << 8);
            return;
        }
#pragma unroll
        for (int j = 0; j < NP; ++j)
            pr[j] = carrier_u8<M>(ip0[j], tp0[j], a, b, c, mg) | (carrier_u8<M>(ip0[j] + 1, tp1[j], a, b, c, mg) << 8);
    };
    uint32_t ta0 = 0, ta1 = 0, tb0 = 0, tb1 = 0;
    auto build_tables = [&]() CQ_INLINE {
        if constexpr (B == 3) {
            ta0 = TB ? tw0 : ((pr[0] << 8) | 0x7f000000u);  // r0 r1 r2 r3
            const uint32_t neg = (0x80808080u - ta0) ^ 0x80808080u;  // 0 -r1 -r2 -r3
            tb0 = perm(neg, neg, 0x01020300u);                      // 0 -r3 -r2 -r1
            return;
        }
        if constexpr (TB) {
            ta0 = tw0;
            ta1 = tw1;
            w4_negative_table(ta0, ta1, tb0, tb1);
            return;
        }
        uint32_t P[4];
        if constexpr (Q == 4) {
            P[0] = quad_bcast<0x00>(pr[0]);
            P[1] = quad_bcast<0x55>(pr[0]);
            P[2] = quad_bcast<0xaa>(pr[0]);
            P[3] = quad_bcast<0xff>(pr[0]);
        } else {
            P[0] = quad_bcast<0xa0>(pr[0]);
            P[1] = quad_bcast<0xf5>(pr[0]);
            P[2] = quad_bcast<0xa0>(pr[1]);
            P[3] = quad_bcast<0xf5>(pr[1]);
        }
        ta0 = P[0] | (P[1] << 16);  // r0 r1 r2 r3
        ta1 = P[2] | (P[3] << 16);  // r4 r5 r6 r7
        w4_negative_table(ta0, ta1, tb0, tb1);
    };

    // Activation bytes of a step go to LDS unchanged; code words are decoded
    // to carriers first.
    auto store_acts = [&](int buf, auto slot_c) CQ_INLINE {
        constexpr int SL = decltype(slot_c)::value;
        int8_t *ap = &As[buf][xr * kStride + xc];
#pragma unroll
        for (int q = 0; q < XB / 16; ++q) lds_store16(ap + 16 * q, xw[SL] + 4 * q);
    };
    auto store_codes = [&](int buf, auto slot_c) CQ_INLINE {
        constexpr int SL = decltype(slot_c)::value;
        uint32_t cr[CPT / 4];
        if constexpr (B == 4) {
#pragma unroll
            for (int i = 0; i < CPT / 8; ++i) w4_word_carriers(cw[SL][i], ta0, ta1, tb0, tb1, cr[2 * i], cr[2 * i + 1]);
        } else {
            const uint64_t win = ((uint64_t(cw[SL][1]) << 32) | cw[SL][0]) >> (8u * ((6u * uint32_t(lq)) & 3u));
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t x = uint32_t(win >> (12 * q)) & 0xfffu;  // four 3-bit fields
                const uint32_t sel = (x & 7u) | ((x << 5) & 0x700u) | ((x << 10) & 0x70000u) | ((x << 15) & 0x7000000u);
                cr[q] = perm(tb0, ta0, sel);
            }
        }
        int8_t *bp = &Bs[buf][lr * kStride + CPT * lq];
#pragma unroll
        for (int q = 0; q < CPT / 16; ++q) lds_store16(bp + 16 * q, cr + 4 * q);
    };

    i32x4 acc[4][4];
    float accf[4][4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) accf[i][j][e] = 0.f;

    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    const int nsteps = k / kKS;
    unroll_positions<0, kCodeSlots>([&](auto p_c) CQ_INLINE {
        constexpr int P = decltype(p_c)::value;
        load_codes(min(P, nsteps - 1), p_c);
    });
    load_acts(0, S0{});
    load_acts(min(1, nsteps - 1), S1{});
    load_ab(0);
    load_scales(0);
    eval_carriers();
    build_tables();
    // carriers of the group that starts at step 1 (G = 64 only: later group
    // starts are evaluated two steps ahead inside the loop)
    load_ab(min(1, ng - 1));
    if constexpr (SPG == 1) {
        eval_carriers();
        load_ab(min(2, ng - 1));
    }
    store_acts(0, S0{});
    store_codes(0, S0{});
    __syncthreads();

    // One K step at position P of the unrolled period: matrix work on LDS
    // buffer P % 2 (step st); step st + 1 goes to the other buffer (its
    // activations first, then its decoded codes); the slots step st came
    // from receive the requests for steps st + kCodeSlots (codes) and
    // st + 2 (activations).  At the last step of a group the next group's
    // tables are assembled (its first step is decoded now), the partials are
    // rescaled and the next group's scales requested.  Two steps before a
    // group starts, its carriers are evaluated at the end of the step, and
    // the (a, b) of the group after it requested.  Requests past the last
    // step or group repeat the last one (in bounds; their data is unused).
    // The last period may be partial (G < 256); its missing steps are skipped.
    constexpr int PER = SPG >= kCodeSlots ? SPG : kCodeSlots;  // steps per period
    auto do_step = [&](int st, auto p_c) CQ_INLINE {
        constexpr int P = decltype(p_c)::value;
        constexpr int BUF = P % 2;
        constexpr bool kFirst = P % SPG == 0;
        constexpr bool kLast = P % SPG == SPG - 1;
        load_codes(min(st + kCodeSlots, nsteps - 1), std::integral_constant<int, P % kCodeSlots>{});
        load_acts(min(st + 2, nsteps - 1), std::integral_constant<int, BUF>{});
        i32x4 af[4], bf[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            af[i] = *reinterpret_cast<const i32x4 *>(&As[BUF][(wm + 16 * i + (lane & 15)) * kStride + 16 * (lane >> 4)]);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            bf[j] = *reinterpret_cast<const i32x4 *>(&Bs[BUF][(wn + 16 * j + (lane & 15)) * kStride + 16 * (lane >> 4)]);
        // LDS writes are several times slower than reads: the activations of
        // step st + 1 need no decode and go out before the matrix work
        store_acts(BUF ^ 1, std::integral_constant<int, BUF ^ 1>{});
        if constexpr (kFirst) {
            // first step of a group: the partials start from zero
            const i32x4 zero = {0, 0, 0, 0};
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[i], bf[j], zero, 0, 0, 0);
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[i], bf[j], acc[i][j], 0, 0, 0);
        }
        const int g = st / SPG;
        if constexpr (kLast) build_tables();  // group g + 1
        store_codes(BUF ^ 1, std::integral_constant<int, (P + 1) % kCodeSlots>{});
        if constexpr (kLast) {
            // group complete: FP32 rescale of the exact partials
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
            load_scales(g + 1);  // reads zero past the last group
        }
        if constexpr (!DUMP) interleave_step<3, 4>();
        if constexpr ((P + 2) % SPG == 0) {
            // the group starting at step st + 2
            const int gn = (st + 2) / SPG;
            eval_carriers();
            load_ab(min(gn + 1, ng - 1));
        }
        __syncthreads();
    };

    static_assert(PER % kCodeSlots == 0 && PER % SPG == 0 && PER % 2 == 0, "period must hold whole slots");
    for (int st = 0; st < nsteps; st += PER)
        unroll_positions<0, PER>([&](auto p_c) CQ_INLINE {
            if (p_c == 0 || st + p_c < nsteps) do_step(st + p_c, p_c);
        });

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

template <int B, int WM, int WN, int UPG, int YDT, bool DUMP, bool TB>
static hipError_t a8_mfma_launch(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                                 int32_t *partials, const int8_t *ctab, hipStream_t stream) {
    const int tiles_m = int((m + 64 * WM - 1) / (64 * WM));
    const int tiles_n = int((w.n + 64 * WN - 1) / (64 * WN));
    const int64_t nwg = int64_t(tiles_m) * tiles_n;
    if (nwg > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemm_a8_mfma<B, WM, WN, UPG, YDT, DUMP, TB>), dim3(unsigned(nwg)), dim3(64 * WM * WN), 0, stream,
                       w.codes, w.scale, w.a, w.b, int(w.n), int(w.k), x8, dx, int(m), y, partials, tiles_m, tiles_n,
                       ctab);
    return hipGetLastError();
}

template <int B, int YDT, bool TB>
static hipError_t a8_mfma_group(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                                int32_t *partials, const int8_t *ctab, hipStream_t stream) {
    // The partials dump (a test path) runs four waves per workgroup, which
    // leaves room for its extra registers; the fast path runs eight.
    if (partials) {
        if constexpr (B != 4) {
            return hipErrorNotSupported;  // W3 partials: the 64x64 kernel
        } else {
        switch (w.group) {
            case 64: return a8_mfma_launch<B, 2, 2, 2, YDT, true, TB>(w, x8, dx, m, y, partials, ctab, stream);
            case 128: return a8_mfma_launch<B, 2, 2, 4, YDT, true, TB>(w, x8, dx, m, y, partials, ctab, stream);
            case 256: return a8_mfma_launch<B, 2, 2, 8, YDT, true, TB>(w, x8, dx, m, y, partials, ctab, stream);
            case 512: return a8_mfma_launch<B, 2, 2, 16, YDT, true, TB>(w, x8, dx, m, y, partials, ctab, stream);
        }
        return hipErrorNotSupported;
        }
    }
    switch (w.group) {
        case 64: return a8_mfma_launch<B, 4, 2, 2, YDT, false, TB>(w, x8, dx, m, y, partials, ctab, stream);
        case 128: return a8_mfma_launch<B, 4, 2, 4, YDT, false, TB>(w, x8, dx, m, y, partials, ctab, stream);
        case 256: return a8_mfma_launch<B, 4, 2, 8, YDT, false, TB>(w, x8, dx, m, y, partials, ctab, stream);
        case 512: return a8_mfma_launch<B, 4, 2, 16, YDT, false, TB>(w, x8, dx, m, y, partials, ctab, stream);
    }
    return hipErrorNotSupported;
}

bool gemm_a8_mfma_supported(const cq_weight &w, int64_t m) {
    const int64_t lim = int64_t(1) << 31;
    return (w.bits == 4 || w.bits == 3) && w.group >= 64 && m * w.k < lim &&
           stream_fits(w.n, w.k, w.bits, w.group) && w.n < lim && m < lim;
}

template <bool TB>
static hipError_t a8_mfma_dispatch(const cq_weight &w, const int8_t *ctab, const int8_t *x8, const float *dx,
                                   int64_t m, void *y, int y_dt, int32_t *partials, hipStream_t stream) {
    if (w.bits == 3) {
        if (y_dt == 0) return a8_mfma_group<3, 0, TB>(w, x8, dx, m, y, partials, ctab, stream);
        if (y_dt == 1) return a8_mfma_group<3, 1, TB>(w, x8, dx, m, y, partials, ctab, stream);
        return a8_mfma_group<3, 2, TB>(w, x8, dx, m, y, partials, ctab, stream);
    }
    if (y_dt == 0) return a8_mfma_group<4, 0, TB>(w, x8, dx, m, y, partials, ctab, stream);
    if (y_dt == 1) return a8_mfma_group<4, 1, TB>(w, x8, dx, m, y, partials, ctab, stream);
    return a8_mfma_group<4, 2, TB>(w, x8, dx, m, y, partials, ctab, stream);
}

// x-tile height for m rows when the caller does not name one: the smallest
// of 32, 64, 128 that holds m (gemm_a8_tile.hip), else 256 (this file)
static int a8_mfma_tile_rows(int64_t m) { return m <= 32 ? 32 : m <= 64 ? 64 : m <= 128 ? 128 : 256; }

hipError_t launch_gemm_a8_mfma(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y, int y_dt,
                               int32_t *partials, int tile_rows, hipStream_t stream) {
    // the partials dump is written by the 256-row kernel's four-wave variant
    const int tr = partials ? 256 : (tile_rows ? tile_rows : a8_mfma_tile_rows(m));
    if (tr != 256) return launch_gemm_a8_tile(w, nullptr, x8, dx, m, y, y_dt, tr, stream);
    return a8_mfma_dispatch<false>(w, nullptr, x8, dx, m, y, y_dt, partials, stream);
}

hipError_t launch_gemm_a8_mfma_tab(const cq_weight &w, const int8_t *ctab, const int8_t *x8, const float *dx,
                                   int64_t m, void *y, int y_dt, hipStream_t stream) {
    const int tr = a8_mfma_tile_rows(m);
    if (tr != 256) return launch_gemm_a8_tile(w, ctab, x8, dx, m, y, y_dt, tr, stream);
    return a8_mfma_dispatch<true>(w, ctab, x8, dx, m, y, y_dt, nullptr, stream);
}

}  // namespace cq
