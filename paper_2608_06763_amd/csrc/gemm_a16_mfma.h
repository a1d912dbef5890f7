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
// allows it.  FP16 activations always use one FP16 operand.  Folding s_g
// into the reconstructed operand is a regrouping of the group sum: no
// per-group rescale is needed and accumulation runs across groups in the MFMA.
//
// Tiling.  A workgroup owns a TM x TN tile of y (rows of x by rows of W);
// each of its waves owns a block of 16 x 16 MFMA tiles of it and issues
// v_mfma_f32_16x16x32_{bf16,f16}.  Many rows of x take 256 x 128 tiles (8
// waves of 64 x 64), so every decoded weight feeds 256 rows; few rows take
// tiles of 128, 64 or 32 rows, so no matrix work is spent on absent rows and
// the narrower weight tiles of the shorter ones put more workgroups on the
// chip.  K advances one 32-code unit per step through two LDS buffers; while
// the matrix cores work on one, every thread decodes its codes of the next
// step into the other, so one barrier per step suffices.  Code words,
// activations and group metadata of a step are requested R steps ahead into
// one of R register slots (2 for the 256-row tile, whose steps are long; 8
// for the short tiles); loads complete in issue order, so activations
// requested later than the codes would make every step wait for all codes
// in flight.
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
#pragma once

#include "cq_device.h"
#include "cq_internal.h"
#include "stream_common.h"

#include <type_traits>

namespace cq {

namespace a16_mfma {

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

// f(integral_constant<P>) for P = P0 .. PN - 1, in order
template <int P0, int PN, typename F>
__device__ __forceinline__ void unroll_slots(F &&f) {
    if constexpr (P0 < PN) {
        f(std::integral_constant<int, P0>{});
        unroll_slots<P0 + 1, PN>(f);
    }
}

// Keep the vector-memory reads of successive ring slots in program order
// (the scheduler may move anything else across): the wait before a slot is
// used counts the loads issued after it, so a slot requested later must not
// be issued earlier.
__device__ __forceinline__ void vmem_order() { __builtin_amdgcn_sched_barrier(0x78f); }

__device__ __forceinline__ void lds_fence_wave() {
    // LDS operations of one wavefront complete in issue order; keeping the
    // compiler from reordering them is enough for the quad that shares a table.
    __asm__ __volatile__("" ::: "memory");
    __builtin_amdgcn_wave_barrier();
}

}  // namespace a16_mfma

// Tile configurations.  A workgroup of WM x WN waves owns a TM x TN tile of
// y (TM = 16 BI WM rows of x, TN = 16 BJ WN rows of W); every wave owns a
// (16 BI) x (16 BJ) block of it.  Q = threads / TN threads share a weight row
// and decode 32 / Q of its codes per step.  Code words are requested R steps
// ahead (R register slots): with few rows of x a step is short, and the
// weight stream needs many steps in flight to cover the memory latency.
template <int WM_, int WN_, int BI_, int BJ_, int R_>
struct a16_tile {
    static constexpr int WM = WM_, WN = WN_, BI = BI_, BJ = BJ_, R = R_;
    static constexpr int NT = 64 * WM * WN;
    static constexpr int TM = 16 * BI * WM, TN = 16 * BJ * WN;
};
// x-tile height 256 (many rows), 128, 64 and 32 (few rows)
using tile256 = a16_tile<4, 2, 4, 4, 2>;
using tile128 = a16_tile<2, 4, 4, 2, 8>;
using tile64 = a16_tile<1, 4, 4, 1, 8>;
using tile32 = a16_tile<1, 4, 2, 1, 8>;

using namespace a16_mfma;

template <int B, int UPG, int XDT, int YDT, bool ONE, class T>
__global__ void __launch_bounds__(T::NT) gemm_a16_mfma(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int n, int k, const uint16_t *__restrict__ x, int m, void *__restrict__ y, int tiles_m, int tiles_n) {
    constexpr int M = max_code(B);
    constexpr int WN = T::WN, BI = T::BI, BJ = T::BJ, R = T::R, NT = T::NT;
    constexpr int TM = T::TM, TN = T::TN;
    constexpr int Q = NT / TN;                // threads per weight row
    constexpr int CPT = kKS / Q;              // codes per thread per step
    constexpr int XPT = TM * kKS * 2 / NT;    // activation bytes per thread per step
    constexpr int XTR = kKS * 2 / XPT;        // threads per activation row
    constexpr int SPG = UPG;                  // steps (units) per group
    constexpr int NE = 1 << B;                // table entries (fields)
    constexpr int EPT = NE >= Q ? NE / Q : 1; // entries built per thread
    constexpr int TSTR = NE + 1;              // table words per row (padded)
    constexpr bool SPLIT = (XDT == 0) && !ONE;
    static_assert(NT % TN == 0 && Q == 4, "four threads per weight row");
    static_assert(XPT % 4 == 0 && XPT <= 32 && XTR * XPT == kKS * 2, "activation loader shape");
    static_assert(R >= 2 && R % 2 == 0, "an even number of code slots");
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
    const int wm = (wave / WN) * (16 * BI);
    const int wn = (wave % WN) * (16 * BJ);

    const int ng = k / (32 * UPG);
    const uint32_t row_bytes = uint32_t(k) * B / 8u;
    const auto rc = make_rsrc(codes, uint32_t(n) * row_bytes);
    const auto rs = make_rsrc(scale, uint32_t(n) * ng * 4u);
    const auto ra = make_rsrc(a16, uint32_t(n) * ng * 2u);
    const auto rb = make_rsrc(b16, uint32_t(n) * ng * 2u);
    const auto rx = make_rsrc(x, uint32_t(m) * uint32_t(k) * 2u);

    // loader roles
    const int lr = tid / Q;                  // weight row of the tile
    const int lq = tid % Q;                  // which CPT-code part of the unit
    const int wrow = n0 + lr;
    const bool wok = wrow < n;
    const int xr = tid / XTR;                // activation row of the tile
    const int xc = (tid % XTR) * (XPT / 2);  // first K element of this thread
    const int xrow = m0 + xr;
    const bool xok = xrow < m;

    // Ring of R register slots, one per step: the step's code words, its
    // activations and, for a step that may start a group, the group's
    // metadata.  Every load is unconditional (indices past the last step
    // repeat it), so the loads of a step are waited for only when that step
    // is decoded, R - 1 steps after they were issued.
    constexpr int MSTEP = SPG < R ? SPG : R;  // slots whose step can start a group
    // A thread's 8 codes are the 8B bits at bit 8B lq of the unit (4B bytes).
    // It loads the aligned 8-byte window of the unit that holds them (the
    // whole unit for W1) and shifts them down by cs bits, so every field then
    // sits at a compile-time position.
    constexpr int CW = B == 1 ? 1 : 2;        // words per thread and step
    const uint32_t wbyte = B == 1 ? 0u : uint32_t(min((B * lq) & ~3, 4 * B - 8));
    const uint32_t cs = uint32_t(8 * B * lq) - 8u * wbyte;
    uint32_t cw[R][CW];
    uint32_t xw[R][XPT / 4];
    float sv[R];
    uint32_t av[R], bv[R];

    auto load_slot = [&](int st, auto slot_c) {
        constexpr int SL = decltype(slot_c)::value;
        load_words<CW>(rc, wok ? uint32_t(wrow) * row_bytes + uint32_t(st) * (4u * B) + wbyte : kOobOffset, cw[SL]);
        if constexpr (SL % MSTEP == 0) {
            const uint32_t gi = uint32_t(wrow) * ng + st / SPG;
            sv[SL] = load_f32(rs, wok ? gi * 4u : kOobOffset);
            av[SL] = load_u16(ra, wok ? gi * 2u : kOobOffset);
            bv[SL] = load_u16(rb, wok ? gi * 2u : kOobOffset);
        }
        const uint32_t off = xok ? (uint32_t(xrow) * uint32_t(k) + uint32_t(st) * kKS + xc) * 2u : kOobOffset;
        load_words<XPT / 4>(rx, off, xw[SL]);
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
            const int f = lq + Q * e;
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

    // decode the codes of slot SL into weight buffer `buf`, copy its activations
    auto store_step = [&](auto buf_c, auto slot_c) {
        constexpr int buf = decltype(buf_c)::value;
        constexpr int SL = decltype(slot_c)::value;
        uint64_t win;
        if constexpr (CW == 1) win = uint64_t(cw[SL][0] >> cs);
        else win = ((uint64_t(cw[SL][1]) << 32) | cw[SL][0]) >> cs;
        const uint32_t f0 = uint32_t(win), f1 = uint32_t(win >> 32);
        uint32_t ent[CPT];
#pragma unroll
        for (int e = 0; e < CPT; ++e) {
            const int bit = B * e;  // compile-time after unrolling
            uint32_t v;
            if (bit + B <= 32) v = f0 >> bit;
            else if (bit >= 32) v = f1 >> (bit - 32);
            else v = __builtin_amdgcn_alignbit(f1, f0, bit);
            ent[e] = tab[tbase + (v & uint32_t(NE - 1))];
        }
        uint32_t hi[CPT / 2], lo[CPT / 2];
#pragma unroll
        for (int p = 0; p < CPT / 2; ++p) {
            hi[p] = __builtin_amdgcn_perm(ent[2 * p + 1], ent[2 * p], 0x05040100u);
            lo[p] = __builtin_amdgcn_perm(ent[2 * p + 1], ent[2 * p], 0x07060302u);
        }
#pragma unroll
        for (int q = 0; q < CPT / 8; ++q) {
            *reinterpret_cast<u32x4 *>(&Bh[buf][lr * kRowB + 2 * CPT * lq + 16 * q]) =
                u32x4{hi[4 * q], hi[4 * q + 1], hi[4 * q + 2], hi[4 * q + 3]};
            if constexpr (SPLIT)
                *reinterpret_cast<u32x4 *>(&Bl[buf][lr * kRowB + 2 * CPT * lq + 16 * q]) =
                    u32x4{lo[4 * q], lo[4 * q + 1], lo[4 * q + 2], lo[4 * q + 3]};
        }
        uint8_t *ap = &As[buf][xr * kRowB + 2 * xc];
        const uint32_t *xs = xw[SL];
        if constexpr (XPT >= 16) {
#pragma unroll
            for (int q = 0; q < XPT / 16; ++q)
                *reinterpret_cast<u32x4 *>(ap + 16 * q) = u32x4{xs[4 * q], xs[4 * q + 1], xs[4 * q + 2], xs[4 * q + 3]};
        } else if constexpr (XPT == 8) {
            typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
            *reinterpret_cast<u32x2 *>(ap) = u32x2{xs[0], xs[1]};
        } else {
            *reinterpret_cast<uint32_t *>(ap) = xs[0];
        }
    };

    f32x4_t acc[BI][BJ];
#pragma unroll
    for (int i = 0; i < BI; ++i)
#pragma unroll
        for (int j = 0; j < BJ; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    using S0 = std::integral_constant<int, 0>;
    const int nsteps = k / kKS;
    // prologue: steps 0 .. R - 1 requested into their slots, step 0 decoded
    unroll_slots<0, R>([&](auto p_c) {
        constexpr int P = decltype(p_c)::value;
        load_slot(min(P, nsteps - 1), p_c);
        vmem_order();
    });
    build_table(S0{});
    store_step(S0{}, S0{});
    __syncthreads();

    // Step st works on LDS buffer st % 2.  Its slot st % R was decoded in the
    // previous step and now receives the request for step st + R; step st + 1
    // (slot (st + 1) % R) is decoded into the other buffer, with its row
    // tables rebuilt first when it starts a group.  The last period may run
    // steps past the end: they decode repeated data and skip the matrix work.
    auto do_step = [&](int st, auto p_c) {
        constexpr int P = decltype(p_c)::value;  // st % R
        constexpr int buf = P % 2;
        constexpr int SN = (P + 1) % R;           // slot of step st + 1
        load_slot(min(st + R, nsteps - 1), p_c);
        vmem_order();
        if (st < nsteps) {
            u32x4 af[BI], bh[BJ], bl[BJ];
#pragma unroll
            for (int i = 0; i < BI; ++i)
                af[i] = *reinterpret_cast<const u32x4 *>(&As[buf][(wm + 16 * i + (lane & 15)) * kRowB + 16 * (lane >> 4)]);
#pragma unroll
            for (int j = 0; j < BJ; ++j) {
                bh[j] = *reinterpret_cast<const u32x4 *>(&Bh[buf][(wn + 16 * j + (lane & 15)) * kRowB + 16 * (lane >> 4)]);
                if constexpr (SPLIT)
                    bl[j] = *reinterpret_cast<const u32x4 *>(&Bl[buf][(wn + 16 * j + (lane & 15)) * kRowB + 16 * (lane >> 4)]);
            }
#pragma unroll
            for (int i = 0; i < BI; ++i)
#pragma unroll
                for (int j = 0; j < BJ; ++j) {
                    acc[i][j] = mma<XDT>(af[i], bh[j], acc[i][j]);
                    if constexpr (SPLIT) acc[i][j] = mma<XDT>(af[i], bl[j], acc[i][j]);
                }
        }
        if constexpr (SPG <= R && R % SPG == 0) {
            if constexpr ((P + 1) % SPG == 0) build_table(std::integral_constant<int, SN>{});
        } else {
            if ((st + 1) % SPG == 0) build_table(std::integral_constant<int, SN>{});
        }
        store_step(std::integral_constant<int, 1 - buf>{}, std::integral_constant<int, SN>{});
        __syncthreads();
    };

    for (int st = 0; st < nsteps; st += R)
        unroll_slots<0, R>([&](auto p_c) {
            constexpr int P = decltype(p_c)::value;
            do_step(st + P, p_c);
        });

#pragma unroll
    for (int i = 0; i < BI; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int row = m0 + wm + 16 * i + 4 * (lane >> 4) + e;
            if (row >= m) continue;
#pragma unroll
            for (int j = 0; j < BJ; ++j) {
                const int col = n0 + wn + 16 * j + (lane & 15);
                if (col < n) store_out<YDT>(y, int64_t(row) * n + col, acc[i][j][e]);
            }
        }
}

template <int B, int UPG, int XDT, int YDT, bool ONE, class T>
static hipError_t a16_mfma_launch(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    const int64_t tiles_m = (m + T::TM - 1) / T::TM;
    const int64_t tiles_n = (w.n + T::TN - 1) / T::TN;
    const int64_t nwg = tiles_m * tiles_n;
    if (nwg > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemm_a16_mfma<B, UPG, XDT, YDT, ONE, T>), dim3(unsigned(nwg)), dim3(T::NT), 0, stream,
                       w.codes, w.scale, w.a, w.b, int(w.n), int(w.k), static_cast<const uint16_t *>(x), int(m), y,
                       int(tiles_m), int(tiles_n));
    return hipGetLastError();
}

template <int B, int XDT, int YDT, bool ONE, class T>
static hipError_t a16_mfma_group(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    switch (w.group) {
        case 32: return a16_mfma_launch<B, 1, XDT, YDT, ONE, T>(w, x, m, y, stream);
        case 64: return a16_mfma_launch<B, 2, XDT, YDT, ONE, T>(w, x, m, y, stream);
        case 128: return a16_mfma_launch<B, 4, XDT, YDT, ONE, T>(w, x, m, y, stream);
        case 256: return a16_mfma_launch<B, 8, XDT, YDT, ONE, T>(w, x, m, y, stream);
        case 512: return a16_mfma_launch<B, 16, XDT, YDT, ONE, T>(w, x, m, y, stream);
    }
    return hipErrorNotSupported;
}

template <int XDT, int YDT, bool ONE, class T>
static hipError_t a16_mfma_bits(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    switch (w.bits) {
        case 1: return a16_mfma_group<1, XDT, YDT, ONE, T>(w, x, m, y, stream);
        case 2: return a16_mfma_group<2, XDT, YDT, ONE, T>(w, x, m, y, stream);
        case 3: return a16_mfma_group<3, XDT, YDT, ONE, T>(w, x, m, y, stream);
        case 4: return a16_mfma_group<4, XDT, YDT, ONE, T>(w, x, m, y, stream);
        case 5: return a16_mfma_group<5, XDT, YDT, ONE, T>(w, x, m, y, stream);
    }
    return hipErrorNotSupported;
}

template <bool ONE, class T>
static hipError_t a16_mfma_dtypes(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                  hipStream_t stream) {
    if (x_dt == 0) {
        if (y_dt == 0) return a16_mfma_bits<0, 0, ONE, T>(w, x, m, y, stream);
        return a16_mfma_bits<0, 2, ONE, T>(w, x, m, y, stream);
    }
    // FP16 activations: one FP16 operand in every instantiation
    if (y_dt == 1) return a16_mfma_bits<1, 1, false, T>(w, x, m, y, stream);
    return a16_mfma_bits<1, 2, false, T>(w, x, m, y, stream);
}

// Launch of one tile configuration for every width, group and dtype pair
// (each configuration is instantiated in a file of its own).
hipError_t launch_a16_tile32(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt, bool one,
                             hipStream_t stream);
hipError_t launch_a16_tile64(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt, bool one,
                             hipStream_t stream);
hipError_t launch_a16_tile128(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt, bool one,
                              hipStream_t stream);
hipError_t launch_a16_tile256(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt, bool one,
                              hipStream_t stream);

}  // namespace cq
