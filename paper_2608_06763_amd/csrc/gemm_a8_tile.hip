// Dynamic-A8 tiled GEMM for moderate row counts (m <= 128) on gfx950 int8
// matrix cores, W3 and W4 (Sec. 5.4; the regime between the single-row GEMV
// and the many-row GEMM of Sec. 5.5).
//
// Numerics are those of gemm_a8_mfma.hip (eq. a8-output): exact INT8
// carriers (eq. carrier) times INT8 activations accumulate into exact INT32
// group partials (eq. a8-int32-bound), each rescaled by s_g in FP32 at the
// group's last step; the row factor d_x / 127 multiplies the sum.
//
// Tiling.  A workgroup owns a TM x TN tile of y (TM = 32, 64 or 128 rows of
// x, so no matrix work is spent on absent rows, and TN = 64 or 128 rows of W,
// which puts hundreds of workgroups on the chip even for a single x tile).
// Its waves each own a (16 BI) x (16 BJ) block and issue
// v_mfma_i32_16x16x64_i8.  K advances 64 codes per step through two LDS
// buffers with one barrier per step: every thread decodes its 16 codes of
// the next step to carriers (four threads of a quad per weight row, the
// register tables of a8_carriers.h) while the matrix cores work on the
// current one.
//
// Loads.  A step's code window, activations and, where the step starts a
// group, that group's (a, b) (or load-time carrier table words) and the
// previous group's scales for the wave's output columns are requested R
// steps ahead into one of R register slots (a slot is decoded one step before
// its own step and refilled at the start of it, so a group's scales ride in
// the slot of the step after its last).  Every load is unconditional (requests past the
// last step repeat it) and their order is pinned, because loads complete in
// issue order for the wait counter: the wait before a step is then for loads
// issued R - 1 steps earlier.
#include "cq_device.h"
#include "cq_internal.h"
#include "stream_common.h"
#include "a8_carriers.h"

#include <atomic>
#include <type_traits>

#define CQ_INLINE __attribute__((always_inline))

namespace cq {

namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kKS = 64;              // K step
constexpr int kStride = kKS + 16;    // LDS bytes per tile row (padded)

// KSM: at most this many K-groups per workgroup (the launch picks the count).
// Each K-group is a full set of the tile's waves with its own LDS buffers and a
// contiguous range of K steps; all of them pass the same per-step barrier, and
// their FP32 sums meet in LDS at the end.  More waves per workgroup hide the
// step's latency chain when a short tile leaves few workgroups on the chip.
template <int WM_, int WN_, int BI_, int BJ_, int R_, int KSM_>
struct a8_tile {
    static constexpr int WM = WM_, WN = WN_, BI = BI_, BJ = BJ_, R = R_, KSM = KSM_;
    static constexpr int NT = 64 * WM * WN;  // threads of one K-group
    static constexpr int TM = 16 * BI * WM, TN = 16 * BJ * WN;
    static constexpr int LDS = 2 * (TM + TN) * 80;  // bytes of one K-group's buffers
};
using a8_tile32 = a8_tile<1, 4, 2, 1, 8, 4>;    // 32 x 64, four waves of 32 x 16, up to four K-groups
using a8_tile64 = a8_tile<1, 4, 4, 1, 8, 2>;    // 64 x 64, four waves of 64 x 16, up to two K-groups
using a8_tile128 = a8_tile<2, 4, 4, 2, 8, 1>;   // 128 x 128, eight waves of 64 x 32

template <int P0, int PN, typename F>
__device__ __forceinline__ void unroll_slots(F &&f) {
    if constexpr (P0 < PN) {
        f(std::integral_constant<int, P0>{});
        unroll_slots<P0 + 1, PN>(f);
    }
}

// Keep the vector-memory reads of successive ring slots in issue order.
__device__ __forceinline__ void vmem_order() { __builtin_amdgcn_sched_barrier(0x78f); }

}  // namespace

template <int B, int SPG, int YDT, bool TB, class T>
__global__ void __launch_bounds__(T::NT * T::KSM) gemm_a8_tile(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int n, int k, const int8_t *__restrict__ x8, const float *__restrict__ dx, int m,
    void *__restrict__ y, int tiles_m, int tiles_n, const int8_t *__restrict__ ctab) {
    constexpr int M = max_code(B);
    constexpr int WN = T::WN, BI = T::BI, BJ = T::BJ, R = T::R, NT = T::NT;
    constexpr int TM = T::TM, TN = T::TN;
    constexpr int Q = NT / TN;              // threads per weight row
    constexpr int XB = TM * kKS / NT;       // activation bytes per thread per step
    constexpr int XTR = kKS / XB;           // threads per activation row
    static_assert(Q == 4, "a quad of threads per weight row");
    static_assert(XB == 8 || XB == 16, "activation loader shape");
    static_assert(R % SPG == 0 && R % 2 == 0, "group boundaries at fixed ring slots");
    static_assert(B == 3 || B == 4, "W3 and W4");
    // one K-group's double buffers per K-group (dynamic, KS x T::LDS bytes)
    extern __shared__ __attribute__((aligned(16))) int8_t lds_raw[];
    static_assert(T::KSM == 1 || 16 * NT * BI * BJ <= T::LDS, "K-group sums fit in a group's buffers");
    static_assert(T::LDS == 2 * (TM + TN) * kStride, "buffer size");
    const int KS = int(blockDim.x) / NT;

    // ---- tile: the workgroups of one XCD take consecutive indices
    const int nwg = tiles_m * tiles_n;
    int wg = blockIdx.x;
    if (nwg % 8 == 0) wg = (wg % 8) * (nwg / 8) + wg / 8;
    const int m0 = (wg / tiles_n) * TM;
    const int n0 = (wg % tiles_n) * TN;

    const int kg = T::KSM == 1 ? 0 : __builtin_amdgcn_readfirstlane(int(threadIdx.x) / NT);  // K-group
    const int tid = int(threadIdx.x) - kg * NT;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    typedef int8_t tile_buf[2][TM * kStride];
    typedef int8_t wtile_buf[2][TN * kStride];
    tile_buf &As = *reinterpret_cast<tile_buf *>(lds_raw + kg * 2 * (TM + TN) * kStride);
    wtile_buf &Bs = *reinterpret_cast<wtile_buf *>(lds_raw + kg * 2 * (TM + TN) * kStride + 2 * TM * kStride);
    const int wm = (wave / WN) * (16 * BI);
    const int wn = (wave % WN) * (16 * BJ);

    const int ng = k / (kKS * SPG);
    const uint32_t row_bytes = uint32_t(k) * B / 8u;
    const auto rc = make_rsrc(codes, uint32_t(n) * row_bytes);
    const auto rs = make_rsrc(scale, uint32_t(n) * ng * 4u);
    const auto ra = make_rsrc(a16, uint32_t(n) * ng * 2u);
    const auto rb = make_rsrc(b16, uint32_t(n) * ng * 2u);
    const auto rt = make_rsrc(ctab, TB ? uint32_t(n) * ng * (1u << (B - 1)) : 0u);
    const auto rx = make_rsrc(x8, uint32_t(m) * uint32_t(k));

    // decode roles: the quad lr serves weight row lr of the tile, thread lq
    // codes 16 lq .. +15 of every step
    const int lr = tid / Q, lq = tid % Q;
    const int wrow = n0 + lr;
    const bool wok = wrow < n;
    // W4: the 8 code bytes at byte 8 lq of the step's 32; W3: the 6 bytes at
    // byte 6 lq of its 24, inside the aligned 8-byte window that holds them
    const uint32_t wbyte = B == 4 ? 8u * uint32_t(lq) : (6u * uint32_t(lq)) & ~3u;
    const uint32_t cs = B == 4 ? 0u : 8u * ((6u * uint32_t(lq)) & 3u);
    const uint32_t cbase = uint32_t(wrow) * row_bytes + wbyte;
    const int xr = tid / XTR;                // activation row of the tile
    const int xc = (tid % XTR) * XB;         // byte offset inside the step
    const int xrow = m0 + xr;
    const bool xok = xrow < m;
    // W4 carriers this thread evaluates: magnitudes 2 lq, 2 lq + 1
    const int i0 = 2 * lq;
    const float t0 = float(i0) / float(M), t1 = float(i0 + 1) / float(M);

    uint32_t cw[R][2];
    uint32_t xw[R][XB / 4];
    uint32_t av[R], bv[R];
    float sj[R][BJ];

    // st: the step whose data the slot receives (requests past the last step
    // repeat it); su: the same step unclamped, which names the group whose
    // scales ride in a group-start slot (the group ending just before it)
    auto load_slot = [&](int st, int su, auto slot_c) CQ_INLINE {
        constexpr int SL = decltype(slot_c)::value;
        load_words<2>(rc, wok ? cbase + uint32_t(st) * (8u * B) : kOobOffset, cw[SL]);
        const int g = st / SPG;
        if constexpr (SL % SPG == 0) {
            // the group's shape (a, b) or its load-time carrier words
            const uint32_t gi = uint32_t(wrow) * ng + uint32_t(g);
            if constexpr (TB && B == 4) {
                uint32_t t[2];
                load_words<2>(rt, wok ? gi * 8u : kOobOffset, t);
                av[SL] = t[0];
                bv[SL] = t[1];
            } else if constexpr (TB) {
                av[SL] = __builtin_amdgcn_raw_buffer_load_b32(rt, wok ? gi * 4u : kOobOffset, 0, 0);
            } else {
                av[SL] = load_u16(ra, wok ? gi * 2u : kOobOffset);
                bv[SL] = load_u16(rb, wok ? gi * 2u : kOobOffset);
            }
        }
        if constexpr (SL % SPG == 0) {
            // scales of the wave's output columns for the group that ends at
            // step su - 1: it is rescaled while this slot is decoded, before
            // the slot is requested again
            const int gp = min(max(su / SPG - 1, 0), ng - 1);
#pragma unroll
            for (int j = 0; j < BJ; ++j) {
                const int col = n0 + wn + 16 * j + (lane & 15);
                sj[SL][j] = load_f32(rs, col < n ? (uint32_t(col) * ng + uint32_t(gp)) * 4u : kOobOffset);
            }
        }
        load_words<XB / 4>(rx, xok ? uint32_t(xrow) * uint32_t(k) + uint32_t(st) * kKS + uint32_t(xc) : kOobOffset,
                           xw[SL]);
    };

    // carrier tables of the group starting at the step in slot SL
    uint32_t ta0 = 0, ta1 = 0, tb0 = 0, tb1 = 0;
    auto build_tables = [&](auto slot_c) CQ_INLINE {
        constexpr int SL = decltype(slot_c)::value;
        if constexpr (B == 4) {
            if constexpr (TB) {
                ta0 = av[SL];
                ta1 = bv[SL];
            } else {
                const float a = f16_to_f32(uint16_t(av[SL])), b = f16_to_f32(uint16_t(bv[SL]));
                const float c = 1.f - a - b;
                const float mg = carrier_margin(a, b, c);
                const uint32_t pr = carrier_u8<M>(i0, t0, a, b, c, mg) | (carrier_u8<M>(i0 + 1, t1, a, b, c, mg) << 8);
                // the quad's four pairs: r0 r1 | r2 r3 | r4 r5 | r6 r7
                ta0 = quad_bcast<0x00>(pr) | (quad_bcast<0x55>(pr) << 16);
                ta1 = quad_bcast<0xaa>(pr) | (quad_bcast<0xff>(pr) << 16);
            }
            w4_negative_table(ta0, ta1, tb0, tb1);
        } else {
            if constexpr (TB) {
                ta0 = av[SL];  // r0 r1 r2 r3
            } else {
                const float a = f16_to_f32(uint16_t(av[SL])), b = f16_to_f32(uint16_t(bv[SL]));
                const float c = 1.f - a - b;
                const float mg = carrier_margin(a, b, c);
                const uint32_t pr = carrier_u8<M>(1, 1.f / 3.f, a, b, c, mg) | (carrier_u8<M>(2, 2.f / 3.f, a, b, c, mg) << 8);
                ta0 = (pr << 8) | 0x7f000000u;  // r0 r1 r2 r3
            }
            const uint32_t neg = (0x80808080u - ta0) ^ 0x80808080u;  // 0 -r1 -r2 -r3
            tb0 = perm(neg, neg, 0x01020300u);                      // 0 -r3 -r2 -r1
        }
    };

    // decode slot SL into buffer `buf`: carriers of the thread's 16 codes and
    // the step's activation bytes
    auto store_step = [&](auto buf_c, auto slot_c) CQ_INLINE {
        constexpr int buf = decltype(buf_c)::value;
        constexpr int SL = decltype(slot_c)::value;
        uint32_t cr[4];
        if constexpr (B == 4) {
            w4_word_carriers(cw[SL][0], ta0, ta1, tb0, tb1, cr[0], cr[1]);
            w4_word_carriers(cw[SL][1], ta0, ta1, tb0, tb1, cr[2], cr[3]);
        } else {
            const uint64_t win = ((uint64_t(cw[SL][1]) << 32) | cw[SL][0]) >> cs;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t x3 = uint32_t(win >> (12 * q)) & 0xfffu;  // four 3-bit fields
                const uint32_t sel = (x3 & 7u) | ((x3 << 5) & 0x700u) | ((x3 << 10) & 0x70000u) | ((x3 << 15) & 0x7000000u);
                cr[q] = perm(tb0, ta0, sel);
            }
        }
        *reinterpret_cast<u32x4 *>(&Bs[buf][lr * kStride + 16 * lq]) = u32x4{cr[0], cr[1], cr[2], cr[3]};
        int8_t *ap = &As[buf][xr * kStride + xc];
        if constexpr (XB == 16)
            *reinterpret_cast<u32x4 *>(ap) = u32x4{xw[SL][0], xw[SL][1], xw[SL][2], xw[SL][3]};
        else
            *reinterpret_cast<u32x2 *>(ap) = u32x2{xw[SL][0], xw[SL][1]};
    };

    i32x4 acc[BI][BJ];
    f32x4 accf[BI][BJ];
#pragma unroll
    for (int i = 0; i < BI; ++i)
#pragma unroll
        for (int j = 0; j < BJ; ++j) {
            acc[i][j] = i32x4{0, 0, 0, 0};
            accf[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        }

    using S0 = std::integral_constant<int, 0>;
    const int nsteps = k / kKS;
    // this K-group's steps: [s0, s1), s0 a multiple of the ring length (so
    // ring positions and group boundaries stay compile-time); every group runs
    // `per` steps, the ones past s1 without matrix work
    const int per = ((nsteps + KS - 1) / KS + R - 1) / R * R;
    const int s0 = kg * per;
    const int s1 = min(s0 + per, nsteps);
    unroll_slots<0, R>([&](auto p_c) CQ_INLINE {
        constexpr int P = decltype(p_c)::value;
        load_slot(min(s0 + P, nsteps - 1), s0 + P, p_c);
        vmem_order();
    });
    build_tables(S0{});
    store_step(S0{}, S0{});
    __syncthreads();

    // Step st works on buffer st % 2 with slot st % R (decoded in the previous
    // step), requests step st + R into that slot and decodes step st + 1 into
    // the other buffer.  Steps past the end (the last period) skip the matrix
    // work.
    auto do_step = [&](int st, auto p_c) CQ_INLINE {
        constexpr int P = decltype(p_c)::value;
        constexpr int buf = P % 2;
        constexpr int SN = (P + 1) % R;
        load_slot(min(st + R, nsteps - 1), st + R, p_c);
        vmem_order();
        if (st < s1) {
            i32x4 af[BI], bf[BJ];
#pragma unroll
            for (int i = 0; i < BI; ++i)
                af[i] = *reinterpret_cast<const i32x4 *>(&As[buf][(wm + 16 * i + (lane & 15)) * kStride + 16 * (lane >> 4)]);
#pragma unroll
            for (int j = 0; j < BJ; ++j)
                bf[j] = *reinterpret_cast<const i32x4 *>(&Bs[buf][(wn + 16 * j + (lane & 15)) * kStride + 16 * (lane >> 4)]);
            const i32x4 zero = {0, 0, 0, 0};
#pragma unroll
            for (int i = 0; i < BI; ++i)
#pragma unroll
                for (int j = 0; j < BJ; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[i], bf[j], P % SPG == 0 ? zero : acc[i][j], 0,
                                                                      0, 0);
            if constexpr (P % SPG == SPG - 1) {
                // group complete: FP32 rescale of the exact partials
#pragma unroll
                for (int j = 0; j < BJ; ++j)
#pragma unroll
                    for (int i = 0; i < BI; ++i)
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            accf[i][j][e] = __builtin_fmaf(sj[SN][j], float(acc[i][j][e]), accf[i][j][e]);
            }
        }
        if constexpr (SN % SPG == 0) build_tables(std::integral_constant<int, SN>{});
        store_step(std::integral_constant<int, 1 - buf>{}, std::integral_constant<int, SN>{});
        __syncthreads();
    };

    for (int st = s0; st < s0 + per; st += R)
        unroll_slots<0, R>([&](auto p_c) CQ_INLINE {
            constexpr int P = decltype(p_c)::value;
            do_step(st + P, p_c);
        });

    if (T::KSM > 1 && KS > 1) {
        // the K-groups' sums meet in LDS (the step buffers are free after the
        // last barrier); K-group 0 adds them in group order and stores
        f32x4 *red = reinterpret_cast<f32x4 *>(lds_raw);
#pragma unroll
        for (int i = 0; i < BI; ++i)
#pragma unroll
            for (int j = 0; j < BJ; ++j) red[((kg * BI + i) * BJ + j) * NT + tid] = accf[i][j];
        __syncthreads();
        if (kg != 0) return;
#pragma unroll
        for (int i = 0; i < BI; ++i)
#pragma unroll
            for (int j = 0; j < BJ; ++j)
                for (int g = 1; g < KS; ++g) accf[i][j] += red[((g * BI + i) * BJ + j) * NT + tid];
    }

#pragma unroll
    for (int i = 0; i < BI; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int row = m0 + wm + 16 * i + 4 * (lane >> 4) + e;
            if (row >= m) continue;
            const float f = dx[row] / 127.0f;
#pragma unroll
            for (int j = 0; j < BJ; ++j) {
                const int col = n0 + wn + 16 * j + (lane & 15);
                if (col < n) store_out<YDT>(y, int64_t(row) * n + col, accf[i][j][e] * f);
            }
        }
}

namespace {

// K-groups per workgroup: the most (up to KSM, at least 4 K steps each) with
// which every workgroup is resident in one round, by the runtime's occupancy
// for that block size (cached per kernel, device and count)
template <class K, class T>
int a8_tile_groups(K kernel, int64_t nwg, int64_t nsteps) {
    static std::atomic<int> fit[64][T::KSM + 1];  // workgroups per CU + 1; 0: not yet asked
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1;
    const int64_t cus = device_cu_count();
    for (int ks = T::KSM; ks > 1; ks /= 2) {
        if (nsteps < 4 * ks) continue;
        int f = fit[dev][ks].load(std::memory_order_relaxed) - 1;
        if (f < 0) {
            int nb = 0;
            if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kernel, T::NT * ks, size_t(ks) * T::LDS) != hipSuccess)
                nb = 0;
            fit[dev][ks].store(nb + 1, std::memory_order_relaxed);
            f = nb;
        }
        if (f > 0 && nwg <= int64_t(f) * cus) return ks;
    }
    return 1;
}

template <int B, int SPG, int YDT, bool TB, class T>
hipError_t a8_tile_launch(const cq_weight &w, const int8_t *ctab, const int8_t *x8, const float *dx, int64_t m,
                          void *y, hipStream_t stream) {
    const int64_t tiles_m = (m + T::TM - 1) / T::TM;
    const int64_t tiles_n = (w.n + T::TN - 1) / T::TN;
    const int64_t nwg = tiles_m * tiles_n;
    if (nwg > 0x7fffffff) return hipErrorInvalidValue;
    auto kernel = gemm_a8_tile<B, SPG, YDT, TB, T>;
    const int ks = T::KSM == 1 ? 1 : a8_tile_groups<decltype(kernel), T>(kernel, nwg, w.k / kKS);
    hipLaunchKernelGGL(kernel, dim3(unsigned(nwg)), dim3(T::NT * ks), size_t(ks) * T::LDS, stream, w.codes,
                       w.scale, w.a, w.b, int(w.n), int(w.k), x8, dx, int(m), y, int(tiles_m), int(tiles_n), ctab);
    return hipGetLastError();
}

template <int B, int YDT, bool TB, class T>
hipError_t a8_tile_group(const cq_weight &w, const int8_t *ctab, const int8_t *x8, const float *dx, int64_t m,
                         void *y, hipStream_t stream) {
    switch (w.group) {
        case 64: return a8_tile_launch<B, 1, YDT, TB, T>(w, ctab, x8, dx, m, y, stream);
        case 128: return a8_tile_launch<B, 2, YDT, TB, T>(w, ctab, x8, dx, m, y, stream);
        case 256: return a8_tile_launch<B, 4, YDT, TB, T>(w, ctab, x8, dx, m, y, stream);
        case 512: return a8_tile_launch<B, 8, YDT, TB, T>(w, ctab, x8, dx, m, y, stream);
    }
    return hipErrorNotSupported;
}

template <bool TB, class T>
hipError_t a8_tile_dtypes(const cq_weight &w, const int8_t *ctab, const int8_t *x8, const float *dx, int64_t m,
                          void *y, int y_dt, hipStream_t stream) {
    if (w.bits == 3) {
        if (y_dt == 0) return a8_tile_group<3, 0, TB, T>(w, ctab, x8, dx, m, y, stream);
        if (y_dt == 1) return a8_tile_group<3, 1, TB, T>(w, ctab, x8, dx, m, y, stream);
        return a8_tile_group<3, 2, TB, T>(w, ctab, x8, dx, m, y, stream);
    }
    if (y_dt == 0) return a8_tile_group<4, 0, TB, T>(w, ctab, x8, dx, m, y, stream);
    if (y_dt == 1) return a8_tile_group<4, 1, TB, T>(w, ctab, x8, dx, m, y, stream);
    return a8_tile_group<4, 2, TB, T>(w, ctab, x8, dx, m, y, stream);
}

template <bool TB>
hipError_t a8_tile_rows(const cq_weight &w, const int8_t *ctab, const int8_t *x8, const float *dx, int64_t m, void *y,
                        int y_dt, int tile_rows, hipStream_t stream) {
    switch (tile_rows) {
        case 32: return a8_tile_dtypes<TB, a8_tile32>(w, ctab, x8, dx, m, y, y_dt, stream);
        case 64: return a8_tile_dtypes<TB, a8_tile64>(w, ctab, x8, dx, m, y, y_dt, stream);
        case 128: return a8_tile_dtypes<TB, a8_tile128>(w, ctab, x8, dx, m, y, y_dt, stream);
    }
    return hipErrorNotSupported;
}

}  // namespace

hipError_t launch_gemm_a8_tile(const cq_weight &w, const int8_t *ctab, const int8_t *x8, const float *dx, int64_t m,
                               void *y, int y_dt, int tile_rows, hipStream_t stream) {
    return ctab ? a8_tile_rows<true>(w, ctab, x8, dx, m, y, y_dt, tile_rows, stream)
                : a8_tile_rows<false>(w, ctab, x8, dx, m, y, y_dt, tile_rows, stream);
}

}  // namespace cq
