// Model-dtype single-row GEMV, streaming table-decode family (Sec. 5.2
// strategy 2 and Sec. 5.3 narrow-row tactic) for m == 1.
//
// Numerics follow the paper's narrow-row GEMV: the activation and the
// normalised level are multiplied in FP32; the FP32 group scale multiplies
// each 32-code sub-reduction of the group (a regrouping of the group
// reduction, identical up to rounding order).
//
// Work mapping (coalescing first).  K is cut into column blocks of 64 units of
// 32 codes (2048 codes; a unit is exactly B 32-bit words of the row).  Lane l
// of a wave always owns unit l of its column block, so one wavefront load of a
// row reads 64 * 4B contiguous bytes.  A workgroup owns RW rows; its waves take
// different column blocks of those rows and are reduced through LDS at the
// end.  A wave requests the codes, metadata and activations of its next item
// (RW rows of one column block) before it decodes the current one, and the
// activations of an item are converted to FP32 once for all RW rows.
//
// Decode.  Every lane reads one entry per weight of a table of the 2^B signed
// normalised levels (0 for the reserved pattern) in its own LDS column, at
// byte (field << 8) + lane * 4 + slot base, which is free of bank conflicts,
// and writes that whole column itself (writing one value into the columns of
// all lanes of a group would put those lanes' stores of different fields on
// the same four banks).  W4/W5 at G = 128 evaluate a quarter of the
// magnitudes per lane and gather the group's others through DPP, other
// widths and groups evaluate all of them.  W1 and W2, whose levels are -1,
// 0 and +1 for every shape, skip the table: a code pair's levels are formed
// in the activation dtype from the code bits and meet the activation pair in
// a two-term dot product (Sec. 5.2 strategy 1).  For W4 the address is assembled by one byte permute per
// weight, and the reads are issued 16 weights ahead of the products that
// consume them.  B >= 6 evaluates the cubic in registers instead of keeping a
// 64..256-entry table.
#include <algorithm>

#include "cq_device.h"
#include "cq_internal.h"
#include "stream_common.h"

#define CQ_INLINE __attribute__((always_inline))

namespace cq {

namespace {

typedef __attribute__((address_space(3))) float lds_f;
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float lds_ld(uint32_t a) { return *reinterpret_cast<const lds_f *>(uintptr_t(a)); }
__device__ __forceinline__ void lds_st(uint32_t a, float v) { *reinterpret_cast<lds_f *>(uintptr_t(a)) = v; }

__device__ __forceinline__ void wave_lds_fence() {
    // LDS instructions of one wavefront execute in issue order, so ordering the
    // compiler's memory operations is enough for cross-lane LDS visibility within
    // a wavefront; no hardware wait (which would also drain pending HBM loads).
    __asm__ __volatile__("" ::: "memory");
    __builtin_amdgcn_wave_barrier();
}

}  // namespace

// XRES (resident activations, not routed): the workgroup has one wave per
// column block and every wave keeps its block for the whole launch, so the
// wave converts its slice of x to FP32 once and then streams only codes and
// metadata, tile after tile; the per-tile sums of the waves meet in LDS in
// batches of kResBatch tiles (two alternating buffers, one barrier a batch).
//
// ROUTED: a bank of n_experts matrices of n rows each (expert e at row e * n)
// and `routes` (token, expert) pairs; route r computes x[token] W_expert^T
// into row r of y, every route streaming its expert's weights (the decode
// case of a few routes per expert).  Routes naming a token or expert out of
// range are skipped and their output row is not written.
constexpr int kResBatch = 4;

template <int B, int UPG, int RW, int XDT, int YDT, bool ROUTED, bool XRES>
__global__ void __launch_bounds__(XRES ? 512 : 256) gemv_a16_stream(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int n, int k, const uint16_t *__restrict__ x, void *__restrict__ y,
    const int32_t *__restrict__ rtok, const int32_t *__restrict__ rexp, int routes, int tokens, int n_experts) {
    static_assert(!(XRES && ROUTED), "resident activations serve the single-matrix product");
    constexpr int G = UPG * 32;
    constexpr int M = max_code(B);
    // W1/W2 levels are -1, 0, +1 whatever the shape: mapped directly (DIRECT),
    // no table; W3..W5 use the LDS tables; B >= 6 evaluates the cubic
    constexpr bool DIRECT = (B <= 2);
    constexpr bool LUT = (B >= 3 && B <= 5);
    constexpr int NT = LUT ? (1 << B) : 1;
    // every lane owns a full column of the table (no replicated stores, whose
    // lanes of one group all hit the same four banks)
    constexpr bool OWN = LUT;
    // LDS (dynamic, starting at address 0): one NT x 256-byte table per wave,
    // then the cross-wave partial sums.  The W4 address build relies on bits
    // 8..15 of the table base being zero.
    extern __shared__ __attribute__((aligned(16))) float tab[];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));  // uniform: rows stay scalar
    const int nwaves = blockDim.x >> 6;  // the host keeps nwaves <= ncb (XRES: == ncb)
    // cross-wave sums: [nwaves][RW], XRES [2][nwaves][kResBatch * RW]
    float *red = tab + nwaves * RW * NT * 64;
    const int ntiles = (n + RW - 1) / RW;
    // item space: the row tiles, or (route, row tile) pairs, route-major
    const int nitems_t = ROUTED ? ntiles * routes : ntiles;
    const int units = k >> 5;
    const int ncb = (units + 63) >> 6;
    const int ng = k / G;
    const uint32_t row_bytes = uint32_t(k) * B / 8;
    const uint32_t bank_rows = ROUTED ? uint32_t(n) * uint32_t(n_experts) : uint32_t(n);
    const auto rc = make_rsrc(codes, bank_rows * row_bytes);
    const auto rs = make_rsrc(scale, bank_rows * ng * 4u);
    const auto ra = make_rsrc(a16, bank_rows * ng * 2u);
    const auto rb = make_rsrc(b16, bank_rows * ng * 2u);
    const auto rx = make_rsrc(x, uint32_t(ROUTED ? tokens : 1) * uint32_t(k) * 2u);
    const uint32_t tbase = uint32_t(uintptr_t((lds_f *)tab));
    // one table per (wave, row of the tile): slot index wave * RW + r
    const uint32_t col = tbase + uint32_t(wave * RW) * (NT * 256u) + uint32_t(lane) * 4u;
    const uint32_t wtag = uint32_t(wave * RW) * 0x10101010u;

    // magnitudes this lane evaluates for its group's table, and their t = i/M
    constexpr int MPL = (B == 1) ? 1 : (M + 1 + UPG - 1) / UPG;
    int mag[MPL];
    float tq[MPL];
#pragma unroll
    for (int t = 0; t < MPL; ++t) {
        mag[t] = (B == 1) ? (lane % UPG == 0 ? 1 : M + 1) : lane % UPG + UPG * t;
        tq[t] = float(mag[t]) * (1.0f / float(M));
    }

    // An item is (row tile, column block).  A workgroup walks the tiles
    // blockIdx.x + j * gridDim.x; its wave w takes column blocks w, w + nwaves,
    // ... of each tile.  Row offsets are wave-uniform (scalar offsets); rows
    // past the matrix repeat its last row and are never stored; lanes past the
    // row's units load an out-of-range offset and read zeros.
    //
    // Two register sets alternate: the codes, metadata and activations of the
    // next item are requested into one set before the item in the other set
    // is decoded, so every wait is for loads issued a whole item earlier
    // (vector-memory loads complete in issue order for the wait counter).
    struct Item {
        uint32_t w[RW][B];
        float s[RW];
        uint32_t a[RW], b[RW];
        uint32_t x[XRES ? 1 : 16];
        bool ok;  // routed: the route names a valid token and expert
    };
    // route and row tile of an item (routed), else the row tile itself
    auto split = [&](int ti, int &route, int &t) CQ_INLINE {
        if constexpr (ROUTED) {
            route = ti / ntiles;
            t = ti - route * ntiles;
        } else {
            route = 0;
            t = ti;
        }
    };
    // An item past the last tile (ok false) still issues its loads, at an
    // out-of-range offset that reads zeros: every path through the loop then
    // has the same loads in flight, and the waits stay exact.
    auto fetch = [&](Item &it, int ti, int c, bool ok) CQ_INLINE {
        int route, t;
        split(ti, route, t);
        uint32_t row_base = 0, x_base = 0;
        if constexpr (ROUTED) {
            const int rr = ok ? route : 0;
            const int tok = __builtin_amdgcn_readfirstlane(rtok[rr]);
            const int ex = __builtin_amdgcn_readfirstlane(rexp[rr]);
            ok = ok && tok >= 0 && tok < tokens && ex >= 0 && ex < n_experts;
            row_base = ok ? uint32_t(ex) * uint32_t(n) : 0u;
            x_base = ok ? uint32_t(tok) * uint32_t(k) * 2u : 0u;
        }
        it.ok = ok;
        const int u = c * 64 + lane;
        const bool uok = ok && u < units;
        const uint32_t vc = uok ? uint32_t(u) * (4 * B) : kOobOffset;
        const uint32_t vm = uok ? uint32_t(u) / UPG * 4u : kOobOffset;
        const uint32_t vh = uok ? uint32_t(u) / UPG * 2u : kOobOffset;
        const uint32_t xo = uok ? uint32_t(u) * 64u : kOobOffset;
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            const uint32_t row = row_base + uint32_t(min(t * RW + r, n - 1));  // t may be past the last tile
            const uint32_t gi = row * uint32_t(ng);
            load_words_s<B>(rc, vc, row * row_bytes, it.w[r]);
            it.s[r] = load_f32_s(rs, vm, gi * 4u);
            it.a[r] = load_u16_s(ra, vh, gi * 2u);
            it.b[r] = load_u16_s(rb, vh, gi * 2u);
        }
        if constexpr (!XRES) load_words_s<16>(rx, xo, x_base, it.x);
    };

    // DIRECT: the unit's activations as 16 pairs (x_j, x_{j+16}) in the
    // activation dtype, the operands of a two-term dot product whose other
    // operand holds the levels of codes j and j + 16
    auto pair_x = [&](const uint32_t (&xw)[16], uint32_t (&xp)[16]) CQ_INLINE {
#pragma unroll
        for (int j = 0; j < 16; ++j)
            xp[j] = __builtin_amdgcn_perm(xw[8 + j / 2], xw[j / 2], (j & 1) ? 0x07060302u : 0x05040100u);
    };
    // XRES: the wave's slice of x (column block `wave`), FP32 (DIRECT: pairs),
    // for the launch
    float xr[XRES && !DIRECT ? 32 : 1];
    uint32_t xrp[XRES && DIRECT ? 16 : 1];
    if constexpr (XRES) {
        const int u = wave * 64 + lane;
        uint32_t xw[16];
        load_words_s<16>(rx, u < units ? uint32_t(u) * 64u : kOobOffset, 0u, xw);
        if constexpr (DIRECT) {
            pair_x(xw, xrp);
        } else {
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                xr[2 * e] = act_to_f32<XDT>(uint16_t(xw[e] & 0xffffu));
                xr[2 * e + 1] = act_to_f32<XDT>(uint16_t(xw[e] >> 16));
            }
        }
    }
    int slot = 0, flushes = 0;  // XRES: tiles recorded in the current batch, batches done

    float acc[RW];
#pragma unroll
    for (int i = 0; i < RW; ++i) acc[i] = 0.f;

    auto process = [&](const Item &it, int ti, bool last_cb, bool final) CQ_INLINE {
        int route, tile;
        split(ti, route, tile);
        // ---- activations of this unit, FP32 in registers
        float xu[XRES || DIRECT ? 1 : 32];
        if constexpr (!XRES && !DIRECT) {
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                xu[2 * e] = act_to_f32<XDT>(uint16_t(it.x[e] & 0xffffu));
                xu[2 * e + 1] = act_to_f32<XDT>(uint16_t(it.x[e] >> 16));
            }
        }
        auto xf = [&](int i) CQ_INLINE {
            if constexpr (XRES) return xr[i];
            else return xu[i];
        };
        if constexpr (DIRECT) {
            // Levels -1, 0, +1 (Sec. 5.2 strategy 1): the pair of levels of
            // codes j and j + 16 is built in the activation dtype from the
            // code bits and fed with the pair (x_j, x_{j+16}) to a two-term
            // dot product with FP32 accumulation (products of a level +-1 or 0
            // are exact).  W1: code 1 -> +1, 0 -> -1; bit j and bit j + 16 of
            // the unit's word go to the two sign bits with one shift.  W2:
            // codes 0, 1, 2 (reserved), 3 -> 0, +1, 0, -1; the two 2-bit codes
            // (as bytes f, f + 4) select the level bytes from two 4-byte tables.
            uint32_t xpl[XRES ? 1 : 16];
            if constexpr (!XRES) pair_x(it.x, xpl);
            auto xpair = [&](int j) CQ_INLINE {
                if constexpr (XRES) return xrp[j];
                else return xpl[j];
            };
            constexpr uint32_t kOne = XDT == 0 ? 0x3f803f80u : 0x3c003c00u;
            constexpr uint32_t kLo = XDT == 0 ? 0x80008000u : 0u;          // low bytes of 0, +1, 0, -1
            constexpr uint32_t kHi = XDT == 0 ? 0xbf003f00u : 0xbc003c00u;  // high bytes
            auto dot2 = [&](uint32_t xa, uint32_t lv, float c) CQ_INLINE {
                if constexpr (XDT == 0)
                    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, xa),
                                                           __builtin_bit_cast(bf16x2_t, lv), c, false);
                else
                    return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2_t, xa), __builtin_bit_cast(f16x2_t, lv),
                                                  c, false);
            };
#pragma unroll
            for (int r = 0; r < RW; ++r) {
                float p0 = 0.f, p1 = 0.f;
                if constexpr (B == 1) {
                    const uint32_t nw = ~it.w[r][0];
#pragma unroll
                    for (int j = 0; j < 16; ++j) {
                        const uint32_t lv = ((nw << (15 - j)) & 0x80008000u) | kOne;
                        if (j & 1) p1 = dot2(xpair(j), lv, p1);
                        else p0 = dot2(xpair(j), lv, p0);
                    }
                } else {
                    // codes j < 8 and j + 16 in the low and high halves of c0,
                    // codes 8..15 and 24..31 in those of c1
                    const uint32_t c0 = __builtin_amdgcn_perm(it.w[r][1], it.w[r][0], 0x05040100u);
                    const uint32_t c1 = __builtin_amdgcn_perm(it.w[r][1], it.w[r][0], 0x07060302u);
#pragma unroll
                    for (int j = 0; j < 16; ++j) {
                        const uint32_t f = ((j < 8 ? c0 : c1) >> (2 * (j & 7))) & 0x00030003u;
                        const uint32_t lv = __builtin_amdgcn_perm(kHi, kLo, f * 0x0101u + 0x04000400u);
                        if (j & 1) p1 = dot2(xpair(j), lv, p1);
                        else p0 = dot2(xpair(j), lv, p0);
                    }
                }
                acc[r] = __builtin_fmaf(it.s[r], p0 + p1, acc[r]);
            }
        }
        // ---- level tables of all rows of the tile first (one slot per row), so
        // that the LDS writes of one row overlap the reads of the previous one
        float al_r[RW], be_r[RW], ga_r[RW];
        if constexpr (LUT) wave_lds_fence();  // the previous item's reads are issued
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            float a = 1.f, b = 0.f;
            if constexpr (B >= 3) {
                a = f16_to_f32(uint16_t(it.a[r]));
                b = f16_to_f32(uint16_t(it.b[r]));
            }
            const float cc = 1.f - a - b;
            al_r[r] = a * (1.0f / float(M));
            be_r[r] = b * (1.0f / float(M * M));
            ga_r[r] = cc * (1.0f / float(M * M * M));
            if constexpr (OWN) {
                // every lane writes its own column: +q at field i and -q at field
                // NT - i for i = 1 .. M - 1 (fields 0 and NT/2 hold 0 and fields M
                // and NT - M hold +1 and -1, all written once before the loop)
                if constexpr (B >= 3) {
                    float qa[M + 1];
                    if constexpr (B >= 4 && UPG == 4) {
                        // the group is one DPP quad: lane j evaluates magnitudes j,
                        // j + 4, ..., and every lane gathers all of them
                        constexpr int NQ = (M + 1) / 4;
                        float qv[NQ];
#pragma unroll
                        for (int t = 0; t < NQ; ++t) {
                            qv[t] = tq[t] * __builtin_fmaf(tq[t], __builtin_fmaf(tq[t], cc, b), a);
                        }
#pragma unroll
                        for (int t = 0; t < NQ; ++t) {
                            const int u = int(__float_as_uint(qv[t]));
                            qa[4 * t + 0] = __uint_as_float(uint32_t(__builtin_amdgcn_mov_dpp(u, 0x00, 0xf, 0xf, true)));
                            qa[4 * t + 1] = __uint_as_float(uint32_t(__builtin_amdgcn_mov_dpp(u, 0x55, 0xf, 0xf, true)));
                            qa[4 * t + 2] = __uint_as_float(uint32_t(__builtin_amdgcn_mov_dpp(u, 0xaa, 0xf, 0xf, true)));
                            qa[4 * t + 3] = __uint_as_float(uint32_t(__builtin_amdgcn_mov_dpp(u, 0xff, 0xf, 0xf, true)));
                        }
                    } else {
#pragma unroll
                        for (int i = 1; i < M; ++i) {
                            const float t = float(i) * (1.0f / float(M));
                            qa[i] = t * __builtin_fmaf(t, __builtin_fmaf(t, cc, b), a);
                        }
                    }
                    const uint32_t own = col + uint32_t(r) * (NT * 256u);
#pragma unroll
                    for (int i = 1; i < M; ++i) {
                        lds_st(own + uint32_t(i) * 256u, qa[i]);
                        lds_st(own + uint32_t(NT - i) * 256u, -qa[i]);
                    }
                }
            }
        }
        if constexpr (LUT) wave_lds_fence();
        // ---- decode
        if constexpr (DIRECT) {
        } else if constexpr (B == 4) {
            // The 64 weights of the item (both rows) in chunks of 16: the table
            // reads of chunk c + 1 are issued before the products of chunk c, so
            // a wave keeps 16 to 32 LDS reads in flight.
            constexpr int BT = 16;
            // the nibble mask lives in a vector register, so that mask and slot
            // tag fold into one v_and_or_b32 (a literal and a scalar tag would
            // exceed the one scalar operand a VOP3 instruction may read)
            uint32_t nmask;
            __asm__("v_mov_b32 %0, 0x0f0f0f0f" : "=v"(nmask));
            constexpr int CH = RW * 32 / BT;
            float lvb[2][BT];
            float pp[RW][2];
#pragma unroll
            for (int r = 0; r < RW; ++r) pp[r][0] = pp[r][1] = 0.f;
            auto reads = [&](int c, float *dst) CQ_INLINE {
#pragma unroll
                for (int e = 0; e < BT; ++e) {
                    // weight i of row r: byte i / 2 % 4 of code word i / 8, low
                    // nibble for even i
                    const int wi = c * BT + e;
                    const int r = wi / 32, i = wi % 32;
                    const uint32_t wd = it.w[r][i / 8];
                    const uint32_t nib =
                        ((i & 1) ? ((wd >> 4) & nmask) : (wd & nmask)) | (wtag + uint32_t(r) * 0x10101010u);
                    const uint32_t sel = 0x03020000u | (uint32_t(4 + (i % 8) / 2) << 8);
                    dst[e] = lds_ld(__builtin_amdgcn_perm(nib, col + uint32_t(r) * (NT * 256u), sel));
                }
            };
            auto products = [&](int c, const float *src) CQ_INLINE {
#pragma unroll
                for (int e = 0; e < BT; ++e) {
                    const int wi = c * BT + e;
                    const int r = wi / 32, i = wi % 32;
                    pp[r][i & 1] = __builtin_fmaf(xf(i), src[e], pp[r][i & 1]);
                }
            };
            reads(0, lvb[0]);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                if (c + 1 < CH) reads(c + 1, lvb[(c + 1) & 1]);
                __builtin_amdgcn_sched_barrier(0);
                products(c, lvb[c & 1]);
                __builtin_amdgcn_sched_barrier(0);
            }
#pragma unroll
            for (int r = 0; r < RW; ++r) acc[r] = __builtin_fmaf(it.s[r], pp[r][0] + pp[r][1], acc[r]);
        } else {
#pragma unroll
            for (int r = 0; r < RW; ++r) {
                const uint32_t colr = col + uint32_t(r) * (NT * 256u);
                const float al = al_r[r], be = be_r[r], ga = ga_r[r];
                float p0 = 0.f, p1 = 0.f;
#pragma unroll
                for (int i8 = 0; i8 < 4; ++i8) {
                    float lv[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int i = i8 * 8 + e;
                        const int bit = i * B;
                        const int wd = bit >> 5, sh = bit & 31;
                        uint32_t v;
                        if (sh + B <= 32) v = it.w[r][wd] >> sh;
                        else v = __builtin_amdgcn_alignbit(it.w[r][wd + 1], it.w[r][wd], sh);
                        if constexpr (LUT) {
                            lv[e] = lds_ld(((v & uint32_t(NT - 1)) << 8) + colr);
                        } else {
                            const int kk = __builtin_amdgcn_sbfe(int(v), 0, B);
                            const float kf = float(kk);
                            const float ak = __builtin_fabsf(kf);
                            const float lvv = kf * __builtin_fmaf(ak, __builtin_fmaf(ak, ga, be), al);
                            lv[e] = (kk == -(1 << (B - 1))) ? 0.f : lvv;
                        }
                    }
#pragma unroll
                    for (int e = 0; e < 8; e += 2) {
                        p0 = __builtin_fmaf(xf(i8 * 8 + e), lv[e], p0);
                        p1 = __builtin_fmaf(xf(i8 * 8 + e + 1), lv[e + 1], p1);
                    }
                }
                acc[r] = __builtin_fmaf(it.s[r], p0 + p1, acc[r]);
            }
        }
        if (last_cb) {
            const int row0 = tile * RW;
            static_assert(RW == 2, "the output store writes row pairs");
            // one lane stores the tile's row pair (routed: row route * n + row,
            // two single stores, as that index can be odd; invalid routes store
            // nothing)
            auto store = [&](float v0, float v1) CQ_INLINE {
                if constexpr (ROUTED) {
                    if (!it.ok) return;
                    const int64_t o = int64_t(route) * n + row0;
                    store_out<YDT>(y, o, v0);
                    if (row0 + 1 < n) store_out<YDT>(y, o + 1, v1);
                } else {
                    store_row_pair<YDT>(y, row0, v0, v1, row0 + 1 < n);
                }
            };
            if constexpr (XRES) {
                // record the wave's sums of this tile; every kResBatch tiles
                // (and after the last) the first wave adds the waves' sums
                float *rb = red + (flushes & 1) * (nwaves * kResBatch * RW);
#pragma unroll
                for (int r = 0; r < RW; ++r) {
                    const float v = wave_sum(acc[r]);
                    acc[r] = 0.f;
                    if (lane == 0) rb[wave * (kResBatch * RW) + slot * RW + r] = v;
                }
                ++slot;
                if (slot == kResBatch || final) {
                    __syncthreads();
                    if (wave == 0 && lane < slot * RW) {
                        float v = 0.f;
                        for (int wv = 0; wv < nwaves; ++wv) v += rb[wv * (kResBatch * RW) + lane];
                        const int j = lane / RW, r = lane - j * RW;
                        const int row = (tile - (slot - 1 - j) * int(gridDim.x)) * RW + r;
                        if (row < n) store_out<YDT>(y, row, v);
                    }
                    // the other buffer takes the next batch: the barrier of
                    // that batch orders these reads before its reuse
                    ++flushes;
                    slot = 0;
                }
            } else if (nwaves == 1) {
                const float v0 = wave_sum(acc[0]);
                const float v1 = wave_sum(acc[1]);
                acc[0] = 0.f;
                acc[1] = 0.f;
                if (lane == 0 && row0 < n) store(v0, v1);
            } else {
#pragma unroll
                for (int r = 0; r < RW; ++r) {
                    const float v = wave_sum(acc[r]);
                    acc[r] = 0.f;
                    if (lane == 0) red[wave * RW + r] = v;
                }
                __syncthreads();
                if (wave == 0 && lane == 0 && row0 < n) {
                    float v0 = 0.f, v1 = 0.f;
                    for (int wv = 0; wv < nwaves; ++wv) {
                        v0 += red[wv * RW];
                        v1 += red[wv * RW + 1];
                    }
                    store(v0, v1);
                }
                __syncthreads();  // red is reused by the next tile
            }
        }
    };

    // the item after (tile, cb): the wave's next column block of the tile,
    // else its first column block of the workgroup's next tile
    auto advance = [&](int &tile, int &cb) CQ_INLINE {
        cb += nwaves;
        if (cb >= ncb) {
            cb = wave;
            tile += int(gridDim.x);
        }
    };

    Item ia, ib;
    int tile = blockIdx.x, cb = wave;
    if (tile >= nitems_t) return;
    if constexpr (OWN) {
        // the entries no item rewrites
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            const uint32_t own = col + uint32_t(r) * (NT * 256u);
            {
                lds_st(own, 0.f);
                lds_st(own + uint32_t(NT / 2) * 256u, 0.f);
                lds_st(own + uint32_t(M) * 256u, 1.f);
                lds_st(own + uint32_t(NT - M) * 256u, -1.f);
            }
        }
        wave_lds_fence();
    }
    fetch(ia, tile, cb, true);
    while (true) {
        int t1 = tile, c1 = cb;
        advance(t1, c1);
        const bool last0 = t1 != tile;
        const bool have1 = t1 < nitems_t;
        fetch(ib, t1, c1, have1);
        process(ia, tile, last0, !have1);
        if (!have1) break;
        int t2 = t1, c2 = c1;
        advance(t2, c2);
        const bool last1 = t2 != t1;
        const bool have2 = t2 < nitems_t;
        fetch(ia, t2, c2, have2);
        process(ib, t1, last1, !have2);
        if (!have2) break;
        tile = t2;
        cb = c2;
    }
}

// route map of the routed mode (unused otherwise)
struct StreamRoutes {
    const int32_t *tok = nullptr, *exp = nullptr;
    int routes = 0, tokens = 0, n_experts = 0;
};

template <int B, int UPG, int RW, int XDT, int YDT, bool ROUTED>
static hipError_t stream_waves(const cq_weight &w, const void *x, void *y, const StreamRoutes &rt,
                               hipStream_t stream) {
    const int64_t ncb = ((w.k >> 5) + 63) >> 6;
    constexpr int NT = (B >= 3 && B <= 5) ? (1 << B) : 1;
    constexpr int kMaxW = NT >= 32 ? 2 : 4;  // keep the tables within 32 KB and the W4 slot tag in 4 bits
    // Rows of up to two column blocks: one wave per tile walks them in turn
    // (no cross-wave reduction); longer rows split their column blocks over two
    // waves (measured on the Llama-3-8B layer shapes).
    int nw = ncb > 2 ? 2 : 1;
    if (nw > kMaxW) nw = kMaxW;
    const size_t lds = sizeof(float) * (size_t(nw) * RW * NT * 64 + size_t(nw) * RW);
    const int64_t tiles = (w.n + RW - 1) / RW * (ROUTED ? rt.routes : 1);
    if (tiles < 1) return hipSuccess;
    // one workgroup per tile up to 64 per CU; the kernel strides over the rest
    int64_t blocks = int64_t(device_cu_count()) * 64;
    if (blocks > tiles) blocks = tiles;
    hipLaunchKernelGGL((gemv_a16_stream<B, UPG, RW, XDT, YDT, ROUTED, false>), dim3(unsigned(blocks)), dim3(nw * 64), lds,
                       stream, w.codes, w.scale, w.a, w.b, int(w.n), int(w.k), static_cast<const uint16_t *>(x), y,
                       rt.tok, rt.exp, rt.routes, rt.tokens, rt.n_experts);
    return hipGetLastError();
}

// Resident-activation launch: one wave per column block (at most 8), and
// about 16 waves per compute unit, each workgroup walking a multiple of
// kResBatch row tiles.
constexpr int kRowsRW = 2;

static size_t rows_lds_bytes(int bits, int64_t ncb) {
    const int64_t nt = (bits >= 3 && bits <= 5) ? (int64_t(1) << bits) : 1;
    return sizeof(float) * size_t(ncb * kRowsRW * nt * 64 + 2 * ncb * kResBatch * kRowsRW);
}

template <int B, int UPG, int XDT, int YDT>
static hipError_t rows_waves(const cq_weight &w, const void *x, void *y, hipStream_t stream) {
    const int64_t ncb = ((w.k >> 5) + 63) >> 6;
    const int64_t tiles = (w.n + kRowsRW - 1) / kRowsRW;
    if (tiles < 1) return hipSuccess;
    int64_t nb = int64_t(device_cu_count()) * 16 / ncb;
    if (nb < 1) nb = 1;
    int64_t per = (tiles + nb - 1) / nb;
    per = (per + kResBatch - 1) / kResBatch * kResBatch;
    const int64_t blocks = (tiles + per - 1) / per;
    hipLaunchKernelGGL((gemv_a16_stream<B, UPG, kRowsRW, XDT, YDT, false, true>), dim3(unsigned(blocks)),
                       dim3(unsigned(ncb * 64)), rows_lds_bytes(B, ncb), stream, w.codes, w.scale, w.a, w.b, int(w.n),
                       int(w.k), static_cast<const uint16_t *>(x), y, nullptr, nullptr, 0, 0, 0);
    return hipGetLastError();
}

template <int B, int UPG, int XDT, int YDT, bool ROUTED>
static hipError_t stream_rows(const cq_weight &w, const void *x, void *y, const StreamRoutes &rt,
                              hipStream_t stream) {
    // two rows per workgroup: the smallest tile keeps the most workgroups in
    // flight, which is what hides the load latency of a streaming GEMV
    return stream_waves<B, UPG, 2, XDT, YDT, ROUTED>(w, x, y, rt, stream);
}

template <int B, int XDT, int YDT>
static hipError_t rows_group(const cq_weight &w, const void *x, void *y, hipStream_t stream) {
    switch (w.group) {
        case 32: return rows_waves<B, 1, XDT, YDT>(w, x, y, stream);
        case 64: return rows_waves<B, 2, XDT, YDT>(w, x, y, stream);
        case 128: return rows_waves<B, 4, XDT, YDT>(w, x, y, stream);
        case 256: return rows_waves<B, 8, XDT, YDT>(w, x, y, stream);
        case 512: return rows_waves<B, 16, XDT, YDT>(w, x, y, stream);
    }
    return hipErrorNotSupported;
}

template <int XDT, int YDT>
static hipError_t rows_bits(const cq_weight &w, const void *x, void *y, hipStream_t stream) {
    switch (w.bits) {
        case 1: return rows_group<1, XDT, YDT>(w, x, y, stream);
        case 2: return rows_group<2, XDT, YDT>(w, x, y, stream);
        case 3: return rows_group<3, XDT, YDT>(w, x, y, stream);
        case 4: return rows_group<4, XDT, YDT>(w, x, y, stream);
        case 5: return rows_group<5, XDT, YDT>(w, x, y, stream);
        case 6: return rows_group<6, XDT, YDT>(w, x, y, stream);
        case 7: return rows_group<7, XDT, YDT>(w, x, y, stream);
        case 8: return rows_group<8, XDT, YDT>(w, x, y, stream);
    }
    return hipErrorNotSupported;
}

template <int B, int XDT, int YDT, bool ROUTED>
static hipError_t stream_group(const cq_weight &w, const void *x, void *y, const StreamRoutes &rt,
                               hipStream_t stream) {
    switch (w.group) {
        case 32: return stream_rows<B, 1, XDT, YDT, ROUTED>(w, x, y, rt, stream);
        case 64: return stream_rows<B, 2, XDT, YDT, ROUTED>(w, x, y, rt, stream);
        case 128: return stream_rows<B, 4, XDT, YDT, ROUTED>(w, x, y, rt, stream);
        case 256: return stream_rows<B, 8, XDT, YDT, ROUTED>(w, x, y, rt, stream);
        case 512: return stream_rows<B, 16, XDT, YDT, ROUTED>(w, x, y, rt, stream);
    }
    return hipErrorNotSupported;
}

template <int XDT, int YDT, bool ROUTED>
static hipError_t stream_bits(const cq_weight &w, const void *x, void *y, const StreamRoutes &rt,
                              hipStream_t stream) {
    switch (w.bits) {
        case 1: return stream_group<1, XDT, YDT, ROUTED>(w, x, y, rt, stream);
        case 2: return stream_group<2, XDT, YDT, ROUTED>(w, x, y, rt, stream);
        case 3: return stream_group<3, XDT, YDT, ROUTED>(w, x, y, rt, stream);
        case 4: return stream_group<4, XDT, YDT, ROUTED>(w, x, y, rt, stream);
        case 5: return stream_group<5, XDT, YDT, ROUTED>(w, x, y, rt, stream);
        case 6: return stream_group<6, XDT, YDT, ROUTED>(w, x, y, rt, stream);
        case 7: return stream_group<7, XDT, YDT, ROUTED>(w, x, y, rt, stream);
        case 8: return stream_group<8, XDT, YDT, ROUTED>(w, x, y, rt, stream);
    }
    return hipErrorNotSupported;
}

template <bool ROUTED>
static hipError_t stream_dtypes(const cq_weight &w, const void *x, int x_dt, void *y, int y_dt,
                                const StreamRoutes &rt, hipStream_t stream) {
    if (x_dt == 0) {
        if (y_dt == 0) return stream_bits<0, 0, ROUTED>(w, x, y, rt, stream);
        return stream_bits<0, 2, ROUTED>(w, x, y, rt, stream);
    }
    if (y_dt == 1) return stream_bits<1, 1, ROUTED>(w, x, y, rt, stream);
    return stream_bits<1, 2, ROUTED>(w, x, y, rt, stream);
}

bool gemv_a16_stream_supported(const cq_weight &w, int64_t m) {
    return m == 1 && stream_fits(w.n, w.k, w.bits, w.group);
}

hipError_t launch_gemv_a16_stream(const cq_weight &w, const void *x, int x_dt, void *y, int y_dt,
                                  hipStream_t stream) {
    return stream_dtypes<false>(w, x, x_dt, y, y_dt, StreamRoutes{}, stream);
}

bool gemv_a16_rows_supported(const cq_weight &w, int64_t m) {
    // a wave per column block within one workgroup of at most 8 waves (and
    // the W4 table slot tag), tables and batch sums within 64 KB of LDS
    const int64_t ncb = ((w.k >> 5) + 63) >> 6;
    return m == 1 && stream_fits(w.n, w.k, w.bits, w.group) && ncb <= 8 &&
           rows_lds_bytes(w.bits, ncb) <= size_t(64) * 1024;
}

bool gemv_a16_rows_preferred(const cq_weight &w, int64_t m) {
    if (!gemv_a16_rows_supported(w, m)) return false;
    // the resident slice pays off once each workgroup walks three or more row
    // tiles (measured on Llama-3-8B-shaped layers: faster on 4096 x 28672 and
    // 14336 x 4096, slower on 4096 x 4096 and 4096 x 6144)
    const int64_t ncb = ((w.k >> 5) + 63) >> 6;
    const int64_t nb = std::max<int64_t>(1, int64_t(256) * 16 / ncb);
    return (w.n + kRowsRW - 1) / kRowsRW >= 3 * nb;
}

hipError_t launch_gemv_a16_rows(const cq_weight &w, const void *x, int x_dt, void *y, int y_dt,
                                hipStream_t stream) {
    if (x_dt == 0) {
        if (y_dt == 0) return rows_bits<0, 0>(w, x, y, stream);
        return rows_bits<0, 2>(w, x, y, stream);
    }
    if (y_dt == 1) return rows_bits<1, 1>(w, x, y, stream);
    return rows_bits<1, 2>(w, x, y, stream);
}

bool gemv_a16_stream_routed_supported(const cq_weight &w, int64_t n_experts, int64_t tokens, int64_t routes) {
    const int64_t lim = int64_t(1) << 31;
    return stream_fits(w.n * n_experts, w.k, w.bits, w.group) && tokens * w.k * 2 < lim && routes * w.n < lim &&
           (w.n + 1) / 2 * routes < lim / 2;
}

hipError_t launch_gemv_a16_stream_routed(const cq_weight &w, int n_experts, const void *x, int x_dt, int64_t tokens,
                                         const int32_t *token, const int32_t *expert, int64_t routes, void *y,
                                         int y_dt, hipStream_t stream) {
    StreamRoutes rt;
    rt.tok = token;
    rt.exp = expert;
    rt.routes = int(routes);
    rt.tokens = int(tokens);
    rt.n_experts = n_experts;
    return stream_dtypes<true>(w, x, x_dt, y, y_dt, rt, stream);
}

}  // namespace cq
