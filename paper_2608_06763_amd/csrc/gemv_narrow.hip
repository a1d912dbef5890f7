// Narrow-row products (2 <= m <= 16) on gfx950 matrix cores, both paths.
//
// With m <= 16 activation rows every group is a dense m x G x 16 contraction
// for 16 weight rows, so the narrow-row regime (Sec. 5.3 and 5.4) maps onto
// 16 x 16 MFMA blocks whose weight operand is decoded straight into registers:
// no LDS staging of decoded weights, and the decode cost per weight does not
// depend on m.
//
// Work mapping.  A workgroup owns a strip of 16 weight rows; its 4..16 waves
// (chosen by the host so that the grid holds about eight waves per SIMD) take
// the groups of K round-robin and add their 16 x 16 FP32 partial tiles
// through LDS at the end.  In a wave, lane l serves weight row l % 16
// (the MFMA column) and K slots 16 (l / 16) .. +15 of a 64-slot step (A8) or
// 8 (l / 16) .. +7 of a 32-slot step (model dtype).  Activation rows past m
// and weight rows past n load out-of-range offsets and read zeros.
//
// Dynamic-A8 (eq. a8-output), W4, G >= 64: each lane decodes its 16 codes to
// exact INT8 carriers with the register tables of a8_carriers.h (the four
// lanes of a row each evaluate two of the row's carriers and gather the rest
// with ds_bpermute); v_mfma_i32_16x16x64_i8 accumulates exact INT32 group
// partials, which are scaled by s_g in FP32 at the end of each group.
//
// Model dtype (Sec. 5.3), B <= 5: the four lanes of a row build the row's
// table of the 2^B levels s_g sign(k) q(|k|/M) for each group in LDS, each an
// unevaluated hi + lo pair in the activation dtype (16 or 22 significant bits,
// so the products keep the FP32 quality of the narrow-row tactic); every code
// costs one LDS read and both halves feed v_mfma_f32_16x16x32_{bf16,f16}.
#include <algorithm>

#include "cq_device.h"
#include "cq_internal.h"
#include "stream_common.h"
#include "a8_carriers.h"

namespace cq {

namespace {

typedef int i32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));

constexpr int kMaxWaves = 16;  // waves per workgroup (one 16-row strip), chosen by the host

__device__ __forceinline__ uint32_t lane_read(uint32_t v, int src_lane) {
    return uint32_t(__builtin_amdgcn_ds_bpermute(src_lane << 2, int(v)));
}

__device__ __forceinline__ void wave_lds_order() {
    __asm__ __volatile__("" ::: "memory");
    __builtin_amdgcn_wave_barrier();
}

// Sum the waves' 16 x 16 tiles (lane l holds rows 4 (l / 16) + i, column
// l % 16) and store rows < m of the 16-row strip.
template <int YDT>
__device__ __forceinline__ void reduce_store(float (*red)[16][17], const float v[4], int lane, int wave, int nwaves,
                                             int n0, int n, int m, const float *row_factor, void *y,
                                             const int *out_row = nullptr) {
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][4 * (lane >> 4) + i][lane & 15] = v[i];
    __syncthreads();
    for (int e = threadIdx.x; e < 256; e += blockDim.x) {
        const int r = e >> 4, c = e & 15;
        if (r < m && n0 + c < n) {
            float s = 0.f;
            for (int w = 0; w < nwaves; ++w) s += red[w][r][c];
            if (row_factor) s *= row_factor[r];
            store_out<YDT>(y, int64_t(out_row ? out_row[r] : r) * n + n0 + c, s);
        }
    }
}

// Route map of a routed product, grouped by expert (see routed.hip).  The
// routed kernel keeps its route chunk state in registers: at most 8 waves.
constexpr int kMaxRoutedWaves = 8;
struct route_groups {
    const int32_t *token;    // [R] activation row of each route
    const int32_t *order;    // route ids grouped by expert
    const int32_t *offsets;  // [E + 1] first entry of each expert in order
    int strips;              // 16-row strips per expert
};

}  // namespace

// ---------------------------------------------------------------- Dynamic-A8, W3 and W4

// W3: a lane's 16 codes of a step are 6 bytes at an even byte offset, inside
// one aligned 8-byte window; every lane evaluates the two interior carriers
// r(1), r(2) of its group itself, and four fields at a time, spread into
// selector bytes, index the pair [r0 r1 r2 r3 | 0 -r3 -r2 -r1] with one byte
// permute (the reserved pattern selects the 0), giving carriers in field order.
// XB = 2 (17..32 rows): every decoded weight operand feeds the MFMAs of two
// 16-row blocks of x; at most 8 waves per strip.
template <int B, int UPG, int YDT, int XB>
__global__ void __launch_bounds__(UPG >= 16 || XB == 2 ? 512 : 1024) gemv_a8_narrow(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int n, int k, const int8_t *__restrict__ x8, const float *__restrict__ dx, int m, void *__restrict__ y) {
    static_assert(B == 3 || B == 4, "narrow-row A8 widths");
    static_assert(XB == 1 || XB == 2, "one or two 16-row blocks of x");
    constexpr int M = max_code(B);
    constexpr int SPG = UPG / 2;  // 64-slot steps per group
    constexpr int kRedWaves = (UPG >= 16 || XB == 2) ? 8 : kMaxWaves;
    __shared__ float red[kRedWaves][16 * XB][17];
    __shared__ float fac[16 * XB];

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int nwaves = blockDim.x >> 6;
    const int n0 = blockIdx.x * 16;
    const int col = lane & 15;     // weight row of the strip / activation row
    const int part = lane >> 4;    // K part of a step
    const int wrow = n0 + col;
    const bool wok = wrow < n;
    const int ng = k / (32 * UPG);
    const uint32_t row_bytes = uint32_t(k) * B / 8u;
    const auto rc = make_rsrc(codes, uint32_t(n) * row_bytes);
    const auto rs = make_rsrc(scale, uint32_t(n) * ng * 4u);
    const auto ra = make_rsrc(a16, uint32_t(n) * ng * 2u);
    const auto rb = make_rsrc(b16, uint32_t(n) * ng * 2u);
    const auto rx = make_rsrc(x8, uint32_t(m) * uint32_t(k));
    if (threadIdx.x < 16 * XB) fac[threadIdx.x] = int(threadIdx.x) < m ? dx[threadIdx.x] / 127.0f : 0.f;

    // carriers of pair `part` of the row: magnitudes 2 part, 2 part + 1
    const int i0 = 2 * part;
    const float t0 = float(i0) / float(M), t1 = float(i0 + 1) / float(M);

    // A wave takes a contiguous run of groups.  Per group it loads the
    // strip's code bytes as whole pieces (PS bytes; consecutive lanes on
    // consecutive bytes of a row, so each quad of lanes reads one run of a
    // row), writes them to its own LDS staging rows and reads each lane's
    // slice back; only the wave touches its staging rows, so program order
    // orders the writes and reads.  The group metadata of the strip come in
    // batches of four groups (lane l: row l / 4, group l % 4) and reach their
    // lanes by ds_bpermute.  The codes and activations of the next group, and
    // the metadata of the next batch, are requested before the current group
    // is decoded (two register stages, the loop unrolled by two).
    constexpr int GB = 32 * UPG * B / 8;         // code bytes of one row in one group
    constexpr int PS = GB % 16 == 0 ? 16 : 8;    // bytes per piece
    constexpr int PPR = GB / PS;                 // pieces per row
    constexpr int NP = 16 * PPR;                 // pieces per group
    constexpr int NL = (NP + 63) / 64;           // piece loads per lane
    constexpr int RS = GB + 16;                  // staged row stride (bytes)
    constexpr int kStgWaves = kRedWaves;
    __shared__ __attribute__((aligned(16))) uint32_t stg[kStgWaves * 16 * RS / 4];
    uint8_t *const mystg = reinterpret_cast<uint8_t *>(stg) + wave * (16 * RS);
    const int gper = (ng + nwaves - 1) / nwaves;
    const int gbeg = min(ng, wave * gper), gend = min(ng, gbeg + gper);

    struct Stage {
        uint32_t pc[NL][PS / 4];
        u32x4_t xa[XB][SPG];
    };
    auto load = [&](int g, Stage &st) {
#pragma unroll
        for (int t = 0; t < NL; ++t) {
            const int pi = t * 64 + lane;
            const int wr = n0 + pi / PPR;
            const bool ok = pi < NP && wr < n;
            load_words<PS / 4>(rc, ok ? uint32_t(wr) * row_bytes + uint32_t(g) * GB + uint32_t(pi % PPR) * PS
                                      : kOobOffset, st.pc[t]);
        }
#pragma unroll
        for (int bx = 0; bx < XB; ++bx) {
            const int xrow = 16 * bx + col;
#pragma unroll
            for (int q = 0; q < SPG; ++q) {
                const uint32_t kk = uint32_t(g) * (32u * UPG) + 64u * q + 16u * part;
                uint32_t xv[4];
                load_words<4>(rx, xrow < m ? uint32_t(xrow) * uint32_t(k) + kk : kOobOffset, xv);
                st.xa[bx][q] = u32x4_t{xv[0], xv[1], xv[2], xv[3]};
            }
        }
    };
    // metadata of groups gb .. gb + 3 of the strip: scale, and a | b << 16
    float ms_c = 0.f, ms_n = 0.f;
    uint32_t mab_c = 0, mab_n = 0;
    auto load_meta = [&](int gb, float &ms, uint32_t &mab) {
        const int r = n0 + (lane >> 2), gg = gb + (lane & 3);
        const bool ok = r < n && gg < ng;
        const uint32_t gi = uint32_t(r) * ng + gg;
        ms = load_f32(rs, ok ? gi * 4u : kOobOffset);
        mab = load_u16(ra, ok ? gi * 2u : kOobOffset) | (load_u16(rb, ok ? gi * 2u : kOobOffset) << 16);
    };
    float accf[XB][4];
#pragma unroll
    for (int bx = 0; bx < XB; ++bx)
#pragma unroll
        for (int i = 0; i < 4; ++i) accf[bx][i] = 0.f;
    auto process = [&](int g, const Stage &st) {
        const int j = (g - gbeg) & 3;
        if (j == 0 && g != gbeg) {
            ms_c = ms_n;
            mab_c = mab_n;
            if (g + 4 < gend) load_meta(g + 4, ms_n, mab_n);
        }
        const float s = __int_as_float(int(lane_read(__float_as_uint(ms_c), 4 * col + j)));
        const uint32_t ab = lane_read(mab_c, 4 * col + j);
        const float a = f16_to_f32(uint16_t(ab & 0xffffu)), b = f16_to_f32(uint16_t(ab >> 16));
        // stage the group's code pieces, then read this lane's slices
#pragma unroll
        for (int t = 0; t < NL; ++t) {
            const int pi = t * 64 + lane;
            if (pi < NP) {
                uint8_t *dst = mystg + (pi / PPR) * RS + (pi % PPR) * PS;
                if constexpr (PS == 16)
                    *reinterpret_cast<u32x4_t *>(dst) = u32x4_t{st.pc[t][0], st.pc[t][1], st.pc[t][2], st.pc[t][3]};
                else
                    *reinterpret_cast<uint2 *>(dst) = make_uint2(st.pc[t][0], st.pc[t][1]);
            }
        }
        wave_lds_order();
        uint32_t cw[SPG][2];
#pragma unroll
        for (int q = 0; q < SPG; ++q) {
            // W4: 8 code bytes at 32 q + 8 part; W3: the aligned window of the
            // 6 code bytes at 24 q + 6 part
            const int o = B == 4 ? 32 * q + 8 * part : (24 * q + 6 * part) & ~3;
            const uint32_t *src = reinterpret_cast<const uint32_t *>(mystg + col * RS + o);
            cw[q][0] = src[0];
            cw[q][1] = src[1];
        }
        wave_lds_order();
        const float c = 1.f - a - b;
        const float mg = carrier_margin(a, b, c);
        i32x4_t acc[XB];
#pragma unroll
        for (int bx = 0; bx < XB; ++bx) acc[bx] = i32x4_t{0, 0, 0, 0};
        if constexpr (B == 4) {
            const uint32_t pr = carrier_u8<M>(i0, t0, a, b, c, mg) | (carrier_u8<M>(i0 + 1, t1, a, b, c, mg) << 8);
            const uint32_t p0 = lane_read(pr, col), p1 = lane_read(pr, col + 16);
            const uint32_t p2 = lane_read(pr, col + 32), p3 = lane_read(pr, col + 48);
            const uint32_t ta0 = p0 | (p1 << 16), ta1 = p2 | (p3 << 16);
            uint32_t tb0, tb1;
            w4_negative_table(ta0, ta1, tb0, tb1);
#pragma unroll
            for (int q = 0; q < SPG; ++q) {
                uint32_t cr[4];
                w4_word_carriers(cw[q][0], ta0, ta1, tb0, tb1, cr[0], cr[1]);
                w4_word_carriers(cw[q][1], ta0, ta1, tb0, tb1, cr[2], cr[3]);
                const i32x4_t bop = {int(cr[0]), int(cr[1]), int(cr[2]), int(cr[3])};
#pragma unroll
                for (int bx = 0; bx < XB; ++bx)
                    acc[bx] = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4_t, st.xa[bx][q]), bop, acc[bx],
                                                                    0, 0, 0);
            }
        } else {
            const uint32_t r12 = carrier_u8<M>(1, 1.f / 3.f, a, b, c, mg) | (carrier_u8<M>(2, 2.f / 3.f, a, b, c, mg) << 8);
            const uint32_t ta = (r12 << 8) | 0x7f000000u;             // r0 r1 r2 r3
            const uint32_t neg = (0x80808080u - ta) ^ 0x80808080u;  // 0 -r1 -r2 -r3
            const uint32_t tb = perm(neg, neg, 0x01020300u);        // 0 -r3 -r2 -r1
            // the window starts at the 6 code bytes, or 2 bytes before them
            const uint32_t sh = (part & 1) ? 16u : 0u;
#pragma unroll
            for (int q = 0; q < SPG; ++q) {
                const uint32_t lo = __builtin_amdgcn_alignbit(cw[q][1], cw[q][0], sh);  // fields 0..10
                const uint32_t hi = cw[q][1] >> sh;                                     // bits 32..47
                uint32_t cr[4];
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    uint32_t x;
                    if (t < 2) x = lo >> (12 * t);
                    else if (t == 2) x = __builtin_amdgcn_alignbit(hi, lo, 24);
                    else x = hi >> 4;
                    x &= 0xfffu;  // fields 4t .. 4t + 3
                    const uint32_t sel =
                        (x & 7u) | ((x << 5) & 0x700u) | ((x << 10) & 0x70000u) | ((x << 15) & 0x7000000u);
                    cr[t] = perm(tb, ta, sel);
                }
                const i32x4_t bop = {int(cr[0]), int(cr[1]), int(cr[2]), int(cr[3])};
#pragma unroll
                for (int bx = 0; bx < XB; ++bx)
                    acc[bx] = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4_t, st.xa[bx][q]), bop, acc[bx],
                                                                    0, 0, 0);
            }
        }
        // rows of acc are activation rows, its column this lane's weight row
#pragma unroll
        for (int bx = 0; bx < XB; ++bx)
#pragma unroll
            for (int i = 0; i < 4; ++i) accf[bx][i] = __builtin_fmaf(s, float(acc[bx][i]), accf[bx][i]);
    };
    Stage s0, s1;
    if (gbeg < gend) {
        load_meta(gbeg, ms_c, mab_c);
        if (gbeg + 4 < gend) load_meta(gbeg + 4, ms_n, mab_n);
        load(gbeg, s0);
    }
    for (int g = gbeg; g < gend; g += 2) {
        if (g + 1 < gend) load(g + 1, s1);
        process(g, s0);
        if (g + 1 >= gend) break;
        if (g + 2 < gend) load(g + 2, s0);
        process(g + 1, s1);
    }
    // the scale loaded above is this lane's column (weight row), so the
    // rescale above is s_{n,g} P_g for output (row 16 bx + 4 part + i, column
    // col); the waves' tiles meet in LDS
#pragma unroll
    for (int bx = 0; bx < XB; ++bx)
#pragma unroll
        for (int i = 0; i < 4; ++i) red[wave][16 * bx + 4 * part + i][col] = accf[bx][i];
    __syncthreads();
    for (int e = threadIdx.x; e < 256 * XB; e += blockDim.x) {
        const int r = e >> 4, c = e & 15;
        if (r < m && n0 + c < n) {
            float sum = 0.f;
            for (int wv = 0; wv < nwaves; ++wv) sum += red[wv][r][c];
            store_out<YDT>(y, int64_t(r) * n + n0 + c, sum * fac[r]);
        }
    }
}

// ---------------------------------------------------------------- model dtype, B <= 5

// ROUTED: a bank of experts of n rows each, stacked; block b serves strip
// b % strips of expert b / strips for all routes of that expert, 16 routes
// (gathered activation rows) at a time; outputs are route-major rows.  x then
// has m rows (tokens).
template <int B, int UPG, int XDT, int YDT, bool ROUTED>
__global__ void __launch_bounds__(ROUTED ? 64 * kMaxRoutedWaves : 1024) gemv_a16_narrow(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int n, int k, const uint16_t *__restrict__ x, int m, void *__restrict__ y, route_groups rg) {
    constexpr int M = max_code(B);
    constexpr int NE = 1 << B;
    constexpr int EPT = NE >= 4 ? NE / 4 : 1;
    constexpr int TSTR = NE + 1;
    __shared__ float red[kMaxWaves][16][17];
    __shared__ uint32_t tab[kMaxWaves][16 * TSTR];

    __shared__ int out_row[16];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int nwaves = blockDim.x >> 6;
    const int ng = k / (32 * UPG);
    const uint32_t row_bytes = uint32_t(k) * B / 8u;
    int strip = blockIdx.x, r_begin = 0, r_end = m;
    if constexpr (ROUTED) {
        const int e = blockIdx.x / rg.strips;
        strip = blockIdx.x % rg.strips;
        r_begin = rg.offsets[e];
        r_end = rg.offsets[e + 1];
        codes += size_t(e) * n * row_bytes;
        scale += size_t(e) * n * ng;
        a16 += size_t(e) * n * ng;
        b16 += size_t(e) * n * ng;
    }
    const int n0 = strip * 16;
    const int col = lane & 15;
    const int part = lane >> 4;
    const int wrow = n0 + col;
    const bool wok = wrow < n;
    const auto rc = make_rsrc(codes, uint32_t(n) * row_bytes);
    const auto rs = make_rsrc(scale, uint32_t(n) * ng * 4u);
    const auto ra = make_rsrc(a16, uint32_t(n) * ng * 2u);
    const auto rb = make_rsrc(b16, uint32_t(n) * ng * 2u);
    const auto rx = make_rsrc(x, uint32_t(m) * uint32_t(k) * 2u);
    uint32_t *mytab = tab[wave] + col * TSTR;
    // activation row of this lane's MFMA row in the current chunk of routes
    int xrow = col;
    bool xok = col < m;

    // Items are (group, batch of at most four units); a wave walks the items
    // of its groups g = wave, wave + 4, ... and requests the next item's codes,
    // activations and metadata before decoding the current one (two register
    // stages, the loop unrolled by two).
    constexpr int QB = UPG < 4 ? UPG : 4;   // units per item
    constexpr int NB = UPG / QB;            // items per group
    // The 8 codes of this lane in a unit are the B bytes at byte B * part of
    // the unit; an aligned 8-byte window holds them (B <= 5), so each unit
    // costs one 64-bit load and the fields come out with 64-bit shifts.
    struct Stage {
        uint32_t cw[QB][2];
        u32x4_t xa[QB];
        float s, a, b;
    };
    const uint32_t part_byte = uint32_t(B * part);
    const uint32_t win_shift = 8u * (part_byte & 3u);   // bit of the first field in the window
    const int my_groups = wave < ng ? (ng - 1 - wave) / nwaves + 1 : 0;
    const int items = my_groups * NB;
    auto load = [&](int it, Stage &st) {
        const int g = wave + (it / NB) * nwaves;
        const int q0 = (it % NB) * QB;
        {
            // every item carries its group's metadata (a cache hit after the first batch)
            const uint32_t gi = uint32_t(wrow) * ng + g;
            st.s = load_f32(rs, wok ? gi * 4u : kOobOffset);
            st.a = 1.f;
            st.b = 0.f;
            if constexpr (B >= 3) {
                st.a = f16_to_f32(uint16_t(load_u16(ra, wok ? gi * 2u : kOobOffset)));
                st.b = f16_to_f32(uint16_t(load_u16(rb, wok ? gi * 2u : kOobOffset)));
            }
        }
#pragma unroll
        for (int q = 0; q < QB; ++q) {
            const uint32_t u = uint32_t(g) * UPG + q0 + q;  // unit index along K
            const uint32_t byte0 = uint32_t(wrow) * row_bytes + u * (4u * B) + part_byte;
            load_words<2>(rc, wok ? (byte0 & ~3u) : kOobOffset, st.cw[q]);
            uint32_t xv[4];
            load_words<4>(rx, xok ? (uint32_t(xrow) * uint32_t(k) + u * 32u + 8u * part) * 2u : kOobOffset, xv);
            st.xa[q] = u32x4_t{xv[0], xv[1], xv[2], xv[3]};
        }
    };
    f32x4_t acc;
    auto process = [&](int it, const Stage &st) {
        if (it % NB == 0) {
            // the row's level table: lane part of the row writes fields part, part + 4, ...
            const float a = st.a, b = st.b;
            const float c = 1.f - a - b;
            wave_lds_order();  // the previous group's reads are issued
#pragma unroll
            for (int e = 0; e < EPT; ++e) {
                const int f = part + 4 * e;
                if (f < NE) {
                    const int kc = field_to_code(uint32_t(f), B);
                    const float v = st.s * ((B == 1) ? float(kc) : signed_level(kc, M, a, b, c));
                    uint32_t ent;
                    if constexpr (XDT == 0) {
                        const __bf16 hi = __bf16(v);
                        const __bf16 lo = __bf16(v - float(hi));
                        ent = uint32_t(__builtin_bit_cast(uint16_t, hi)) |
                              (uint32_t(__builtin_bit_cast(uint16_t, lo)) << 16);
                    } else {
                        const _Float16 hi = _Float16(v);
                        const _Float16 lo = _Float16(v - float(hi));
                        ent = uint32_t(__builtin_bit_cast(uint16_t, hi)) |
                              (uint32_t(__builtin_bit_cast(uint16_t, lo)) << 16);
                    }
                    mytab[f] = ent;
                }
            }
            wave_lds_order();
        }
#pragma unroll
        for (int q = 0; q < QB; ++q) {
            uint32_t ent[8];
            const uint64_t win = (uint64_t(st.cw[q][1]) << 32) | st.cw[q][0];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const uint32_t v = uint32_t(win >> (win_shift + uint32_t(B * e)));
                ent[e] = mytab[v & uint32_t(NE - 1)];
            }
            u32x4_t hi, lo;
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                hi[p] = __builtin_amdgcn_perm(ent[2 * p + 1], ent[2 * p], 0x05040100u);
                lo[p] = __builtin_amdgcn_perm(ent[2 * p + 1], ent[2 * p], 0x07060302u);
            }
            if constexpr (XDT == 0) {
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, st.xa[q]),
                                                              __builtin_bit_cast(bf16x8_t, hi), acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, st.xa[q]),
                                                              __builtin_bit_cast(bf16x8_t, lo), acc, 0, 0, 0);
            } else {
                acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, st.xa[q]),
                                                             __builtin_bit_cast(f16x8_t, hi), acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, st.xa[q]),
                                                             __builtin_bit_cast(f16x8_t, lo), acc, 0, 0, 0);
            }
        }
    };
    auto run_rows = [&](int mc) {
        acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
        Stage s0, s1;
        if (items > 0) load(0, s0);
        for (int it = 0; it < items; it += 2) {
            if (it + 1 < items) load(it + 1, s1);
            process(it, s0);
            if (it + 1 >= items) break;
            if (it + 2 < items) load(it + 2, s0);
            process(it + 1, s1);
        }
        const float v[4] = {acc[0], acc[1], acc[2], acc[3]};
        reduce_store<YDT>(red, v, lane, wave, nwaves, n0, n, mc, nullptr, y, ROUTED ? out_row : nullptr);
    };
    if constexpr (ROUTED) {
        for (int j = r_begin; j < r_end; j += 16) {
            const int mc = min(16, r_end - j);
            const int rid = col < mc ? rg.order[j + col] : 0;
            xrow = col < mc ? rg.token[rid] : 0;
            xok = col < mc;
            if (threadIdx.x < 16) out_row[threadIdx.x] = threadIdx.x < mc ? rg.order[j + threadIdx.x] : 0;
            run_rows(mc);
            __syncthreads();  // red, the tables and out_row are reused by the next chunk
        }
    } else {
        run_rows(m);
    }
}

// ---------------------------------------------------------------- launchers

// Waves per 16-row strip: enough strips x waves to give every SIMD about eight
// waves of work (latency hiding), at least four, at most sixteen, and no more
// than there are groups along K.
static int narrow_waves(const cq_weight &w, int max_waves = kMaxWaves) {
    const int64_t strips = (w.n + 15) / 16;
    const int64_t ng = w.k / w.group;
    int64_t want = (int64_t(device_cu_count()) * 4 * 8 + strips - 1) / strips;
    int nw = 4;
    while (nw < max_waves && nw < want) nw *= 2;
    while (nw > 1 && nw > ng) nw /= 2;
    return nw;
}

template <int B, int UPG, int YDT, int XB>
static hipError_t a8_narrow_launch_x(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                                     hipStream_t stream) {
    const int64_t blocks = (w.n + 15) / 16;
    // G = 512 keeps two stages of eight 64-code steps in registers: at most 8 waves;
    // each wave takes a contiguous run of groups, and its metadata come in
    // batches of four: at most one wave per four groups (measured: qkv-sized
    // layers 20% faster with four groups per wave than with two)
    const int64_t ng = w.k / w.group;
    const int cap = int(std::min<int64_t>(UPG >= 16 || XB == 2 ? 8 : kMaxWaves, std::max<int64_t>(4, ng / 4)));
    int nw = narrow_waves(w, cap);
    if constexpr (B == 4 && UPG == 4 && XB == 1) {
        // W4 G128, one x block: fewer, longer runs where the grid still holds
        // three or more waves per SIMD, down to about eight groups per wave
        // (measured on 4096 x 28672: 22.6 -> 21.0 us at 4 rows with four waves
        // instead of eight; 8192 x 28672, 14336 x 4096 and 4096 x 6144 keep
        // the count above)
        const int64_t strips = (w.n + 15) / 16;
        const int64_t need = std::max<int64_t>(ng / 8, (int64_t(device_cu_count()) * 4 * 3 + strips - 1) / strips);
        int lean = 4;
        while (lean < nw && lean < need) lean *= 2;
        nw = std::min(nw, lean);
    }
    hipLaunchKernelGGL((gemv_a8_narrow<B, UPG, YDT, XB>), dim3(unsigned(blocks)), dim3(64 * nw), 0, stream, w.codes, w.scale,
                       w.a, w.b, int(w.n), int(w.k), x8, dx, int(m), y);
    return hipGetLastError();
}

template <int B, int UPG, int YDT>
static hipError_t a8_narrow_launch(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                                   hipStream_t stream) {
    if (m > 16) return a8_narrow_launch_x<B, UPG, YDT, 2>(w, x8, dx, m, y, stream);
    return a8_narrow_launch_x<B, UPG, YDT, 1>(w, x8, dx, m, y, stream);
}

template <int B, int YDT>
static hipError_t a8_narrow_group(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                                  hipStream_t stream) {
    switch (w.group) {
        case 64: return a8_narrow_launch<B, 2, YDT>(w, x8, dx, m, y, stream);
        case 128: return a8_narrow_launch<B, 4, YDT>(w, x8, dx, m, y, stream);
        case 256: return a8_narrow_launch<B, 8, YDT>(w, x8, dx, m, y, stream);
        case 512: return a8_narrow_launch<B, 16, YDT>(w, x8, dx, m, y, stream);
    }
    return hipErrorNotSupported;
}

template <int YDT>
static hipError_t a8_narrow_bits(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                                 hipStream_t stream) {
    if (w.bits == 3) return a8_narrow_group<3, YDT>(w, x8, dx, m, y, stream);
    if (w.bits == 4) return a8_narrow_group<4, YDT>(w, x8, dx, m, y, stream);
    return hipErrorNotSupported;
}

bool gemv_a8_narrow_supported(const cq_weight &w, int64_t m) {
    return m >= 2 && m <= 32 && (w.bits == 3 || w.bits == 4) && w.group >= 64 && stream_fits(w.n, w.k, w.bits, w.group) &&
           m * w.k < (int64_t(1) << 31);
}

hipError_t launch_gemv_a8_narrow(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y, int y_dt,
                                 hipStream_t stream) {
    if (y_dt == 0) return a8_narrow_bits<0>(w, x8, dx, m, y, stream);
    if (y_dt == 1) return a8_narrow_bits<1>(w, x8, dx, m, y, stream);
    return a8_narrow_bits<2>(w, x8, dx, m, y, stream);
}

template <int B, int UPG, int XDT, int YDT>
static hipError_t a16_narrow_launch(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    const int64_t blocks = (w.n + 15) / 16;
    hipLaunchKernelGGL((gemv_a16_narrow<B, UPG, XDT, YDT, false>), dim3(unsigned(blocks)), dim3(64 * narrow_waves(w)), 0,
                       stream, w.codes, w.scale, w.a, w.b, int(w.n), int(w.k), static_cast<const uint16_t *>(x), int(m), y,
                       route_groups{});
    return hipGetLastError();
}

template <int B, int XDT, int YDT>
static hipError_t a16_narrow_group(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    switch (w.group) {
        case 32: return a16_narrow_launch<B, 1, XDT, YDT>(w, x, m, y, stream);
        case 64: return a16_narrow_launch<B, 2, XDT, YDT>(w, x, m, y, stream);
        case 128: return a16_narrow_launch<B, 4, XDT, YDT>(w, x, m, y, stream);
        case 256: return a16_narrow_launch<B, 8, XDT, YDT>(w, x, m, y, stream);
        case 512: return a16_narrow_launch<B, 16, XDT, YDT>(w, x, m, y, stream);
    }
    return hipErrorNotSupported;
}

template <int XDT, int YDT>
static hipError_t a16_narrow_bits(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    switch (w.bits) {
        case 1: return a16_narrow_group<1, XDT, YDT>(w, x, m, y, stream);
        case 2: return a16_narrow_group<2, XDT, YDT>(w, x, m, y, stream);
        case 3: return a16_narrow_group<3, XDT, YDT>(w, x, m, y, stream);
        case 4: return a16_narrow_group<4, XDT, YDT>(w, x, m, y, stream);
        case 5: return a16_narrow_group<5, XDT, YDT>(w, x, m, y, stream);
    }
    return hipErrorNotSupported;
}

bool gemv_a16_narrow_supported(const cq_weight &w, int64_t m) {
    return m >= 2 && m <= 16 && w.bits <= 5 && stream_fits(w.n, w.k, w.bits, w.group) &&
           m * w.k * 2 < (int64_t(1) << 31);
}

template <int B, int UPG, int XDT, int YDT>
static hipError_t a16_routed_launch(const cq_weight &w, int n_experts, const void *x, int64_t tokens,
                                    const int32_t *token, const int32_t *order, const int32_t *offsets, void *y,
                                    hipStream_t stream) {
    const int strips = int((w.n + 15) / 16);
    const int64_t blocks = int64_t(strips) * n_experts;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemv_a16_narrow<B, UPG, XDT, YDT, true>), dim3(unsigned(blocks)),
                       dim3(64 * narrow_waves(w, kMaxRoutedWaves)), 0,
                       stream, w.codes, w.scale, w.a, w.b, int(w.n), int(w.k), static_cast<const uint16_t *>(x),
                       int(tokens), y, route_groups{token, order, offsets, strips});
    return hipGetLastError();
}

template <int B, int XDT, int YDT>
static hipError_t a16_routed_group(const cq_weight &w, int n_experts, const void *x, int64_t tokens,
                                   const int32_t *token, const int32_t *order, const int32_t *offsets, void *y,
                                   hipStream_t stream) {
    switch (w.group) {
        case 32: return a16_routed_launch<B, 1, XDT, YDT>(w, n_experts, x, tokens, token, order, offsets, y, stream);
        case 64: return a16_routed_launch<B, 2, XDT, YDT>(w, n_experts, x, tokens, token, order, offsets, y, stream);
        case 128: return a16_routed_launch<B, 4, XDT, YDT>(w, n_experts, x, tokens, token, order, offsets, y, stream);
        case 256: return a16_routed_launch<B, 8, XDT, YDT>(w, n_experts, x, tokens, token, order, offsets, y, stream);
        case 512: return a16_routed_launch<B, 16, XDT, YDT>(w, n_experts, x, tokens, token, order, offsets, y, stream);
    }
    return hipErrorNotSupported;
}

template <int XDT, int YDT>
static hipError_t a16_routed_bits(const cq_weight &w, int n_experts, const void *x, int64_t tokens,
                                  const int32_t *token, const int32_t *order, const int32_t *offsets, void *y,
                                  hipStream_t stream) {
    switch (w.bits) {
        case 1: return a16_routed_group<1, XDT, YDT>(w, n_experts, x, tokens, token, order, offsets, y, stream);
        case 2: return a16_routed_group<2, XDT, YDT>(w, n_experts, x, tokens, token, order, offsets, y, stream);
        case 3: return a16_routed_group<3, XDT, YDT>(w, n_experts, x, tokens, token, order, offsets, y, stream);
        case 4: return a16_routed_group<4, XDT, YDT>(w, n_experts, x, tokens, token, order, offsets, y, stream);
        case 5: return a16_routed_group<5, XDT, YDT>(w, n_experts, x, tokens, token, order, offsets, y, stream);
    }
    return hipErrorNotSupported;
}

bool gemv_a16_routed_supported(const cq_weight &w, int64_t tokens) {
    return w.bits <= 5 && stream_fits(w.n, w.k, w.bits, w.group) && tokens * w.k * 2 < (int64_t(1) << 31);
}

hipError_t launch_gemv_a16_routed(const cq_weight &w, int n_experts, const void *x, int x_dt, int64_t tokens,
                                  const int32_t *token, const int32_t *order, const int32_t *offsets, void *y,
                                  int y_dt, hipStream_t stream) {
    if (x_dt == 0) {
        if (y_dt == 0) return a16_routed_bits<0, 0>(w, n_experts, x, tokens, token, order, offsets, y, stream);
        return a16_routed_bits<0, 2>(w, n_experts, x, tokens, token, order, offsets, y, stream);
    }
    if (y_dt == 1) return a16_routed_bits<1, 1>(w, n_experts, x, tokens, token, order, offsets, y, stream);
    return a16_routed_bits<1, 2>(w, n_experts, x, tokens, token, order, offsets, y, stream);
}

hipError_t launch_gemv_a16_narrow(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                  hipStream_t stream) {
    if (x_dt == 0) {
        if (y_dt == 0) return a16_narrow_bits<0, 0>(w, x, m, y, stream);
        return a16_narrow_bits<0, 2>(w, x, m, y, stream);
    }
    if (y_dt == 1) return a16_narrow_bits<1, 1>(w, x, m, y, stream);
    return a16_narrow_bits<1, 2>(w, x, m, y, stream);
}

}  // namespace cq
