// Dynamic-A8 single-row GEMV, streaming byte-permute family (Sec. 5.4) for
// m == 1 and every B.
//
// Numerics are those of eq. a8-output: every weight contributes the INT8
// carrier r(k) = sign(k) RNE(127 q(|k|/M)) (eq. carrier, Appendix A item 7)
// times the INT8 activation, summed exactly in INT32 over a 32-code unit (a
// K-tile partial of the group partial P_g, which Sec. 5.4 allows); each unit
// partial is converted to FP32 and weighted by s_g, and the row factor
// d_x / 127 multiplies the FP32 sum.
//
// Work mapping: identical to the model-dtype streaming GEMV (lane l owns unit
// l of a 2048-code column block, RW rows per workgroup tile, waves split the
// column blocks and meet in LDS, the next item's codes are requested before
// the current item is decoded).
//
// Decode without memory tables: W4 carriers come from two 8-byte tables held
// in registers and looked up with byte permutes (a8_carriers.h), multiplied
// with four activations at a time by v_dot4_i32_i8.  The carriers of a group
// are computed once per (row, group): the group's lanes each evaluate two
// magnitudes and share them through quad DPP moves.  W3: every lane evaluates
// the two interior carriers itself; a field indexes the 8-byte pair
// [r0 r1 r2 r3 | 0 -r3 -r2 -r1] directly once four fields are spread into
// bytes, and the carriers come out in field order.  W2 and W1 use constant
// tables ({0, 127, 0, -127} and {-127, 127}).  W5..W8 (16..128 magnitudes per
// group, more than a group's 32-code unit uses) evaluate each weight's carrier
// from its own magnitude, exact near ties as everywhere else.
//
// Fused quantization (FX >= 0, B <= 4): the kernel takes the BF16/FP16 activation row
// itself and forms its carriers in a prologue, so that a single-row A8 product
// is one launch (the activation encoding is the fixed cost of the single-row
// A8 path, Sec. 6).  Every workgroup reduces the whole row to its maximum
// magnitude (order-free, so every workgroup gets the same d_x): wave w of a
// workgroup owns column block w for the whole launch, so the 32 activations of
// each lane's unit, read once, give both the row maximum and the carriers,
// which are formed with the standalone quantizer's results (a8_quant.h: a
// reciprocal product, exact division near rounding boundaries) and kept in
// registers.  The codes of the first tile are requested before the
// prologue.
#include "cq_device.h"
#include "cq_internal.h"
#include "stream_common.h"
#include "a8_carriers.h"
#include "a8_quant.h"

namespace cq {

namespace {

// Byte transpose of a 4 x 4 byte matrix held in four words: out[s] byte b =
// in[b] byte s.
__device__ __forceinline__ void transpose4(const uint32_t in[4], uint32_t out[4]) {
    const uint32_t t0 = perm(in[1], in[0], 0x05010400u);  // in0.b0 in1.b0 in0.b1 in1.b1
    const uint32_t t1 = perm(in[1], in[0], 0x07030602u);  // in0.b2 in1.b2 in0.b3 in1.b3
    const uint32_t t2 = perm(in[3], in[2], 0x05010400u);
    const uint32_t t3 = perm(in[3], in[2], 0x07030602u);
    out[0] = perm(t2, t0, 0x05040100u);  // in0.b0 in1.b0 in2.b0 in3.b0
    out[1] = perm(t2, t0, 0x07060302u);
    out[2] = perm(t3, t1, 0x05040100u);
    out[3] = perm(t3, t1, 0x07060302u);
}

// Activations of one unit (32 INT8 values in 8 words), rearranged in the byte
// order in which the decode produces carriers.
template <int B>
__device__ __forceinline__ void arrange_x(const uint32_t xw[8], uint32_t xa[8]) {
    if constexpr (B == 3 || B >= 5) {
        // carriers come out in field order
#pragma unroll
        for (int i = 0; i < 8; ++i) xa[i] = xw[i];
    } else if constexpr (B == 4) {
        // word i of codes holds fields 8i..8i+7; the even fields come out as
        // bytes (8i, 8i+2, 8i+4, 8i+6), the odd ones as (8i+1, ...)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            xa[2 * i] = perm(xw[2 * i + 1], xw[2 * i], 0x06040200u);
            xa[2 * i + 1] = perm(xw[2 * i + 1], xw[2 * i], 0x07050301u);
        }
    } else if constexpr (B == 2) {
        // word i of codes holds fields 16i..16i+15; shift s gives fields
        // (16i + s, +4, +8, +12), i.e. byte s of x words 4i..4i+3
#pragma unroll
        for (int i = 0; i < 2; ++i) transpose4(xw + 4 * i, xa + 4 * i);
    } else {
        // one word of codes holds all 32 fields; shift s gives fields
        // (s, 8 + s, 16 + s, 24 + s): byte s%4 of x words s/4, 2 + s/4, 4 + s/4, 6 + s/4
        const uint32_t ev[4] = {xw[0], xw[2], xw[4], xw[6]};
        const uint32_t od[4] = {xw[1], xw[3], xw[5], xw[7]};
        uint32_t te[4], to[4];
        transpose4(ev, te);
        transpose4(od, to);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            xa[s] = te[s];
            xa[4 + s] = to[s];
        }
    }
}

}  // namespace

// FX < 0: xin holds the INT8 carriers and dxv their d_x.  FX = 0 / 1: xin is
// the BF16 / FP16 row, quantized here; block 0 writes the carriers to x8_out
// (if given) and d_x to dxv.  With FX >= 0 the host launches one wave per
// column block (at most kMaxFusedWaves).
constexpr int kMaxFusedWaves = 8;

template <int B, int UPG, int RW, int YDT, int FX>
__global__ void __launch_bounds__(FX >= 0 ? 64 * kMaxFusedWaves : 256) gemv_a8_stream(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int n, int k, const void *__restrict__ xin, float *__restrict__ dxv, int8_t *__restrict__ x8_out,
    void *__restrict__ y) {
    constexpr int M = max_code(B);
    constexpr bool kFused = FX >= 0;
    __shared__ float red[kMaxFusedWaves * RW];

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int nwaves = blockDim.x >> 6;  // the host keeps nwaves <= ncb
    const int ntiles = (n + RW - 1) / RW;
    const int units = k >> 5;
    const int ncb = (units + 63) >> 6;
    const int ng = k / (UPG * 32);
    const uint32_t row_bytes = uint32_t(k) * B / 8;
    const auto rc = make_rsrc(codes, uint32_t(n) * row_bytes);
    const auto rs = make_rsrc(scale, uint32_t(n) * ng * 4u);
    const auto ra = make_rsrc(a16, uint32_t(n) * ng * 2u);
    const auto rb = make_rsrc(b16, uint32_t(n) * ng * 2u);
    const auto rx = make_rsrc(xin, uint32_t(k) * (kFused ? 2u : 1u));

    // W4 carrier pairs evaluated by this lane: pair p covers magnitudes 2p, 2p+1.
    // Q lanes of a quad share a group; lane j of them evaluates pairs j, j+Q, ...
    constexpr int Q = UPG >= 4 ? 4 : UPG;
    constexpr int NP = 4 / Q;
    float tp0[NP], tp1[NP];
    int ip0[NP];
#pragma unroll
    for (int j = 0; j < NP; ++j) {
        ip0[j] = 2 * ((lane % Q) + Q * j);
        tp0[j] = float(ip0[j]) / float(M);
        tp1[j] = float(ip0[j] + 1) / float(M);
    }

    // An item is (row tile, column block).  A workgroup walks the tiles
    // blockIdx.x + j * gridDim.x; its wave w takes column blocks w, w + nwaves,
    // ... of each tile.  Rows and lanes past the matrix load an out-of-range
    // offset and read zeros (zero scale, so they add nothing).
    uint32_t wn[RW][B];
    float sn[RW];
    uint32_t an[RW], bn[RW];
    auto fetch = [&](int t, int c) {
        const int u = c * 64 + lane;
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            const int row = t * RW + r;
            const bool ok = (u < units) && (row < n);
            const uint32_t gi = uint32_t(row) * ng + uint32_t(u) / UPG;
            load_words<B>(rc, ok ? uint32_t(row) * row_bytes + uint32_t(u) * (4 * B) : kOobOffset, wn[r]);
            sn[r] = load_f32(rs, ok ? gi * 4u : kOobOffset);
            if constexpr (B >= 3) {
                an[r] = load_u16(ra, ok ? gi * 2u : kOobOffset);
                bn[r] = load_u16(rb, ok ? gi * 2u : kOobOffset);
            }
        }
    };

    float acc[RW];
#pragma unroll
    for (int i = 0; i < RW; ++i) acc[i] = 0.f;
    int tile = blockIdx.x, cb = wave;
    bool have = tile < ntiles;
    if (have) fetch(tile, cb);

    // fused quantization: d_x of the row and this lane's fixed carriers.  The
    // waves of a workgroup own all column blocks, so the lanes' own units are
    // the whole row: one read gives both the maximum and the values.
    uint32_t xq[8];
    float fac_fused = 0.f;
    if constexpr (kFused) {
        const int u = cb * 64 + lane;
        const uint32_t xo = u < units ? uint32_t(u) * 64u : kOobOffset;
        uint4 xv[4];
        float mx = 0.f;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            uint32_t p[4];
            load_words<4>(rx, xo + 16u * q, p);
            xv[q] = make_uint4(p[0], p[1], p[2], p[3]);
            mx = absmax8<FX>(xv[q], mx);
        }
        mx = wave_max(mx);
        if (lane == 0) red[wave] = mx;
        __syncthreads();
        mx = red[0];
        for (int wv = 1; wv < nwaves; ++wv) mx = fmaxf(mx, red[wv]);
        __syncthreads();  // red is reused by the tile reduction
        const float d = a8_row_scale(mx);
        const float rcp = __fdiv_rn(1.0f, d);
        fac_fused = d / 127.0f;
        uint32_t xw[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint2 c = quantize8_rcp<FX>(xv[q], d, rcp);
            xw[2 * q] = c.x;
            xw[2 * q + 1] = c.y;
        }
        if (blockIdx.x == 0) {
            if (x8_out && u < units) {
                typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
                u32x4_t *o = reinterpret_cast<u32x4_t *>(x8_out + size_t(u) * 32u);
                o[0] = u32x4_t{xw[0], xw[1], xw[2], xw[3]};
                o[1] = u32x4_t{xw[4], xw[5], xw[6], xw[7]};
            }
            if (threadIdx.x == 0) dxv[0] = d;
        }
        arrange_x<B>(xw, xq);
    }

    while (have) {
        uint32_t w[RW][B];
        float s[RW];
        uint32_t av[RW], bv[RW];
#pragma unroll
        for (int r = 0; r < RW; ++r) {
#pragma unroll
            for (int i = 0; i < B; ++i) w[r][i] = wn[r][i];
            s[r] = sn[r];
            av[r] = an[r];
            bv[r] = bn[r];
        }
        int cb_next = cb + nwaves, tile_next = tile;
        const bool last_cb = kFused || cb_next >= ncb;
        if (last_cb) {
            cb_next = wave;
            tile_next = tile + int(gridDim.x);
        }
        const bool have_next = tile_next < ntiles;
        if (have_next) fetch(tile_next, cb_next);

        uint32_t xa[8];
        if constexpr (kFused) {
#pragma unroll
            for (int i = 0; i < 8; ++i) xa[i] = xq[i];
        } else {
            const int u = cb * 64 + lane;
            uint32_t xw[8];
            const uint32_t xo = u < units ? uint32_t(u) * 32u : kOobOffset;
            load_words<4>(rx, xo, xw);
            load_words<4>(rx, xo + 16u, xw + 4);
            arrange_x<B>(xw, xa);
        }

#pragma unroll
        for (int r = 0; r < RW; ++r) {
            int p = 0;
            if constexpr (B == 4) {
                const float a = f16_to_f32(uint16_t(av[r]));
                const float b = f16_to_f32(uint16_t(bv[r]));
                const float c = 1.f - a - b;
                const float margin = carrier_margin(a, b, c);
                uint32_t pr[NP];
#pragma unroll
                for (int j = 0; j < NP; ++j) {
                    pr[j] = carrier_u8<M>(ip0[j], tp0[j], a, b, c, margin) |
                            (carrier_u8<M>(ip0[j] + 1, tp1[j], a, b, c, margin) << 8);
                }
                uint32_t P[4];
                if constexpr (Q == 4) {
                    P[0] = quad_bcast<0x00>(pr[0]);
                    P[1] = quad_bcast<0x55>(pr[0]);
                    P[2] = quad_bcast<0xaa>(pr[0]);
                    P[3] = quad_bcast<0xff>(pr[0]);
                } else if constexpr (Q == 2) {
                    P[0] = quad_bcast<0xa0>(pr[0]);
                    P[1] = quad_bcast<0xf5>(pr[0]);
                    P[2] = quad_bcast<0xa0>(pr[1]);
                    P[3] = quad_bcast<0xf5>(pr[1]);
                } else {
#pragma unroll
                    for (int j = 0; j < 4; ++j) P[j] = pr[j];
                }
                const uint32_t ta0 = P[0] | (P[1] << 16);  // r0 r1 r2 r3
                const uint32_t ta1 = P[2] | (P[3] << 16);  // r4 r5 r6 r7
                uint32_t tb0, tb1;
                w4_negative_table(ta0, ta1, tb0, tb1);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint32_t wd = w[r][i];
                    const uint32_t f2[2] = {wd & 0x0f0f0f0fu, (wd >> 4) & 0x0f0f0f0fu};
#pragma unroll
                    for (int h = 0; h < 2; ++h)
                        p = __builtin_amdgcn_sdot4(int(w4_lookup(f2[h], ta0, ta1, tb0, tb1)), int(xa[2 * i + h]), p,
                                                   false);
                }
            } else if constexpr (B == 3) {
                const float a = f16_to_f32(uint16_t(av[r]));
                const float b = f16_to_f32(uint16_t(bv[r]));
                const float c = 1.f - a - b;
                const float margin = carrier_margin(a, b, c);
                const uint32_t r12 = carrier_u8<M>(1, 1.f / 3.f, a, b, c, margin) |
                                     (carrier_u8<M>(2, 2.f / 3.f, a, b, c, margin) << 8);
                const uint32_t ta = (r12 << 8) | 0x7f000000u;             // r0 r1 r2 r3
                const uint32_t neg = (0x80808080u - ta) ^ 0x80808080u;  // 0 -r1 -r2 -r3
                const uint32_t tb = perm(neg, neg, 0x01020300u);        // 0 -r3 -r2 -r1
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const int bit = 12 * q, wi = bit >> 5, sh = bit & 31;
                    uint32_t x;
                    if (sh + 12 <= 32) x = w[r][wi] >> sh;
                    else x = __builtin_amdgcn_alignbit(w[r][wi + 1], w[r][wi], sh);
                    x &= 0xfffu;  // fields 4q .. 4q + 3
                    const uint32_t sel =
                        (x & 7u) | ((x << 5) & 0x700u) | ((x << 10) & 0x70000u) | ((x << 15) & 0x7000000u);
                    p = __builtin_amdgcn_sdot4(int(perm(tb, ta, sel)), int(xa[q]), p, false);
                }
            } else if constexpr (B >= 5) {
                // 16..128 magnitudes per group: every weight's carrier comes
                // from its own code, four fields to a word in field order.
                // The FP32 estimate 127 q(|k|/M) sign(k) uses coefficients
                // prescaled by 127 / M^j (its error stays below a third of
                // the doubled margin); when any estimate of the unit lies
                // within the margin of a half-integer, the unit's carriers
                // are formed again with the exact test of carrier_u8.
                const float a = f16_to_f32(uint16_t(av[r]));
                const float b = f16_to_f32(uint16_t(bv[r]));
                const float c = 1.f - a - b;
                const float margin = 2.f * carrier_margin(a, b, c);
                const float ca = a * (127.0f / float(M));
                const float cb = b * (127.0f / float(M * M));
                const float cc = c * (127.0f / float(M * M * M));
                auto field = [&](int i) __attribute__((always_inline)) {
                    const int bit = i * B, wi = bit >> 5, sh = bit & 31;
                    uint32_t v;
                    if (sh + B <= 32) v = w[r][wi] >> sh;
                    else v = __builtin_amdgcn_alignbit(w[r][wi + 1], w[r][wi], sh);
                    const int kk = __builtin_amdgcn_sbfe(int(v), 0, B);
                    return kk == -(M + 1) ? 0 : kk;  // the reserved pattern carries 0
                };
                uint32_t words[8];
                float worst = 0.f;
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    uint32_t word = 0;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float kf = float(field(4 * q + e));
                        const float ak = __builtin_fabsf(kf);
                        const float f = kf * __builtin_fmaf(ak, __builtin_fmaf(ak, cc, cb), ca);
                        const float rr = __builtin_rintf(f);
                        worst = __builtin_fmaxf(worst, __builtin_fabsf(f - rr));
                        const int cr = int(__builtin_fminf(__builtin_fmaxf(rr, -127.f), 127.f));
                        word |= (uint32_t(cr) & 0xffu) << (8 * e);
                    }
                    words[q] = word;
                }
                if (__builtin_expect(worst > 0.5f - margin, 0)) {
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        uint32_t word = 0;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int kk = field(4 * q + e);
                            const int mag = kk < 0 ? -kk : kk;
                            const int cr = int(carrier_u8<M>(mag, float(mag) / float(M), a, b, c,
                                                             carrier_margin(a, b, c)));
                            word |= (uint32_t(kk < 0 ? -cr : cr) & 0xffu) << (8 * e);
                        }
                        words[q] = word;
                    }
                }
#pragma unroll
                for (int q = 0; q < 8; ++q) p = __builtin_amdgcn_sdot4(int(words[q]), int(xa[q]), p, false);
            } else if constexpr (B == 2) {
                // fields 0 -> 0, 1 -> +127, 2 (reserved) -> 0, 3 -> -127
                constexpr uint32_t T = 0x81007f00u;
#pragma unroll
                for (int i = 0; i < 2; ++i) {
#pragma unroll
                    for (int sft = 0; sft < 4; ++sft) {
                        const uint32_t sel = (w[r][i] >> (2 * sft)) & 0x03030303u;
                        p = __builtin_amdgcn_sdot4(int(perm(T, T, sel)), int(xa[4 * i + sft]), p, false);
                    }
                }
            } else {
                // bit 1 -> +127, bit 0 -> -127
                constexpr uint32_t T = 0x00007f81u;
#pragma unroll
                for (int sft = 0; sft < 8; ++sft) {
                    const uint32_t sel = (w[r][0] >> sft) & 0x01010101u;
                    p = __builtin_amdgcn_sdot4(int(perm(T, T, sel)), int(xa[sft]), p, false);
                }
            }
            acc[r] = __builtin_fmaf(s[r], float(p), acc[r]);
        }
        if (last_cb) {
            const int row0 = tile * RW;
            const float fac = kFused ? fac_fused : dxv[0] / 127.0f;
            static_assert(RW == 2, "the output store writes row pairs");
            if (nwaves == 1) {
                const float v0 = wave_sum(acc[0]);
                const float v1 = wave_sum(acc[1]);
                acc[0] = 0.f;
                acc[1] = 0.f;
                if (lane == 0 && row0 < n) store_row_pair<YDT>(y, row0, v0 * fac, v1 * fac, row0 + 1 < n);
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
                    store_row_pair<YDT>(y, row0, v0 * fac, v1 * fac, row0 + 1 < n);
                }
                __syncthreads();  // red is reused by the next tile
            }
        }
        tile = tile_next;
        cb = cb_next;
        have = have_next;
    }
}

template <int B, int UPG, int YDT, int FX>
static hipError_t a8_stream_launch(const cq_weight &w, const void *xin, float *dxv, int8_t *x8_out, void *y,
                                   hipStream_t stream) {
    constexpr int RW = 2;
    const int64_t ncb = ((w.k >> 5) + 63) >> 6;
    // unfused: up to two column blocks a single wave per tile is fastest (no
    // LDS reduction); longer rows split their column blocks over two waves.
    // Fused: one wave per column block.
    const int nw = FX >= 0 ? int(ncb) : (ncb > 2 ? 2 : 1);
    if (nw > kMaxFusedWaves) return hipErrorNotSupported;
    const int64_t tiles = (w.n + RW - 1) / RW;
    const int64_t cus = device_cu_count();
    // unfused: one workgroup per tile up to 64 per CU.  Fused: every workgroup
    // quantizes the whole row once, so fewer, longer-lived workgroups (per CU:
    // 2 with four or more waves, 4 up to 8192 tiles, 12 beyond; measured on
    // the Llama-3-8B decode layers)
    int64_t per_cu = 64;
    if (FX >= 0) per_cu = nw >= 4 ? 2 : (tiles > 8192 ? 12 : 4);
    int64_t blocks = cus * per_cu;
    if (blocks > tiles) blocks = tiles;
    hipLaunchKernelGGL((gemv_a8_stream<B, UPG, RW, YDT, FX>), dim3(unsigned(blocks)), dim3(nw * 64), 0, stream,
                       w.codes, w.scale, w.a, w.b, int(w.n), int(w.k), xin, dxv, x8_out, y);
    return hipGetLastError();
}

template <int B, int YDT, int FX>
static hipError_t a8_stream_group(const cq_weight &w, const void *xin, float *dxv, int8_t *x8_out, void *y,
                                  hipStream_t stream) {
    switch (w.group) {
        case 32: return a8_stream_launch<B, 1, YDT, FX>(w, xin, dxv, x8_out, y, stream);
        case 64: return a8_stream_launch<B, 2, YDT, FX>(w, xin, dxv, x8_out, y, stream);
        case 128: return a8_stream_launch<B, 4, YDT, FX>(w, xin, dxv, x8_out, y, stream);
        case 256: return a8_stream_launch<B, 8, YDT, FX>(w, xin, dxv, x8_out, y, stream);
        case 512: return a8_stream_launch<B, 16, YDT, FX>(w, xin, dxv, x8_out, y, stream);
    }
    return hipErrorNotSupported;
}

template <int YDT, int FX>
static hipError_t a8_stream_bits(const cq_weight &w, const void *xin, float *dxv, int8_t *x8_out, void *y,
                                 hipStream_t stream) {
    switch (w.bits) {
        case 1: return a8_stream_group<1, YDT, FX>(w, xin, dxv, x8_out, y, stream);
        case 2: return a8_stream_group<2, YDT, FX>(w, xin, dxv, x8_out, y, stream);
        case 3: return a8_stream_group<3, YDT, FX>(w, xin, dxv, x8_out, y, stream);
        case 4: return a8_stream_group<4, YDT, FX>(w, xin, dxv, x8_out, y, stream);
    }
    if constexpr (FX < 0) {
        switch (w.bits) {
            case 5: return a8_stream_group<5, YDT, FX>(w, xin, dxv, x8_out, y, stream);
            case 6: return a8_stream_group<6, YDT, FX>(w, xin, dxv, x8_out, y, stream);
            case 7: return a8_stream_group<7, YDT, FX>(w, xin, dxv, x8_out, y, stream);
            case 8: return a8_stream_group<8, YDT, FX>(w, xin, dxv, x8_out, y, stream);
        }
    }
    return hipErrorNotSupported;
}

template <int FX>
static hipError_t a8_stream_ydt(const cq_weight &w, const void *xin, float *dxv, int8_t *x8_out, void *y, int y_dt,
                                hipStream_t stream) {
    if (y_dt == 0) return a8_stream_bits<0, FX>(w, xin, dxv, x8_out, y, stream);
    if (y_dt == 1) return a8_stream_bits<1, FX>(w, xin, dxv, x8_out, y, stream);
    return a8_stream_bits<2, FX>(w, xin, dxv, x8_out, y, stream);
}

bool gemv_a8_stream_supported(const cq_weight &w, int64_t m) {
    return m == 1 && stream_fits(w.n, w.k, w.bits, w.group);
}

bool gemv_a8_fused_supported(const cq_weight &w, int64_t m) {
    return gemv_a8_stream_supported(w, m) && w.bits <= 4 && (((w.k >> 5) + 63) >> 6) <= kMaxFusedWaves;
}

hipError_t launch_gemv_a8_stream(const cq_weight &w, const int8_t *x8, const float *dx, void *y, int y_dt,
                                 hipStream_t stream) {
    return a8_stream_ydt<-1>(w, x8, const_cast<float *>(dx), nullptr, y, y_dt, stream);
}

hipError_t launch_gemv_a8_fused(const cq_weight &w, const void *x, int x_dt, int8_t *x8_out, float *dx_out, void *y,
                                int y_dt, hipStream_t stream) {
    if (x_dt == 0) return a8_stream_ydt<0>(w, x, dx_out, x8_out, y, y_dt, stream);
    return a8_stream_ydt<1>(w, x, dx_out, x8_out, y, y_dt, stream);
}

}  // namespace cq
