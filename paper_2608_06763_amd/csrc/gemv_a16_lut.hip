// Model-dtype narrow-row GEMV, table-decode family (Sec. 5.2 strategy 2, a
// signed level table per group; Sec. 5.3 narrow-row tactic).
//
// Numerics follow the paper's narrow-row GEMV: activations and normalised
// levels are multiplied in FP32 and s_g is applied in FP32 to the group's
// reduction.
//
// Work mapping.  A workgroup owns R output rows; K is walked in chunks of P
// groups (R * P = 64).  Lane l of a wave handles row (l % R) and group
// (l / R) of a chunk; the waves of a workgroup take every WAVES-th chunk and
// are reduced through LDS at the end.  Every wave keeps the packed codes,
// metadata and activations of its next chunk in registers, loaded before the
// current chunk is decoded, so HBM reads overlap decoding.
//
// Decode.  For its group a lane evaluates the cubic once per magnitude and
// writes one FP32 value per raw B-bit field u (the signed normalised level,
// 0 for the reserved pattern) into its wave's table at byte
// u * 256 + lane * 4.  Every lane owns a 4-byte column, so the per-weight table
// read is free of bank conflicts.  For W4 the read address is built with one
// byte permute per weight: the nibbles of a code word are spread into bytes,
// tagged with the wave number, and each byte is dropped into bits 8..15 of the
// lane's address.  Wider payloads (B >= 6) evaluate the cubic directly (a
// 64..256-entry table per group would cost more than it saves).
#include "cq_device.h"
#include "cq_internal.h"

namespace cq {

namespace {
constexpr int WAVES = 4;
constexpr int THREADS = WAVES * 64;

__device__ __forceinline__ void wave_sync_lds() {
    // LDS instructions of one wavefront execute in issue order, so ordering the
    // compiler's memory operations is enough for cross-lane LDS visibility within
    // a wavefront; no hardware wait (which would also drain pending HBM loads).
    __asm__ __volatile__("" ::: "memory");
    __builtin_amdgcn_wave_barrier();
}

typedef __attribute__((address_space(3))) float lds_float;

__device__ __forceinline__ float lds_load(uint32_t byte_addr) {
    return *reinterpret_cast<const lds_float *>(static_cast<uintptr_t>(byte_addr));
}
__device__ __forceinline__ void lds_store(uint32_t byte_addr, float v) {
    *reinterpret_cast<lds_float *>(static_cast<uintptr_t>(byte_addr)) = v;
}
}  // namespace

template <int B, int UPG, int R, int MR, int XDT, int YDT>
__global__ void __launch_bounds__(THREADS) gemv_a16_lut(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int64_t n, int64_t k, const uint16_t *__restrict__ x, int m_rows, void *__restrict__ y) {
    constexpr int G = UPG * 32;
    constexpr int P = 64 / R;                     // groups per chunk
    constexpr int M = max_code(B);
    constexpr bool LUT = (B <= 5);
    constexpr int NT = LUT ? (1 << B) : 1;
    constexpr int XROW = G + 4;                   // floats per staged group (pad spreads banks)
    constexpr int XWAVE = MR * P * XROW;          // floats per wave
    constexpr int V8 = G / 8;                     // 16-byte activation vectors per group
    constexpr int SLOTS = (P * V8 + 63) / 64;     // staging vectors per lane per row
    static_assert(SLOTS == 1 || MR == 1, "multi-slot staging only for one row");
    // the W4 address build needs bits 8..15 of the table base to be zero
    __shared__ __attribute__((aligned(B == 4 ? 65536 : 1024))) float tab[WAVES * NT * 64];
    __shared__ __attribute__((aligned(16))) float xs_all[WAVES * XWAVE];
    __shared__ float red[WAVES * R * MR];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int r = lane % R;
    const int p = lane / R;
    const int64_t row = int64_t(blockIdx.x) * R + r;
    const bool row_ok = row < n;
    const int64_t ng = k / G;
    const int64_t nchunks = (ng + P - 1) / P;
    const int64_t row_words = (k * B) >> 5;
    // byte address of this lane's table column; wave w's table starts NT*256 bytes after wave w-1's
    const uint32_t tab_base = uint32_t(uintptr_t((lds_float *)tab));
    const uint32_t col = tab_base + uint32_t(wave) * (NT * 256u) + uint32_t(lane) * 4u;
    float *xs = xs_all + wave * XWAVE;

    auto fetch = [&](int64_t c, uint32_t (&w)[UPG][B], float &s, uint32_t &aa, uint32_t &bb,
                     uint4 (&xv)[MR][SLOTS]) {
        const int64_t g = c * P + p;
        if (c < nchunks && row_ok && g < ng) {
            const uint32_t *wp = reinterpret_cast<const uint32_t *>(codes) + row * row_words + g * (UPG * B);
#pragma unroll
            for (int t = 0; t < UPG; ++t)
#pragma unroll
                for (int i = 0; i < B; ++i) w[t][i] = __builtin_nontemporal_load(wp + t * B + i);
            const int64_t gi = row * ng + g;
            s = scale[gi];
            aa = a16[gi];
            bb = b16[gi];
        } else {
            s = 0.f;
            aa = 0x3c00;  // 1.0
            bb = 0;
#pragma unroll
            for (int t = 0; t < UPG; ++t)
#pragma unroll
                for (int i = 0; i < B; ++i) w[t][i] = 0u;
        }
#pragma unroll
        for (int sl = 0; sl < SLOTS; ++sl) {
            const int idx = lane + sl * 64;
            const int pp = idx / V8;
            const int j8 = idx - pp * V8;
            const int64_t gx = c * P + pp;
#pragma unroll
            for (int mr = 0; mr < MR; ++mr) {
                uint4 v = make_uint4(0, 0, 0, 0);
                if (c < nchunks && idx < P * V8 && mr < m_rows && gx < ng)
                    v = *reinterpret_cast<const uint4 *>(x + int64_t(mr) * k + gx * G + j8 * 8);
                xv[mr][sl] = v;
            }
        }
    };

    uint32_t wc[UPG][B], wn[UPG][B];
    float sc = 0.f, sn = 0.f;
    uint32_t ac = 0, bc = 0, an = 0, bn = 0;  // 32-bit: no packed-half merging of loads
    uint4 xc[MR][SLOTS], xn[MR][SLOTS];
    float acc[MR];
#pragma unroll
    for (int i = 0; i < MR; ++i) acc[i] = 0.f;

    const int cpw = int((nchunks + WAVES - 1) / WAVES);  // chunk slots per wave
    fetch(wave, wn, sn, an, bn, xn);
    for (int ci = 0; ci < cpw; ++ci) {
        const int64_t c = wave + int64_t(ci) * WAVES;
#pragma unroll
        for (int t = 0; t < UPG; ++t)
#pragma unroll
            for (int i = 0; i < B; ++i) wc[t][i] = wn[t][i];
        sc = sn; ac = an; bc = bn;
#pragma unroll
        for (int mr = 0; mr < MR; ++mr)
#pragma unroll
            for (int sl = 0; sl < SLOTS; ++sl) xc[mr][sl] = xn[mr][sl];
        if (ci + 1 < cpw) fetch(c + WAVES, wn, sn, an, bn, xn);
        if (c >= nchunks) break;  // wave-uniform

        // ---- stage this chunk's activations as FP32
#pragma unroll
        for (int sl = 0; sl < SLOTS; ++sl) {
            const int idx = lane + sl * 64;
            if (idx < P * V8) {
                const int pp = idx / V8;
                const int j8 = idx - pp * V8;
#pragma unroll
                for (int mr = 0; mr < MR; ++mr) {
                    const uint32_t vw[4] = {xc[mr][sl].x, xc[mr][sl].y, xc[mr][sl].z, xc[mr][sl].w};
                    float f[8];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        f[2 * e] = act_to_f32<XDT>(uint16_t(vw[e] & 0xffffu));
                        f[2 * e + 1] = act_to_f32<XDT>(uint16_t(vw[e] >> 16));
                    }
                    float4 *dst = reinterpret_cast<float4 *>(xs + (mr * P + pp) * XROW + j8 * 8);
                    dst[0] = make_float4(f[0], f[1], f[2], f[3]);
                    dst[1] = make_float4(f[4], f[5], f[6], f[7]);
                }
            }
        }
        wave_sync_lds();

        float a = 1.f, b = 0.f;
        if constexpr (B >= 3) {
            a = f16_to_f32(uint16_t(ac));
            b = f16_to_f32(uint16_t(bc));
        }
        const float cc = 1.f - a - b;
        if constexpr (LUT) {
            if constexpr (B == 1) {
                lds_store(col, -1.f);
                lds_store(col + 256u, 1.f);
            } else {
                lds_store(col, 0.f);
                lds_store(col + (NT / 2) * 256u, 0.f);  // reserved pattern
#pragma unroll
                for (int i = 1; i <= M; ++i) {
                    const float t = float(i) * (1.0f / float(M));
                    const float q = (i == M) ? 1.f : t * __builtin_fmaf(t, __builtin_fmaf(t, cc, b), a);
                    lds_store(col + uint32_t(i) * 256u, q);
                    lds_store(col + uint32_t(NT - i) * 256u, -q);
                }
            }
        }
        // direct path: sign(k) q(|k|/M) = k (al + |k| (be + |k| ga))
        const float al = a * (1.0f / float(M));
        const float be = b * (1.0f / float(M * M));
        const float ga = cc * (1.0f / float(M * M * M));
        // W4 address build: the bytes of ev/od (nibble | wave << 4) land in bits 8..15 of col
        const uint32_t wtag = uint32_t(wave) * 0x10101010u;
        float part[MR];
#pragma unroll
        for (int i = 0; i < MR; ++i) part[i] = 0.f;
        const float *xg = xs + p * XROW;
#pragma unroll
        for (int t = 0; t < UPG; ++t) {
#pragma unroll
            for (int i8 = 0; i8 < 4; ++i8) {   // 8 codes per step
                float lv[8];
                if constexpr (B == 4) {
                    const uint32_t wd = wc[t][i8];
                    const uint32_t ev = (wd & 0x0f0f0f0fu) | wtag;         // codes 0, 2, 4, 6
                    const uint32_t od = ((wd >> 4) & 0x0f0f0f0fu) | wtag;  // codes 1, 3, 5, 7
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        // result bytes 0, 2, 3 from col, byte 1 from byte j of the tag word
                        const uint32_t sel = 0x03020000u | (uint32_t(4 + j) << 8);
                        lv[2 * j] = lds_load(__builtin_amdgcn_perm(ev, col, sel));
                        lv[2 * j + 1] = lds_load(__builtin_amdgcn_perm(od, col, sel));
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int i = i8 * 8 + e;
                        const int bit = i * B;
                        const int wd = bit >> 5, sh = bit & 31;
                        uint32_t v;
                        if (sh + B <= 32) v = wc[t][wd] >> sh;
                        else v = __builtin_amdgcn_alignbit(wc[t][wd + 1], wc[t][wd], sh);
                        if constexpr (LUT) {
                            lv[e] = lds_load(((v & uint32_t(NT - 1)) << 8) + col);
                        } else {
                            const int kk = __builtin_amdgcn_sbfe(int(v), 0, B);
                            const float kf = float(kk);
                            const float ak = __builtin_fabsf(kf);
                            const float lvv = kf * __builtin_fmaf(ak, __builtin_fmaf(ak, ga, be), al);
                            lv[e] = (kk == -(1 << (B - 1))) ? 0.f : lvv;
                        }
                    }
                }
#pragma unroll
                for (int mr = 0; mr < MR; ++mr) {
                    const float4 x0 = *reinterpret_cast<const float4 *>(xg + mr * P * XROW + t * 32 + i8 * 8);
                    const float4 x1 = *reinterpret_cast<const float4 *>(xg + mr * P * XROW + t * 32 + i8 * 8 + 4);
                    float p0 = part[mr];
                    float p1 = 0.f;
                    p0 = __builtin_fmaf(x0.x, lv[0], p0);
                    p1 = __builtin_fmaf(x0.y, lv[1], p1);
                    p0 = __builtin_fmaf(x0.z, lv[2], p0);
                    p1 = __builtin_fmaf(x0.w, lv[3], p1);
                    p0 = __builtin_fmaf(x1.x, lv[4], p0);
                    p1 = __builtin_fmaf(x1.y, lv[5], p1);
                    p0 = __builtin_fmaf(x1.z, lv[6], p0);
                    p1 = __builtin_fmaf(x1.w, lv[7], p1);
                    part[mr] = p0 + p1;
                }
            }
        }
#pragma unroll
        for (int mr = 0; mr < MR; ++mr) acc[mr] = __builtin_fmaf(sc, part[mr], acc[mr]);
        wave_sync_lds();
    }
    // ---- reduce the P group lanes of each row, then the waves
#pragma unroll
    for (int mr = 0; mr < MR; ++mr) {
        float v = acc[mr];
#pragma unroll
        for (int off = R; off < 64; off <<= 1) v += __shfl_xor(v, off, 64);
        acc[mr] = v;
    }
    if (p == 0) {
#pragma unroll
        for (int mr = 0; mr < MR; ++mr) red[(wave * R + r) * MR + mr] = acc[mr];
    }
    __syncthreads();
    if (wave == 0 && p == 0 && row_ok) {
#pragma unroll
        for (int mr = 0; mr < MR; ++mr) {
            float v = red[r * MR + mr];
#pragma unroll
            for (int wv = 1; wv < WAVES; ++wv) v += red[(wv * R + r) * MR + mr];
            if (mr < m_rows) store_out<YDT>(y, int64_t(mr) * n + row, v);
        }
    }
}

constexpr size_t lut_lds_bytes_of(int B, int UPG, int R, int MR) {
    return sizeof(float) * ((B <= 5 ? (size_t(1) << B) * THREADS : THREADS) +
                            size_t(WAVES) * MR * (64 / R) * (UPG * 32 + 4) + size_t(WAVES) * R * MR);
}

template <int B, int UPG, int R, int MR>
constexpr size_t lut_lds_bytes() {
    return lut_lds_bytes_of(B, UPG, R, MR);
}

template <int B, int UPG, int R, int MR, int XDT, int YDT>
static hipError_t run_lut(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    if constexpr (lut_lds_bytes<B, UPG, R, MR>() > 65536) {
        return hipErrorNotSupported;  // caller falls back to the conservative GEMV
    } else {
        const int64_t blocks = (w.n + R - 1) / R;
        if (blocks > 0x7fffffff) return hipErrorInvalidValue;
        hipLaunchKernelGGL((gemv_a16_lut<B, UPG, R, MR, XDT, YDT>), dim3(unsigned(blocks)), dim3(THREADS), 0, stream,
                           w.codes, w.scale, w.a, w.b, w.n, w.k, static_cast<const uint16_t *>(x), int(m), y);
        return hipGetLastError();
    }
}

template <int B, int UPG, int XDT, int YDT>
static hipError_t lut_rows(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    if constexpr (UPG >= 8) {
        return run_lut<B, UPG, 16, 1, XDT, YDT>(w, x, m, y, stream);
    } else {
        if (m <= 1) return run_lut<B, UPG, 8, 1, XDT, YDT>(w, x, m, y, stream);
        if (m <= 2) return run_lut<B, UPG, 16, 2, XDT, YDT>(w, x, m, y, stream);
        return run_lut<B, UPG, 16, 4, XDT, YDT>(w, x, m, y, stream);
    }
}

template <int B, int XDT, int YDT>
static hipError_t lut_group(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    switch (w.group) {
        case 32: return lut_rows<B, 1, XDT, YDT>(w, x, m, y, stream);
        case 64: return lut_rows<B, 2, XDT, YDT>(w, x, m, y, stream);
        case 128: return lut_rows<B, 4, XDT, YDT>(w, x, m, y, stream);
        case 256: return lut_rows<B, 8, XDT, YDT>(w, x, m, y, stream);
    }
    return hipErrorNotSupported;
}

template <int XDT, int YDT>
static hipError_t lut_bits(const cq_weight &w, const void *x, int64_t m, void *y, hipStream_t stream) {
    switch (w.bits) {
        case 1: return lut_group<1, XDT, YDT>(w, x, m, y, stream);
        case 2: return lut_group<2, XDT, YDT>(w, x, m, y, stream);
        case 3: return lut_group<3, XDT, YDT>(w, x, m, y, stream);
        case 4: return lut_group<4, XDT, YDT>(w, x, m, y, stream);
        case 5: return lut_group<5, XDT, YDT>(w, x, m, y, stream);
        case 6: return lut_group<6, XDT, YDT>(w, x, m, y, stream);
        case 7: return lut_group<7, XDT, YDT>(w, x, m, y, stream);
        case 8: return lut_group<8, XDT, YDT>(w, x, m, y, stream);
    }
    return hipErrorNotSupported;
}

bool gemv_a16_lut_supported(const cq_weight &w, int64_t m) {
    if (!(w.group <= 128 ? m <= 4 : (w.group == 256 && m <= 1))) return false;
    // the (R, MR) configuration lut_rows picks must fit 64 KB of LDS
    const int upg = w.group / 32;
    const int r = upg >= 8 ? 16 : (m <= 1 ? 8 : 16);
    const int mr = upg >= 8 ? 1 : (m <= 1 ? 1 : (m <= 2 ? 2 : 4));
    return lut_lds_bytes_of(w.bits, upg, r, mr) <= 65536;
}

hipError_t launch_gemv_a16_lut(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                               hipStream_t stream) {
    if (x_dt == 0) {
        if (y_dt == 0) return lut_bits<0, 0>(w, x, m, y, stream);
        return lut_bits<0, 2>(w, x, m, y, stream);
    }
    if (y_dt == 1) return lut_bits<1, 1>(w, x, m, y, stream);
    return lut_bits<1, 2>(w, x, m, y, stream);
}

}  // namespace cq
