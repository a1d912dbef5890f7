// Building blocks of the single-row streaming GEMV kernels (gfx950).
//
// Buffer loads: the packed codes and the group metadata are read through
// buffer resources, so offsets are 32-bit and any load whose byte range ends
// past the resource's size returns zero instead of touching memory; lanes and
// rows beyond the matrix simply load an out-of-range offset.  A tensor must
// therefore be smaller than 2 GiB for these kernels (checked by the host).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cq_device.h"

namespace cq {

// Byte offset that lies past the end of every resource used here.
constexpr uint32_t kOobOffset = 0x80000000u;

// Resource word 3 for gfx9-family raw buffers (32-bit data format, no swizzle).
constexpr int kBufferFlags = 0x00020000;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, int(bytes), kBufferFlags);
}

template <int WORDS>
struct words_t {
    uint32_t v[WORDS];
};

// Load WORDS (1..8) consecutive 32-bit words at a 4-byte aligned byte offset.
template <int WORDS>
__device__ __forceinline__ void load_words(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t *out) {
    if constexpr (WORDS >= 4) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
        out[0] = v[0]; out[1] = v[1]; out[2] = v[2]; out[3] = v[3];
        if constexpr (WORDS > 4) load_words<WORDS - 4>(r, off + 16u, out + 4);
    } else if constexpr (WORDS == 3) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b96(r, off, 0, 0);
        out[0] = v[0]; out[1] = v[1]; out[2] = v[2];
    } else if constexpr (WORDS == 2) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
        out[0] = v[0]; out[1] = v[1];
    } else {
        out[0] = __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
    }
}

// The same with a wave-uniform part of the offset in a scalar register (the
// caller keeps voff + soff below 2^32; an out-of-range voff still reads zero).
template <int WORDS>
__device__ __forceinline__ void load_words_s(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, uint32_t *out) {
    if constexpr (WORDS >= 4) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
        out[0] = v[0]; out[1] = v[1]; out[2] = v[2]; out[3] = v[3];
        if constexpr (WORDS > 4) load_words_s<WORDS - 4>(r, voff + 16u, soff, out + 4);
    } else if constexpr (WORDS == 3) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b96(r, voff, soff, 0);
        out[0] = v[0]; out[1] = v[1]; out[2] = v[2];
    } else if constexpr (WORDS == 2) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
        out[0] = v[0]; out[1] = v[1];
    } else {
        out[0] = __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
    }
}

__device__ __forceinline__ float load_f32_s(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}

__device__ __forceinline__ uint32_t load_u16_s(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return uint32_t(__builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0));
}

__device__ __forceinline__ float load_f32(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

__device__ __forceinline__ uint32_t load_u16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return uint32_t(__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0));
}

// Store the outputs of two consecutive rows (row0 even, so a bf16/fp16 pair is
// 4-byte aligned and an FP32 pair 8-byte aligned) with one write; a lone last
// row is written alone.
template <int YDT>
__device__ __forceinline__ void store_row_pair(void *y, int row0, float v0, float v1, bool has1) {
    if constexpr (YDT == 2) {
        float *p = static_cast<float *>(y) + row0;
        if (has1) {
            typedef float f2_t __attribute__((ext_vector_type(2)));
            *reinterpret_cast<f2_t *>(p) = f2_t{v0, v1};
        } else {
            p[0] = v0;
        }
    } else {
        uint16_t *p = static_cast<uint16_t *>(y) + row0;
        const uint32_t h0 = YDT == 0 ? f32_to_bf16(v0) : f32_to_f16(v0);
        if (has1) {
            const uint32_t h1 = YDT == 0 ? f32_to_bf16(v1) : f32_to_f16(v1);
            *reinterpret_cast<uint32_t *>(p) = h0 | (h1 << 16);
        } else {
            p[0] = uint16_t(h0);
        }
    }
}

// Host check: every buffer a streaming kernel reads (codes, FP32 scales,
// activations of up to 2 bytes) is addressable with 31-bit offsets.
inline bool stream_fits(int64_t n, int64_t k, int bits, int group) {
    const int64_t lim = int64_t(1) << 31;
    return n * (k * bits / 8) < lim && n * (k / group) * 4 < lim && k * 2 < lim;
}

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}

// Sum over the 64 lanes of a wavefront (every lane active); the result is
// wave-uniform.  Lanes are added pairwise within quads, then across the two
// halves of each 8-lane and 16-lane row by mirrored DPP moves, and the four
// row sums are read out with readlane.
__device__ __forceinline__ float wave_sum(float v) {
    v += dpp_f32<0xb1>(v);   // quad_perm [1,0,3,2]
    v += dpp_f32<0x4e>(v);   // quad_perm [2,3,0,1]
    v += dpp_f32<0x141>(v);  // row_half_mirror
    v += dpp_f32<0x140>(v);  // row_mirror
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return (r0 + r1) + (r2 + r3);
}

}  // namespace cq
