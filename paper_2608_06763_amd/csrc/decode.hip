// Materialising reference decode (cq_decode_ref): one thread per weight.
//
// Unpack with the byte/shift rule of eq. gpu-packed-extraction, sign-extend,
// reserved pattern -> 0, W1 -> 2u - 1 (Sec. 2.1, Sec. 5.2), then reconstruct
// sign(k) s q(|k|/M) in FP32 with the Horner form of eq. gpu-horner.
#include "cq_device.h"
#include "cq_internal.h"

namespace cq {

__global__ void __launch_bounds__(256) decode_ref_kernel(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const uint16_t *__restrict__ a16, const uint16_t *__restrict__ b16,
    int bits, int group, int64_t n, int64_t k,
    int8_t *__restrict__ codes_out, float *__restrict__ w_out) {
    const int64_t total = n * k;
    const int64_t row_bytes = (k * bits) >> 3;
    const int64_t ng = k / group;
    const int m = max_code(bits);
    for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
         idx += int64_t(gridDim.x) * blockDim.x) {
        const int64_t r = idx / k;
        const int64_t j = idx - r * k;
        const uint32_t u = extract_field(codes + r * row_bytes, j, bits);
        const int code = field_to_code(u, bits);
        if (codes_out) codes_out[idx] = int8_t(code);
        if (w_out) {
            const int64_t gi = r * ng + j / group;
            const float s = scale[gi];
            float v;
            if (bits == 1) {
                v = float(code) * s;
            } else {
                const float a = f16_to_f32(a16[gi]);
                const float b = f16_to_f32(b16[gi]);
                const float c = 1.0f - a - b;
                v = s * signed_level(code, m, a, b, c);
            }
            w_out[idx] = v;
        }
    }
}

hipError_t launch_decode_ref(const cq_weight &w, int8_t *codes_out, float *w_out, hipStream_t stream) {
    const int64_t total = w.n * w.k;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(decode_ref_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream, w.codes, w.scale, w.a,
                       w.b, w.bits, w.group, w.n, w.k, codes_out, w_out);
    return hipGetLastError();
}

}  // namespace cq
