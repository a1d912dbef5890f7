// Load-time INT8 carrier tables for the Dynamic-A8 path (Sec. 4.3 eq.
// carrier; the interior carriers precomputed at load, Sec. 5.2).
//
// For every (row, group) the table holds r(i) = RNE(127 q(i/M)) for the
// magnitudes i = 0 .. 2^(B-1) - 1 (r(0) = 0, r(M) = 127, exact from the FP16
// shapes: exact_carrier), one int8 each, 2^(B-1) bytes per group.  For W4 the
// 8 bytes are exactly the first register table of the in-kernel W4 decode
// (a8_carriers.h), so the A8 kernels can load them instead of evaluating the
// cubic; W3 needs 4 bytes of which the two interior carriers carry
// information.  The table is built once per weight and depends only on (a, b):
// it changes neither the codes nor the stored metadata.
#include "cq_device.h"
#include "cq_internal.h"

namespace cq {

template <int B>
__global__ void __launch_bounds__(256) build_carriers_kernel(const uint16_t *__restrict__ a16,
                                                             const uint16_t *__restrict__ b16, int64_t groups,
                                                             int8_t *__restrict__ out) {
    constexpr int M = max_code(B);
    constexpr int T = 1 << (B - 1);
    const int64_t gi = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (gi >= groups) return;
    const double a = (B == 2) ? 1.0 : double(f16_to_f32(a16[gi]));
    const double b = (B == 2) ? 0.0 : double(f16_to_f32(b16[gi]));
    int8_t *o = out + gi * T;
#pragma unroll 4
    for (int i = 0; i < T; ++i) o[i] = int8_t(i <= M ? exact_carrier(i, M, a, b) : 0);
}

int carrier_table_bytes(int bits) { return bits >= 2 ? (1 << (bits - 1)) : 0; }

hipError_t launch_build_carriers(const cq_weight &w, int8_t *out, hipStream_t stream) {
    const int64_t groups = w.n * (w.k / w.group);
    const int64_t blocks = (groups + 255) / 256;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    const dim3 grid(static_cast<uint32_t>(blocks)), block(256);
    switch (w.bits) {
        case 2: hipLaunchKernelGGL(build_carriers_kernel<2>, grid, block, 0, stream, w.a, w.b, groups, out); break;
        case 3: hipLaunchKernelGGL(build_carriers_kernel<3>, grid, block, 0, stream, w.a, w.b, groups, out); break;
        case 4: hipLaunchKernelGGL(build_carriers_kernel<4>, grid, block, 0, stream, w.a, w.b, groups, out); break;
        case 5: hipLaunchKernelGGL(build_carriers_kernel<5>, grid, block, 0, stream, w.a, w.b, groups, out); break;
        case 6: hipLaunchKernelGGL(build_carriers_kernel<6>, grid, block, 0, stream, w.a, w.b, groups, out); break;
        case 7: hipLaunchKernelGGL(build_carriers_kernel<7>, grid, block, 0, stream, w.a, w.b, groups, out); break;
        case 8: hipLaunchKernelGGL(build_carriers_kernel<8>, grid, block, 0, stream, w.a, w.b, groups, out); break;
        default: return hipSuccess;  // W1 has no table
    }
    return hipGetLastError();
}

}  // namespace cq
