// Instantiations of the model-dtype matrix-core GEMM for the x-tile height
// of 64 rows (kernel in gemm_a16_mfma.h).
#include "gemm_a16_mfma.h"

namespace cq {

hipError_t launch_a16_tile64(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt, bool one,
                             hipStream_t stream) {
    if (one) return hipErrorNotSupported;  // the rounded operand runs the 256-row tile only
    return a16_mfma_dtypes<false, tile64>(w, x, x_dt, m, y, y_dt, stream);
}

}  // namespace cq
