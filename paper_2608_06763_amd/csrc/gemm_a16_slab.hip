// Few-row model-dtype GEMM with lane-decoded operands: support and shape
// choice (the kernel is in gemm_a16_slab.h).
#include "gemm_a16_slab.h"

namespace cq {

bool gemm_a16_slab_supported(const cq_weight &w, int64_t m) {
    return w.bits <= 5 && m >= 1 && m <= kSlabMaxRows && stream_fits(w.n, w.k, w.bits, w.group) &&
           m * w.k * 2 < (int64_t(1) << 31);
}

hipError_t launch_gemm_a16_slab(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                hipStream_t stream) {
    // up to 16 rows: a wave serves 32 weight rows with each activation load
    // when there are enough weight rows to keep the chip busy (measured
    // faster from 6144 rows, slower at 4096), else 16; more rows take two
    // x-row blocks
    if (m <= 16 && w.n < 6144) return launch_a16_slab_1x1(w, x, x_dt, m, y, y_dt, stream);
    if (m <= 16) return launch_a16_slab_1x2(w, x, x_dt, m, y, y_dt, stream);
    return launch_a16_slab_2x1(w, x, x_dt, m, y, y_dt, stream);
}

}  // namespace cq
