// Few-row model-dtype GEMM, 16 rows of x and 32 weight rows per wave.
#include "gemm_a16_slab.h"

namespace cq {

hipError_t launch_a16_slab_1x2(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                               hipStream_t stream) {
    return a16_slab::slab_dtypes<1, 2>(w, x, x_dt, m, y, y_dt, stream);
}

}  // namespace cq
