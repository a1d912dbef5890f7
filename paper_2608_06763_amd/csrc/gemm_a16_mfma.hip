// Model-dtype many-row GEMM on gfx950 matrix cores: host dispatch over the
// tile configurations (kernel and its description in gemm_a16_mfma.h).
#include "gemm_a16_mfma.h"

namespace cq {

// x-tile height for m rows when the caller does not name one: the smallest
// of 32, 64, 128 that holds m, else 256
int a16_mfma_tile_rows(int64_t m) { return m <= 32 ? 32 : m <= 64 ? 64 : m <= 128 ? 128 : 256; }

bool gemm_a16_mfma_supported(const cq_weight &w, int64_t m) {
    const int64_t lim = int64_t(1) << 31;
    return w.bits <= 5 && m * w.k * 2 < lim && stream_fits(w.n, w.k, w.bits, w.group) && m < lim;
}

hipError_t launch_gemm_a16_mfma(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                int tile_rows, hipStream_t stream) {
    switch (tile_rows ? tile_rows : a16_mfma_tile_rows(m)) {
        case 32: return launch_a16_tile32(w, x, x_dt, m, y, y_dt, false, stream);
        case 64: return launch_a16_tile64(w, x, x_dt, m, y, y_dt, false, stream);
        case 128: return launch_a16_tile128(w, x, x_dt, m, y, y_dt, false, stream);
        case 256: return launch_a16_tile256(w, x, x_dt, m, y, y_dt, false, stream);
    }
    return hipErrorNotSupported;
}

// the single-rounded operand (an opt-in family) on the 256-row tile
hipError_t launch_gemm_a16_mfma_rounded(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                        hipStream_t stream) {
    return launch_a16_tile256(w, x, x_dt, m, y, y_dt, true, stream);
}

}  // namespace cq
