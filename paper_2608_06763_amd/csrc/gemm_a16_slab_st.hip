// Few-row model-dtype GEMM, staged variant (16 rows of x, 16 weight rows per wave).
#include "gemm_a16_slab.h"

namespace cq {

bool a16_slab_st_fits(const cq_weight &w, int64_t m) {
    return m <= 32 && w.bits <= 5 && w.group <= 128 && w.group * w.bits <= 512 && (w.k / w.group) % 4 == 0;
}

bool gemm_a16_slab_staged_supported(const cq_weight &w, int64_t m) {
    return gemm_a16_slab_supported(w, m) && a16_slab_st_fits(w, m);
}

bool gemm_a16_slab_staged_preferred(const cq_weight &w, int64_t m) {
    if (!gemm_a16_slab_staged_supported(w, m)) return false;
    // the second x-row block pays for itself on short K too once it is
    // mostly full, and from 17 rows on more than 4096 weight rows (measured
    // on 4096 and 6144 weight rows over K = 4096: 6144 rows at 17-23 rows
    // 20.1-20.2 us against 21.1-24.4 for the plain kernel, 4096 rows slower)
    if (m >= 28 || (m > 16 && w.n > 4096)) return true;
    // two or more sweeps per wave when K is split over about 16 waves per
    // compute unit, at most 8 with the transposing activation loads (above 8
    // rows), a wave serving 32 rows above 16 (the test as it was measured;
    // the launch itself now runs fewer waves with longer runs)
    const int64_t tiles = (w.n + 15) / 16 * (m > 16 ? 1 : (m + 15) / 16);
    int64_t s = int64_t(256) * 16 / tiles;
    const int64_t s_max = m > 8 ? 8 : 16;
    if (s > s_max) s = s_max;
    if (s < 1) s = 1;
    const int64_t nsw = w.k / w.group / 4;
    return (nsw + s - 1) / s >= 2;
}

hipError_t launch_gemm_a16_slab_staged(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                       hipStream_t stream) {
    return launch_a16_slab_st(w, x, x_dt, m, y, y_dt, stream);
}

bool gemm_a16_slab_routed_supported(const cq_weight &w, int64_t tokens) {
    return w.bits <= 5 && w.group <= 128 && w.group * w.bits <= 512 && (w.k / w.group) % 4 == 0 &&
           stream_fits(w.n, w.k, w.bits, w.group) && tokens * w.k * 2 < (int64_t(1) << 31);
}

hipError_t launch_gemm_a16_slab_routed(const cq_weight &w, int n_experts, const void *x, int x_dt, int64_t tokens,
                                       int64_t routes, const int32_t *token, const int32_t *order,
                                       const int32_t *offsets, void *y, int y_dt, hipStream_t stream) {
    using namespace a16_slab;
    if (x_dt == 0) {
        if (y_dt == 0) return slab_st_routed_bits<0, 0>(w, n_experts, x, tokens, routes, token, order, offsets, y, stream);
        return slab_st_routed_bits<0, 2>(w, n_experts, x, tokens, routes, token, order, offsets, y, stream);
    }
    if (y_dt == 1) return slab_st_routed_bits<1, 1>(w, n_experts, x, tokens, routes, token, order, offsets, y, stream);
    return slab_st_routed_bits<1, 2>(w, n_experts, x, tokens, routes, token, order, offsets, y, stream);
}

hipError_t launch_a16_slab_st(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                              hipStream_t stream) {
    using namespace a16_slab;
    if (x_dt == 0) {
        if (y_dt == 0) return slab_st_bits<0, 0>(w, x, m, y, stream);
        return slab_st_bits<0, 2>(w, x, m, y, stream);
    }
    if (y_dt == 1) return slab_st_bits<1, 1>(w, x, m, y, stream);
    return slab_st_bits<1, 2>(w, x, m, y, stream);
}

}  // namespace cq
