// Kernel-family predicates, the built-in row-regime rules and the measured
// selection table (Sec. 5.5-5.6).  Host code only: nothing here touches device
// memory, so the choice for a call can be queried without a GPU.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <memory>
#include <mutex>
#include <vector>

#include "cq_internal.h"

namespace cq {

bool family_supported(int path, int family, const cq_weight &w, int64_t m) {
    if (m < 1) return false;
    if (path == CQ_PATH_MODEL_DTYPE) {
        switch (family) {
            case CQ_FAMILY_GEMV_STREAM: return gemv_a16_stream_supported(w, m);
            case CQ_FAMILY_GEMV_LUT: return gemv_a16_lut_supported(w, m);
            case CQ_FAMILY_GEMV_NARROW: return gemv_a16_narrow_supported(w, m);
            case CQ_FAMILY_GEMV_GENERIC: return m <= kGemvMaxRows;
            case CQ_FAMILY_GEMM_MFMA: return gemm_a16_mfma_supported(w, m);
            case CQ_FAMILY_GEMM_TILED: return m <= int64_t(65535) * 64;
            case CQ_FAMILY_GEMM_MFMA_ROUNDED: return gemm_a16_mfma_supported(w, m);
            case CQ_FAMILY_GEMM_MFMA_M32:
            case CQ_FAMILY_GEMM_MFMA_M64:
            case CQ_FAMILY_GEMM_MFMA_M128:
            case CQ_FAMILY_GEMM_MFMA_M256: return gemm_a16_mfma_supported(w, m);
            case CQ_FAMILY_GEMM_SLAB: return gemm_a16_slab_supported(w, m);
            case CQ_FAMILY_GEMM_SLAB_STAGED: return gemm_a16_slab_staged_supported(w, m);
            case CQ_FAMILY_GEMV_ROWS: return gemv_a16_rows_supported(w, m);
        }
        return false;
    }
    if (path == CQ_PATH_A8) {
        switch (family) {
            case CQ_FAMILY_GEMV_STREAM: return gemv_a8_stream_supported(w, m);
            case CQ_FAMILY_GEMV_NARROW: return gemv_a8_narrow_supported(w, m);
            case CQ_FAMILY_GEMV_GENERIC: return m <= kGemvMaxRows;
            case CQ_FAMILY_GEMM_MFMA: return gemm_a8_mfma_supported(w, m);
            case CQ_FAMILY_GEMM_TILED: return m <= int64_t(65535) * 64;
            case CQ_FAMILY_GEMM_MFMA_M32:
            case CQ_FAMILY_GEMM_MFMA_M64:
            case CQ_FAMILY_GEMM_MFMA_M128:
            case CQ_FAMILY_GEMM_MFMA_M256: return gemm_a8_mfma_supported(w, m);
        }
        return false;
    }
    return false;
}

int default_family(int path, const cq_weight &w, int64_t m, int64_t gemv_max_rows, bool partials) {
    const bool gemv = m <= gemv_max_rows && m <= kGemvMaxRows;
    if (path == CQ_PATH_MODEL_DTYPE) {
        if (gemv) {
            // one row: the resident-activation form on layers with enough
            // row tiles per workgroup, else the streaming GEMV
            if (gemv_a16_rows_preferred(w, m)) return CQ_FAMILY_GEMV_ROWS;
            if (gemv_a16_stream_supported(w, m)) return CQ_FAMILY_GEMV_STREAM;
            // 2..16 rows: the lane-decoded matrix-core GEMM measured faster
            // than the table-decode and narrow-row families on every decode
            // and crossover shape, staged when each wave gets at least two
            // sweeps; B >= 6 keeps the GEMV families
            if (gemm_a16_slab_staged_preferred(w, m)) return CQ_FAMILY_GEMM_SLAB_STAGED;
            if (gemm_a16_slab_supported(w, m)) return CQ_FAMILY_GEMM_SLAB;
            if (gemv_a16_lut_supported(w, m)) return CQ_FAMILY_GEMV_LUT;
            if (gemv_a16_narrow_supported(w, m)) return CQ_FAMILY_GEMV_NARROW;
            return CQ_FAMILY_GEMV_GENERIC;
        }
        // 17..32 rows: the lane-decoded GEMM splits K over the waves of a
        // workgroup, which the tiled GEMM lacks (2-3x on up to 14336 weight
        // rows); its staged two-block form leads wherever the K split leaves
        // each wave two or more sweeps (28672 weight rows included)
        if (m > kGemvMaxRows && gemm_a16_slab_staged_preferred(w, m)) return CQ_FAMILY_GEMM_SLAB_STAGED;
        if (m > kGemvMaxRows && gemm_a16_slab_supported(w, m)) return CQ_FAMILY_GEMM_SLAB;
        return gemm_a16_mfma_supported(w, m) ? CQ_FAMILY_GEMM_MFMA : CQ_FAMILY_GEMM_TILED;
    }
    // Dynamic A8: a partials dump is written by the generic GEMV, the W4
    // matrix-core GEMM and the 64 x 64 GEMM only
    if (gemv) {
        if (!partials && gemv_a8_stream_supported(w, m)) return CQ_FAMILY_GEMV_STREAM;
        if (!partials && gemv_a8_narrow_supported(w, m)) return CQ_FAMILY_GEMV_NARROW;
        return CQ_FAMILY_GEMV_GENERIC;
    }
    // 17..32 rows (with the GEMV threshold at its maximum): the narrow-row
    // kernel with two 16-row blocks of x per decoded operand (measured ahead
    // of the 32-row tile on every decode and crossover shape, 1.2-3.4x)
    if (!partials && m > kGemvMaxRows && gemv_max_rows >= kGemvMaxRows && gemv_a8_narrow_supported(w, m))
        return CQ_FAMILY_GEMV_NARROW;
    return gemm_a8_mfma_supported(w, m) && (w.bits == 4 || !partials) ? CQ_FAMILY_GEMM_MFMA : CQ_FAMILY_GEMM_TILED;
}

hipError_t run_family_a16(int family, const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                          hipStream_t stream) {
    switch (family) {
        case CQ_FAMILY_GEMV_STREAM: return launch_gemv_a16_stream(w, x, x_dt, y, y_dt, stream);
        case CQ_FAMILY_GEMV_LUT: return launch_gemv_a16_lut(w, x, x_dt, m, y, y_dt, stream);
        case CQ_FAMILY_GEMV_NARROW: return launch_gemv_a16_narrow(w, x, x_dt, m, y, y_dt, stream);
        case CQ_FAMILY_GEMV_GENERIC: return launch_gemv_a16_generic(w, x, x_dt, m, y, y_dt, stream);
        case CQ_FAMILY_GEMM_MFMA: return launch_gemm_a16_mfma(w, x, x_dt, m, y, y_dt, 0, stream);
        case CQ_FAMILY_GEMM_TILED: return launch_gemm_a16_tiled(w, x, x_dt, m, y, y_dt, stream);
        case CQ_FAMILY_GEMM_MFMA_ROUNDED: return launch_gemm_a16_mfma_rounded(w, x, x_dt, m, y, y_dt, stream);
        case CQ_FAMILY_GEMM_MFMA_M32:
        case CQ_FAMILY_GEMM_MFMA_M64:
        case CQ_FAMILY_GEMM_MFMA_M128:
        case CQ_FAMILY_GEMM_MFMA_M256:
            return launch_gemm_a16_mfma(w, x, x_dt, m, y, y_dt, family_tile_rows(family), stream);
        case CQ_FAMILY_GEMM_SLAB: return launch_gemm_a16_slab(w, x, x_dt, m, y, y_dt, stream);
        case CQ_FAMILY_GEMM_SLAB_STAGED: return launch_gemm_a16_slab_staged(w, x, x_dt, m, y, y_dt, stream);
        case CQ_FAMILY_GEMV_ROWS: return launch_gemv_a16_rows(w, x, x_dt, y, y_dt, stream);
    }
    return hipErrorInvalidValue;
}

hipError_t run_family_a8(int family, const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                         int y_dt, int32_t *partials, hipStream_t stream) {
    switch (family) {
        case CQ_FAMILY_GEMV_STREAM: return launch_gemv_a8_stream(w, x8, dx, y, y_dt, stream);
        case CQ_FAMILY_GEMV_NARROW: return launch_gemv_a8_narrow(w, x8, dx, m, y, y_dt, stream);
        case CQ_FAMILY_GEMV_GENERIC: return launch_gemv_a8_generic(w, x8, dx, m, y, y_dt, partials, stream);
        case CQ_FAMILY_GEMM_MFMA: return launch_gemm_a8_mfma(w, x8, dx, m, y, y_dt, partials, 0, stream);
        case CQ_FAMILY_GEMM_TILED: return launch_gemm_a8_tiled(w, x8, dx, m, y, y_dt, partials, stream);
        case CQ_FAMILY_GEMM_MFMA_M32:
        case CQ_FAMILY_GEMM_MFMA_M64:
        case CQ_FAMILY_GEMM_MFMA_M128:
        case CQ_FAMILY_GEMM_MFMA_M256:
            return launch_gemm_a8_mfma(w, x8, dx, m, y, y_dt, partials, family_tile_rows(family), stream);
    }
    return hipErrorInvalidValue;
}

// ---------------------------------------------------------------- selection table

namespace {

// The installed table is sorted by (path, bits, group, n, k, m_lo), so a lookup
// is a binary search for the shape followed by a scan of that shape's few
// row ranges.
using Table = std::vector<cq_select_entry>;

bool shape_less(const cq_select_entry &a, const cq_select_entry &b) {
    if (a.path != b.path) return a.path < b.path;
    if (a.bits != b.bits) return a.bits < b.bits;
    if (a.group != b.group) return a.group < b.group;
    if (a.n != b.n) return a.n < b.n;
    return a.k < b.k;
}

bool entry_less(const cq_select_entry &a, const cq_select_entry &b) {
    if (shape_less(a, b)) return true;
    if (shape_less(b, a)) return false;
    return a.m_lo < b.m_lo;
}

std::mutex g_table_mutex;               // serialises writers
std::shared_ptr<const Table> g_table;   // read with std::atomic_load
std::atomic<bool> g_table_nonempty{false};

bool entry_matches(const cq_select_entry &e, int path, const cq_weight &w, int x_dt, int64_t m) {
    return e.path == path && e.bits == w.bits && e.group == w.group && e.n == w.n && e.k == w.k &&
           (e.x_dtype < 0 || e.x_dtype == x_dt) && m >= e.m_lo && m <= e.m_hi;
}

}  // namespace

int table_family(int path, const cq_weight &w, int x_dt, int64_t m) {
    if (!g_table_nonempty.load(std::memory_order_acquire)) return CQ_FAMILY_AUTO;
    const std::shared_ptr<const Table> t = std::atomic_load(&g_table);
    if (!t) return CQ_FAMILY_AUTO;
    cq_select_entry probe{};
    probe.path = path;
    probe.bits = w.bits;
    probe.group = w.group;
    probe.n = w.n;
    probe.k = w.k;
    const auto range = std::equal_range(t->begin(), t->end(), probe, shape_less);
    for (auto it = range.first; it != range.second; ++it)
        if (entry_matches(*it, path, w, x_dt, m)) return it->family;
    return CQ_FAMILY_AUTO;
}

bool select_entry_valid(const cq_select_entry &e) {
    if (e.path != CQ_PATH_MODEL_DTYPE && e.path != CQ_PATH_A8) return false;
    if (e.family < CQ_FAMILY_GEMV_STREAM || e.family > CQ_FAMILY_GEMV_ROWS) return false;
    if (e.path == CQ_PATH_A8 && (e.family == CQ_FAMILY_GEMV_LUT || e.family == CQ_FAMILY_GEMM_MFMA_ROUNDED ||
                                 e.family == CQ_FAMILY_GEMM_SLAB || e.family == CQ_FAMILY_GEMM_SLAB_STAGED ||
                                 e.family == CQ_FAMILY_GEMV_ROWS))
        return false;
    if (e.bits < 1 || e.bits > 8) return false;
    if (e.group < 32 || e.group > 512 || e.group % 32) return false;
    if (e.n < 1 || e.k < 1) return false;
    if (e.m_lo < 1 || e.m_hi < e.m_lo) return false;
    if (e.x_dtype < -1 || e.x_dtype > 1 || (e.path == CQ_PATH_A8 && e.x_dtype != -1)) return false;
    return e.reserved == 0;
}

bool select_sort_disjoint(std::vector<cq_select_entry> &entries) {
    std::sort(entries.begin(), entries.end(), entry_less);
    // Within one shape, the entries that a model-dtype call with activations
    // of dtype d can match (x_dtype d or any) must have disjoint row ranges;
    // A8 entries all carry x_dtype -1, so one pass covers them.
    for (size_t lo = 0; lo < entries.size();) {
        size_t hi = lo + 1;
        while (hi < entries.size() && !shape_less(entries[lo], entries[hi])) ++hi;
        for (int d = 0; d <= 1; ++d) {
            bool any = false;
            int64_t reach = 0;
            for (size_t i = lo; i < hi; ++i) {
                const cq_select_entry &e = entries[i];
                if (e.x_dtype >= 0 && e.x_dtype != d) continue;
                if (any && e.m_lo <= reach) return false;
                reach = any ? std::max(reach, e.m_hi) : e.m_hi;
                any = true;
            }
        }
        lo = hi;
    }
    return true;
}

void select_install(std::vector<cq_select_entry> entries) {
    std::lock_guard<std::mutex> lock(g_table_mutex);
    const bool nonempty = !entries.empty();
    std::shared_ptr<const Table> t = nonempty ? std::make_shared<const Table>(std::move(entries)) : nullptr;
    std::atomic_store(&g_table, t);
    g_table_nonempty.store(nonempty, std::memory_order_release);
}

}  // namespace cq
