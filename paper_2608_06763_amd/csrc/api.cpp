// Host side of the C ABI: argument validation, the host packer and the
// row-regime dispatch between the GEMV and tiled-GEMM kernel families.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>

#include "cq_internal.h"

namespace {

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// exact binary16 -> binary64 widening
double half_to_double(uint16_t h) {
    const int sign = (h >> 15) & 1;
    const int exp = (h >> 10) & 0x1f;
    const int man = h & 0x3ff;
    double v;
    if (exp == 0) v = std::ldexp(double(man), -24);
    else if (exp == 31) v = man ? NAN : INFINITY;
    else v = std::ldexp(double(man | 0x400), exp - 25);
    return sign ? -v : v;
}

// m(a, b) = min over t in [0, 1] of q'(t) = a + 2bt + 3ct^2, c = 1 - a - b
// (Sec. 3.1, eq. shape-domain).
double shape_margin(double a, double b) {
    const double c = 1.0 - a - b;
    double m = std::fmin(a, 3.0 - 2.0 * a - b);
    if (c > 0.0 && -3.0 * c < b && b < 0.0) m = std::fmin(m, a - b * b / (3.0 * c));
    return m;
}

// cq_gemm_a8_fused: 1 = single fused launch for one row, 0 = two launches
std::atomic<int32_t> g_a8_fused_single{0};
std::atomic<int64_t> g_gemv_max_rows[2] = {{-1}, {-1}};
constexpr int64_t kDefaultGemvMaxRows[2] = {cq::kGemvMaxRows, cq::kGemvMaxRows};

int64_t gemv_max_rows(int path) {
    const int64_t v = g_gemv_max_rows[path].load(std::memory_order_relaxed);
    return v < 0 ? kDefaultGemvMaxRows[path] : v;
}

cq_status check_weight(const cq_weight *w) {
    if (!w || !w->codes || !w->scale || !w->a || !w->b) return CQ_ERR_ARG;
    if (w->bits < 1 || w->bits > 8) return CQ_ERR_ARG;
    if (w->group < 32 || w->group > 512 || (w->group % 32) != 0) return CQ_ERR_ARG;
    if (w->n < 1 || w->k < 1) return CQ_ERR_ARG;
    if (w->k % w->group) return CQ_ERR_SHAPE;
    if ((w->k * w->bits) % 128) return CQ_ERR_SHAPE;
    if (w->n > (int64_t(1) << 40) / w->k) return CQ_ERR_SHAPE;
    if (!aligned16(w->codes) || !aligned16(w->scale) || !aligned16(w->a) || !aligned16(w->b)) return CQ_ERR_ALIGN;
    return CQ_OK;
}

cq_status hip_status(hipError_t e) { return e == hipSuccess ? CQ_OK : CQ_ERR_HIP; }

// Table entry if it names a family that can take the call, else the built-in
// rules (a partials dump always takes the built-in rules).
int choose_family(int path, const cq_weight &w, int x_dt, int64_t m, bool partials) {
    if (!partials) {
        const int f = cq::table_family(path, w, x_dt, m);
        if (f != CQ_FAMILY_AUTO && cq::family_supported(path, f, w, m)) return f;
    }
    return cq::default_family(path, w, m, gemv_max_rows(path), partials);
}

}  // namespace

extern "C" {

const char *cq_status_str(cq_status s) {
    switch (s) {
        case CQ_OK: return "CQ_OK";
        case CQ_ERR_ARG: return "CQ_ERR_ARG: invalid argument";
        case CQ_ERR_SHAPE: return "CQ_ERR_SHAPE: unsupported shape";
        case CQ_ERR_ALIGN: return "CQ_ERR_ALIGN: device pointer not 16-byte aligned";
        case CQ_ERR_META: return "CQ_ERR_META: invalid scale or shape metadata";
        case CQ_ERR_CODE: return "CQ_ERR_CODE: code out of range";
        case CQ_ERR_DTYPE: return "CQ_ERR_DTYPE: unsupported dtype";
        case CQ_ERR_HIP: return "CQ_ERR_HIP: HIP runtime error";
        case CQ_ERR_UNSUPPORTED: return "CQ_ERR_UNSUPPORTED: no kernel for this request";
    }
    return "unknown cq_status";
}

cq_status cq_pack_groups(int32_t bits, int32_t group, int64_t n, int64_t k, const int8_t *codes,
                         const float *scale, const uint16_t *a, const uint16_t *b, uint8_t *packed_out,
                         int64_t *bad_index) {
    if (!codes || !scale || !a || !b || !packed_out) return CQ_ERR_ARG;
    if (bits < 1 || bits > 8 || group < 1 || n < 1 || k < 1) return CQ_ERR_ARG;
    if ((int64_t(group) * bits) % 8 || k % group) return CQ_ERR_SHAPE;
    if (n > (int64_t(1) << 40) / k) return CQ_ERR_SHAPE;
    const int mcode = bits == 1 ? 1 : (1 << (bits - 1)) - 1;
    const int64_t ng = k / group;
    // codes
    for (int64_t i = 0; i < n * k; ++i) {
        const int c = codes[i];
        const bool ok = bits == 1 ? (c == 1 || c == -1) : (c >= -mcode && c <= mcode);
        if (!ok) {
            if (bad_index) *bad_index = i;
            return CQ_ERR_CODE;
        }
    }
    // metadata, group by group
    for (int64_t gi = 0; gi < n * ng; ++gi) {
        const float s = scale[gi];
        const double av = half_to_double(a[gi]), bv = half_to_double(b[gi]);
        bool ok = std::isfinite(s) && s >= 0.0f && std::isfinite(av) && std::isfinite(bv);
        if (ok && s == 0.0f && bits >= 2) {
            const int8_t *cg = codes + (gi / ng) * k + (gi % ng) * group;
            for (int j = 0; j < group; ++j) ok = ok && cg[j] == 0;
        }
        if (ok && bits >= 3) ok = shape_margin(av, bv) > 0.0;
        if (!ok) {
            if (bad_index) *bad_index = gi;
            return CQ_ERR_META;
        }
    }
    // pack: field j of a row occupies stream bits [jB, jB+B), LSB first
    const int64_t rb = (k * bits + 7) / 8;
    std::memset(packed_out, 0, size_t(n * rb));
    for (int64_t r = 0; r < n; ++r) {
        uint8_t *out = packed_out + r * rb;
        const int8_t *cr = codes + r * k;
        for (int64_t j = 0; j < k; ++j) {
            const uint32_t f = bits == 1 ? (cr[j] > 0 ? 1u : 0u) : uint32_t(int(cr[j])) & ((1u << bits) - 1u);
            const int64_t bit = j * bits;
            const int64_t p = bit >> 3;
            const int d = int(bit & 7);
            out[p] |= uint8_t(f << d);
            if (d + bits > 8) out[p + 1] |= uint8_t(f >> (8 - d));
        }
    }
    return CQ_OK;
}

cq_status cq_decode_ref(const cq_weight *w, int8_t *codes_out, float *w_out, void *stream) {
    const cq_status st = check_weight(w);
    if (st != CQ_OK) return st;
    if (!codes_out && !w_out) return CQ_ERR_ARG;
    if ((codes_out && !aligned16(codes_out)) || (w_out && !aligned16(w_out))) return CQ_ERR_ALIGN;
    return hip_status(cq::launch_decode_ref(*w, codes_out, w_out, static_cast<hipStream_t>(stream)));
}

cq_status cq_gemm_model_dtype(const cq_weight *w, const void *x, cq_dtype x_dtype, int64_t m, void *y,
                              cq_dtype y_dtype, void *stream) {
    const cq_status st = check_weight(w);
    if (st != CQ_OK) return st;
    if (!x || !y || m < 1) return CQ_ERR_ARG;
    if (x_dtype != CQ_BF16 && x_dtype != CQ_FP16) return CQ_ERR_DTYPE;
    if (y_dtype != x_dtype && y_dtype != CQ_FP32) return CQ_ERR_DTYPE;
    if (!aligned16(x) || !aligned16(y)) return CQ_ERR_ALIGN;
    if (m > (int64_t(1) << 40) / w->k || m > (int64_t(1) << 40) / w->n) return CQ_ERR_SHAPE;
    if (m > int64_t(65535) * 64) return CQ_ERR_SHAPE;
    const int family = choose_family(CQ_PATH_MODEL_DTYPE, *w, int(x_dtype), m, false);
    return hip_status(
        cq::run_family_a16(family, *w, x, int(x_dtype), m, y, int(y_dtype), static_cast<hipStream_t>(stream)));
}

cq_status cq_quantize_act_a8(const void *x, cq_dtype x_dtype, int64_t m, int64_t k, int8_t *x8, float *dx,
                             void *stream) {
    if (!x || !x8 || !dx || m < 1 || k < 1) return CQ_ERR_ARG;
    if (x_dtype != CQ_BF16 && x_dtype != CQ_FP16) return CQ_ERR_DTYPE;
    if (k % 32) return CQ_ERR_SHAPE;
    if (m > 0x7fffffff || m > (int64_t(1) << 40) / k) return CQ_ERR_SHAPE;
    if (!aligned16(x) || !aligned16(x8) || !aligned16(dx)) return CQ_ERR_ALIGN;
    return hip_status(cq::launch_quant_a8(x, int(x_dtype), m, k, x8, dx, static_cast<hipStream_t>(stream)));
}

cq_status cq_gemm_a8(const cq_weight *w, const int8_t *x8, const float *dx, int64_t m, void *y, cq_dtype y_dtype,
                     int32_t *partials_dbg, void *stream) {
    const cq_status st = check_weight(w);
    if (st != CQ_OK) return st;
    if (!x8 || !dx || !y || m < 1) return CQ_ERR_ARG;
    if (y_dtype != CQ_BF16 && y_dtype != CQ_FP16 && y_dtype != CQ_FP32) return CQ_ERR_DTYPE;
    if (!aligned16(x8) || !aligned16(dx) || !aligned16(y) || (partials_dbg && !aligned16(partials_dbg)))
        return CQ_ERR_ALIGN;
    if (m > (int64_t(1) << 40) / w->k || m > (int64_t(1) << 40) / w->n) return CQ_ERR_SHAPE;
    if (m > int64_t(65535) * 64) return CQ_ERR_SHAPE;
    const int family = choose_family(CQ_PATH_A8, *w, -1, m, partials_dbg != nullptr);
    return hip_status(cq::run_family_a8(family, *w, x8, dx, m, y, int(y_dtype), partials_dbg,
                                        static_cast<hipStream_t>(stream)));
}

cq_status cq_gemm_a8_fused(const cq_weight *w, const void *x, cq_dtype x_dtype, int64_t m, int8_t *x8, float *dx,
                           void *y, cq_dtype y_dtype, void *stream) {
    const cq_status st = check_weight(w);
    if (st != CQ_OK) return st;
    if (!x || !x8 || !dx || !y || m < 1) return CQ_ERR_ARG;
    if (x_dtype != CQ_BF16 && x_dtype != CQ_FP16) return CQ_ERR_DTYPE;
    if (y_dtype != CQ_BF16 && y_dtype != CQ_FP16 && y_dtype != CQ_FP32) return CQ_ERR_DTYPE;
    if (!aligned16(x) || !aligned16(x8) || !aligned16(dx) || !aligned16(y)) return CQ_ERR_ALIGN;
    if (m > (int64_t(1) << 40) / w->k || m > (int64_t(1) << 40) / w->n) return CQ_ERR_SHAPE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (g_a8_fused_single.load(std::memory_order_relaxed) && m <= gemv_max_rows(1) &&
        cq::gemv_a8_fused_supported(*w, m))
        return hip_status(cq::launch_gemv_a8_fused(*w, x, int(x_dtype), x8, dx, y, int(y_dtype), s));
    // the default, and every shape the single launch does not take: the two
    // calls, in order on the stream
    const cq_status q = cq_quantize_act_a8(x, x_dtype, m, w->k, x8, dx, stream);
    if (q != CQ_OK) return q;
    return cq_gemm_a8(w, x8, dx, m, y, y_dtype, nullptr, stream);
}

cq_status cq_gemm_routed_model_dtype(const cq_weight *bank, int32_t n_experts, const void *x, cq_dtype x_dtype,
                                     int64_t tokens, const int32_t *route_token, const int32_t *route_expert,
                                     int64_t routes, int32_t *workspace, void *y, cq_dtype y_dtype, void *stream) {
    const cq_status st = check_weight(bank);
    if (st != CQ_OK) return st;
    if (n_experts < 1 || tokens < 1 || routes < 0) return CQ_ERR_ARG;
    if (!x || !route_token || !route_expert || !workspace || !y) return CQ_ERR_ARG;
    if (x_dtype != CQ_BF16 && x_dtype != CQ_FP16) return CQ_ERR_DTYPE;
    if (y_dtype != x_dtype && y_dtype != CQ_FP32) return CQ_ERR_DTYPE;
    if (!aligned16(x) || !aligned16(y)) return CQ_ERR_ALIGN;
    if ((reinterpret_cast<uintptr_t>(route_token) | reinterpret_cast<uintptr_t>(route_expert) |
         reinterpret_cast<uintptr_t>(workspace)) % 4)
        return CQ_ERR_ALIGN;
    if (bank->n > (int64_t(1) << 40) / bank->k / n_experts) return CQ_ERR_SHAPE;
    if (tokens > (int64_t(1) << 40) / bank->k || routes > (int64_t(1) << 40) / bank->n) return CQ_ERR_SHAPE;
    if (!cq::routed_supported(*bank, n_experts, tokens, routes)) return CQ_ERR_UNSUPPORTED;
    if (routes == 0) return CQ_OK;
    return hip_status(cq::launch_routed_model_dtype(*bank, n_experts, x, int(x_dtype), tokens, route_token,
                                                    route_expert, routes, workspace, y, int(y_dtype),
                                                    static_cast<hipStream_t>(stream)));
}

cq_status cq_gemm_routed_model_dtype_noalloc(const cq_weight *bank, int32_t n_experts, const void *x, cq_dtype x_dtype,
                                             int64_t tokens, const int32_t *route_token, const int32_t *route_expert,
                                             int64_t routes, void *y, cq_dtype y_dtype, void *stream) {
    const cq_status st = check_weight(bank);
    if (st != CQ_OK) return st;
    if (n_experts < 1 || tokens < 1 || routes < 0) return CQ_ERR_ARG;
    if (!x || !route_token || !route_expert || !y) return CQ_ERR_ARG;
    if (x_dtype != CQ_BF16 && x_dtype != CQ_FP16) return CQ_ERR_DTYPE;
    if (y_dtype != x_dtype && y_dtype != CQ_FP32) return CQ_ERR_DTYPE;
    if (!aligned16(x) || !aligned16(y)) return CQ_ERR_ALIGN;
    if ((reinterpret_cast<uintptr_t>(route_token) | reinterpret_cast<uintptr_t>(route_expert)) % 4) return CQ_ERR_ALIGN;
    if (bank->n > (int64_t(1) << 40) / bank->k / n_experts) return CQ_ERR_SHAPE;
    if (tokens > (int64_t(1) << 40) / bank->k || routes > (int64_t(1) << 40) / bank->n) return CQ_ERR_SHAPE;
    // the grouping needs n_experts + 1 + routes ints of the library's scratch
    if (int64_t(n_experts) + 1 + routes > cq::kNoAllocRoutedInts) return CQ_ERR_SHAPE;
    if (!cq::routed_supported(*bank, n_experts, tokens, routes)) return CQ_ERR_UNSUPPORTED;
    if (routes == 0) return CQ_OK;
    return hip_status(cq::launch_routed_model_dtype_noalloc(*bank, n_experts, x, int(x_dtype), tokens, route_token,
                                                            route_expert, routes, y, int(y_dtype),
                                                            static_cast<hipStream_t>(stream)));
}

cq_status cq_build_carriers(const cq_weight *w, int8_t *carriers, void *stream) {
    const cq_status st = check_weight(w);
    if (st != CQ_OK) return st;
    if (w->bits == 1) return CQ_OK;  // W1 carriers are +-127: no table
    if (!carriers) return CQ_ERR_ARG;
    if (!aligned16(carriers)) return CQ_ERR_ALIGN;
    return hip_status(cq::launch_build_carriers(*w, carriers, static_cast<hipStream_t>(stream)));
}

cq_status cq_gemm_a8_carriers(const cq_weight *w, const int8_t *carriers, const int8_t *x8, const float *dx,
                              int64_t m, void *y, cq_dtype y_dtype, void *stream) {
    const cq_status st = check_weight(w);
    if (st != CQ_OK) return st;
    if (!x8 || !dx || !y || m < 1 || (w->bits > 1 && !carriers)) return CQ_ERR_ARG;
    if (y_dtype != CQ_BF16 && y_dtype != CQ_FP16 && y_dtype != CQ_FP32) return CQ_ERR_DTYPE;
    if (!aligned16(x8) || !aligned16(dx) || !aligned16(y) || (carriers && !aligned16(carriers))) return CQ_ERR_ALIGN;
    if (m > (int64_t(1) << 40) / w->k || m > (int64_t(1) << 40) / w->n) return CQ_ERR_SHAPE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (m <= gemv_max_rows(1) && m <= cq::kGemvMaxRows)
        return hip_status(cq::launch_gemv_a8_tab(*w, carriers, x8, dx, m, y, int(y_dtype), s));
    // 17..32 rows: the narrow-row kernel of the built-in rules (its register
    // decode forms the same carriers as the table)
    if (gemv_max_rows(1) >= cq::kGemvMaxRows && cq::gemv_a8_narrow_supported(*w, m))
        return hip_status(cq::launch_gemv_a8_narrow(*w, x8, dx, m, y, int(y_dtype), s));
    if (m > int64_t(65535) * 64) return CQ_ERR_SHAPE;
    return hip_status(cq::launch_gemm_a8_tab(*w, carriers, x8, dx, m, y, int(y_dtype), s));
}

cq_status cq_set_a8_fused_launch(int32_t single) {
    if (single != 0 && single != 1) return CQ_ERR_ARG;
    g_a8_fused_single.store(single, std::memory_order_relaxed);
    return CQ_OK;
}

int32_t cq_get_a8_fused_launch(void) { return g_a8_fused_single.load(std::memory_order_relaxed); }

cq_status cq_set_gemv_max_rows(int32_t path, int64_t max_rows) {
    if (path != 0 && path != 1) return CQ_ERR_ARG;
    g_gemv_max_rows[path].store(max_rows < 0 ? -1 : max_rows, std::memory_order_relaxed);
    return CQ_OK;
}

int64_t cq_get_gemv_max_rows(int32_t path) {
    if (path != 0 && path != 1) return -1;
    return gemv_max_rows(path);
}

int32_t cq_family_supported(int32_t path, int32_t family, const cq_weight *w, int64_t m) {
    if (check_weight(w) != CQ_OK) return 0;
    return cq::family_supported(path, family, *w, m) ? 1 : 0;
}

cq_status cq_gemm_model_dtype_family(const cq_weight *w, const void *x, cq_dtype x_dtype, int64_t m, void *y,
                                     cq_dtype y_dtype, int32_t family, void *stream) {
    if (family == CQ_FAMILY_AUTO) return cq_gemm_model_dtype(w, x, x_dtype, m, y, y_dtype, stream);
    const cq_status st = check_weight(w);
    if (st != CQ_OK) return st;
    if (!x || !y || m < 1) return CQ_ERR_ARG;
    if (x_dtype != CQ_BF16 && x_dtype != CQ_FP16) return CQ_ERR_DTYPE;
    if (y_dtype != x_dtype && y_dtype != CQ_FP32) return CQ_ERR_DTYPE;
    if (!aligned16(x) || !aligned16(y)) return CQ_ERR_ALIGN;
    if (m > (int64_t(1) << 40) / w->k || m > (int64_t(1) << 40) / w->n) return CQ_ERR_SHAPE;
    if (!cq::family_supported(CQ_PATH_MODEL_DTYPE, family, *w, m)) return CQ_ERR_UNSUPPORTED;
    const hipError_t e =
        cq::run_family_a16(family, *w, x, int(x_dtype), m, y, int(y_dtype), static_cast<hipStream_t>(stream));
    return e == hipErrorNotSupported ? CQ_ERR_UNSUPPORTED : hip_status(e);
}

cq_status cq_gemm_a8_family(const cq_weight *w, const int8_t *x8, const float *dx, int64_t m, void *y,
                            cq_dtype y_dtype, int32_t family, void *stream) {
    if (family == CQ_FAMILY_AUTO) return cq_gemm_a8(w, x8, dx, m, y, y_dtype, nullptr, stream);
    const cq_status st = check_weight(w);
    if (st != CQ_OK) return st;
    if (!x8 || !dx || !y || m < 1) return CQ_ERR_ARG;
    if (y_dtype != CQ_BF16 && y_dtype != CQ_FP16 && y_dtype != CQ_FP32) return CQ_ERR_DTYPE;
    if (!aligned16(x8) || !aligned16(dx) || !aligned16(y)) return CQ_ERR_ALIGN;
    if (m > (int64_t(1) << 40) / w->k || m > (int64_t(1) << 40) / w->n) return CQ_ERR_SHAPE;
    if (!cq::family_supported(CQ_PATH_A8, family, *w, m)) return CQ_ERR_UNSUPPORTED;
    const hipError_t e = cq::run_family_a8(family, *w, x8, dx, m, y, int(y_dtype), nullptr,
                                           static_cast<hipStream_t>(stream));
    return e == hipErrorNotSupported ? CQ_ERR_UNSUPPORTED : hip_status(e);
}

cq_status cq_select_set(const cq_select_entry *entries, int64_t count) {
    if (count < 0 || count > 65536 || (count > 0 && !entries)) return CQ_ERR_ARG;
    std::vector<cq_select_entry> t(entries, entries + count);
    for (int64_t i = 0; i < count; ++i)
        if (!cq::select_entry_valid(t[i])) return CQ_ERR_ARG;
    if (!cq::select_sort_disjoint(t)) return CQ_ERR_ARG;
    cq::select_install(std::move(t));
    return CQ_OK;
}

cq_status cq_probe_read(const void *buf, int64_t bytes, uint32_t *sink, void *stream) {
    if (!buf || !sink || bytes < 0) return CQ_ERR_ARG;
    if (bytes % 16) return CQ_ERR_ARG;
    if (!aligned16(buf) || (reinterpret_cast<uintptr_t>(sink) & 3u)) return CQ_ERR_ALIGN;
    return hip_status(cq::launch_read_probe(buf, bytes, sink, static_cast<hipStream_t>(stream)));
}

cq_status cq_select_query(int32_t path, const cq_weight *w, cq_dtype x_dtype, int64_t m, int32_t *family) {
    const cq_status st = check_weight(w);
    if (st != CQ_OK) return st;
    if (!family || m < 1 || (path != CQ_PATH_MODEL_DTYPE && path != CQ_PATH_A8)) return CQ_ERR_ARG;
    if (path == CQ_PATH_MODEL_DTYPE && x_dtype != CQ_BF16 && x_dtype != CQ_FP16) return CQ_ERR_DTYPE;
    *family = choose_family(path, *w, path == CQ_PATH_A8 ? -1 : int(x_dtype), m, false);
    return CQ_OK;
}

}  // extern "C"
