// Internal launcher declarations shared by the host API and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "../../include/cq.h"
#include "../../include/cq_measure.h"

namespace cq {

// Dtype codes used as template arguments: 0 = bf16, 1 = fp16, 2 = fp32.

hipError_t launch_decode_ref(const cq_weight &w, int8_t *codes_out, float *w_out, hipStream_t stream);

// Conservative model-dtype GEMV (every B and G, m <= 16).
hipError_t launch_gemv_a16_generic(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                   hipStream_t stream);

// Model-dtype single-row streaming GEMV (m == 1, every B, G <= 512).
bool gemv_a16_stream_supported(const cq_weight &w, int64_t m);
hipError_t launch_gemv_a16_stream(const cq_weight &w, const void *x, int x_dt, void *y, int y_dt,
                                  hipStream_t stream);
// The same kernel with the activation slice resident in registers (one wave
// per 2048-code column block, K <= 16384).
bool gemv_a16_rows_supported(const cq_weight &w, int64_t m);
bool gemv_a16_rows_preferred(const cq_weight &w, int64_t m);
hipError_t launch_gemv_a16_rows(const cq_weight &w, const void *x, int x_dt, void *y, int y_dt,
                                hipStream_t stream);

// Model-dtype table-decode GEMV (m <= 4); see gemv_a16_lut.hip.
bool gemv_a16_lut_supported(const cq_weight &w, int64_t m);
hipError_t launch_gemv_a16_lut(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                               hipStream_t stream);

// Narrow-row (2 <= m <= 16) matrix-core products; see gemv_narrow.hip.
bool gemv_a16_narrow_supported(const cq_weight &w, int64_t m);
hipError_t launch_gemv_a16_narrow(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                  hipStream_t stream);
bool gemv_a8_narrow_supported(const cq_weight &w, int64_t m);
hipError_t launch_gemv_a8_narrow(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y, int y_dt,
                                 hipStream_t stream);

// Model-dtype many-row GEMM for B <= 5 (tensors below 2 GiB).  tile_rows is
// the x-tile height (32, 64, 128 or 256), 0 for the built-in choice by m.
bool gemm_a16_mfma_supported(const cq_weight &w, int64_t m);
int a16_mfma_tile_rows(int64_t m);
hipError_t launch_gemm_a16_mfma(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                int tile_rows, hipStream_t stream);
// The same GEMM with the decoded weight rounded once to the activation dtype
// (one MFMA per product for BF16; FP16 is the default kernel).
hipError_t launch_gemm_a16_mfma_rounded(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                        hipStream_t stream);

// Model-dtype GEMM for few rows (1 <= m <= kSlabMaxRows, B <= 5) that decodes
// each weight into the matrix-core operand of the decoding lane, with split-K
// over the waves of a workgroup.
constexpr int64_t kSlabMaxRows = 32;
bool gemm_a16_slab_supported(const cq_weight &w, int64_t m);
hipError_t launch_gemm_a16_slab(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                hipStream_t stream);
// The staged variant (codes and metadata through LDS, contiguous K per wave)
// and the built-in preference for it: the waves of the K split get two or
// more sweeps each (host only, sized for 256 compute units).
bool gemm_a16_slab_staged_supported(const cq_weight &w, int64_t m);
bool gemm_a16_slab_staged_preferred(const cq_weight &w, int64_t m);
hipError_t launch_gemm_a16_slab_staged(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                       hipStream_t stream);
// Its routed form: one workgroup per (expert, 16 weight rows) over the grouped
// route list, 16 routes at a time (G <= 128, G B <= 512, K / G a multiple of 4).
bool gemm_a16_slab_routed_supported(const cq_weight &w, int64_t tokens);
hipError_t launch_gemm_a16_slab_routed(const cq_weight &w, int n_experts, const void *x, int x_dt, int64_t tokens,
                                       int64_t routes, const int32_t *token, const int32_t *order,
                                       const int32_t *offsets, void *y, int y_dt, hipStream_t stream);

// Dynamic-A8 activation quantizer.
hipError_t launch_quant_a8(const void *x, int x_dt, int64_t m, int64_t k, int8_t *x8, float *dx,
                           hipStream_t stream);

// Dynamic-A8 single-row streaming GEMV (m == 1, B <= 4, no partials dump).
bool gemv_a8_stream_supported(const cq_weight &w, int64_t m);
bool gemv_a8_fused_supported(const cq_weight &w, int64_t m);
bool gemv_a16_routed_supported(const cq_weight &w, int64_t tokens);
hipError_t launch_gemv_a16_routed(const cq_weight &w, int n_experts, const void *x, int x_dt, int64_t tokens,
                                  const int32_t *token, const int32_t *order, const int32_t *offsets, void *y,
                                  int y_dt, hipStream_t stream);
bool routed_supported(const cq_weight &w, int64_t n_experts, int64_t tokens, int64_t routes);
// Routed product with every route streaming its expert (few routes per expert).
bool gemv_a16_stream_routed_supported(const cq_weight &w, int64_t n_experts, int64_t tokens, int64_t routes);
hipError_t launch_gemv_a16_stream_routed(const cq_weight &w, int n_experts, const void *x, int x_dt, int64_t tokens,
                                         const int32_t *token, const int32_t *expert, int64_t routes, void *y,
                                         int y_dt, hipStream_t stream);
int carrier_table_bytes(int bits);
hipError_t launch_build_carriers(const cq_weight &w, int8_t *out, hipStream_t stream);
hipError_t launch_gemv_a8_tab(const cq_weight &w, const int8_t *ctab, const int8_t *x8, const float *dx, int64_t m,
                              void *y, int y_dt, hipStream_t stream);
hipError_t launch_gemm_a8_tab(const cq_weight &w, const int8_t *ctab, const int8_t *x8, const float *dx, int64_t m,
                              void *y, int y_dt, hipStream_t stream);
hipError_t launch_gemm_a8_mfma_tab(const cq_weight &w, const int8_t *ctab, const int8_t *x8, const float *dx,
                                   int64_t m, void *y, int y_dt, hipStream_t stream);
hipError_t launch_routed_model_dtype(const cq_weight &w, int n_experts, const void *x, int x_dt, int64_t tokens,
                                     const int32_t *token, const int32_t *expert, int64_t routes, int32_t *workspace,
                                     void *y, int y_dt, hipStream_t stream);
// The same with the library's per-device scratch array as the workspace
// (n_experts + 1 + routes <= kNoAllocRoutedInts; checked by the caller).
constexpr int64_t kNoAllocRoutedInts = int64_t(1) << 20;
hipError_t routed_scratch(int32_t **ptr);
hipError_t launch_routed_model_dtype_noalloc(const cq_weight &w, int n_experts, const void *x, int x_dt,
                                             int64_t tokens, const int32_t *token, const int32_t *expert,
                                             int64_t routes, void *y, int y_dt, hipStream_t stream);
hipError_t launch_gemv_a8_fused(const cq_weight &w, const void *x, int x_dt, int8_t *x8_out, float *dx_out, void *y,
                                int y_dt, hipStream_t stream);
hipError_t launch_gemv_a8_stream(const cq_weight &w, const int8_t *x8, const float *dx, void *y, int y_dt,
                                 hipStream_t stream);

// Dynamic-A8 many-row GEMM for W3 and W4, G >= 64 (tensors below 2 GiB).
// tile_rows: x-tile height 32, 64, 128 (gemm_a8_tile.hip) or 256, 0 for the
// built-in choice by m; a partials dump always takes the 256-row kernel.
bool gemm_a8_mfma_supported(const cq_weight &w, int64_t m);
hipError_t launch_gemm_a8_mfma(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y, int y_dt,
                               int32_t *partials, int tile_rows, hipStream_t stream);
hipError_t launch_gemm_a8_tile(const cq_weight &w, const int8_t *ctab, const int8_t *x8, const float *dx, int64_t m,
                               void *y, int y_dt, int tile_rows, hipStream_t stream);

// Largest row count each GEMV family accepts.
constexpr int64_t kGemvMaxRows = 16;

// x-tile height of a fixed-tile matrix-core family (CQ_FAMILY_GEMM_MFMA_M32
// .. _M256), 0 for any other family.
inline int family_tile_rows(int family) {
    switch (family) {
        case CQ_FAMILY_GEMM_MFMA_M32: return 32;
        case CQ_FAMILY_GEMM_MFMA_M64: return 64;
        case CQ_FAMILY_GEMM_MFMA_M128: return 128;
        case CQ_FAMILY_GEMM_MFMA_M256: return 256;
    }
    return 0;
}

// Single families, for the measured kernel selection.
hipError_t launch_gemm_a16_tiled(const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                                 hipStream_t stream);
hipError_t launch_gemm_a8_tiled(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y, int y_dt,
                                int32_t *partials, hipStream_t stream);
hipError_t launch_gemv_a8_generic(const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y, int y_dt,
                                  int32_t *partials, hipStream_t stream);

// Family predicates, defaults and launches (select.cpp).  Families are the
// CQ_FAMILY_* values; path 0 = model dtype, 1 = Dynamic A8.
bool family_supported(int path, int family, const cq_weight &w, int64_t m);
int default_family(int path, const cq_weight &w, int64_t m, int64_t gemv_max_rows, bool partials);
// table entry for this call, or CQ_FAMILY_AUTO
int table_family(int path, const cq_weight &w, int x_dt, int64_t m);
hipError_t run_family_a16(int family, const cq_weight &w, const void *x, int x_dt, int64_t m, void *y, int y_dt,
                          hipStream_t stream);
hipError_t run_family_a8(int family, const cq_weight &w, const int8_t *x8, const float *dx, int64_t m, void *y,
                         int y_dt, int32_t *partials, hipStream_t stream);
bool select_entry_valid(const cq_select_entry &e);
// sort the entries into table order; false if two of them can match one call
bool select_sort_disjoint(std::vector<cq_select_entry> &entries);
// replace the table (empty clears it)
void select_install(std::vector<cq_select_entry> entries);

// Pure streaming read (measurement aid).
hipError_t launch_read_probe(const void *buf, int64_t bytes, uint32_t *sink, hipStream_t stream);

}  // namespace cq
