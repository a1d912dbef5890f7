/*
 * cq.h -- C ABI of the CubicQuant hot path on AMD Instinct MI355X (gfx950).
 *
 * CubicQuant (arXiv 2608.06763) stores a weight matrix W of logical shape
 * N x K (output rows x input channels) as:
 *   - a packed B-bit code stream, B in 1..8 (Sec. 2.1, eq. codes): codes
 *     k in [-M, M] with M = 2^(B-1) - 1, stored as two's-complement B-bit
 *     fields; the pattern -2^(B-1) is reserved and decodes to zero; W1 stores
 *     one bit per weight, 1 meaning +1 and 0 meaning -1.  Fields are laid out
 *     row-major as one continuous bitstream per row, least significant bit
 *     first: field j of a row occupies stream bits [jB, jB+B), and stream bit
 *     p is bit (p mod 8) of byte floor(p/8) (Sec. 2.1, Sec. 5.2
 *     eq. gpu-packed-extraction).  Fields may straddle bytes (W3, W5..W7).
 *   - per [1, G] group along K (Sec. 2.3): one FP32 scale s and two FP16
 *     shape values a, b, as three row-major N x (K/G) tensors.  c = 1 - a - b
 *     is derived.  64 bits of metadata per group, B + 64/G bits per weight
 *     (eq. effective-bits).
 * A code k of a group decodes to w = sign(k) s q(|k|/M) with
 * q(t) = t [a + t (b + c t)] (Sec. 2.2, eq. cubic); W1 decodes to k s.
 *
 * Conventions for every call:
 *   - All pointers marked "device" are HIP device pointers; the caller owns
 *     every buffer and keeps it alive until the stream has finished the call.
 *     The library allocates no memory in any call declared here and keeps no
 *     state besides a per-device property cache and the scratch array of
 *     cq_gemm_routed_model_dtype_noalloc.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Device calls are asynchronous and stream ordered; they validate their
 *     arguments on the host in O(1) and return a status synchronously.  A
 *     launch failure is reported as CQ_ERR_HIP.  A fault inside a kernel
 *     surfaces at the caller's next synchronisation.
 *   - Device pointers must be 16-byte aligned (CQ_ERR_ALIGN otherwise).
 *   - Row strides are dense: codes rows are K*B/8 bytes, metadata rows K/G
 *     entries, activations rows K elements, outputs rows N elements.
 *   - Hot calls assume metadata validated by cq_pack_groups (finite,
 *     admissible shapes); they never read outside the described buffers for
 *     any metadata values.
 *   - All calls are thread safe.
 */
#ifndef CQ_H
#define CQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CQ_OK = 0,
    CQ_ERR_ARG = 1,          /* null pointer, bad width, bad group, m or k <= 0  */
    CQ_ERR_SHAPE = 2,        /* K % G != 0, K*B % 128 != 0, size overflow        */
    CQ_ERR_ALIGN = 3,        /* a device pointer is not 16-byte aligned          */
    CQ_ERR_META = 4,         /* scale or shape values rejected by cq_pack_groups */
    CQ_ERR_CODE = 5,         /* code outside [-M, M] (W1: outside {-1, +1})      */
    CQ_ERR_DTYPE = 6,        /* unsupported activation / output dtype            */
    CQ_ERR_HIP = 7,          /* a HIP runtime call or a kernel launch failed     */
    CQ_ERR_UNSUPPORTED = 8   /* valid request this build has no kernel for       */
} cq_status;

typedef enum { CQ_BF16 = 0, CQ_FP16 = 1, CQ_FP32 = 2 } cq_dtype;

/* Borrowed description of one packed weight matrix (never retained). */
typedef struct {
    int32_t bits;            /* B in 1..8                                        */
    int32_t group;           /* G: multiple of 32, 32 <= G <= 512                */
    int64_t n;               /* N output rows                                    */
    int64_t k;               /* K input channels; K % G == 0, K*B % 128 == 0     */
    const uint8_t *codes;    /* device, N x (K*B/8) bytes                        */
    const float *scale;      /* device, N x (K/G) FP32                           */
    const uint16_t *a;       /* device, N x (K/G) FP16 bit patterns              */
    const uint16_t *b;       /* device, N x (K/G) FP16 bit patterns              */
} cq_weight;

/* Human-readable name of a status code (static string, never NULL). */
const char *cq_status_str(cq_status s);

/*
 * cq_pack_groups -- validate one quantized matrix and pack its codes (host).
 *
 * Implements the storage format of Sec. 2.1-2.3 and Appendix A.  Every
 * pointer is a HOST pointer.
 *   codes      N x K signed codes, row-major: [-M, M] for B >= 2 (the reserved
 *              pattern is never emitted), {-1, +1} for B = 1.
 *   scale      N x (K/G) FP32; finite and >= 0; 0 only for a group whose codes
 *              are all zero (B >= 2).
 *   a, b       N x (K/G) FP16 bit patterns; finite.  For B >= 3 the curve must
 *              be strictly monotone: m(a, b) > 0 evaluated in float64 on the
 *              FP16 values (Sec. 3.1, eq. shape-domain; Appendix A item 5).
 *   packed_out N x (K*B/8) bytes, written only when the call succeeds.
 *   bad_index  optional; on CQ_ERR_CODE receives the flat index of the first
 *              bad code, on CQ_ERR_META the flat index of the first bad group.
 * Group constraints: G*B % 8 == 0, K % G == 0 (CQ_ERR_SHAPE otherwise).  The
 * host packer accepts any G >= 1 with those properties; device calls further
 * require G % 32 == 0, G <= 512 and K*B % 128 == 0.
 * Integer-only and bit exact; O(N K); runs on the calling thread.
 */
cq_status cq_pack_groups(int32_t bits, int32_t group, int64_t n, int64_t k,
                         const int8_t *codes, const float *scale,
                         const uint16_t *a, const uint16_t *b,
                         uint8_t *packed_out, int64_t *bad_index);

/*
 * cq_decode_ref -- materialising decode of a packed matrix (device).
 *
 * Unpacks every field with the byte/shift rule of eq. gpu-packed-extraction,
 * sign-extends it and maps the reserved pattern to 0 (W1: 2u - 1), and
 * reconstructs w = sign(k) s q(|k|/M) in FP32 (Sec. 5.2, Horner form
 * eq. gpu-horner).  This is the test reference for the fused kernels and the
 * "expand, then multiply" baseline; the hot calls never use it.
 *   codes_out  optional device int8 [N, K]: the signed codes (bit exact).
 *   w_out      optional device float [N, K]: the FP32 reconstruction.
 * At least one output must be non-NULL.
 */
cq_status cq_decode_ref(const cq_weight *w, int8_t *codes_out, float *w_out, void *stream);

/*
 * cq_gemm_model_dtype -- y = x W_hat^T with BF16/FP16 activations (device).
 *
 * Model-dtype execution of Sec. 5.3: the packed payload and group metadata
 * are decoded inside the kernel and consumed immediately; no expanded weight
 * is written.  Narrow row counts use a weight-streaming GEMV; many rows use a
 * tiled matrix-core GEMM that forms s*q as a BF16/FP16 operand (the dense
 * rounding point of Sec. 5.3).  Accumulation is FP32.
 *   x        device [M, K] in x_dtype (CQ_BF16 or CQ_FP16), row-major.
 *   m        rows of x, >= 1.
 *   y        device [M, N] in y_dtype: x_dtype, or CQ_FP32 (diagnostics).
 * The result is deterministic for a given device, shape and dtype.
 */
cq_status cq_gemm_model_dtype(const cq_weight *w, const void *x, cq_dtype x_dtype, int64_t m,
                              void *y, cq_dtype y_dtype, void *stream);

/*
 * cq_quantize_act_a8 -- dynamic per-row INT8 activation carrier (device).
 *
 * Sec. 5.4, eq. a8-activation-scale and eq. a8-activation-quantization:
 *   xbar = max(max_j |x_j|, eps), eps = 1e-10 rounded to FP32,
 *   d_x = xbar / 127 (IEEE FP32 division),
 *   x8_j = clip(round_half_away(x_j / d_x), -127, 127) (IEEE FP32 division).
 *   x    device [M, K] in x_dtype (CQ_BF16 or CQ_FP16).
 *   x8   device int8 [M, K];  dx  device float [M].
 * Bit exact.  An all-zero row yields zero carriers and d_x = eps/127.
 */
cq_status cq_quantize_act_a8(const void *x, cq_dtype x_dtype, int64_t m, int64_t k,
                             int8_t *x8, float *dx, void *stream);

/*
 * cq_gemm_a8 -- Dynamic-A8 product from INT8 activation carriers (device).
 *
 * Sec. 5.4, eq. a8-output: every weight maps to the INT8 carrier
 * r(k) = sign(k) RNE(127 q(|k|/M)) (Sec. 4.3 eq. carrier; round to nearest
 * even of the exact value from the FP16 shapes, Appendix A item 7; W1 +-127),
 * each group forms the exact INT32 partial P_g = sum_j x8_j r(k_j)
 * (|P_g| <= G 127^2, eq. a8-int32-bound), and
 *   y = sum_g (d_x s_g / 127) P_g
 * with the rescale and the cross-group sum in FP32.
 *   x8, dx        outputs of cq_quantize_act_a8 for the same M and K.
 *   y             device [M, N] in y_dtype (CQ_BF16, CQ_FP16 or CQ_FP32).
 *   partials_dbg  optional device int32 [M, N, K/G] receiving every P_g
 *                 (a debugging output; it slows the call down).
 */
cq_status cq_gemm_a8(const cq_weight *w, const int8_t *x8, const float *dx, int64_t m,
                     void *y, cq_dtype y_dtype, int32_t *partials_dbg, void *stream);

/*
 * cq_gemm_a8_fused -- Dynamic-A8 product from model-dtype activations (device).
 *
 * Same result as cq_quantize_act_a8 followed by cq_gemm_a8 (Sec. 5.4): x8 and
 * dx receive the carriers and d_x, bit-exact; y follows eq. a8-output.  By
 * default it runs exactly those two calls in order on the stream, which
 * measured faster on MI355X than the single launch on every decode layer.
 * With cq_set_a8_fused_launch(1), a single row (m == 1, B <= 4, K <= 16384,
 * and m within the A8 GEMV threshold) is one launch instead: the GEMV forms
 * the row's carriers itself in a prologue, which removes the separate
 * encoding pass the paper names as the fixed cost of the single-row A8 path
 * (Sec. 6).  The FP32 summation order of the single launch can differ from
 * cq_gemm_a8's for the same row, so its y agrees with the two calls' to
 * rounding, not bit for bit.
 *   x        device [M, K] in x_dtype (CQ_BF16 or CQ_FP16).
 *   x8, dx   device int8 [M, K] and float [M], written (caller-owned).
 *   y        device [M, N] in y_dtype (CQ_BF16, CQ_FP16 or CQ_FP32).
 * Errors as cq_quantize_act_a8 and cq_gemm_a8.
 */
cq_status cq_gemm_a8_fused(const cq_weight *w, const void *x, cq_dtype x_dtype, int64_t m,
                           int8_t *x8, float *dx, void *y, cq_dtype y_dtype, void *stream);

/*
 * How cq_gemm_a8_fused runs a single row: 0 (default) the quantizer and the
 * product as two launches, 1 the single fused launch where it applies.  Other
 * values are CQ_ERR_ARG.  Host only, process wide; a call already past its
 * dispatch is not affected.
 */
cq_status cq_set_a8_fused_launch(int32_t single);
int32_t cq_get_a8_fused_launch(void);

/*
 * cq_build_carriers -- load-time INT8 carrier tables (device).
 *
 * Sec. 4.3 eq. carrier, precomputed once per weight (the interior carriers
 * of Sec. 5.2): for every (row, group) the table holds r(i) = RNE(127 q(i/M))
 * for i = 0 .. 2^(B-1) - 1, exact from the FP16 shapes (r(0) = 0, r(M) = 127),
 * one int8 each.  It depends only on (a, b): codes and metadata are unchanged.
 *   carriers  device int8 [N, K/G, 2^(B-1)], 16-byte aligned (caller-owned).
 *             W1 has no table (its carriers are +-127): nothing is written and
 *             carriers may be NULL.
 */
cq_status cq_build_carriers(const cq_weight *w, int8_t *carriers, void *stream);

/*
 * cq_gemm_a8_carriers -- Dynamic-A8 product with load-time carriers (device).
 *
 * Same result as cq_gemm_a8 (without the partials dump), bit for bit: the
 * kernels read the carriers of cq_build_carriers for the same weight instead
 * of forming them (the many-row W4 matrix-core GEMM and the generic kernels
 * of the other widths; the single-row kernels and the W3/W4 narrow-row
 * kernels, up to 32 rows, keep their register decode, which gives the same
 * carriers).
 *   carriers  the table of cq_build_carriers (NULL allowed for W1).
 * Errors as cq_gemm_a8.
 */
cq_status cq_gemm_a8_carriers(const cq_weight *w, const int8_t *carriers, const int8_t *x8,
                              const float *dx, int64_t m, void *y, cq_dtype y_dtype, void *stream);

/*
 * cq_gemm_routed_model_dtype -- routed (mixture-of-experts) product (device).
 *
 * Sec. 5.5 (workload regimes and routed execution): for every route
 * r = (route_token[r], route_expert[r]) of a route map supplied by the
 * caller, y[r] = x[route_token[r]] W_e^T with W_e = expert route_expert[r]
 * of the bank, in the model-dtype arithmetic of cq_gemm_model_dtype (FP32
 * products and accumulation).  Outputs are route-major; routing weights and
 * expert choice stay with the caller.  No host synchronisation: with at
 * most one route per expert on average (routes <= n_experts, the decode
 * case) every route streams its expert's weights through the single-row
 * kernel; otherwise routes are grouped by expert on the device and every
 * decoded weight tile serves all routes of its expert (Sec. 5.5's
 * compaction and grouping).
 *   bank          n_experts experts of equal shape stacked along the rows:
 *                 bank->n is the row count of ONE expert, and codes, scale, a
 *                 and b hold n_experts * bank->n rows (expert e first at row
 *                 e * bank->n).  B <= 5 (otherwise CQ_ERR_UNSUPPORTED).
 *   x             device [tokens, K] in x_dtype (CQ_BF16 or CQ_FP16).
 *   route_token   device int32 [routes]; route_expert  device int32 [routes].
 *                 Routes naming a token outside [0, tokens) or an expert
 *                 outside [0, n_experts) are dropped: their rows of y are not
 *                 written.
 *   workspace     device int32 [n_experts + 1 + routes], caller-owned scratch
 *                 (expert offsets and the grouped route order; not touched
 *                 in the streaming case).
 *   y             device [routes, bank->n] in y_dtype: x_dtype or CQ_FP32.
 * Deterministic: a route's output does not depend on the other routes.
 */
cq_status cq_gemm_routed_model_dtype(const cq_weight *bank, int32_t n_experts, const void *x,
                                     cq_dtype x_dtype, int64_t tokens, const int32_t *route_token,
                                     const int32_t *route_expert, int64_t routes, int32_t *workspace,
                                     void *y, cq_dtype y_dtype, void *stream);

/*
 * cq_gemm_routed_model_dtype_noalloc -- the routed product without a caller
 * workspace, for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation).
 *
 * Arguments, result and routing rules as cq_gemm_routed_model_dtype, minus
 * `workspace`: the expert grouping uses a scratch array that the library
 * holds on each device for the life of the process (4 MiB per device, found
 * on the first call on a device).  Limit: n_experts + 1 + routes <= 2^20
 * (CQ_ERR_SHAPE otherwise, before anything is launched).  The call allocates
 * nothing.  All calls on one device share its scratch: calls that can overlap
 * on that device (other streams, other host threads) race on it and must be
 * ordered by the caller; calls on one stream are ordered.  Nothing in the
 * scratch needs to start at zero (every entry read is first written by the
 * same call).
 */
cq_status cq_gemm_routed_model_dtype_noalloc(const cq_weight *bank, int32_t n_experts, const void *x,
                                             cq_dtype x_dtype, int64_t tokens, const int32_t *route_token,
                                             const int32_t *route_expert, int64_t routes, void *y,
                                             cq_dtype y_dtype, void *stream);

/*
 * Row-regime kernel selection (Sec. 5.5-5.6).  Each path picks the GEMV
 * family for m <= its threshold and the tiled GEMM family above it.  The
 * defaults come from measurements on MI355X.  cq_set_gemv_max_rows
 * overrides the threshold for one path (0 = model dtype, 1 = Dynamic A8);
 * a negative value restores the default.  Intended for tests and
 * benchmarks; process wide.
 */
cq_status cq_set_gemv_max_rows(int32_t path, int64_t max_rows);
int64_t cq_get_gemv_max_rows(int32_t path);

/*
 * Measured shape- and device-dependent kernel selection (Sec. 5.6).
 *
 * The paper treats the choice of kernel family as an optimisation over the
 * operator signature (B, G, M, N, K, activation dtype) on the measured device:
 * candidates are filtered by width, dtype and structural constraints, the
 * valid ones are timed on representative row counts, and the winner is a
 * deterministic function of signature and device.  Selection changes neither
 * codes nor metadata.  These calls expose the families (for a tuner to time
 * them) and a process-wide table that the dispatcher of cq_gemm_model_dtype
 * and cq_gemm_a8 consults before its built-in rules.
 *
 * Paths: CQ_PATH_MODEL_DTYPE (cq_gemm_model_dtype), CQ_PATH_A8 (cq_gemm_a8).
 * Families (CQ_FAMILY_AUTO = the built-in rules):
 *   GEMV_STREAM   single-row streaming GEMV (m == 1)
 *   GEMV_LUT      model dtype only, per-wave level tables (m <= 4, G <= 128;
 *                 m == 1 at G == 256)
 *   GEMV_NARROW   matrix-core narrow-row GEMV (model dtype 2 <= m <= 16,
 *                 B <= 5; A8 2 <= m <= 32, W3 and W4 with G >= 64, two
 *                 16-row blocks of x per decoded operand above 16 rows)
 *   GEMV_GENERIC  conservative one-wave-per-row GEMV (m <= 16, every B, G)
 *   GEMM_MFMA     tiled matrix-core GEMM (model dtype B <= 5; A8 W3/W4 with
 *                 G >= 64)
 *   GEMM_TILED    conservative 64 x 64 tiled GEMM (every B, G)
 *   GEMM_MFMA_ROUNDED  model dtype only: the tiled matrix-core GEMM with the
 *                 decoded weight s_g q rounded once to the activation dtype
 *                 before the dot, the dense rounding point of Sec. 5.3 (BF16:
 *                 one MFMA per product; GEMM_MFMA carries the BF16 operand as
 *                 hi + lo).  Every weight then carries a relative error of up
 *                 to 2^-8: measured 0.7e-3 to 2.1e-3 of max|y| on the
 *                 benchmark layers (hi + lo: about 1e-6), above the 2e-3
 *                 budget on some, so the built-in rules never pick it; a
 *                 caller's selection table may.
 *   GEMM_MFMA_M32, _M64, _M128, _M256  GEMM_MFMA with a fixed x-tile height
 *                 (rows of x per workgroup tile; the tile-height dimension of
 *                 the selection in Sec. 5.6).  GEMM_MFMA picks the smallest of
 *                 32, 64, 128 that holds m, else 256 (an A8 partials dump
 *                 always runs the 256-row tile).  Same widths as GEMM_MFMA.
 *   GEMM_SLAB     model dtype only, 1 <= m <= 32, B <= 5: matrix-core GEMM for
 *                 few rows in which every lane decodes its codes straight into
 *                 its own MFMA operand (no decoded tile in LDS, no barrier in
 *                 the K loop) and the waves of a workgroup split K; numerics
 *                 as GEMM_MFMA (hi + lo operand in the activation dtype, FP32
 *                 accumulation).
 *   GEMM_SLAB_STAGED  model dtype only, 1 <= m <= 32, G <= 128, G B <= 512,
 *                 K / G a multiple of 4: GEMM_SLAB whose waves each take a
 *                 contiguous K range and bring codes and group metadata in
 *                 through LDS with whole-cache-line loads; same numerics.
 *                 Above 16 rows each wave serves two 16-row blocks of x.
 *                 The built-in rules pick it when the K split gives the
 *                 waves two or more sweeps of four groups each.
 *   GEMV_ROWS     model dtype only, m == 1, K <= 16384: GEMV_STREAM with one
 *                 wave per 2048-code column block of K in every workgroup;
 *                 each wave converts its slice of x once and streams only
 *                 codes and metadata over many row tiles, and the waves'
 *                 sums meet in LDS; numerics as GEMV_STREAM.  The built-in
 *                 rules pick it when every workgroup gets three or more row
 *                 tiles.
 * Families that read 32-bit buffer offsets also need tensors below 2 GiB.
 */
typedef enum { CQ_PATH_MODEL_DTYPE = 0, CQ_PATH_A8 = 1 } cq_path;
typedef enum {
    CQ_FAMILY_AUTO = 0,
    CQ_FAMILY_GEMV_STREAM = 1,
    CQ_FAMILY_GEMV_LUT = 2,
    CQ_FAMILY_GEMV_NARROW = 3,
    CQ_FAMILY_GEMV_GENERIC = 4,
    CQ_FAMILY_GEMM_MFMA = 5,
    CQ_FAMILY_GEMM_TILED = 6,
    CQ_FAMILY_GEMM_MFMA_ROUNDED = 7,
    CQ_FAMILY_GEMM_MFMA_M32 = 8,
    CQ_FAMILY_GEMM_MFMA_M64 = 9,
    CQ_FAMILY_GEMM_MFMA_M128 = 10,
    CQ_FAMILY_GEMM_MFMA_M256 = 11,
    CQ_FAMILY_GEMM_SLAB = 12,
    CQ_FAMILY_GEMM_SLAB_STAGED = 13,
    CQ_FAMILY_GEMV_ROWS = 14
} cq_family;

/*
 * 1 if `family` can run `path` for this weight and row count, else 0 (also 0
 * for invalid arguments).  Host only: reads the descriptor's fields, never
 * its device memory.
 */
int32_t cq_family_supported(int32_t path, int32_t family, const cq_weight *w, int64_t m);

/*
 * cq_gemm_model_dtype / cq_gemm_a8 forced onto one family (for timing and
 * for checking that every family computes the same product).  Arguments and
 * results as in those calls (no partials dump); CQ_ERR_UNSUPPORTED, before
 * anything is launched, when cq_family_supported would return 0.
 * CQ_FAMILY_AUTO runs the ordinary dispatch.
 */
cq_status cq_gemm_model_dtype_family(const cq_weight *w, const void *x, cq_dtype x_dtype, int64_t m,
                                     void *y, cq_dtype y_dtype, int32_t family, void *stream);
cq_status cq_gemm_a8_family(const cq_weight *w, const int8_t *x8, const float *dx, int64_t m, void *y,
                            cq_dtype y_dtype, int32_t family, void *stream);

/*
 * One row of the selection table: calls on `path` with exactly this (bits,
 * group, n, k), activation dtype x_dtype (CQ_BF16 or CQ_FP16; -1 matches
 * both; A8 entries take -1) and m_lo <= m <= m_hi run `family`.
 */
typedef struct {
    int32_t path, family;
    int32_t bits, group;
    int64_t n, k;
    int64_t m_lo, m_hi;
    int32_t x_dtype;
    int32_t reserved; /* must be 0 */
} cq_select_entry;

/*
 * Replace the process-wide table with a copy of entries[0 .. count) (count 0
 * clears it).  Host only.  CQ_ERR_ARG, with the previous table kept, if an
 * entry is malformed (unknown path or family, CQ_FAMILY_AUTO, the LUT,
 * ROUNDED or either SLAB family on the A8 path, bits outside 1..8, a group that is not a multiple of 32 in
 * 32..512, n or k < 1, m_lo < 1 or m_hi < m_lo, a bad x_dtype, reserved != 0)
 * or if two entries of the same path, shape and dtype overlap in m; count
 * above 65536 is CQ_ERR_ARG too.  With overlaps rejected, at most one entry
 * matches a call (found by binary search over the shape, so large tables cost
 * no more per call than small ones); when its family cannot take the call
 * (cq_family_supported is 0) the built-in rules decide.  The table does not apply to a cq_gemm_a8 call that asks for the
 * partials dump, nor to cq_gemm_a8_fused, cq_gemm_a8_carriers or the routed
 * product.  Safe to call while other threads launch products; a call already
 * past its dispatch is not affected.
 */
cq_status cq_select_set(const cq_select_entry *entries, int64_t count);

/*
 * The family the dispatcher would run for this call (table first, then the
 * built-in rules, including the cq_set_gemv_max_rows threshold), written to
 * *family.  Host only.
 */
cq_status cq_select_query(int32_t path, const cq_weight *w, cq_dtype x_dtype, int64_t m, int32_t *family);

#ifdef __cplusplus
}
#endif

#endif /* CQ_H */
