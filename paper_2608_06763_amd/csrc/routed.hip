// Routed (mixture-of-experts) product, model dtype (Sec. 5.5, workload regimes
// and routed execution): every active route (token t, expert e) of a route
// map supplied by the caller gives one route-major output row
// y[r] = x[t] W_e^T, W_e the packed expert e of a bank of equally shaped
// experts stacked along the rows.
//
// Routes are compacted and grouped by expert on the device, so the call
// needs no host synchronisation and can be captured in a graph: one
// workgroup histograms the routes by expert in LDS, scans the counts into
// offsets and scatters the route ids into an expert-grouped order (the order
// inside an expert is that of the atomics: the rows of a chunk are independent
// in the product, so it changes no output bit).  Routes naming a token or an
// expert outside the inputs are dropped and their output rows left
// unwritten.  The product then runs the narrow-row matrix-core GEMV with one
// workgroup per (expert, 16-row strip): every decoded weight tile serves all
// routes of its expert, 16 gathered activation rows at a time.
#include "cq_device.h"
#include "cq_internal.h"

#include <mutex>

namespace cq {

constexpr int kRouteThreads = 1024;

// Device scratch of the no-allocation routed call: the expert offsets and the
// grouped route order (n_experts + 1 + routes ints), one array per device,
// held until the process ends.  Host code never names it directly: its device
// address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) int32_t scratch[kNoAllocRoutedInts];

// offsets: [E + 1]; order: [R].  counters in dynamic LDS: E + 1 ints, the last
// one counts dropped routes.
__global__ void __launch_bounds__(kRouteThreads) route_group_kernel(const int32_t *__restrict__ token,
                                                                    const int32_t *__restrict__ expert, int routes,
                                                                    int n_experts, int tokens,
                                                                    int32_t *__restrict__ offsets,
                                                                    int32_t *__restrict__ order) {
    extern __shared__ int cnt[];
    __shared__ int scan[kRouteThreads];
    const int tid = threadIdx.x;
    for (int e = tid; e <= n_experts; e += kRouteThreads) cnt[e] = 0;
    __syncthreads();
    auto bucket = [&](int r) {
        const int t = token[r], e = expert[r];
        return (t >= 0 && t < tokens && e >= 0 && e < n_experts) ? e : n_experts;
    };
    for (int r = tid; r < routes; r += kRouteThreads) atomicAdd(&cnt[bucket(r)], 1);
    __syncthreads();
    // exclusive scan of the E expert counts: each thread sums a contiguous
    // chunk, the chunk sums are scanned in LDS, then each chunk is written
    const int per = (n_experts + kRouteThreads - 1) / kRouteThreads;
    const int lo = min(tid * per, n_experts), hi = min(lo + per, n_experts);
    int sum = 0;
    for (int e = lo; e < hi; ++e) sum += cnt[e];
    scan[tid] = sum;
    __syncthreads();
    for (int d = 1; d < kRouteThreads; d <<= 1) {
        const int v = tid >= d ? scan[tid - d] : 0;
        __syncthreads();
        scan[tid] += v;
        __syncthreads();
    }
    int run = scan[tid] - sum;  // exclusive prefix of this chunk
    for (int e = lo; e < hi; ++e) {
        const int c = cnt[e];
        offsets[e] = run;
        cnt[e] = run;  // becomes the expert's write cursor
        run += c;
    }
    if (tid == kRouteThreads - 1) offsets[n_experts] = scan[tid];
    __syncthreads();
    for (int r = tid; r < routes; r += kRouteThreads) {
        const int e = bucket(r);
        if (e < n_experts) order[atomicAdd(&cnt[e], 1)] = r;
    }
}

bool routed_supported(const cq_weight &w, int64_t n_experts, int64_t tokens, int64_t routes) {
    return n_experts >= 1 && n_experts <= 16384 && routes <= 0x7fffffff && tokens <= 0x7fffffff &&
           gemv_a16_routed_supported(w, tokens);
}

hipError_t launch_routed_model_dtype(const cq_weight &w, int n_experts, const void *x, int x_dt, int64_t tokens,
                                     const int32_t *token, const int32_t *expert, int64_t routes, int32_t *workspace,
                                     void *y, int y_dt, hipStream_t stream) {
    // At most one route per two experts (decode of one or two tokens): every
    // route streams its expert's weights once, with no grouping pass.  More
    // routes: the expert-grouped matrix-core path decodes each weight tile
    // once for up to 16 routes of its expert, which wins as soon as experts
    // share routes (and on skewed maps, where streaming would read one expert
    // once per route).
    if (2 * routes <= n_experts && gemv_a16_stream_routed_supported(w, n_experts, tokens, routes))
        return launch_gemv_a16_stream_routed(w, n_experts, x, x_dt, tokens, token, expert, routes, y, y_dt, stream);
    int32_t *offsets = workspace;
    int32_t *order = workspace + n_experts + 1;
    const size_t lds = sizeof(int) * size_t(n_experts + 1);
    hipLaunchKernelGGL(route_group_kernel, dim3(1), dim3(kRouteThreads), lds, stream, token, expert, int(routes),
                       n_experts, int(tokens), offsets, order);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (gemm_a16_slab_routed_supported(w, tokens))
        return launch_gemm_a16_slab_routed(w, n_experts, x, x_dt, tokens, routes, token, order, offsets, y, y_dt,
                                           stream);
    return launch_gemv_a16_routed(w, n_experts, x, x_dt, tokens, token, order, offsets, y, y_dt, stream);
}

namespace {

constexpr int kMaxScratchDevices = 64;
struct scratch_slot {
    std::once_flag once;
    int32_t *ptr = nullptr;
    hipError_t err = hipSuccess;
};
scratch_slot g_scratch[kMaxScratchDevices];

}  // namespace

hipError_t routed_scratch(int32_t **ptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
    scratch_slot &s = g_scratch[dev];
    // first call on this device, with it current: the array's address there
    std::call_once(s.once, [&s] {
        void *p = nullptr;
        s.err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (s.err == hipSuccess) s.ptr = static_cast<int32_t *>(p);
    });
    *ptr = s.ptr;
    return s.err;
}

hipError_t launch_routed_model_dtype_noalloc(const cq_weight &w, int n_experts, const void *x, int x_dt,
                                             int64_t tokens, const int32_t *token, const int32_t *expert,
                                             int64_t routes, void *y, int y_dt, hipStream_t stream) {
    int32_t *ws = nullptr;
    const hipError_t e = routed_scratch(&ws);
    if (e != hipSuccess) return e;
    return launch_routed_model_dtype(w, n_experts, x, x_dt, tokens, token, expert, routes, ws, y, y_dt, stream);
}

}  // namespace cq
