// Measurement aid: a pure streaming read of a device buffer, the HBM ceiling
// that the weight-streaming kernels are compared with.  Each workgroup reads
// one contiguous chunk (measured faster than a grid-stride walk, which opens
// many more DRAM pages at once), eight 16-byte vectors in flight per thread,
// and folds them into one word; the word is stored only if it equals a fixed
// constant, which keeps the loads alive without write traffic.
#include "cq_device.h"
#include "cq_internal.h"

namespace cq {

namespace {

constexpr int kProbeUnroll = 8;

__global__ void __launch_bounds__(256) read_probe(const uint4 *__restrict__ p, int64_t n16, int64_t per_block,
                                                  uint32_t *sink) {
    const int64_t beg = int64_t(blockIdx.x) * per_block;
    const int64_t end = beg + per_block < n16 ? beg + per_block : n16;
    uint32_t acc = 0;
    int64_t i = beg + threadIdx.x;
    for (; i + (kProbeUnroll - 1) * 256 < end; i += kProbeUnroll * 256) {
        uint4 v[kProbeUnroll];
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) v[u] = p[i + u * 256];
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < end; i += 256) {
        const uint4 a = p[i];
        acc ^= a.x ^ a.y ^ a.z ^ a.w;
    }
    if (acc == 0x9e3779b9u) sink[0] = acc;
}

}  // namespace

hipError_t launch_read_probe(const void *buf, int64_t bytes, uint32_t *sink, hipStream_t stream) {
    const int64_t n16 = bytes / 16;
    if (n16 < 1) return hipSuccess;
    // 32 workgroups per CU (measured best from 4 to 32), each one chunk
    int64_t blocks = int64_t(device_cu_count()) * 32;
    if (blocks > n16) blocks = n16;
    const int64_t per_block = (n16 + blocks - 1) / blocks;
    blocks = (n16 + per_block - 1) / per_block;
    hipLaunchKernelGGL(read_probe, dim3(unsigned(blocks)), dim3(256), 0, stream, static_cast<const uint4 *>(buf), n16,
                       per_block, sink);
    return hipGetLastError();
}

}  // namespace cq
