// hx_probe.hip -- a measurement probe, not part of the scoring path: the LDS read bandwidth the
// chip sustains, the measured ceiling beside the datasheet one for the LDS-resident kernels
// (the max-flow residual graphs, the refinement closure).
//
// Each workgroup fills 16 KB of LDS, then every lane reads 16 bytes per load, the 64 lanes of a
// wavefront on consecutive 16-byte words (no bank conflicts), eight loads in flight at eight
// distinct addresses (so that none can be merged with another), for `reps` rounds.  The XOR of everything read is stored only if it equals a value the data cannot give,
// so the loads stay and nothing is written.
#include "hx_internal.h"

namespace hx {
namespace {

constexpr int kProbeBlock = 256;
constexpr int kProbeWords = 1024;  // 16-byte words: 16 KB per workgroup
constexpr int kProbeUnroll = 8;

__global__ void __launch_bounds__(kProbeBlock) lds_probe_kernel(int32_t reps, uint32_t* sink) {
    __shared__ uint4 buf[kProbeWords];
    for (int i = threadIdx.x; i < kProbeWords; i += kProbeBlock)
        buf[i] = make_uint4((uint32_t)i, (uint32_t)i * 3u + 1u, (uint32_t)i * 5u + 7u, (uint32_t)i ^ 0x55u);
    __syncthreads();
    uint4 acc = make_uint4(0u, 0u, 0u, 0u);
    int idx = threadIdx.x;
    for (int r = 0; r < reps; ++r) {
        uint4 v[kProbeUnroll];
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) v[u] = buf[(idx + u * (kProbeWords / kProbeUnroll)) & (kProbeWords - 1)];
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) {
            acc.x ^= v[u].x;
            acc.y ^= v[u].y;
            acc.z ^= v[u].z;
            acc.w ^= v[u].w;
        }
        idx = (idx + 64) & (kProbeWords - 1);
    }
    // every word's x and y halves are below 2^13, so their XOR never has the top bit set
    if ((acc.x & acc.y) == 0xFFFFFFFFu) sink[(int64_t)blockIdx.x * kProbeBlock + threadIdx.x] = acc.z ^ acc.w;
}

}  // namespace

hipError_t launch_lds_probe(int32_t blocks, int32_t reps, uint32_t* sink, hipStream_t s) {
    hipLaunchKernelGGL(lds_probe_kernel, dim3(blocks), dim3(kProbeBlock), 0, s, reps, sink);
    return hipGetLastError();
}

int64_t lds_probe_bytes(int32_t blocks, int32_t reps) {
    return (int64_t)blocks * kProbeBlock * 16 * kProbeUnroll * reps;
}

}  // namespace hx
