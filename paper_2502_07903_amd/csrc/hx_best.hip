// hx_best.hip -- the best candidate: highest flow value, lowest index on ties (the Sec. 3.1
// objective; Sec. 3.4 keeps the placement with the larger max-flow).
//
// One workgroup of 1024 lanes: each lane scans a strided slice with coalesced loads, keeping
// its first maximum; the wavefront reduces with cross-lane shuffles and the 16 wavefront
// winners meet in LDS.  Order of comparison makes the result independent of the launch shape.
#include <limits.h>

#include "hx_internal.h"

namespace hx {
namespace {

constexpr int kBestBlock = 1024;

__device__ __forceinline__ void take(int32_t& bv, int32_t& bi, int32_t v, int32_t i) {
    if (v > bv || (v == bv && i < bi)) {
        bv = v;
        bi = i;
    }
}

__global__ void __launch_bounds__(kBestBlock) best_kernel(const int32_t* __restrict__ v, int32_t n, int32_t* best) {
    __shared__ int32_t wv[kBestBlock / 64], wi[kBestBlock / 64];
    const int tid = threadIdx.x;
    int32_t bv = INT_MIN, bi = INT_MAX;
    // Eight independent coalesced loads in flight per lane, then the compares in index order.
    constexpr int kUnroll = 8;
    int64_t i = tid;
    for (; i + (kUnroll - 1) * kBestBlock < n; i += kUnroll * kBestBlock) {
        int32_t x[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) x[k] = v[i + k * kBestBlock];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) take(bv, bi, x[k], (int32_t)(i + k * kBestBlock));
    }
    for (; i < n; i += kBestBlock) take(bv, bi, v[i], (int32_t)i);
    for (int off = 32; off > 0; off >>= 1) {
        const int32_t ov = __shfl_down(bv, off, 64);
        const int32_t oi = __shfl_down(bi, off, 64);
        take(bv, bi, ov, oi);
    }
    const int w = tid >> 6, lane = tid & 63;
    if (lane == 0) {
        wv[w] = bv;
        wi[w] = bi;
    }
    __syncthreads();
    if (tid == 0) {
        int32_t gv = wv[0], gi = wi[0];
        for (int k = 1; k < kBestBlock / 64; ++k) take(gv, gi, wv[k], wi[k]);
        best[0] = gi;
        best[1] = gv;
    }
}

}  // namespace

hipError_t launch_best(const int32_t* flow_value, int32_t n, int32_t* best, hipStream_t s) {
    hipLaunchKernelGGL(best_kernel, dim3(1), dim3(kBestBlock), 0, s, flow_value, n, best);
    return hipGetLastError();
}

}  // namespace hx
