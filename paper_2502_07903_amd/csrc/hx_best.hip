// hx_best.hip -- the best candidate: highest flow value, lowest index on ties (the Sec. 3.1
// objective; Sec. 3.4 keeps the placement with the larger max-flow).
//
// One workgroup of 1024 lanes: each lane scans a strided slice with coalesced loads, keeping
// its first maximum; the wavefront reduces with cross-lane shuffles and the 16 wavefront
// winners meet in LDS.  Order of comparison makes the result independent of the launch shape.
#include <limits.h>
#include <stdint.h>

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
    // Lane t reads 16-byte vectors t, t + 1024, ... (coalesced), eight of them in flight per
    // batch, then compares in index order; a ragged head and tail are read one by one.
    const int head = (int)(((16 - ((uintptr_t)v & 15)) & 15) / 4);
    const int64_t h = head < n ? head : n;
    for (int64_t i = tid; i < h; i += kBestBlock) take(bv, bi, v[i], (int32_t)i);
    const int4* v4 = reinterpret_cast<const int4*>(v + h);
    const int64_t n4 = (n - h) / 4;
    constexpr int kUnroll = 8;
    int64_t q = tid;
    for (; q + (kUnroll - 1) * kBestBlock < n4; q += kUnroll * kBestBlock) {
        int4 x[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) x[k] = v4[q + k * kBestBlock];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int32_t base = (int32_t)(h + 4 * (q + k * kBestBlock));
            take(bv, bi, x[k].x, base);
            take(bv, bi, x[k].y, base + 1);
            take(bv, bi, x[k].z, base + 2);
            take(bv, bi, x[k].w, base + 3);
        }
    }
    for (; q < n4; q += kBestBlock) {
        const int4 x = v4[q];
        const int32_t base = (int32_t)(h + 4 * q);
        take(bv, bi, x.x, base);
        take(bv, bi, x.y, base + 1);
        take(bv, bi, x.z, base + 2);
        take(bv, bi, x.w, base + 3);
    }
    for (int64_t i = h + 4 * n4 + tid; i < n; i += kBestBlock) take(bv, bi, v[i], (int32_t)i);
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
    prof_mark(kKBest, false, s);
    hipLaunchKernelGGL(best_kernel, dim3(1), dim3(kBestBlock), 0, s, flow_value, n, best);
    prof_mark(kKBest, true, s);
    return hipGetLastError();
}

}  // namespace hx
