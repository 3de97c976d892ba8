// hx_best.hip -- the best candidate: highest flow value, lowest index on ties (the Sec. 3.1
// objective; Sec. 3.4 keeps the placement with the larger max-flow).
//
// One workgroup of 1024 lanes: each lane scans a strided slice with coalesced loads, keeping
// its first maximum; the wavefront reduces with cross-lane shuffles and the 16 wavefront
// winners meet in LDS.  Order of comparison makes the result independent of the launch shape.
// With a scratch area (hx_score_batch), up to 256 workgroups of 256 lanes each take a
// contiguous slice, and the last workgroup to finish reduces their winners.
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

constexpr int kPartBlock = 256;
constexpr int kPartMax = 256;        // workgroups of best_parts_kernel, at most
constexpr int kPartPerLane = 4;      // candidates per lane before another workgroup is added

__device__ __forceinline__ void wave_take(int32_t& bv, int32_t& bi) {
    for (int off = 32; off > 0; off >>= 1) {
        const int32_t ov = __shfl_down(bv, off, 64);
        const int32_t oi = __shfl_down(bi, off, 64);
        take(bv, bi, ov, oi);
    }
}

// Workgroup b takes candidates [b chunk, (b + 1) chunk); its winner goes to part[b] as
// value << 32 | index.  The workgroup whose ticket is the last reads every part (after the
// others' release fences) and writes best.
__global__ void __launch_bounds__(kPartBlock) best_parts_kernel(const int32_t* __restrict__ v, int32_t n, int32_t chunk,
                                                                int32_t* best, int32_t* counter, uint64_t* part) {
    __shared__ int32_t wv[kPartBlock / 64], wi[kPartBlock / 64];
    __shared__ int32_t last;
    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
    const int64_t lo = (int64_t)blockIdx.x * chunk;
    const int64_t hi = lo + chunk < n ? lo + chunk : n;
    int32_t bv = INT_MIN, bi = INT_MAX;
    // eight loads in flight per lane, the ones past the slice predicated off
    constexpr int kUnroll = 8;
    for (int64_t i = lo + tid; i < hi; i += kUnroll * kPartBlock) {
        int32_t x[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) x[k] = i + k * kPartBlock < hi ? v[i + k * kPartBlock] : INT_MIN;
#pragma unroll
        for (int k = 0; k < kUnroll; ++k)
            if (i + k * kPartBlock < hi) take(bv, bi, x[k], (int32_t)(i + k * kPartBlock));
    }
    wave_take(bv, bi);
    if (lane == 0) {
        wv[w] = bv;
        wi[w] = bi;
    }
    __syncthreads();
    if (tid == 0) {
        int32_t gv = wv[0], gi = wi[0];
        for (int k = 1; k < kPartBlock / 64; ++k) take(gv, gi, wv[k], wi[k]);
        __hip_atomic_store(&part[blockIdx.x], ((uint64_t)(uint32_t)gv << 32) | (uint32_t)gi, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
        __threadfence();
        last = atomicAdd(counter, 1) == (int32_t)gridDim.x - 1;
        __threadfence();
    }
    __syncthreads();
    if (!last) return;
    __threadfence();
    bv = INT_MIN;
    bi = INT_MAX;
    for (int b = tid; b < (int)gridDim.x; b += kPartBlock) {
        const uint64_t k = __hip_atomic_load(&part[b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        take(bv, bi, (int32_t)(uint32_t)(k >> 32), (int32_t)(uint32_t)k);
    }
    wave_take(bv, bi);
    if (lane == 0) {
        wv[w] = bv;
        wi[w] = bi;
    }
    __syncthreads();
    if (tid == 0) {
        int32_t gv = wv[0], gi = wi[0];
        for (int k = 1; k < kPartBlock / 64; ++k) take(gv, gi, wv[k], wi[k]);
        best[0] = gi;
        best[1] = gv;
        *counter = 0;
    }
}

// The fused argmax's last step: kFinalLanes lanes, each over every kFinalLanes-th slot, the
// largest key (argmax_key order) decoded to {index, value}.
constexpr int kFinalLanes = 1024;
static_assert(kArgSlots % kFinalLanes == 0, "whole slot rows per lane");
__global__ void __launch_bounds__(kFinalLanes) best_final_kernel(const unsigned long long* __restrict__ slots,
                                                                 int32_t* best) {
    __shared__ unsigned long long wk[kFinalLanes / 64];
    unsigned long long key = 0;
#pragma unroll
    for (int i = 0; i < kArgSlots / kFinalLanes; ++i) {
        const unsigned long long v = slots[i * kFinalLanes + threadIdx.x];
        key = v > key ? v : key;
    }
    for (int off = 32; off > 0; off >>= 1) {
        const unsigned long long o = __shfl_xor(key, off, 64);
        key = o > key ? o : key;
    }
    if ((threadIdx.x & 63) == 0) wk[threadIdx.x >> 6] = key;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kFinalLanes / 64; ++w) key = wk[w] > key ? wk[w] : key;
        best[0] = (int32_t)(0xFFFFFFFFu - (uint32_t)key);
        best[1] = (int32_t)((uint32_t)(key >> 32) ^ 0x80000000u);
    }
}

}  // namespace

hipError_t launch_best_final(const unsigned long long* slots, int32_t* best, hipStream_t s) {
    prof_mark(kKBest, false, s);
    hipLaunchKernelGGL(best_final_kernel, dim3(1), dim3(kFinalLanes), 0, s, slots, best);
    prof_mark(kKBest, true, s);
    return hipGetLastError();
}

hipError_t launch_best(const int32_t* flow_value, int32_t n, int32_t* best, hipStream_t s) {
    prof_mark(kKBest, false, s);
    hipLaunchKernelGGL(best_kernel, dim3(1), dim3(kBestBlock), 0, s, flow_value, n, best);
    prof_mark(kKBest, true, s);
    return hipGetLastError();
}

size_t best_parts_bytes() { return sizeof(uint64_t) * (kPartMax > kArgSlots ? kPartMax : kArgSlots); }

hipError_t launch_best_parts(const int32_t* flow_value, int32_t n, int32_t* best, int32_t* counter, uint64_t* part,
                             hipStream_t s) {
    const int64_t per = (int64_t)kPartBlock * kPartPerLane;
    int64_t blocks = (n + per - 1) / per;
    blocks = blocks < 1 ? 1 : blocks > kPartMax ? kPartMax : blocks;
    const int32_t chunk = (int32_t)((n + blocks - 1) / blocks);
    blocks = (n + chunk - 1) / chunk;  // every workgroup has a candidate
    prof_mark(kKBest, false, s);
    hipLaunchKernelGGL(best_parts_kernel, dim3((unsigned)blocks), dim3(kPartBlock), 0, s, flow_value, n, chunk, best,
                       counter, part);
    prof_mark(kKBest, true, s);
    return hipGetLastError();
}

}  // namespace hx
