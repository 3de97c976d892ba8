// hx_partition.hip -- the graph-partition phase of Sec. 3.2 as a candidate generator, on gfx950.
//
// The device graph has the GPUs as nodes, weighted by memory, and the links as edges, weighted by
// bandwidth.  Edge weights are whole MB/s of the symmetrised bandwidth (clamped to 2^47, which
// keeps every cut of a graph of up to 255 GPUs below 2^62), so every cut, gain and coarsened
// weight is an exact 64-bit integer sum and does not depend on the order of the additions; only
// the spectral step is floating point, and it sums in ascending index order.
//
//   graph_kernel      one lane per GPU pair: w = floor(((beta_de + beta_ed) * 0.5) / 1e6);
//   spectral_kernel   one workgroup: power iteration on (cap I - Lap) for the Fiedler direction,
//                     a lane per row (ascending products); the mean and the squared norm summed
//                     in ascending order by one lane (255 dependent additions, twice per
//                     iteration; the order depends only on the cluster, so a search computes it
//                     once); the GPUs ranked by (x, id);
//   partition_kernel  one workgroup per candidate: (i) the rotated spectral order cut into K
//                     memory-balanced groups, then Kernighan-Lin passes: a lane per pair of GPUs
//                     scores the swap from per-GPU group sums kept in LDS, a workgroup maximum
//                     picks the largest reduction (negative ones too; lowest pair on ties), the
//                     swap is made tentatively and its two GPUs locked; the pass keeps its best
//                     prefix and undoes the rest; (ii) groups coarsened into super nodes (LDS
//                     atomics) and split into prefill and decode by single flips that raise the
//                     cut; (iii) the projection written as the candidate's assign and role columns.
// Graph and integer work: no MFMA.
#include "hx_internal.h"

namespace hx {
namespace {

constexpr int kPgBlock = 256;   // >= HX_MAX_GPUS + 1: a lane per GPU
constexpr int kPgMaxK = 32;     // groups of one candidate
constexpr double kPgWeightMax = 140737488355328.0;  // 2^47 MB/s
constexpr int kKlPasses = 64;   // Kernighan-Lin passes at most

__global__ void graph_kernel(int G, const double* beta, int64_t* w) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)G * G) return;
    const int d = (int)(i / G), e = (int)(i - (int64_t)d * G);
    double v = 0.0;
    if (d != e) {
        v = floor(((beta[(int64_t)d * G + e] + beta[(int64_t)e * G + d]) * 0.5) / 1.0e6);
        if (!(v >= 0.0)) v = 0.0;
        if (v > kPgWeightMax) v = kPgWeightMax;
    }
    w[i] = (int64_t)v;
}

__global__ void __launch_bounds__(kPgBlock) spectral_kernel(int G, const int64_t* w, int iters, int32_t* order,
                                                            double* fiedler) {
    __shared__ double x[kPgBlock], y[kPgBlock], sq[kPgBlock];
    __shared__ double deg[kPgBlock];
    __shared__ double scal[2];
    const int d = threadIdx.x;
    if (d < G) {
        long long s = 0;
        for (int e = 0; e < G; ++e) s += w[(int64_t)e * G + d];  // column = row: w is symmetric
        deg[d] = (double)s;
        x[d] = (double)d - (double)(G - 1) * 0.5;
    }
    __syncthreads();
    if (d == 0) {
        double cap = 0.0;
        for (int e = 0; e < G; ++e)
            if (2.0 * deg[e] > cap) cap = 2.0 * deg[e];
        scal[0] = cap;
    }
    __syncthreads();
    const double cap = scal[0];
    for (int it = 0; it < iters; ++it) {
        if (d < G) {
            double s = 0.0;
            for (int e = 0; e < G; ++e) s = s + (double)w[(int64_t)e * G + d] * x[e];
            y[d] = (cap - deg[d]) * x[d] + s;
        }
        __syncthreads();
        if (d == 0) {
            double tot = 0.0;
            for (int e = 0; e < G; ++e) tot = tot + y[e];
            scal[1] = tot / (double)G;
        }
        __syncthreads();
        double yd = 0.0;
        if (d < G) {
            yd = y[d] - scal[1];
            sq[d] = yd * yd;
        }
        __syncthreads();
        if (d == 0) {
            double ss = 0.0;
            for (int e = 0; e < G; ++e) ss = ss + sq[e];
            scal[0] = sqrt(ss);
        }
        __syncthreads();
        const double nrm = scal[0];
        if (!(nrm > 0.0)) break;  // uniform: every lane read the same value
        if (d < G) x[d] = yd / nrm;
        __syncthreads();
    }
    __syncthreads();
    if (d < G) {
        const double xd = x[d];
        int rank = 0;
        for (int e = 0; e < G; ++e) rank += (x[e] < xd || (x[e] == xd && e < d)) ? 1 : 0;
        order[rank] = d;
        if (fiedler) fiedler[d] = xd;
    }
}

__device__ __forceinline__ void drain_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);  // this wave's LDS operations done (lgkmcnt(0))
    __syncthreads();
}

// (gain, pair) ordered by larger gain, then lower pair index; pair kNoPair = none.
constexpr int kNoPair = 0x7fffffff;
__device__ __forceinline__ bool better(long long g, int p, long long g2, int p2) {
    return p != kNoPair && (p2 == kNoPair || g > g2 || (g == g2 && p < p2));
}

// Workgroup best (gain, pair): every lane receives it.
__device__ void block_best(long long& g, int& p, long long* redg, int* redp) {
    for (int s = 32; s > 0; s >>= 1) {
        const long long og = __shfl_xor(g, s, 64);
        const int op = __shfl_xor(p, s, 64);
        if (better(og, op, g, p)) {
            g = og;
            p = op;
        }
    }
    if ((threadIdx.x & 63) == 0) {
        redg[threadIdx.x >> 6] = g;
        redp[threadIdx.x >> 6] = p;
    }
    __syncthreads();
    g = redg[0];
    p = redp[0];
    for (int k = 1; k < kPgBlock / 64; ++k)
        if (better(redg[k], redp[k], g, p)) {
            g = redg[k];
            p = redp[k];
        }
    __syncthreads();
}

struct PgArgs {
    int G, Kmax, N, L;
    double H, Hkv, B, s_in, s_out;
    const int64_t* w;        // [G][G]
    const int32_t* order;    // [G] spectral order
    const int32_t* gpu_type;
    const double* mem;       // [T] memory limits
    int T;
    const uint64_t* rnd;     // [N]
    uint8_t *assign, *role;  // [G][N], [Kmax][N]
};

// Exchange GPUs u and v (different groups): the per-GPU group sums follow (a lane per GPU), then
// lane 0 moves the two GPUs and the groups' memory.  The same call undoes it.
__device__ void pg_exchange(const PgArgs& a, int u, int v, int* grp, long long* gval, long long* gmem,
                            const long long* memv) {
    const int G = a.G, tid = threadIdx.x;
    const int A = grp[u], B = grp[v];
    if (tid < G) {
        const long long wxu = a.w[(int64_t)u * G + tid], wxv = a.w[(int64_t)v * G + tid];
        gval[tid * kPgMaxK + A] += wxv - wxu;
        gval[tid * kPgMaxK + B] += wxu - wxv;
    }
    __syncthreads();
    if (tid == 0) {
        gmem[A] += memv[v] - memv[u];
        gmem[B] += memv[u] - memv[v];
        grp[u] = B;
        grp[v] = A;
    }
    __syncthreads();
}

// Dynamic LDS of partition_kernel: gval[u][k], the sum of w(u, x) over the GPUs x of group k.
__host__ __device__ inline size_t pg_lds_bytes(int G) { return (size_t)G * kPgMaxK * sizeof(long long); }

__global__ void __launch_bounds__(kPgBlock) partition_kernel(PgArgs a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char pg_sm[];
    long long* gval = reinterpret_cast<long long*>(pg_sm);  // [G][kPgMaxK]
    __shared__ long long memv[kPgBlock];
    __shared__ int grp[kPgBlock];
    __shared__ int locked[kPgBlock];
    __shared__ int su[kPgBlock / 2], sv[kPgBlock / 2];  // a pass's tentative swaps
    __shared__ long long gmem[kPgMaxK];
    __shared__ long long red[kPgBlock / 64];
    __shared__ int redp[kPgBlock / 64];
    __shared__ int first[kPgMaxK], newid[kPgMaxK], side[kPgMaxK];
    __shared__ long long sw[kPgMaxK * kPgMaxK];
    __shared__ long long cum[kPgBlock];
    const int tid = threadIdx.x, n = blockIdx.x;
    const int G = a.G;
    const int64_t N = a.N;
    const uint64_t r = a.rnd[n];
    if (tid < G) {
        const int t = a.gpu_type[tid];
        memv[tid] = (t >= 0 && t < a.T) ? (long long)a.mem[t] : 0;
        grp[tid] = 0;
    }
    __syncthreads();
    // K: floor(total memory / replica memory), the replica holding the weights and the KV
    // caches of 32 requests (Appendix A), shifted by the draw
    long long total = 0;
    double mtot = 0.0;
    for (int e = 0; e < G; ++e) {
        total += memv[e];
        mtot = mtot + (double)memv[e];
    }
    const double Ld = (double)a.L;
    const double rep = 12.0 * a.H * a.H * a.B * Ld + 32.0 * (2.0 * (a.s_in + a.s_out) * a.Hkv * a.B * Ld);
    int kmax = a.Kmax < G ? a.Kmax : G;
    if (kmax > kPgMaxK) kmax = kPgMaxK;
    int K = (int)floor(mtot / rep) + (int)((r & 7) % 5) - 2;
    if (K > kmax) K = kmax;
    if (K < 2) K = 2;
    const int rot = (int)(((r >> 3) & 0xFF) % (uint64_t)G);
    if (total <= 0) total = 1;  // memories all zero: every GPU lands in group 0
    // step (i): the rotated spectral order cut by memory midpoints into K groups
    if (tid == 0) {
        long long run = 0;
        for (int i = 0; i < G; ++i) {
            const int dd = a.order[(i + rot) % G];
            const bool ok = dd >= 0 && dd < G;
            cum[i] = run;
            run += ok ? memv[dd] : 0;
        }
    }
    __syncthreads();
    if (tid < G) {
        const int dd = a.order[(tid + rot) % G];
        if (dd >= 0 && dd < G) {
            const long long k = ((long long)K * (2 * cum[tid] + memv[dd])) / (2 * total);
            grp[dd] = (int)(k < K - 1 ? k : K - 1);
        }
    }
    if (tid < kPgMaxK) gmem[tid] = 0;
    __syncthreads();
    if (tid < G) atomicAdd((unsigned long long*)&gmem[grp[tid]], (unsigned long long)memv[tid]);
    if (tid < G) {
        long long* row = gval + tid * kPgMaxK;
        for (int k = 0; k < kPgMaxK; ++k) row[k] = 0;
        for (int x = 0; x < G; ++x) row[grp[x]] += a.w[(int64_t)x * G + tid];
    }
    drain_barrier();
    // Kernighan-Lin passes: tentative best swaps on unlocked GPUs (negative gains too), then the
    // pass's best prefix is kept and the rest undone; passes repeat while one lowers the cut
    const int pairs = G * G;
    for (int pass = 0; pass < kKlPasses; ++pass) {
        if (tid < G) locked[tid] = 0;
        __syncthreads();
        int n_swaps = 0, kbest = 0;
        long long run = 0, bestsum = 0;
        for (;;) {
            long long bg = 0;
            int bp = kNoPair;
            for (int p = tid; p < pairs; p += kPgBlock) {
                const int u = p / G, v = p - u * G;
                if (v <= u || locked[u] || locked[v]) continue;
                const int A = grp[u], B = grp[v];
                if (A == B) continue;
                const long long d0 = gmem[A] - gmem[B];
                const long long d1 = (gmem[A] - memv[u] + memv[v]) - (gmem[B] - memv[v] + memv[u]);
                if ((d1 < 0 ? -d1 : d1) > (d0 < 0 ? -d0 : d0)) continue;
                const long long wuv = a.w[(int64_t)u * G + v];
                const long long gain = (gval[u * kPgMaxK + B] - gval[u * kPgMaxK + A] - wuv) +
                                       (gval[v * kPgMaxK + A] - gval[v * kPgMaxK + B] - wuv);
                if (better(gain, p, bg, bp)) {
                    bg = gain;
                    bp = p;
                }
            }
            block_best(bg, bp, red, redp);
            if (bp == kNoPair) break;  // uniform: no admissible pair left
            const int u = bp / G, v = bp - u * G;
            pg_exchange(a, u, v, grp, gval, gmem, memv);
            if (tid == 0) {
                locked[u] = locked[v] = 1;
                su[n_swaps] = u;
                sv[n_swaps] = v;
            }
            __syncthreads();
            ++n_swaps;
            run += bg;
            if (run > bestsum) {
                bestsum = run;
                kbest = n_swaps;
            }
        }
        // undo the swaps past the best prefix, last first
        for (int i = n_swaps - 1; i >= kbest; --i) pg_exchange(a, su[i], sv[i], grp, gval, gmem, memv);
        if (kbest == 0) break;  // uniform
    }
    // groups numbered by smallest member
    if (tid < kPgMaxK) first[tid] = 1 << 30;
    __syncthreads();
    if (tid < G) atomicMin(&first[grp[tid]], tid);
    drain_barrier();
    if (tid < kPgMaxK) {
        int id = 0;
        for (int k = 0; k < kPgMaxK; ++k) id += first[k] < first[tid] ? 1 : 0;
        newid[tid] = id;
    }
    __syncthreads();
    int used = 0;
    for (int k = 0; k < kPgMaxK; ++k) used += first[k] < (1 << 30) ? 1 : 0;
    if (tid < G) grp[tid] = newid[grp[tid]];
    for (int i = tid; i < kPgMaxK * kPgMaxK; i += kPgBlock) sw[i] = 0;
    __syncthreads();
    // step (ii): coarsened weights and the max-cut split
    for (int p = tid; p < pairs; p += kPgBlock) {
        const int dd = p / G, e = p - dd * G;
        const int gd = grp[dd], ge = grp[e];
        if (gd != ge) atomicAdd((unsigned long long*)&sw[gd * kPgMaxK + ge], (unsigned long long)a.w[p]);
    }
    if (tid < kPgMaxK) side[tid] = tid < used ? (int)((r >> (11 + tid)) & 1) : 0;
    drain_barrier();
    int n1 = 0;
    for (int k = 0; k < used; ++k) n1 += side[k];
    __syncthreads();
    if (n1 == 0 || n1 == used) {
        if (tid == 0) side[used - 1] ^= 1;
        n1 += (n1 == 0) ? 1 : -1;
    }
    __syncthreads();
    for (int step = 0; step < used * used; ++step) {
        long long bg = 0;
        int bk = kNoPair;
        if (tid < used) {
            const bool blocked = (side[tid] && n1 == 1) || (!side[tid] && n1 == used - 1);
            if (!blocked) {
                long long gain = 0;
                for (int l = 0; l < used; ++l) {
                    if (l == tid) continue;
                    const long long s = sw[tid * kPgMaxK + l];
                    gain += side[l] == side[tid] ? s : -s;
                }
                if (gain > 0) {  // largest gain, then lowest super node
                    bg = gain;
                    bk = tid;
                }
            }
        }
        block_best(bg, bk, red, redp);
        if (bk == kNoPair) break;  // uniform
        const int k = bk;
        n1 += side[k] ? -1 : 1;
        __syncthreads();
        if (tid == 0) side[k] ^= 1;
        __syncthreads();
    }
    // step (iii): the projection
    if (tid < G) a.assign[(int64_t)tid * N + n] = (uint8_t)grp[tid];
    for (int k = tid; k < a.Kmax; k += kPgBlock)
        a.role[(int64_t)k * N + n] = k < used ? (uint8_t)(side[k] ? HX_DECODE : HX_PREFILL) : (uint8_t)HX_UNUSED;
}

}  // namespace

hipError_t launch_spectral(int32_t G, const double* beta, int64_t* w, int32_t iters, int32_t* order, double* fiedler,
                           hipStream_t s) {
    const int64_t cells = (int64_t)G * G;
    hipLaunchKernelGGL(graph_kernel, dim3((unsigned)((cells + 255) / 256)), dim3(256), 0, s, G, beta, w);
    prof_mark(kKSpectral, false, s);
    hipLaunchKernelGGL(spectral_kernel, dim3(1), dim3(kPgBlock), 0, s, G, w, iters, order, fiedler);
    prof_mark(kKSpectral, true, s);
    return hipGetLastError();
}

hipError_t launch_partition(const Problem& p, int64_t* w, const int32_t* order, const uint64_t* rnd, uint8_t* assign,
                            uint8_t* role, hipStream_t s) {
    const int64_t cells = (int64_t)p.G * p.G;
    hipLaunchKernelGGL(graph_kernel, dim3((unsigned)((cells + 255) / 256)), dim3(256), 0, s, p.G, p.beta, w);
    PgArgs a{p.G, p.Kmax, p.N, p.L, p.H, p.Hkv, p.B, p.s_in, p.s_out, w, order, p.gpu_type, p.mem, p.T, rnd,
             assign, role};
    prof_mark(kKPartition, false, s);
    // gval of 255 GPUs (65,280 bytes) takes the workgroup past 64 KB of LDS, which gfx950 allows
    // (160 KB per workgroup) once the kernel's dynamic limit is raised
    const size_t lds = pg_lds_bytes(p.G);
    if (lds > 32 * 1024) {
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(partition_kernel),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(partition_kernel, dim3((unsigned)p.N), dim3(kPgBlock), lds, s, a);
    prof_mark(kKPartition, true, s);
    return hipGetLastError();
}

}  // namespace hx
