// hx_cost.hip -- Table 1 cost model and Appendix A node capacities on gfx950.
//
// The cost of a group depends on its role and size (which strategies exist, how many
// stages, how many TP peers); mixing sizes in one wavefront serialises every size's loop
// nest.  So the batch is first sorted, globally, into work units bucketed by (size, role),
// largest groups first so that the longest lanes start at once, and the costing kernel then
// runs one unit per lane with a wavefront-uniform control path:
//
//   decode_kernel   one lane per candidate: each group's member set as a GPU bitmask (an
//                   output: the flow-network build reuses it), absent slots zeroed, and a
//                   per-workgroup histogram of units per bucket added to the global one;
//   scan_kernel     one wavefront: exclusive scan of the histogram into bucket offsets;
//   scatter_kernel  one lane per candidate: each present group's unit record
//                   (candidate, slot, role, member mask) written into its bucket, a workgroup
//                   reserving its range of each bucket with one atomic;
//   eval_kernel     one lane per unit: every admissible TP x PP strategy, prefill keeping its
//                   latency-optimal and decode its throughput-optimal one (Sec. 3.3,
//                   "Compute nodes").  The unit's mask is expanded into the lane's own LDS
//                   column of member ids (ascending), from which stage j of (tp, pp) is the
//                   slice [j*tp, (j+1)*tp); for tp in {1, 2, 4, 8} the stage's ids sit in
//                   registers and each device's peer loop is unrolled.
// Per-GPU parameters, and the alpha/beta tables when they fit, are staged in LDS.  The
// arithmetic is FP64 scalar work, not a dense contraction, so there is no MFMA here.
//
// Every expression follows the evaluation order documented in hx.h; a stage's max over
// devices of X/(t*c_d) is taken as X/(t*min c_d), the same binary64 value because rounding
// is monotone (likewise the memory limit on the stage's smallest memory).
#include "hx_internal.h"

namespace hx {
namespace {

constexpr int kTableMaxG = 40;  // alpha and beta staged in LDS up to 2 * 40^2 doubles (25.6 KB)


// ------------------------------------------------------------------ one strategy

struct Tables {
    const double *gfl, *ghb, *gme, *alpha, *beta;
};

struct StrategyCost {
    double bmax, lat, x;
};

// Costs strategy (tp, pp) of a group whose r-th member (ascending id) is mem[r * stride].
// Returns false when the memory limit admits no batch of 1.  TPC > 0 fixes tp at compile
// time: a stage's member ids are then held in registers and each device's peer loop is
// unrolled, so its loads and divisions overlap; TPC == 0 is the same arithmetic for any tp.
template <int TPC>
__device__ __forceinline__ bool cost_strategy(const Problem& p, const Tables& tb, const uint8_t* mem, int stride,
                                              int tp_rt, int pp, int role, StrategyCost& out) {
    constexpr int kMax = TPC > 0 ? TPC : HX_MAX_TP;
    const int tp = TPC > 0 ? TPC : tp_rt;
    const double t = (double)tp;
    const double H = p.H, B = p.B;
    const double W12 = 12.0 * H * H * B;
    const double Kkv = 2.0 * (p.s_in + p.s_out) * p.Hkv * B;
    const double Kact = 4.0 * (p.s_in + p.s_out) * H * B;
    const int G = p.G;
    const int lq = p.L / pp, lr = p.L % pp;

    // Memory-limit row: b_j = floor((M_j - A_j)/K_j) on the stage's smallest memory.
    double bmin = kBmaxClamp;
    for (int j = 0; j < pp; ++j) {
        const double l = (double)(lq + (j < lr ? 1 : 0));
        const double A = (W12 / t) * l;
        const double K = (Kkv / t) * l + Kact;
        const uint8_t* S = mem + (j * tp) * stride;
        double Mmin = tb.gme[S[0]];
#pragma unroll
        for (int r = 1; r < kMax; ++r)
            if (TPC > 0 || r < tp) Mmin = dmin(Mmin, tb.gme[S[r * stride]]);
        const double q = (Mmin - A) / K;
        const double b = q >= kBmaxClamp ? kBmaxClamp : (q <= -kBmaxClamp ? -kBmaxClamp : floor(q));
        bmin = dmin(bmin, b);
    }
    out.bmax = bmin;
    if (bmin < 1.0) return false;

    const bool prefill = role == HX_PREFILL;
    const double b = prefill ? 1.0 : bmin;
    const double Xcomp_p = 24.0 * b * p.s_in * H * H;
    const double Xscan_d = 12.0 * H * H * B * p.s_out;
    const double Xcomp_d = 24.0 * b * p.s_out * H * H;
    const double X = prefill ? b * p.s_in * H * B : b * H * B;

    int S[kMax], Sp[kMax];
    double s1 = 0.0, s2 = 0.0;
    for (int j = 0; j < pp; ++j) {
        const double l = (double)(lq + (j < lr ? 1 : 0));
        const uint8_t* Sl = mem + (j * tp) * stride;
#pragma unroll
        for (int r = 0; r < kMax; ++r) S[r] = (TPC > 0 || r < tp) ? Sl[r * stride] : 0;
        double cmin = tb.gfl[S[0]], hmin = tb.ghb[S[0]];
#pragma unroll
        for (int r = 1; r < kMax; ++r)
            if (TPC > 0 || r < tp) {
                cmin = dmin(cmin, tb.gfl[S[r]]);
                hmin = dmin(hmin, tb.ghb[S[r]]);
            }
        const double comp = prefill ? (Xcomp_p / (t * cmin)) * l
                                    : (Xscan_d / (t * hmin)) * l + (Xcomp_d / (t * cmin)) * l;
        // TP row: the device with the largest sum over its peers (ascending peer order).
        double mx = 0.0;
#pragma unroll 1
        for (int r = 0; r < tp; ++r) {
            int d = S[0];
#pragma unroll
            for (int x = 1; x < kMax; ++x)
                if (x == r) d = S[x];
            const double* arow = tb.alpha + d * G;
            const double* brow = tb.beta + d * G;
            double sum = 0.0;
#pragma unroll
            for (int q = 0; q < kMax; ++q) {
                if ((TPC == 0 && q >= tp) || q == r) continue;
                sum = sum + (arow[S[q]] + X / (t * brow[S[q]]));
            }
            if (r == 0 || sum > mx) mx = sum;
        }
        const double tpc = prefill ? (mx * 4.0) * l : ((mx * 4.0) * p.s_out) * l;
        s1 = s1 + (comp + tpc);
        // PP row between stage j-1 and stage j: the fastest link.
        if (j > 0) {
            double mn = 0.0;
#pragma unroll 1
            for (int r = 0; r < tp; ++r) {
                int d = Sp[0];
#pragma unroll
                for (int x = 1; x < kMax; ++x)
                    if (x == r) d = Sp[x];
                const double* arow = tb.alpha + d * G;
                const double* brow = tb.beta + d * G;
#pragma unroll
                for (int q = 0; q < kMax; ++q) {
                    if (TPC == 0 && q >= tp) continue;
                    const double v = arow[S[q]] + X / brow[S[q]];
                    if ((r == 0 && q == 0) || v < mn) mn = v;
                }
            }
            s2 = s2 + (prefill ? mn : mn * p.s_out);
        }
#pragma unroll
        for (int r = 0; r < kMax; ++r) Sp[r] = S[r];
    }
    out.lat = s1 + s2;
    out.x = (1000.0 * b) / out.lat;
    return true;
}

__device__ __forceinline__ bool cost_any(const Problem& p, const Tables& tb, const uint8_t* mem, int stride, int tp,
                                         int pp, int role, StrategyCost& out) {
    switch (tp) {
        case 1: return cost_strategy<1>(p, tb, mem, stride, tp, pp, role, out);
        case 2: return cost_strategy<2>(p, tb, mem, stride, tp, pp, role, out);
        case 4: return cost_strategy<4>(p, tb, mem, stride, tp, pp, role, out);
        case 8: return cost_strategy<8>(p, tb, mem, stride, tp, pp, role, out);
        default: return cost_strategy<0>(p, tb, mem, stride, tp, pp, role, out);
    }
}

// ------------------------------------------------------------------ kernels

struct CostWork {
    int32_t* hist;    // [nb + 1]: per (size, role) unit counts, then offsets; [nb] = total
    int32_t* cursor;  // [nb]
    uint64_t* units;  // [max units][1 + W]: (n << 16 | k << 8 | role), then the member mask words
    uint64_t* gmask;  // [Kmax][W][N] group member bitmasks (the hx_cost_out output)
};

__global__ void fill_kernel(int32_t* a, int n) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) a[i] = 0;
}

// Bucket of a present group: largest sizes first, roles interleaved.
__device__ __forceinline__ int bucket_of(int G, int size, int role) { return (G - size) * 2 + role; }

// One lane per candidate (candidate-fastest, so every [row][n] access coalesces): the member
// bitmask of each group slot, built in the lane's LDS column from its assign column; absent
// slots' zero outputs; a per-workgroup histogram of units per bucket, added to the global one
// with one atomic per bucket.  Slots go in chunks of kSlotChunk whose loads issue together.
constexpr int kSlotChunk = 8;

template <int W>
__global__ void __launch_bounds__(256) decode_kernel(Problem p, CostOut o, CostWork wk) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const int nb = 2 * (p.G + 1);
    int32_t* lhist = reinterpret_cast<int32_t*>(smem);
    uint64_t* ms = reinterpret_cast<uint64_t*>(smem + ((sizeof(int32_t) * nb + 15) & ~(size_t)15));
    const int tid = threadIdx.x, bs = blockDim.x;
    for (int b = tid; b < nb; b += bs) lhist[b] = 0;
    const int n = blockIdx.x * bs + tid;
    const int64_t N = p.N;
    const int Kmax = p.Kmax;
    if (n < N) {
        for (int e = 0; e < Kmax * W; ++e) ms[e * bs + tid] = 0;
#pragma unroll 8
        for (int g = 0; g < p.G; ++g) {
            const int k = p.assign[(int64_t)g * N + n];
            if (k < Kmax) ms[(k * W + (g >> 6)) * bs + tid] |= 1ull << (g & 63);
        }
    }
    __syncthreads();
    if (n < N) {
        for (int k0 = 0; k0 < Kmax; k0 += kSlotChunk) {
            int rl[kSlotChunk];
#pragma unroll
            for (int x = 0; x < kSlotChunk; ++x)
                rl[x] = k0 + x < Kmax ? p.role[(int64_t)(k0 + x) * N + n] : HX_UNUSED;
#pragma unroll
            for (int x = 0; x < kSlotChunk; ++x) {
                const int k = k0 + x;
                if (k >= Kmax) break;
                int size = 0;
#pragma unroll
                for (int i = 0; i < W; ++i) {
                    const uint64_t m = ms[(k * W + i) * bs + tid];
                    wk.gmask[((int64_t)k * W + i) * N + n] = m;
                    size += __popcll(m);
                }
                if (size > 0 && (rl[x] == HX_PREFILL || rl[x] == HX_DECODE)) {
                    atomicAdd(&lhist[bucket_of(p.G, size, rl[x])], 1);
                } else {
                    const int64_t o_ = (int64_t)k * N + n;
                    o.tp[o_] = 0;
                    o.pp[o_] = 0;
                    o.bmax[o_] = 0;
                    o.cap[o_] = 0;
                    o.lat[o_] = 0.0;
                }
            }
        }
    }
    __syncthreads();
    for (int b = tid; b < nb; b += bs)
        if (lhist[b]) atomicAdd(&wk.hist[b], lhist[b]);
}

// Exclusive scan of hist[0..nb) into hist (offsets) and cursor; hist[nb] = total.
__global__ void __launch_bounds__(64) scan_kernel(CostWork wk, int nb) {
    const int lane = threadIdx.x;
    const int per = (nb + 63) / 64;
    const int lo = lane * per, hi = lo + per < nb ? lo + per : nb;
    int32_t s = 0;
    for (int i = lo; i < hi; ++i) s += wk.hist[i];
    int32_t incl = s;
    for (int off = 1; off < 64; off <<= 1) {
        const int32_t v = __shfl_up(incl, off, 64);
        if (lane >= off) incl += v;
    }
    int32_t run = incl - s;
    for (int i = lo; i < hi; ++i) {
        const int32_t v = wk.hist[i];
        wk.hist[i] = run;
        wk.cursor[i] = run;
        run += v;
    }
    if (lane == 63) wk.hist[nb] = incl;
}

// One lane per candidate: every present group becomes a unit record (candidate, slot, role,
// member mask) in its bucket.  Two passes over the slots: count per bucket, reserve the
// workgroup's range of each bucket with one atomic, then write.
template <int W>
__global__ void __launch_bounds__(256) scatter_kernel(Problem p, CostWork wk) {
    __shared__ int32_t lcount[2 * (HX_MAX_GPUS + 1)];
    __shared__ int32_t lbase[2 * (HX_MAX_GPUS + 1)];
    const int nb = 2 * (p.G + 1);
    for (int b = threadIdx.x; b < nb; b += blockDim.x) lcount[b] = 0;
    __syncthreads();
    const int n = blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t N = p.N;
    const int Kmax = p.Kmax;
    for (int pass = 0; pass < 2; ++pass) {
        if (pass == 1) {
            __syncthreads();
            for (int b = threadIdx.x; b < nb; b += blockDim.x) {
                lbase[b] = lcount[b] ? atomicAdd(&wk.cursor[b], lcount[b]) : 0;
                lcount[b] = 0;
            }
            __syncthreads();
        }
        if (n >= N) continue;
        for (int k0 = 0; k0 < Kmax; k0 += kSlotChunk) {
            int rl[kSlotChunk];
            uint64_t m[kSlotChunk][W];
#pragma unroll
            for (int x = 0; x < kSlotChunk; ++x) {
                const bool in = k0 + x < Kmax;
                rl[x] = in ? p.role[(int64_t)(k0 + x) * N + n] : HX_UNUSED;
#pragma unroll
                for (int i = 0; i < W; ++i) m[x][i] = in ? wk.gmask[((int64_t)(k0 + x) * W + i) * N + n] : 0;
            }
#pragma unroll
            for (int x = 0; x < kSlotChunk; ++x) {
                int size = 0;
#pragma unroll
                for (int i = 0; i < W; ++i) size += __popcll(m[x][i]);
                if (size == 0 || (rl[x] != HX_PREFILL && rl[x] != HX_DECODE)) continue;
                const int b = bucket_of(p.G, size, rl[x]);
                const int rank = atomicAdd(&lcount[b], 1);
                if (pass == 1) {
                    uint64_t* rec = wk.units + (int64_t)(lbase[b] + rank) * (1 + W);
                    rec[0] = ((uint64_t)n << 16) | ((uint64_t)(k0 + x) << 8) | (uint64_t)rl[x];
#pragma unroll
                    for (int i = 0; i < W; ++i) rec[1 + i] = m[x][i];
                }
            }
        }
    }
}

template <int W, bool kTables, int kEvalBlock>
__global__ void __launch_bounds__(kEvalBlock) eval_kernel(Problem p, CostOut o, CostWork wk, int nb) {
    extern __shared__ __attribute__((aligned(16))) double dsm[];
    const int G = p.G;
    double* gfl = dsm;
    double* ghb = gfl + G;
    double* gme = ghb + G;
    for (int g = threadIdx.x; g < G; g += kEvalBlock) {
        const int t = p.gpu_type[g];
        const bool ok = t >= 0 && t < p.T;  // an unknown type can hold nothing: infeasible
        gfl[g] = ok ? p.flops[t] : 0.0;
        ghb[g] = ok ? p.hbm[t] : 0.0;
        gme[g] = ok ? p.mem[t] : 0.0;
    }
    Tables tb{gfl, ghb, gme, p.alpha, p.beta};
    double* tb_end = gme + G;
    if (kTables) {
        double* a = gme + G;
        double* b = a + G * G;
        for (int e = threadIdx.x; e < G * G; e += kEvalBlock) {
            a[e] = p.alpha[e];
            b[e] = p.beta[e];
        }
        tb.alpha = a;
        tb.beta = b;
        tb_end = b + G * G;
    }
    __syncthreads();
    const int64_t total = wk.hist[nb];
    const int64_t N = p.N;
    uint8_t* mem = reinterpret_cast<uint8_t*>(tb_end) + threadIdx.x;  // [G][kEvalBlock] member list
    for (int64_t u = (int64_t)blockIdx.x * kEvalBlock + threadIdx.x; u < total; u += (int64_t)gridDim.x * kEvalBlock) {
        const uint64_t* rec = wk.units + u * (1 + W);
        const uint64_t w = rec[0];
        const int n = (int)(w >> 16), k = (int)((w >> 8) & 0xFF), role = (int)(w & 0xFF);
        int cnt = 0;
#pragma unroll
        for (int i = 0; i < W; ++i) {
            uint64_t m = rec[1 + i];
            while (m) {
                mem[(cnt++) * kEvalBlock] = (uint8_t)(i * 64 + __builtin_ctzll(m));
                m &= m - 1;
            }
        }
        bool have = false;
        int best_tp = 0, best_pp = 0;
        double best_b = 0.0, best_lat = 0.0, best_x = 0.0;
        for (int tp = 1; tp <= HX_MAX_TP; ++tp) {
            if (!((p.tp_mask >> (tp - 1)) & 1u) || cnt % tp != 0) continue;
            const int pp = cnt / tp;
            if (pp > HX_MAX_PP || !((p.pp_mask >> (pp - 1)) & 1u) || pp > p.L) continue;
            StrategyCost sc;
            if (!cost_any(p, tb, mem, kEvalBlock, tp, pp, role, sc)) continue;
            const bool better = !have || (role == HX_PREFILL ? sc.lat < best_lat : sc.x > best_x);
            if (better) {
                have = true;
                best_tp = tp;
                best_pp = pp;
                best_b = sc.bmax;
                best_lat = sc.lat;
                best_x = sc.x;
            }
        }
        const int64_t o_ = (int64_t)k * N + n;
        o.tp[o_] = (uint8_t)best_tp;
        o.pp[o_] = (uint8_t)best_pp;
        o.bmax[o_] = (int32_t)best_b;
        o.cap[o_] = have ? quantize(best_x) : 0;
        o.lat[o_] = best_lat;
    }
}

// Units a candidate can contribute: one per group, at most min(Kmax, G).
int64_t max_units(int G, int Kmax, int64_t N) { return (int64_t)(Kmax < G ? Kmax : G) * N; }

template <int W>
hipError_t launch_w(const Problem& p, const CostOut& o, const CostWork& wk, hipStream_t s) {
    const int nb = 2 * (p.G + 1);
    hipLaunchKernelGGL(fill_kernel, dim3((2 * nb + 1 + 255) / 256), dim3(256), 0, s, wk.hist, 2 * nb + 1);
    // decode: the widest workgroup whose per-lane masks fit in 32 KB of LDS
    int bs = 256;
    while (bs > 64 && (size_t)p.Kmax * W * bs * 8 > 32 * 1024) bs /= 2;
    const size_t lds_dec = ((sizeof(int32_t) * nb + 15) & ~(size_t)15) + (size_t)p.Kmax * W * bs * 8;
    hipLaunchKernelGGL(decode_kernel<W>, dim3((p.N + bs - 1) / bs), dim3(bs), lds_dec, s, p, o, wk);
    hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(64), 0, s, wk, nb);
    hipLaunchKernelGGL(scatter_kernel<W>, dim3((p.N + 255) / 256), dim3(256), 0, s, p, wk);
    const bool tables = p.G <= kTableMaxG;
    // A grid-stride loop over the units: enough workgroups to fill the chip several times.
    // 256 lanes per workgroup amortise the staged tables; the per-lane member columns take
    // G bytes per lane, so beyond 128 GPUs the workgroup halves to stay within 64 KB of LDS.
    const int64_t units = max_units(p.G, p.Kmax, p.N);
    const int eb = p.G <= 128 ? 256 : 128;
    const size_t lds_eval =
        sizeof(double) * (3 * (size_t)p.G + (tables ? 2 * (size_t)p.G * p.G : 0)) + (size_t)p.G * eb;
    const int64_t want = (units + eb - 1) / eb;
    const int blocks = (int)(want < 2048 ? want : 2048);
    if (eb == 256) {
        if (tables)
            hipLaunchKernelGGL((eval_kernel<W, true, 256>), dim3(blocks), dim3(256), lds_eval, s, p, o, wk, nb);
        else
            hipLaunchKernelGGL((eval_kernel<W, false, 256>), dim3(blocks), dim3(256), lds_eval, s, p, o, wk, nb);
    } else {
        hipLaunchKernelGGL((eval_kernel<W, false, 128>), dim3(blocks), dim3(128), lds_eval, s, p, o, wk, nb);
    }
    return hipGetLastError();
}

}  // namespace

int mask_words(int32_t n_gpus) { return n_gpus <= 64 ? 1 : (n_gpus <= 128 ? 2 : 4); }

size_t cost_workspace_bytes(int32_t n_gpus, int32_t max_groups, int32_t n_cand) {
    const size_t nb = 2 * ((size_t)n_gpus + 1);
    const size_t head = ((2 * nb + 1) * sizeof(int32_t) + 255) & ~(size_t)255;
    return head + sizeof(uint64_t) * (1 + mask_words(n_gpus)) * (size_t)max_units(n_gpus, max_groups, n_cand);
}

hipError_t launch_cost(const Problem& p, const CostOut& o, void* workspace, hipStream_t s) {
    const size_t nb = 2 * ((size_t)p.G + 1);
    const size_t head = ((2 * nb + 1) * sizeof(int32_t) + 255) & ~(size_t)255;
    CostWork wk;
    wk.hist = reinterpret_cast<int32_t*>(workspace);
    wk.cursor = wk.hist + nb + 1;
    wk.units = reinterpret_cast<uint64_t*>(reinterpret_cast<unsigned char*>(workspace) + head);
    wk.gmask = o.members;
    switch (mask_words(p.G)) {
        case 1: return launch_w<1>(p, o, wk, s);
        case 2: return launch_w<2>(p, o, wk, s);
        default: return launch_w<4>(p, o, wk, s);
    }
}

}  // namespace hx
