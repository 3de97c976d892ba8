// hx_cost.hip -- Table 1 cost model and Appendix A node capacities on gfx950.
//
// The cost of a group depends on its role and size (which strategies exist, how many
// stages, how many TP peers); mixing sizes in one wavefront serialises every size's loop
// nest.  So the batch is first sorted, globally, into work units bucketed by (size, role),
// largest groups first so that the longest lanes start at once, and the costing kernel then
// runs the units with a wavefront-uniform control path:
//
//   setup_kernel    clears the bucket histogram, tabulates the prefill link terms (batch 1
//                   makes them candidate independent) and the memory-row screen;
//   ref_kernel      with HX_HINT_SHARED_GROUPS only: candidate 0's groups, costed once;
//   decode_kernel   one lane per candidate: each group's member set as a GPU bitmask (an
//                   output: the flow-network build reuses it), absent and screened slots
//                   zeroed, groups equal to one of candidate 0's given its outputs, and each
//                   remaining group's bucket code with a per-workgroup histogram of units per
//                   bucket added to the global one;
//   scatter_kernel  one lane per candidate: each workgroup scans the histogram into bucket
//                   offsets, then writes each unit record (candidate, slot, role, member mask)
//                   into its bucket, reserving its range of each bucket with one atomic;
//   eval_kernel     every admissible TP x PP strategy of a unit, prefill keeping its
//                   latency-optimal and decode its throughput-optimal one (Sec. 3.3,
//                   "Compute nodes").  Large groups take several lanes (coop_unit); the others
//                   one lane each, whose mask is expanded into the lane's own LDS column of
//                   member ids (ascending), from which stage j of (tp, pp) is the slice
//                   [j*tp, (j+1)*tp); for tp in {1, 2, 4, 8} the stage's ids sit in registers
//                   and each device's peer loop is unrolled.
// Per-GPU parameters, and the alpha/beta tables when they fit, are staged in LDS.  The
// arithmetic is FP64 scalar work, not a dense contraction, so there is no MFMA here.
//
// Every expression follows the evaluation order documented in hx.h; a stage's max over
// devices of X/(t*c_d) is taken as X/(t*min c_d), the same binary64 value because rounding
// is monotone (likewise the memory limit on the stage's smallest memory).
#include "hx_internal.h"

namespace hx {
namespace {

constexpr int kTableMaxG = 40;  // alpha and beta staged in LDS up to 2 * 40 * 41 doubles (26.2 KB)


// ------------------------------------------------------------------ one strategy

struct Tables {
    const double *gfl, *ghb, *gme, *alpha, *beta;  // alpha, beta: row d at d * ld
    const double* tp_pre;  // [tp - 1][G][G] alpha + X/(tp beta) at batch 1 (prefill), per call
    const double* pp_pre;  // [G][G] alpha + X/beta at batch 1
    int ld;                // row stride of alpha and beta: G in memory, G + 1 staged in LDS
};

struct StrategyCost {
    double bmax, lat, x;
};

// Costs strategy (tp, pp) of a group whose r-th member (ascending id) is mem[r * stride].
// Returns false when the memory limit admits no batch of 1.  TPC > 0 fixes tp at compile
// time: a stage's member ids are then held in registers and each device's peer loop is
// unrolled, so its loads and divisions overlap; TPC == 0 is the same arithmetic for any tp.
// Slowest FLOP/s among stage j's devices, member r at mem[(j*tp + r) * stride].
__device__ __forceinline__ double stage_cmin(const Tables& tb, const uint8_t* mem, int stride, int j, int tp) {
    double c = tb.gfl[mem[(j * tp) * stride]];
    for (int r = 1; r < tp; ++r) c = dmin(c, tb.gfl[mem[(j * tp + r) * stride]]);
    return c;
}

template <bool kAsym>
__device__ __forceinline__ LayerSplit make_split(const Problem& p, const Tables& tb, const uint8_t* mem, int stride,
                                                 int tp, int pp) {
    return layer_split<kAsym>(p.L, pp, [&](int j) { return stage_cmin(tb, mem, stride, j, tp); });
}

// kVar: variant bits.  HX_VARIANT_PIPELINED: a decode replica's x is 1000 b over its slowest
// stage, T_j = (comp_j + TP_j) + PP_j with the link into stage j+1 counted with stage j; the
// latency is the same sum either way.  HX_VARIANT_ASYM: the asymmetric layer split above.
template <int TPC, int kVar>
__device__ __forceinline__ bool cost_strategy(const Problem& p, const Tables& tb, const uint8_t* mem, int stride,
                                              int tp_rt, int pp, int role, StrategyCost& out) {
    constexpr bool kPipe = (kVar & HX_VARIANT_PIPELINED) != 0;
    constexpr bool kAsym = (kVar & HX_VARIANT_ASYM) != 0;
    constexpr int kMax = TPC > 0 ? TPC : HX_MAX_TP;
    const int tp = TPC > 0 ? TPC : tp_rt;
    const double t = (double)tp;
    const double H = p.H, B = p.B;
    const double W12 = 12.0 * H * H * B;
    const double Kkv = 2.0 * (p.s_in + p.s_out) * p.Hkv * B;
    const double Kact = 4.0 * (p.s_in + p.s_out) * H * B;
    const int G = p.G;
    const LayerSplit split = make_split<kAsym>(p, tb, mem, stride, tp, pp);

    // Memory-limit row: b_j = floor((M_j - A_j)/K_j) on the stage's smallest memory.
    double bmin = kBmaxClamp;
    for (int j = 0; j < pp; ++j) {
        const double l = (double)split_layers<kAsym>(split, j, kAsym ? stage_cmin(tb, mem, stride, j, tp) : 0.0);
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
    double tmax = 0.0, prev = 0.0;  // kPipe: slowest stage so far, previous stage's comp + TP
    for (int j = 0; j < pp; ++j) {
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
        const double l = (double)split_layers<kAsym>(split, j, cmin);
        const double comp = prefill ? (Xcomp_p / (t * cmin)) * l
                                    : (Xscan_d / (t * hmin)) * l + (Xcomp_d / (t * cmin)) * l;
        // TP row: the device with the largest sum over its peers (ascending peer order).
        double mx = 0.0;
        if (TPC > 0 && TPC <= 4 && !prefill) {
            // Decode with tp fixed: the pairs (r, q), r < q, in ascending order.  Device r's sum
            // takes its peers q > r here, after its peers q < r arrived from earlier r, so every
            // device's sum is still formed in ascending peer order.  X / (t beta) of a link is
            // computed once for both directions when beta_{dq} and beta_{qd} have the same bits
            // (the same binary64 quotient), and separately otherwise.
            double sum[kMax];
#pragma unroll
            for (int r = 0; r < kMax; ++r) sum[r] = 0.0;
#pragma unroll
            for (int r = 0; r < kMax; ++r) {
                const double* arow = tb.alpha + S[r] * tb.ld;
                const double* brow = tb.beta + S[r] * tb.ld;
#pragma unroll
                for (int q = r + 1; q < kMax; ++q) {
                    const double bf = brow[S[q]], bb = tb.beta[S[q] * tb.ld + S[r]];
                    const double qf = X / (t * bf);
                    double qb = qf;
                    if (__double_as_longlong(bf) != __double_as_longlong(bb)) qb = X / (t * bb);
                    sum[r] = sum[r] + (arow[S[q]] + qf);
                    sum[q] = sum[q] + (tb.alpha[S[q] * tb.ld + S[r]] + qb);
                    // keep each pair's loads and divisions together (bounded live ranges)
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
#pragma unroll
            for (int r = 0; r < kMax; ++r)
                if (r == 0 || sum[r] > mx) mx = sum[r];
        } else {
#pragma unroll 1
            for (int r = 0; r < tp; ++r) {
                int d = S[0];
#pragma unroll
                for (int x = 1; x < kMax; ++x)
                    if (x == r) d = S[x];
                const double* arow = tb.alpha + d * tb.ld;
                const double* brow = tb.beta + d * tb.ld;
                const double* prow = tb.tp_pre + ((size_t)(tp - 1) * G + d) * G;
                double sum = 0.0;
                if (prefill) {
                    // table lookups: the row's loads issued together (S[q] is 0 past tp), then
                    // summed in ascending peer order
                    double v[kMax];
#pragma unroll
                    for (int q = 0; q < kMax; ++q) v[q] = prow[S[q]];
#pragma unroll
                    for (int q = 0; q < kMax; ++q)
                        if (!((TPC == 0 && q >= tp) || q == r)) sum = sum + v[q];
                } else {
#pragma unroll
                    for (int q = 0; q < kMax; ++q) {
                        if ((TPC == 0 && q >= tp) || q == r) continue;
                        sum = sum + (arow[S[q]] + X / (t * brow[S[q]]));
                    }
                }
                if (r == 0 || sum > mx) mx = sum;
            }
        }
        const double tpc = prefill ? (mx * 4.0) * l : ((mx * 4.0) * p.s_out) * l;
        const double stage = comp + tpc;
        s1 = s1 + stage;
        // PP row between stage j-1 and stage j: the fastest link.
        if (j > 0) {
            double mn = 0.0;
#pragma unroll 1
            for (int r = 0; r < tp; ++r) {
                int d = Sp[0];
#pragma unroll
                for (int x = 1; x < kMax; ++x)
                    if (x == r) d = Sp[x];
                const double* arow = tb.alpha + d * tb.ld;
                const double* brow = tb.beta + d * tb.ld;
                const double* prow = tb.pp_pre + (size_t)d * G;
                if (prefill) {
                    double v[kMax];
#pragma unroll
                    for (int q = 0; q < kMax; ++q) v[q] = prow[S[q]];
#pragma unroll
                    for (int q = 0; q < kMax; ++q)
                        if (!(TPC == 0 && q >= tp) && ((r == 0 && q == 0) || v[q] < mn)) mn = v[q];
                } else {
#pragma unroll
                    for (int q = 0; q < kMax; ++q) {
                        if (TPC == 0 && q >= tp) continue;
                        const double v = arow[S[q]] + X / brow[S[q]];
                        if ((r == 0 && q == 0) || v < mn) mn = v;
                    }
                }
            }
            const double ppt = prefill ? mn : mn * p.s_out;
            s2 = s2 + ppt;
            if (kPipe) tmax = dmax(tmax, prev + ppt);
        }
        if (kPipe) prev = stage;
#pragma unroll
        for (int r = 0; r < kMax; ++r) Sp[r] = S[r];
    }
    out.lat = s1 + s2;
    if (kPipe && !prefill)
        out.x = (1000.0 * b) / dmax(tmax, prev);
    else
        out.x = (1000.0 * b) / out.lat;
    return true;
}

template <int kVar>
__device__ __forceinline__ bool cost_any(const Problem& p, const Tables& tb, const uint8_t* mem, int stride, int tp,
                                         int pp, int role, StrategyCost& out) {
    switch (tp) {
        case 1: return cost_strategy<1, kVar>(p, tb, mem, stride, tp, pp, role, out);
        case 2: return cost_strategy<2, kVar>(p, tb, mem, stride, tp, pp, role, out);
        case 4: return cost_strategy<4, kVar>(p, tb, mem, stride, tp, pp, role, out);
        case 8: return cost_strategy<8, kVar>(p, tb, mem, stride, tp, pp, role, out);
        default: return cost_strategy<0, kVar>(p, tb, mem, stride, tp, pp, role, out);
    }
}

// Template bit of the eval kernels (above the HX_VARIANT_* bits): request classes.
constexpr int kVarClasses = 1 << 8;

// The task of class k, and its prefill tables.
__device__ __forceinline__ void class_task(const Problem& p, const Tables& tb, int k, Problem& pk, Tables& tk) {
    const size_t blk = (size_t)(HX_MAX_TP + 1) * p.G * p.G;
    pk = p;
    pk.s_in = p.cls_in[k];
    pk.s_out = p.cls_out[k];
    tk = tb;
    tk.tp_pre = tb.tp_pre + k * blk;
    tk.pp_pre = tb.pp_pre + k * blk;
}

// Strategy (tp, pp) over the request classes: feasible when it is for every class; b_max the
// smallest, latency sum_k w_k lat_k, capacity 1 / sum_k w_k / x_k (class order, left to right).
template <int kVar>
__device__ __forceinline__ bool cost_mix(const Problem& p, const Tables& tb, const uint8_t* mem, int stride, int tp,
                                         int pp, int role, StrategyCost& out) {
    double lat = 0.0, tau = 0.0, bmax = 0.0;
    for (int k = 0; k < p.n_cls; ++k) {
        Problem pk;
        Tables tk;
        class_task(p, tb, k, pk, tk);
        StrategyCost sk;
        if (!cost_any<kVar>(pk, tk, mem, stride, tp, pp, role, sk)) return false;
        lat = lat + p.cls_w[k] * sk.lat;
        tau = tau + p.cls_w[k] / sk.x;
        if (k == 0 || sk.bmax < bmax) bmax = sk.bmax;
    }
    out.bmax = bmax;
    out.lat = lat;
    out.x = 1.0 / tau;
    return true;
}

// The kept strategy of a group of cnt GPUs (member r at mem[r * stride]) with admissible set
// adm: every strategy costed in ascending tp, prefill keeping the strictly lowest latency and
// decode the strictly highest x (Sec. 3.3, "Compute nodes").  have: some strategy was feasible.
struct GroupCost {
    int tp, pp;
    double b, lat, x;
    bool have;
};

__device__ __forceinline__ int stage_count(int c, int tp);

template <int kVar>
__device__ __forceinline__ GroupCost cost_group(const Problem& p, const Tables& tb, const uint8_t* mem, int stride,
                                                uint32_t adm, int cnt, int role) {
    GroupCost r{0, 0, 0.0, 0.0, 0.0, false};
    for (uint32_t am = adm; am; am &= am - 1) {
        const int tp = __ffs(am);
        const int pp = stage_count(cnt, tp);
        StrategyCost sc;
        if constexpr ((kVar & kVarClasses) != 0) {
            if (!cost_mix<kVar & ~kVarClasses>(p, tb, mem, stride, tp, pp, role, sc)) continue;
        } else if (!cost_any<kVar>(p, tb, mem, stride, tp, pp, role, sc)) {
            continue;
        }
        const bool better = !r.have || (role == HX_PREFILL ? sc.lat < r.lat : sc.x > r.x);
        if (better) {
            r.have = true;
            r.tp = tp;
            r.pp = pp;
            r.b = sc.bmax;
            r.lat = sc.lat;
            r.x = sc.x;
        }
    }
    return r;
}

// Admissible strategies of a group of c GPUs, bit tp-1 for each tp of the mask dividing c with
// pp = c/tp in the PP mask and at most L (the strategy list of Sec. 3.2 for that size).
__device__ __forceinline__ uint8_t admissible(const Problem& p, int c) {
    uint8_t a = 0;
    for (int tp = 1; tp <= HX_MAX_TP; ++tp) {
        if (!((p.tp_mask >> (tp - 1)) & 1u) || c % tp != 0) continue;
        const int pp = c / tp;
        if (pp >= 1 && pp <= HX_MAX_PP && ((p.pp_mask >> (pp - 1)) & 1u) && pp <= p.L) a |= (uint8_t)(1u << (tp - 1));
    }
    return a;
}

// c / tp for an admissible strategy (tp divides c <= 255): multiply by ceil(2^16 / tp).
__device__ __forceinline__ int stage_count(int c, int tp) {
    constexpr uint32_t kRecip[HX_MAX_TP + 1] = {0, 65536, 32768, 21846, 16384, 13108, 10923, 9363, 8192};
    return (int)(((uint32_t)c * kRecip[tp]) >> 16);
}

// ------------------------------------------------------------------ kernels

// HX_HINT_SHARED_GROUPS: candidate 0's groups, costed once: member masks [Kmax][W] (4 Kmax
// words reserved), roles [Kmax] (HX_UNUSED for a slot with no member or no role) and outputs
// (a one-candidate table: entry k is slot k's).  One contiguous block of ref_bytes(Kmax), so
// decode can stage it in LDS with one copy and carve it the same way.
struct RefTable {
    uint64_t* m;
    uint8_t* role;
    CostOut out;
};

__host__ __device__ inline size_t ref_bytes(int Kmax) {
    return ((size_t)Kmax * (4 * sizeof(uint64_t) + sizeof(double) + 2 * sizeof(int32_t) + 3) + 15) & ~(size_t)15;
}

__host__ __device__ inline RefTable carve_ref(unsigned char* r, int Kmax) {
    const size_t K = (size_t)Kmax;
    RefTable t;
    t.m = reinterpret_cast<uint64_t*>(r);
    t.out.lat = reinterpret_cast<double*>(r + 4 * sizeof(uint64_t) * K);
    t.out.bmax = reinterpret_cast<int32_t*>(t.out.lat + K);
    t.out.cap = t.out.bmax + K;
    t.out.tp = reinterpret_cast<uint8_t*>(t.out.cap + K);
    t.out.pp = t.out.tp + K;
    t.role = t.out.pp + K;
    t.out.members = nullptr;
    return t;
}

struct CostWork {
    int32_t* hist;    // [nb + 1]: per (size, role) unit counts ([nb] unused)
    int32_t* cursor;  // [nb]: units placed so far per bucket
    uint64_t* units;  // [max units][1 + W]: (n << 16 | k << 8 | role), then the member mask words
    uint64_t* gmask;  // [Kmax][W][N] group member bitmasks (the hx_cost_out output)
    uint64_t* unfit;  // [G + 2][W] the memory-row screen: a row per group size, then wild
    uint16_t* ukey;   // [Kmax][N] bucket of a group to cost (bucket_of), kNoUnit for a group decode settled
    double* tp_pre;   // [HX_MAX_TP][G][G] prefill TP terms (see Tables), class 0
    double* pp_pre;   // [G][G] prefill PP terms, class 0; class k's tables sit k table blocks on
                      // ((HX_MAX_TP + 1) G^2 doubles each)
    unsigned char* ref_base;  // candidate 0's table (RefTable), ref_bytes(Kmax)
    RefTable ref;
    unsigned long long* clear2;  // [n_clear2] more words the first kernel zeroes (or null)
    int n_clear2;
};

// The memory-row screen, a W-word GPU bitmask per group size c = 0..G, then wild (entry G + 1).
// Row c holds the GPUs g that fail the memory row of every admissible strategy of size c on
// their own memory, in some request class: for strategy (tp, pp) with the stage holding
// floor(L/pp) layers, clamp(floor((M_g - A)/K)) < 1 with A, K and the clamp as the memory row
// has them (row c is every GPU when size c has no strategy).  The row is monotone in the stage's
// smallest memory and only gets stricter with one layer more, so a group of size c holding such
// a GPU has no feasible strategy.  Wild: GPUs whose memory is NaN, where the stage minimum
// depends on the member order, so a group holding one is not screened.  One wavefront per word
// (a ballot over its 64 GPUs); the loop bound is wavefront-uniform.
__device__ void unfit_table(const Problem& p, uint64_t* unfit, int W, int64_t tid, int64_t nth) {
    const int lane = (int)(tid & 63);
    const int nt = p.n_cls > 0 ? p.n_cls : 1;
    for (int64_t e = tid >> 6; e < (int64_t)(p.G + 2) * W; e += nth >> 6) {
        const int c = (int)(e / W), g = (int)(e - (int64_t)c * W) * 64 + lane;
        double M = 0.0;
        if (g < p.G) {
            const int t = p.gpu_type[g];
            M = t >= 0 && t < p.T ? p.mem[t] : 0.0;  // an unknown type holds nothing
        }
        bool bit = g < p.G;
        if (c == p.G + 1) {
            bit = bit && isnan(M);
        } else {
            const double H = p.H, B = p.B;
            const double W12 = 12.0 * H * H * B;
            for (uint32_t am = admissible(p, c); am && bit; am &= am - 1) {
                const int tp = __ffs(am), pp = stage_count(c, tp);
                const double t = (double)tp, l = (double)(p.L / pp);
                bool fails = false;
                for (int k = 0; k < nt; ++k) {
                    const double s_in = p.n_cls > 0 ? p.cls_in[k] : p.s_in;
                    const double s_out = p.n_cls > 0 ? p.cls_out[k] : p.s_out;
                    const double Kkv = 2.0 * (s_in + s_out) * p.Hkv * B;
                    const double Kact = 4.0 * (s_in + s_out) * H * B;
                    const double A = (W12 / t) * l;
                    const double K = (Kkv / t) * l + Kact;
                    const double q = (M - A) / K;
                    const double b = q >= kBmaxClamp ? kBmaxClamp : (q <= -kBmaxClamp ? -kBmaxClamp : floor(q));
                    if (b < 1.0) fails = true;
                }
                bit = fails;
            }
        }
        const uint64_t bits = __ballot(bit);
        if (lane == 0) unfit[e] = bits;
    }
}

// True when the screen settles a group of size c (member mask m): no member's memory is NaN
// and a member fails every admissible strategy's memory row, so the costing would keep no
// strategy and the group's outputs are all zero.  (Groups it does not settle are costed
// exactly.)
template <int W>
__device__ __forceinline__ bool screened_out(const uint64_t* unfit, int G, const uint64_t (&m)[W], int c) {
    uint64_t wild = 0, hit = 0;
#pragma unroll
    for (int i = 0; i < W; ++i) {
        wild |= m[i] & unfit[(G + 1) * W + i];
        hit |= m[i] & unfit[c * W + i];
    }
    return hit != 0 && wild == 0;
}

// First kernel of a call: clears the histogram, cursors and argmax counter (n_clear words), tabulates the
// memory-row screen and the prefill link terms.  Prefill runs at batch 1, so its per-link TP and PP terms depend only on
// the cluster and the task: alpha + X/(tp beta) for every TP degree of the mask and
// alpha + X/beta, X = 1*s_in*H*B, evaluated exactly as the costing expressions do (the same
// binary64 values).  With request classes there is one table block per class (its s_in).
__global__ void setup_kernel(Problem p, CostWork wk, int n_clear, int W) {
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t nth = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = tid; i < n_clear; i += nth) wk.hist[i] = 0;
    for (int64_t i = tid; i < wk.n_clear2; i += nth) wk.clear2[i] = 0;
    unfit_table(p, wk.unfit, W, tid, nth);
    const int G = p.G;
    const int64_t gg = (int64_t)G * G;
    const int64_t blk = (HX_MAX_TP + 1) * gg;
    const int nt = p.n_cls > 0 ? p.n_cls : 1;
    for (int64_t i = tid; i < nt * blk; i += nth) {
        const int cls = (int)(i / blk);
        const int64_t ic = i - cls * blk;
        const double X = 1.0 * (p.n_cls > 0 ? p.cls_in[cls] : p.s_in) * p.H * p.B;
        const int slot = (int)(ic / gg);
        const int64_t de = ic - slot * gg;
        if (slot == HX_MAX_TP) {
            wk.pp_pre[cls * blk + de] = p.alpha[de] + X / p.beta[de];
        } else {
            const int tp = slot + 1;
            if (tp >= 2 && ((p.tp_mask >> (tp - 1)) & 1u))
                wk.tp_pre[cls * blk + ic] = p.alpha[de] + X / ((double)tp * p.beta[de]);
        }
    }
}


// Bucket of a present group: largest sizes first, roles interleaved (< 2 (G + 1) <= 512); the
// role is the bucket's low bit.
__device__ __forceinline__ int bucket_of(int G, int size, int role) { return (G - size) * 2 + role; }
constexpr uint16_t kNoUnit = 0xFFFF;  // a slot with no unit to cost

// Workgroup barrier that first drains the calling wave's outstanding LDS operations
// (lgkmcnt(0); the vector-memory and export counters are left at their maxima).  The counting
// pass ends in LDS atomics whose results are unused; the barrier the compiler emits after them
// does not wait for them on every path, and without the wait some increments were measured to
// land after the workgroup had read the counts.
__device__ __forceinline__ void lds_drain_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __syncthreads();
}

// Group slots per chunk whose loads a lane issues together (C slots of 1 + W words each):
// 8, 16 or 32, the smallest covering every slot, with at most 32 mask words in flight.
__host__ inline int slot_chunk(int W, int Kmax) {
    int c = Kmax <= 8 ? 8 : (Kmax <= 16 ? 16 : 32);
    while (c > 8 && c * W > 32) c /= 2;
    return c;
}

// GPUs per chunk of assign rows a lane loads together.
constexpr int kGpuChunk = 32;

// Group slots whose masks decode builds at a time: 128 bytes of LDS columns per lane, so that a
// 256-lane workgroup takes 32 KB and four of them share a CU (16, 8, 4 slots for 1, 2, 4 mask
// words).
template <int W>
__host__ __device__ constexpr int decode_slots() {
    return 128 / (8 * W);
}

// One lane per candidate (candidate-fastest, so every [row][n] access coalesces): the member
// bitmask of each group slot, built in the lane's LDS column from its assign column; absent
// slots' zero outputs; a per-workgroup histogram of units per bucket, added to the global one
// with one atomic per bucket.  The assign column is loaded once, in chunks of kGpuChunk rows
// that issue together, and kept in registers (four GPUs' group ids per word); the slots are
// then built decode_slots<W>() at a time from it, their role rows loaded together per block.
template <int W>
__global__ void __launch_bounds__(256) decode_kernel(Problem p, CostOut o, CostWork wk, bool use_ref) {
    constexpr int Kc = decode_slots<W>();
    constexpr int kWords = 16 * W;  // packed assign words: 64 W GPUs
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const int nb = 2 * (p.G + 1);
    int32_t* lhist = reinterpret_cast<int32_t*>(smem);
    uint64_t* unfit = reinterpret_cast<uint64_t*>(smem + ((sizeof(int32_t) * nb + 15) & ~(size_t)15));
    uint64_t* ms = unfit + (p.G + 2) * W;
    const int tid = threadIdx.x, bs = blockDim.x;
    for (int b = tid; b < nb; b += bs) lhist[b] = 0;
    for (int e = tid; e < (p.G + 2) * W; e += bs) unfit[e] = wk.unfit[e];
    // with the hint: candidate 0's table, after the mask columns
    unsigned char* rbase = reinterpret_cast<unsigned char*>(ms + (size_t)Kc * W * bs);
    const RefTable ref = carve_ref(rbase, p.Kmax);
    if (use_ref) {
        const uint64_t* src = reinterpret_cast<const uint64_t*>(wk.ref_base);
        uint64_t* dst = reinterpret_cast<uint64_t*>(rbase);
        for (int e = tid; e < (int)(ref_bytes(p.Kmax) / 8); e += bs) dst[e] = src[e];
    }
    const bool screen = (p.variant & HX_VARIANT_ASYM) == 0;  // the screen assumes the uniform split
    const int n = blockIdx.x * bs + tid;
    const int64_t N = p.N;
    const int Kmax = p.Kmax;
    __syncthreads();  // lhist cleared, tables staged
    if (n < N) {
    // the lane's assign column: GPU g's group id in byte g % 4 of word g / 4 (HX_UNUSED past G,
    // which no slot block holds: slots are < Kmax <= 255)
    uint32_t pk[kWords];
#pragma unroll
    for (int c = 0; c < kWords / 8; ++c) {
        if (c * kGpuChunk >= p.G) {
#pragma unroll
            for (int w = 0; w < 8; ++w) pk[c * 8 + w] = 0xFFFFFFFFu;
            continue;
        }
        // every load issued (rows past G read row G - 1 and are replaced), so that the chunk's
        // loads are in flight together
        uint32_t a[kGpuChunk];
#pragma unroll
        for (int x = 0; x < kGpuChunk; ++x) {
            const int g = c * kGpuChunk + x;
            a[x] = p.assign[(int64_t)(g < p.G ? g : p.G - 1) * N + n];
        }
#pragma unroll
        for (int x = 0; x < kGpuChunk; ++x)
            if (c * kGpuChunk + x >= p.G) a[x] = HX_UNUSED;
#pragma unroll
        for (int w = 0; w < 8; ++w)
            pk[c * 8 + w] = a[4 * w] | (a[4 * w + 1] << 8) | (a[4 * w + 2] << 16) | (a[4 * w + 3] << 24);
    }
    for (int kc = 0; kc < Kmax; kc += Kc) {
        // slots [kc, ke) in the lane's column, slot k at row k - kc
        const int ke = kc + Kc < Kmax ? kc + Kc : Kmax;
#pragma unroll
        for (int e = 0; e < Kc * W; ++e) ms[e * bs + tid] = 0;
#pragma unroll
        for (int w = 0; w < kWords; ++w) {
            if (4 * w >= p.G) break;
#pragma unroll
            for (int y = 0; y < 4; ++y) {
                const int g = 4 * w + y;
                const uint32_t r = ((pk[w] >> (8 * y)) & 0xFFu) - (uint32_t)kc;
                if (r < (uint32_t)(ke - kc)) ms[(r * W + (g >> 6)) * bs + tid] |= 1ull << (g & 63);
            }
        }
        int rl[Kc];
#pragma unroll
        for (int x = 0; x < Kc; ++x) rl[x] = p.role[(int64_t)(kc + x < ke ? kc + x : ke - 1) * N + n];
#pragma unroll
        for (int x = 0; x < Kc; ++x)
            if (kc + x >= ke) rl[x] = HX_UNUSED;
#pragma unroll
        for (int x = 0; x < Kc; ++x) {
            const int k = kc + x;
            if (k >= ke) break;
            uint64_t m[W];
            int size = 0;
#pragma unroll
            for (int i = 0; i < W; ++i) {
                m[i] = ms[(x * W + i) * bs + tid];
                wk.gmask[((int64_t)k * W + i) * N + n] = m[i];
                size += __popcll(m[i]);
            }
            const bool costed = size > 0 && (rl[x] == HX_PREFILL || rl[x] == HX_DECODE) &&
                                !(screen && screened_out<W>(unfit, p.G, m, size));
            const int64_t o_ = (int64_t)k * N + n;
            // a group of candidate 0 (same members, same role) takes its outputs: costing it
            // again would give the same values.  Groups are looked for in the same slot and
            // the two next to it (slot-wise numbering shifts a slot by one after a merge);
            // the slot index is uniform, so the reads are the same for every lane.
            int hit = -1;
            if (costed && use_ref) {
#pragma unroll
                for (int d = -1; d <= 1; ++d) {
                    const int e = k + d;
                    if (e < 0 || e >= Kmax) continue;
                    bool same = ref.role[e] == rl[x];
#pragma unroll
                    for (int i = 0; i < W; ++i) same = same && ref.m[e * W + i] == m[i];
                    if (same) hit = e;
                }
            }
            if (costed && hit < 0) {
                atomicAdd(&lhist[bucket_of(p.G, size, rl[x])], 1);
            } else if (hit >= 0) {
                o.tp[o_] = ref.out.tp[hit];
                o.pp[o_] = ref.out.pp[hit];
                o.bmax[o_] = ref.out.bmax[hit];
                o.cap[o_] = ref.out.cap[hit];
                o.lat[o_] = ref.out.lat[hit];
            } else {
                o.tp[o_] = 0;
                o.pp[o_] = 0;
                o.bmax[o_] = 0;
                o.cap[o_] = 0;
                o.lat[o_] = 0.0;
            }
            wk.ukey[o_] = costed && hit < 0 ? (uint16_t)bucket_of(p.G, size, rl[x]) : kNoUnit;
        }
    }
    }
    lds_drain_barrier();
    for (int b = tid; b < nb; b += bs)
        if (lhist[b]) atomicAdd(&wk.hist[b], lhist[b]);
}

// Sum of h[0..hi) across one wavefront; every lane receives it.
__device__ __forceinline__ int32_t wave_sum(const int32_t* h, int hi, int lane) {
    int32_t s = 0;
    for (int i = lane; i < hi; i += 64) s += h[i];
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    return s;
}

// One lane per candidate: every group decode left to cost becomes a unit record (candidate,
// slot, role, member mask) in its bucket.  Each workgroup scans the bucket counts into bucket
// offsets itself (a few hundred words from L2).  Two passes over the slots: count per bucket
// (from the slots' bucket codes alone), reserve the workgroup's range of each bucket with one
// atomic on the bucket's cursor, then write, loading the member masks of C slots together.
template <int W, int C>
__global__ void __launch_bounds__(256) scatter_kernel(Problem p, CostWork wk) {
    __shared__ int32_t lcount[2 * (HX_MAX_GPUS + 1)];
    __shared__ int32_t lbase[2 * (HX_MAX_GPUS + 1)];
    __shared__ int32_t loff[2 * (HX_MAX_GPUS + 1)];
    const int nb = 2 * (p.G + 1);
    for (int b = threadIdx.x; b < nb; b += blockDim.x) lcount[b] = 0;
    if (threadIdx.x < 64) {
        // exclusive scan of the bucket counts, each lane over a run of consecutive buckets
        const int lane = threadIdx.x;
        const int per = (nb + 63) / 64;
        const int lo = lane * per, hi = lo + per < nb ? lo + per : nb;
        int32_t sum = 0;
        for (int i = lo; i < hi; ++i) sum += wk.hist[i];
        int32_t incl = sum;
        for (int off = 1; off < 64; off <<= 1) {
            const int32_t v = __shfl_up(incl, off, 64);
            if (lane >= off) incl += v;
        }
        int32_t run = incl - sum;
        for (int i = lo; i < hi; ++i) {
            loff[i] = run;
            run += wk.hist[i];
        }
    }
    __syncthreads();
    const int n = blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t N = p.N;
    const int Kmax = p.Kmax;
    for (int pass = 0; pass < 2; ++pass) {
        if (pass == 1) {
            lds_drain_barrier();
            for (int b = threadIdx.x; b < nb; b += blockDim.x) {
                lbase[b] = lcount[b] ? loff[b] + atomicAdd(&wk.cursor[b], lcount[b]) : 0;
                lcount[b] = 0;
            }
            __syncthreads();
        }
        if (n >= N) continue;
        for (int k0 = 0; k0 < Kmax; k0 += C) {
            // every load issued (slots past Kmax read slot Kmax - 1 and are dropped)
            int bk[C];
#pragma unroll
            for (int x = 0; x < C; ++x) bk[x] = wk.ukey[(int64_t)(k0 + x < Kmax ? k0 + x : Kmax - 1) * N + n];
#pragma unroll
            for (int x = 0; x < C; ++x)
                if (k0 + x >= Kmax) bk[x] = kNoUnit;
            if (pass == 0) {
#pragma unroll
                for (int x = 0; x < C; ++x)
                    if (bk[x] != kNoUnit) atomicAdd(&lcount[bk[x]], 1);
                continue;
            }
            uint64_t m[C][W];
#pragma unroll
            for (int x = 0; x < C; ++x)
#pragma unroll
                for (int i = 0; i < W; ++i)
                    m[x][i] = wk.gmask[((int64_t)(k0 + x < Kmax ? k0 + x : Kmax - 1) * W + i) * N + n];
#pragma unroll
            for (int x = 0; x < C; ++x) {
                if (bk[x] == kNoUnit) continue;
                const int b = bk[x];
                const int rank = atomicAdd(&lcount[b], 1);
                uint64_t* rec = wk.units + (int64_t)(lbase[b] + rank) * (1 + W);
                rec[0] = ((uint64_t)n << 16) | ((uint64_t)(k0 + x) << 8) | (uint64_t)(b & 1);
#pragma unroll
                for (int i = 0; i < W; ++i) rec[1 + i] = m[x][i];
            }
        }
    }
}

// ------------------------------------------------------------------ large groups

// Groups of at least kCoopMin GPUs carry a long serial chain of divisions when one lane costs
// them (hundreds for a 24-GPU decode group), so kCoopLanes lanes of a wavefront cost each:
// lane-parallel over stages for the memory row and the computation term, over (stage,
// device) rows for the TP sums and PP minima; one lane then combines the rows in the
// documented order, so every value is the same binary64 the one-lane path produces.
// Two settings: (12 GPUs, 16 lanes) where the batch keeps the chip busy, and (6 GPUs, 8 lanes)
// for batches small enough that the longest lane chains set the kernel's time (N Kmax <=
// kSmallBatch): more groups then get several lanes, each with a shorter chain.
constexpr int kCoopMin = 12;
constexpr int kCoopLanes = 16;
constexpr int kCoopMinSmall = 6;
constexpr int kCoopLanesSmall = 8;
constexpr int64_t kSmallBatch = int64_t(1) << 21;

__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Per-group LDS: member ids [G], row values tsum/pmin [G] (one per (stage, device)), per stage
// [max_stages(pp_mask)] the computation term (then the stage's whole time) and the PP link time
// into the next stage.
struct CoopLds {
    uint8_t* mem;
    double *tsum, *pmin, *comp, *ppt;
};

// The most pipeline stages a strategy can have: the highest PP of the mask.
__host__ __device__ inline int max_stages(uint32_t pp_mask) {
    int m = 0;
    for (int b = 0; b < 32; ++b)
        if ((pp_mask >> b) & 1u) m = b + 1;
    return m;
}

__host__ __device__ inline size_t coop_group_bytes(int G, int stages) {
    return ((size_t)G + 7) / 8 * 8 + sizeof(double) * (2 * (size_t)G + 2 * (size_t)stages);
}

__device__ __forceinline__ CoopLds carve_coop(unsigned char* base, int G, int stages) {
    CoopLds c;
    c.mem = base;
    c.tsum = reinterpret_cast<double*>(base + ((size_t)G + 7) / 8 * 8);
    c.pmin = c.tsum + G;
    c.comp = c.pmin + G;
    c.ppt = c.comp + stages;
    return c;
}

// One group of kCL lanes (gl = lane within it) costs unit (n, k, role, mask); `live`
// is false for groups past the last large unit (they still join every wave-level sync).  With
// request classes (kVarClasses) each strategy is costed once per class, and the mix kept as
// cost_mix keeps it.
template <int W, int kVar, int kCL>
__device__ void coop_unit(const Problem& p0, const Tables& tb0, const CostOut& o, const CoopLds& c,
                          const uint8_t* adm_tab, int gl, bool live, int n, int k, int role,
                          const uint64_t (&mask)[W]) {
    constexpr bool kPipe = (kVar & HX_VARIANT_PIPELINED) != 0;
    constexpr bool kAsym = (kVar & HX_VARIANT_ASYM) != 0;
    constexpr bool kCls = (kVar & kVarClasses) != 0;
    const int G = p0.G;
    int cnt = 0;
#pragma unroll
    for (int i = 0; i < W; ++i) cnt += live ? __popcll(mask[i]) : 0;
    // member ids ascending: GPU g goes to position (members below g)
    for (int g = gl; g < G && live; g += kCL) {
        const int wd = g >> 6;
        const uint64_t below = (1ull << (g & 63)) - 1;
        int pos = 0;
        bool in = false;
#pragma unroll
        for (int i = 0; i < W; ++i) {
            if (i < wd) pos += __popcll(mask[i]);
            if (i == wd) {
                in = (mask[i] >> (g & 63)) & 1ull;
                pos += __popcll(mask[i] & below);
            }
        }
        if (in) c.mem[pos] = (uint8_t)g;
    }
    wave_sync();
    const double H = p0.H, B = p0.B;
    const double W12 = 12.0 * H * H * B;
    const bool prefill = role == HX_PREFILL;
    bool have = false;
    int best_tp = 0, best_pp = 0;
    double best_b = 0.0, best_lat = 0.0, best_x = 0.0;
    const uint32_t am = live ? adm_tab[cnt] : 0u;
    const int n_task = kCls ? p0.n_cls : 1;
    // the TP degrees some group of the wavefront can take, ascending (the loop holds wavefront
    // operations, so every lane runs it the same number of times)
    uint32_t wave_am = am;
    for (int off = 32; off > 0; off >>= 1) wave_am |= (uint32_t)__shfl_xor((int)wave_am, off, 64);
    for (uint32_t rest = wave_am; rest; rest &= rest - 1) {
        const int tp = __ffs(rest);
        const bool adm = (am >> (tp - 1)) & 1u;
        const int pp = adm ? stage_count(cnt, tp) : 0;
        const double t = (double)tp;
        const LayerSplit split = adm ? make_split<kAsym>(p0, tb0, c.mem, 1, tp, pp) : LayerSplit{0, 0, 0, 0, 0.0};
        // ok: feasible in every task so far (uniform over the group); the mix at gl == 0.
        bool ok = adm;
        double mix_b = 0.0, mix_lat = 0.0, mix_x = 0.0, mix_tau = 0.0;
        for (int task = 0; task < n_task; ++task) {
            Problem p;
            Tables tb;
            if (kCls) {
                class_task(p0, tb0, task, p, tb);
            } else {
                p = p0;
                tb = tb0;
            }
            const double Kkv = 2.0 * (p.s_in + p.s_out) * p.Hkv * B;
            const double Kact = 4.0 * (p.s_in + p.s_out) * H * B;
            // Memory-limit row, one lane per stage, then the group's minimum (exact).
            double bl = kBmaxClamp;
            for (int j = gl; j < pp; j += kCL) {
                const double l = (double)split_layers<kAsym>(split, j, kAsym ? stage_cmin(tb, c.mem, 1, j, tp) : 0.0);
                const double A = (W12 / t) * l;
                const double K = (Kkv / t) * l + Kact;
                const uint8_t* S = c.mem + j * tp;
                double Mmin = tb.gme[S[0]];
                for (int r = 1; r < tp; ++r) Mmin = dmin(Mmin, tb.gme[S[r]]);
                const double q = (Mmin - A) / K;
                const double b = q >= kBmaxClamp ? kBmaxClamp : (q <= -kBmaxClamp ? -kBmaxClamp : floor(q));
                bl = dmin(bl, b);
            }
            for (int off = kCL / 2; off > 0; off >>= 1) bl = dmin(bl, __shfl_xor(bl, off, kCL));
            const bool feas = ok && bl >= 1.0;
            const double b = prefill ? 1.0 : bl;
            const double Xcomp_p = 24.0 * b * p.s_in * H * H;
            const double Xscan_d = 12.0 * H * H * B * p.s_out;
            const double Xcomp_d = 24.0 * b * p.s_out * H * H;
            const double X = prefill ? b * p.s_in * H * B : b * H * B;
            // Rows (stage j, device r): the device's TP sum over its peers (ascending) and its
            // fastest link into stage j+1.
            for (int it = gl; feas && it < cnt; it += kCL) {
                const int j = it / tp, r = it - j * tp;
                const uint8_t* S = c.mem + j * tp;
                const int d = S[r];
                const double* arow = tb.alpha + d * tb.ld;
                const double* brow = tb.beta + d * tb.ld;
                const double* prow = tb.tp_pre + ((size_t)(tp - 1) * G + d) * G;
                const double* qrow = tb.pp_pre + (size_t)d * G;
                double sum = 0.0;
                for (int q = 0; q < tp; ++q) {
                    if (q == r) continue;
                    sum = sum + (prefill ? prow[S[q]] : (arow[S[q]] + X / (t * brow[S[q]])));
                }
                c.tsum[it] = sum;
                if (j + 1 < pp) {
                    const uint8_t* S2 = S + tp;
                    double mn = 0.0;
                    for (int q = 0; q < tp; ++q) {
                        const double v = prefill ? qrow[S2[q]] : arow[S2[q]] + X / brow[S2[q]];
                        if (q == 0 || v < mn) mn = v;
                    }
                    c.pmin[it] = mn;
                }
            }
            for (int j = gl; feas && j < pp; j += kCL) {
                const uint8_t* S = c.mem + j * tp;
                double cmin = tb.gfl[S[0]], hmin = tb.ghb[S[0]];
                for (int r = 1; r < tp; ++r) {
                    cmin = dmin(cmin, tb.gfl[S[r]]);
                    hmin = dmin(hmin, tb.ghb[S[r]]);
                }
                const double l = (double)split_layers<kAsym>(split, j, cmin);
                c.comp[j] = prefill ? (Xcomp_p / (t * cmin)) * l
                                    : (Xscan_d / (t * hmin)) * l + (Xcomp_d / (t * cmin)) * l;
            }
            wave_sync();
            // Per stage, a lane each: the stage's time (computation + TP row maximum, rows in
            // ascending device order) over its comp entry, and the PP link into the next stage.
            for (int j = gl; feas && j < pp; j += kCL) {
                const double l = (double)split_layers<kAsym>(split, j, kAsym ? stage_cmin(tb, c.mem, 1, j, tp) : 0.0);
                double mx = 0.0;
                for (int r = 0; r < tp; ++r) {
                    const double v = c.tsum[j * tp + r];
                    if (r == 0 || v > mx) mx = v;
                }
                const double tpc = prefill ? (mx * 4.0) * l : ((mx * 4.0) * p.s_out) * l;
                double pt = 0.0;
                if (j + 1 < pp) {
                    double mn = 0.0;
                    for (int r = 0; r < tp; ++r) {
                        const double v = c.pmin[j * tp + r];
                        if (r == 0 || v < mn) mn = v;
                    }
                    pt = prefill ? mn : mn * p.s_out;
                }
                c.comp[j] = c.comp[j] + tpc;
                c.ppt[j] = pt;
            }
            wave_sync();
            // one lane sums them in stage order
            if (feas && gl == 0) {
                double s1 = 0.0, s2 = 0.0, tmax = 0.0;
                for (int j = 0; j < pp; ++j) {
                    const double stage = c.comp[j];
                    s1 = s1 + stage;
                    if (kPipe && !prefill) tmax = dmax(tmax, j + 1 < pp ? stage + c.ppt[j] : stage);
                }
                for (int j = 0; j + 1 < pp; ++j) s2 = s2 + c.ppt[j];
                const double lat = s1 + s2;
                const double x = (1000.0 * b) / (kPipe && !prefill ? tmax : lat);
                if (kCls) {
                    mix_lat = mix_lat + p0.cls_w[task] * lat;
                    mix_tau = mix_tau + p0.cls_w[task] / x;
                    if (task == 0 || bl < mix_b) mix_b = bl;
                } else {
                    mix_lat = lat;
                    mix_x = x;
                    mix_b = bl;
                }
            }
            ok = feas;
            wave_sync();
        }
        if (ok && gl == 0) {
            const double x = kCls ? 1.0 / mix_tau : mix_x;
            const bool better = !have || (prefill ? mix_lat < best_lat : x > best_x);
            if (better) {
                have = true;
                best_tp = tp;
                best_pp = pp;
                best_b = mix_b;
                best_lat = mix_lat;
                best_x = x;
            }
        }
    }
    if (live && gl == 0) {
        const int64_t o_ = (int64_t)k * p0.N + n;
        o.tp[o_] = (uint8_t)best_tp;
        o.pp[o_] = (uint8_t)best_pp;
        o.bmax[o_] = (int32_t)best_b;
        o.cap[o_] = have ? quantize(best_x) : 0;
        o.lat[o_] = best_lat;
    }
}

// HX_HINT_SHARED_GROUPS: candidate 0's groups costed once, kCoopLanes lanes per group slot
// with coop_unit (the same binary64 values as the one-lane path), into the one-candidate
// table wk.ref.out; their member masks and roles into wk.ref.m and wk.ref.role.  A wavefront per
// workgroup, 64 / kCoopLanes slots each, so the slots' chains of table loads run side by side.
template <int W, int kVar>
__global__ void __launch_bounds__(64) ref_kernel(Problem p, CostWork wk) {
    constexpr int kCL = kCoopLanes, kPer = 64 / kCL;
    extern __shared__ __attribute__((aligned(16))) double rsm[];
    __shared__ uint8_t adm_tab[HX_MAX_GPUS + 1];
    const int G = p.G, tid = threadIdx.x, grp = tid / kCL, gl = tid % kCL;
    double* gfl = rsm;
    double* ghb = gfl + G;
    double* gme = ghb + G;
    uint8_t* a0 = reinterpret_cast<uint8_t*>(gme + G);  // [G] candidate 0's assign column
    for (int g = tid; g < G; g += 64) {
        const int t = p.gpu_type[g];
        const bool ok = t >= 0 && t < p.T;
        gfl[g] = ok ? p.flops[t] : 0.0;
        ghb[g] = ok ? p.hbm[t] : 0.0;
        gme[g] = ok ? p.mem[t] : 0.0;
        a0[g] = p.assign[(int64_t)g * p.N];
    }
    for (int c = tid; c <= G; c += 64) adm_tab[c] = admissible(p, c);
    __syncthreads();
    const Tables tb{gfl, ghb, gme, p.alpha, p.beta, wk.tp_pre, wk.pp_pre, G};
    const int k = blockIdx.x * kPer + grp;
    // slot k's members: each lane of the slot's lane group marks every kCL-th GPU, then OR
    uint64_t m[W] = {};
    for (int g = gl; g < G && k < p.Kmax; g += kCL)
        if (a0[g] == k) {
#pragma unroll
            for (int i = 0; i < W; ++i)
                if (i == (g >> 6)) m[i] |= 1ull << (g & 63);
        }
    int cnt = 0;
#pragma unroll
    for (int i = 0; i < W; ++i) {
        for (int off = kCL / 2; off > 0; off >>= 1)
            m[i] |= (uint64_t)__shfl_xor((unsigned long long)m[i], off, kCL);
        cnt += __popcll(m[i]);
    }
    const int role = k < p.Kmax ? p.role[(int64_t)k * p.N] : HX_UNUSED;
    const bool live = k < p.Kmax && cnt > 0 && (role == HX_PREFILL || role == HX_DECODE);
    Problem p1 = p;
    p1.N = 1;  // the table holds one candidate
    unsigned char* cbase = a0 + (((size_t)G + 7) & ~(size_t)7);
    const CoopLds c = carve_coop(cbase + grp * coop_group_bytes(G, max_stages(p.pp_mask)), G, max_stages(p.pp_mask));
    coop_unit<W, kVar, kCL>(p1, tb, wk.ref.out, c, adm_tab, gl, live, 0, k, role, m);
    if (k < p.Kmax && gl == 0) {
#pragma unroll
        for (int i = 0; i < W; ++i) wk.ref.m[(int64_t)k * W + i] = m[i];
        wk.ref.role[k] = (uint8_t)(live ? role : HX_UNUSED);
    }
}

// LDS of ref_kernel beyond its static arrays: the per-GPU tables, candidate 0's assign column
// and the slots' coop_unit areas.
__host__ inline size_t ref_lds_bytes(int G, int stages) {
    return sizeof(double) * 3 * (size_t)G + (((size_t)G + 7) & ~(size_t)7) +
           (size_t)(64 / kCoopLanes) * coop_group_bytes(G, stages);
}

// LDS of one eval wavefront: its cooperative groups' rows (kCL lanes a group), or, without the
// cooperative path, its lanes' member columns; the columns (64 G bytes) fit in the rows.
__host__ __device__ inline size_t eval_wave_bytes(int G, bool coop, int kCL, int stages) {
    return coop ? (size_t)(64 / kCL) * coop_group_bytes(G, stages) : (size_t)G * 64;
}

template <int W, bool kTables, int kEvalBlock, int kVar, int kCMin, int kCL>
__global__ void __launch_bounds__(kEvalBlock, 4) eval_kernel(Problem p, CostOut o, CostWork wk, int nb) {
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
    Tables tb{gfl, ghb, gme, p.alpha, p.beta, wk.tp_pre, wk.pp_pre, G};
    double* tb_end = gme + G;
    if (kTables) {
        // rows padded to G + 1 doubles: the lanes of a cooperative group read one column of
        // several rows at once, which an unpadded stride of G doubles maps onto one bank
        // whenever G is a multiple of 32
        const int ld = G + 1;
        double* a = gme + G;
        double* b = a + G * ld;
        for (int e = threadIdx.x; e < G * G; e += kEvalBlock) {
            const int d = e / G, c = e - d * G;
            a[d * ld + c] = p.alpha[e];
            b[d * ld + c] = p.beta[e];
        }
        tb.alpha = a;
        tb.beta = b;
        tb.ld = ld;
        tb_end = b + G * ld;
    }
    // Admissible strategies by group size, for every size up to G.
    __shared__ uint8_t adm_tab[HX_MAX_GPUS + 1];
    for (int c = threadIdx.x; c <= G; c += kEvalBlock) adm_tab[c] = admissible(p, c);
    // Units in all: the sum of the bucket counts.  Units before the (size kCMin - 1)
    // buckets are the large groups (sizes descend).
    __shared__ int32_t counts[2];
    if (threadIdx.x < 64) {
        const int32_t t = wave_sum(wk.hist, nb, threadIdx.x);
        const int32_t f = W == 1 && G >= kCMin ? wave_sum(wk.hist, bucket_of(G, kCMin - 1, 0), threadIdx.x) : 0;
        if (threadIdx.x == 0) {
            counts[0] = t;
            counts[1] = f;
        }
    }
    __syncthreads();
    const int64_t total = counts[0];
    const int64_t N = p.N;
    const int64_t first_small = counts[1];
    // Each wavefront's LDS area: its cooperative groups' rows, which its lanes' member columns
    // ([G][64], one-lane path) reuse once its cooperative items are done.
    const bool coop = W == 1 && G >= kCMin;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int stages = max_stages(p.pp_mask);
    unsigned char* warea = reinterpret_cast<unsigned char*>(tb_end) + wave * eval_wave_bytes(G, coop, kCL, stages);
    uint8_t* mem = warea + lane;
    if (coop) {
        const int grp = lane / kCL, gl = lane % kCL;
        constexpr int kGroupsPerWave = 64 / kCL;
        const CoopLds c = carve_coop(warea + grp * coop_group_bytes(G, stages), G, stages);
        const int64_t waves = (int64_t)gridDim.x * (kEvalBlock / 64);
        for (int64_t base = ((int64_t)blockIdx.x * (kEvalBlock / 64) + wave) * kGroupsPerWave; base < first_small;
             base += waves * kGroupsPerWave) {
            const int64_t u = base + grp;
            const bool live = u < first_small;
            int n = 0, k = 0, role = 0;
            uint64_t mask[W] = {};
            if (live) {
                const uint64_t* rec = wk.units + u * (1 + W);
                const uint64_t w = rec[0];
                n = (int)(w >> 16);
                k = (int)((w >> 8) & 0xFF);
                role = (int)(w & 0xFF);
#pragma unroll
                for (int i = 0; i < W; ++i) mask[i] = rec[1 + i];
            }
            coop_unit<W, kVar, kCL>(p, tb, o, c, adm_tab, gl, live, n, k, role, mask);
        }
        wave_sync();  // the wavefront's member columns overwrite its cooperative rows
    }
    for (int64_t u = first_small + (int64_t)blockIdx.x * kEvalBlock + threadIdx.x; u < total;
         u += (int64_t)gridDim.x * kEvalBlock) {
        const uint64_t* rec = wk.units + u * (1 + W);
        const uint64_t w = rec[0];
        const int n = (int)(w >> 16), k = (int)((w >> 8) & 0xFF), role = (int)(w & 0xFF);
        int cnt = 0;
#pragma unroll
        for (int i = 0; i < W; ++i) {
            uint64_t m = rec[1 + i];
            while (m) {
                mem[(cnt++) * 64] = (uint8_t)(i * 64 + __builtin_ctzll(m));
                m &= m - 1;
            }
        }
        const GroupCost gc = cost_group<kVar>(p, tb, mem, 64, adm_tab[cnt], cnt, role);
        const int64_t o_ = (int64_t)k * N + n;
        o.tp[o_] = (uint8_t)gc.tp;
        o.pp[o_] = (uint8_t)gc.pp;
        o.bmax[o_] = (int32_t)gc.b;
        o.cap[o_] = gc.have ? quantize(gc.x) : 0;
        o.lat[o_] = gc.lat;
    }
}

template <int W, int kVar, int kCMin, int kCL>
void launch_eval_coop(const Problem& p, const CostOut& o, const CostWork& wk, int nb, bool tables, int eb, int blocks,
                      hipStream_t s) {
    const size_t lds = sizeof(double) * (3 * (size_t)p.G + (tables ? 2 * (size_t)p.G * (p.G + 1) : 0)) +
                       (size_t)(eb / 64) * eval_wave_bytes(p.G, W == 1 && p.G >= kCMin, kCL, max_stages(p.pp_mask));
    if (eb == 256) {
        if (tables)
            hipLaunchKernelGGL((eval_kernel<W, true, 256, kVar, kCMin, kCL>), dim3(blocks), dim3(256), lds, s, p, o, wk,
                               nb);
        else
            hipLaunchKernelGGL((eval_kernel<W, false, 256, kVar, kCMin, kCL>), dim3(blocks), dim3(256), lds, s, p, o,
                               wk, nb);
    } else {
        hipLaunchKernelGGL((eval_kernel<W, false, 128, kVar, kCMin, kCL>), dim3(blocks), dim3(128), lds, s, p, o, wk,
                           nb);
    }
}

// Small batches take the small-batch setting (only mask width 1 has the cooperative path),
// unless every group is costed (the asymmetric split has no memory-row screen, and more lanes
// per group then cost more than they save).
__host__ inline bool small_batch(const Problem& p) {
    return (int64_t)p.N * p.Kmax <= kSmallBatch && !(p.variant & HX_VARIANT_ASYM);
}

template <int W, int kVar>
void launch_eval(const Problem& p, const CostOut& o, const CostWork& wk, int nb, bool tables, int eb, int blocks,
                 hipStream_t s) {
    if (W == 1 && small_batch(p))
        launch_eval_coop<W, kVar, kCoopMinSmall, kCoopLanesSmall>(p, o, wk, nb, tables, eb, blocks, s);
    else
        launch_eval_coop<W, kVar, kCoopMin, kCoopLanes>(p, o, wk, nb, tables, eb, blocks, s);
}

// Units a candidate can contribute: one per group, at most min(Kmax, G).
int64_t max_units(int G, int Kmax, int64_t N) { return (int64_t)(Kmax < G ? Kmax : G) * N; }

template <int W>
hipError_t launch_w(const Problem& p, const CostOut& o, const CostWork& wk, hipStream_t s) {
    const int nb = 2 * (p.G + 1);
    {
        // hist, cursor and the argmax counter are contiguous: 2 nb + 2 words to clear
        const int64_t cells = (int64_t)(HX_MAX_TP + 1) * p.G * p.G;
        const int64_t screen = (int64_t)(p.G + 2) * W * 64;  // a wavefront per screen word
        const int64_t most = cells > screen ? cells : screen;
        const int64_t want = (most > 2 * nb + 2 ? most : 2 * nb + 2) + 255;
        const int blocks = (int)(want / 256 < 1024 ? want / 256 : 1024);
        prof_mark(kKSetup, false, s);
        hipLaunchKernelGGL(setup_kernel, dim3(blocks), dim3(256), 0, s, p, wk, 2 * nb + 2, W);
        prof_mark(kKSetup, true, s);
    }
    // decode: 256 lanes, 32 KB of mask columns (decode_slots<W>() slots of W words per lane)
    constexpr int bs = 256;
    // HX_HINT_SHARED_GROUPS: candidate 0's groups costed first, for decode to hand out (decode
    // stages their table after its mask columns)
    const bool use_ref = (p.variant & HX_HINT_SHARED_GROUPS) != 0;
    const size_t lds_dec = ((sizeof(int32_t) * nb + 15) & ~(size_t)15) + sizeof(uint64_t) * (p.G + 2) * W +
                           sizeof(uint64_t) * decode_slots<W>() * W * bs + (use_ref ? ref_bytes(p.Kmax) : 0);
    if (use_ref) {
        const size_t lds_ref = ref_lds_bytes(p.G, max_stages(p.pp_mask));
        const dim3 gref((p.Kmax + 64 / kCoopLanes - 1) / (64 / kCoopLanes));
        prof_mark(kKShared, false, s);
        switch ((p.variant & (HX_VARIANT_PIPELINED | HX_VARIANT_ASYM)) | (p.n_cls > 0 ? kVarClasses : 0)) {
            case 0: hipLaunchKernelGGL((ref_kernel<W, 0>), gref, dim3(64), lds_ref, s, p, wk); break;
            case kVarClasses: hipLaunchKernelGGL((ref_kernel<W, kVarClasses>), gref, dim3(64), lds_ref, s, p, wk); break;
            case kVarClasses | HX_VARIANT_PIPELINED:
                hipLaunchKernelGGL((ref_kernel<W, kVarClasses | HX_VARIANT_PIPELINED>), gref, dim3(64), lds_ref, s, p,
                                   wk);
                break;
            case HX_VARIANT_PIPELINED:
                hipLaunchKernelGGL((ref_kernel<W, HX_VARIANT_PIPELINED>), gref, dim3(64), lds_ref, s, p, wk);
                break;
            case HX_VARIANT_ASYM:
                hipLaunchKernelGGL((ref_kernel<W, HX_VARIANT_ASYM>), gref, dim3(64), lds_ref, s, p, wk);
                break;
            default:
                hipLaunchKernelGGL((ref_kernel<W, HX_VARIANT_PIPELINED | HX_VARIANT_ASYM>), gref, dim3(64), lds_ref, s,
                                   p, wk);
                break;
        }
        prof_mark(kKShared, true, s);
    }
    const dim3 gdec((p.N + bs - 1) / bs), gsc((p.N + 255) / 256);
    prof_mark(kKDecode, false, s);
    hipLaunchKernelGGL((decode_kernel<W>), gdec, dim3(bs), lds_dec, s, p, o, wk, use_ref);
    prof_mark(kKDecode, true, s);
    prof_mark(kKScatter, false, s);
    switch (slot_chunk(W, p.Kmax)) {
        case 8: hipLaunchKernelGGL((scatter_kernel<W, 8>), gsc, dim3(256), 0, s, p, wk); break;
        case 16: hipLaunchKernelGGL((scatter_kernel<W, (W <= 2 ? 16 : 8)>), gsc, dim3(256), 0, s, p, wk); break;
        default: hipLaunchKernelGGL((scatter_kernel<W, (W == 1 ? 32 : 8)>), gsc, dim3(256), 0, s, p, wk); break;
    }
    prof_mark(kKScatter, true, s);
    const bool tables = p.G <= kTableMaxG;
    // A grid-stride loop over the units: enough workgroups to fill the chip several times.
    // 256 lanes per workgroup amortise the staged tables; the per-lane member columns take
    // G bytes per lane, so beyond 128 GPUs the workgroup halves to stay within 64 KB of LDS.
    const int64_t units = max_units(p.G, p.Kmax, p.N);
    const int eb = p.G <= 128 ? 256 : 128;
    const int64_t want = (units + eb - 1) / eb;
    const int blocks = (int)(want < 2048 ? want : 2048);
    prof_mark(kKEval, false, s);
    switch ((p.variant & (HX_VARIANT_PIPELINED | HX_VARIANT_ASYM)) | (p.n_cls > 0 ? kVarClasses : 0)) {
        case 0: launch_eval<W, 0>(p, o, wk, nb, tables, eb, blocks, s); break;
        case kVarClasses: launch_eval<W, kVarClasses>(p, o, wk, nb, tables, eb, blocks, s); break;
        case kVarClasses | HX_VARIANT_PIPELINED:
            launch_eval<W, kVarClasses | HX_VARIANT_PIPELINED>(p, o, wk, nb, tables, eb, blocks, s);
            break;
        case HX_VARIANT_PIPELINED: launch_eval<W, HX_VARIANT_PIPELINED>(p, o, wk, nb, tables, eb, blocks, s); break;
        case HX_VARIANT_ASYM: launch_eval<W, HX_VARIANT_ASYM>(p, o, wk, nb, tables, eb, blocks, s); break;
        default:
            launch_eval<W, HX_VARIANT_PIPELINED | HX_VARIANT_ASYM>(p, o, wk, nb, tables, eb, blocks, s);
            break;
    }
    prof_mark(kKEval, true, s);
    return hipGetLastError();
}

}  // namespace

int mask_words(int32_t n_gpus) { return n_gpus <= 64 ? 1 : (n_gpus <= 128 ? 2 : 4); }

static size_t units_bytes(int32_t n_gpus, int32_t max_groups, int32_t n_cand) {
    const size_t b = sizeof(uint64_t) * (1 + mask_words(n_gpus)) * (size_t)max_units(n_gpus, max_groups, n_cand);
    return (b + 255) & ~(size_t)255;
}

static size_t tables_bytes(int32_t n_gpus) {
    return sizeof(double) * HX_MAX_CLASSES * (HX_MAX_TP + 1) * (size_t)n_gpus * n_gpus;
}

static size_t unfit_bytes(int32_t n_gpus) {
    return sizeof(uint64_t) * ((size_t)n_gpus + 2) * mask_words(n_gpus);
}

// Layout: histogram and cursors, one more word (cleared with them; hx_score_batch's argmax
// counts its finished workgroups there), unit records, prefill link tables, the memory-row
// screen, a key byte per group slot, and (256-byte aligned) candidate 0's reference groups.
static size_t ref_offset(int32_t n_gpus, int32_t max_groups, int32_t n_cand) {
    const size_t nb = 2 * ((size_t)n_gpus + 1);
    const size_t head = ((2 * nb + 2) * sizeof(int32_t) + 255) & ~(size_t)255;
    const size_t end = head + units_bytes(n_gpus, max_groups, n_cand) + tables_bytes(n_gpus) + unfit_bytes(n_gpus) +
                       sizeof(uint16_t) * (size_t)max_groups * n_cand;
    return (end + 255) & ~(size_t)255;
}

size_t cost_workspace_bytes(int32_t n_gpus, int32_t max_groups, int32_t n_cand) {
    return ref_offset(n_gpus, max_groups, n_cand) + ref_bytes(max_groups);
}

int32_t* cost_workspace_counter(void* workspace, int32_t n_gpus) {
    return reinterpret_cast<int32_t*>(workspace) + 4 * ((size_t)n_gpus + 1) + 1;
}

hipError_t launch_cost(const Problem& p, const CostOut& o, void* workspace, hipStream_t s, unsigned long long* clear,
                       int n_clear) {
    const size_t nb = 2 * ((size_t)p.G + 1);
    const size_t head = ((2 * nb + 2) * sizeof(int32_t) + 255) & ~(size_t)255;
    CostWork wk;
    wk.hist = reinterpret_cast<int32_t*>(workspace);
    wk.cursor = wk.hist + nb + 1;
    wk.units = reinterpret_cast<uint64_t*>(reinterpret_cast<unsigned char*>(workspace) + head);
    wk.tp_pre = reinterpret_cast<double*>(reinterpret_cast<unsigned char*>(workspace) + head +
                                          units_bytes(p.G, p.Kmax, p.N));
    wk.pp_pre = wk.tp_pre + (size_t)HX_MAX_TP * p.G * p.G;
    wk.unfit = reinterpret_cast<uint64_t*>(reinterpret_cast<unsigned char*>(wk.tp_pre) + tables_bytes(p.G));
    wk.ukey = reinterpret_cast<uint16_t*>(reinterpret_cast<unsigned char*>(wk.unfit) + unfit_bytes(p.G));
    wk.ref_base = reinterpret_cast<unsigned char*>(workspace) + ref_offset(p.G, p.Kmax, p.N);
    wk.clear2 = clear;
    wk.n_clear2 = clear ? n_clear : 0;
    wk.ref = carve_ref(wk.ref_base, p.Kmax);
    wk.gmask = o.members;
    switch (mask_words(p.G)) {
        case 1: return launch_w<1>(p, o, wk, s);
        case 2: return launch_w<2>(p, o, wk, s);
        default: return launch_w<4>(p, o, wk, s);
    }
}

}  // namespace hx
