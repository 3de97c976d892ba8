// hx_flownet.hip -- the Sec. 3.3 flow network of every candidate, on gfx950.
//
// Both kernels read the group member bitmasks hx_cost_eval wrote, so no kernel here scans
// the assign array for a group's members.  Both run candidate-fastest, so loads and stores
// of the [row][n] arrays coalesce across the wavefront:
//   nodes_kernel  one lane per candidate: lists the prefill and decode nodes (replicas in
//                 ascending group id, or GPUs in ascending id at per-GPU granularity) with
//                 their source, node and sink capacities (Appendix A), and, for the listed KV
//                 path, which replica nodes have a strategy (FlowNet::feas);
//   kv_kernel     one lane per (KV edge, candidate): the edge capacity between prefill node
//                 i and decode node j (connection type 3; Table 1 last row; Appendix A) of
//                 replica nodes, with the stage-order search of Appendix A (kv_order_kernel)
//                 when HX_VARIANT_KV_ORDER is set, and the class mix with request classes;
//   kv_rows_kernel, kv_scan_kernel, kv_compact_kernel, kv_walk_group_kernel  the same edges as
//                 kv_kernel when hx_score_batch hands over scratch for an edge list: one lane per
//                 candidate writes every edge with an infeasible end (0, row by row) and lists
//                 the others, the lists are packed, then 4 lanes per listed edge walk it;
//   kv_gpu_kernel the same for per-GPU nodes, a workgroup per 64 candidates.
// hx_score_batch's per-GPU path (up to 128 GPUs and 128 slots) replaces the last two: a table of
// every link's capacity (link_table_kernel), and nodes_gpu_kernel<W, true>, which settles each
// network whose KV edges all dominate while it counts its nodes and lists the others for the
// max-flow.
#include "hx_internal.h"

namespace hx {
namespace {

constexpr int kNodeBlock = 128;
constexpr int kKvBlock = 64;

template <int W>
__device__ __forceinline__ int mask_size(const uint64_t* gm, int k, int64_t N, int n) {
    int s = 0;
#pragma unroll
    for (int i = 0; i < W; ++i) s += __popcll(gm[((int64_t)k * W + i) * N + n]);
    return s;
}

// Members of group k below GPU g (its rank inside the group).
template <int W>
__device__ __forceinline__ int mask_rank(const uint64_t* gm, int k, int64_t N, int n, int g) {
    int s = 0;
#pragma unroll
    for (int i = 0; i < W; ++i) {
        const uint64_t m = gm[((int64_t)k * W + i) * N + n];
        if (i < (g >> 6)) s += __popcll(m);
        else if (i == (g >> 6)) s += __popcll(m & ((1ull << (g & 63)) - 1));
    }
    return s;
}

template <int W>
__global__ void __launch_bounds__(kNodeBlock) nodes_kernel(Problem p, CostOut o, FlowNet f) {
    const int n = blockIdx.x * blockDim.x + threadIdx.x;
    if (n >= p.N) return;
    const int64_t N = p.N;
    int np = 0, nd = 0;
    if (p.granularity == 0) {
        // Group slots in chunks of 8: the chunk's loads are issued together, then its slots
        // are appended to the node lists in ascending order.
        constexpr int kC = 8;
        uint32_t pf = 0, df = 0;  // nodes whose replica has a strategy (tp > 0), by node index
        for (int k0 = 0; k0 < p.Kmax; k0 += kC) {
            int sz[kC], rl[kC], tq[kC];
            int32_t cp[kC];
            // every load issued (slots past Kmax read slot Kmax - 1 and are replaced), so that
            // the chunk's loads are in flight together
#pragma unroll
            for (int x = 0; x < kC; ++x) {
                const int k = k0 + x < p.Kmax ? k0 + x : p.Kmax - 1;
                sz[x] = mask_size<W>(o.members, k, N, n);
                rl[x] = p.role[(int64_t)k * N + n];
                cp[x] = o.cap[(int64_t)k * N + n];
                tq[x] = o.tp[(int64_t)k * N + n];
            }
#pragma unroll
            for (int x = 0; x < kC; ++x)
                if (k0 + x >= p.Kmax) {
                    sz[x] = 0;
                    rl[x] = HX_UNUSED;
                    cp[x] = 0;
                }
#pragma unroll
            for (int x = 0; x < kC; ++x) {
                if (sz[x] == 0) continue;
                const int k = k0 + x;
                if (rl[x] == HX_PREFILL) {
                    const int64_t e = (int64_t)np * N + n;
                    f.p_slot[e] = k;
                    f.src_cap[e] = p.coord_cap;
                    f.p_cap[e] = cp[x];
                    if (tq[x] > 0 && np < 32) pf |= 1u << np;
                    ++np;
                } else if (rl[x] == HX_DECODE) {
                    const int64_t e = (int64_t)nd * N + n;
                    f.d_slot[e] = k;
                    f.d_cap[e] = cp[x];
                    f.sink_cap[e] = p.coord_cap;
                    if (tq[x] > 0 && nd < 32) df |= 1u << nd;
                    ++nd;
                }
            }
        }
        if (f.feas) f.feas[n] = (uint64_t)pf | ((uint64_t)df << 32);
    } else {
        // Per-GPU nodes: the k-th member (by GPU id) of a replica of sz GPUs and capacity C
        // carries floor(C/sz) + [k < C mod sz].
        for (int g = 0; g < p.G; ++g) {
            const int k = p.assign[(int64_t)g * N + n];
            if (k >= p.Kmax) continue;
            const int r = p.role[(int64_t)k * N + n];
            if (r != HX_PREFILL && r != HX_DECODE) continue;
            const int rk = mask_rank<W>(o.members, k, N, n, g);
            const int sz = mask_size<W>(o.members, k, N, n);
            const int32_t C = o.cap[(int64_t)k * N + n];
            const int32_t share = C / sz + (rk < C % sz ? 1 : 0);
            if (r == HX_PREFILL) {
                const int64_t e = (int64_t)np * N + n;
                f.p_slot[e] = g;
                f.src_cap[e] = p.coord_cap;
                f.p_cap[e] = share;
                ++np;
            } else {
                const int64_t e = (int64_t)nd * N + n;
                f.d_slot[e] = g;
                f.d_cap[e] = share;
                f.sink_cap[e] = p.coord_cap;
                ++nd;
            }
        }
    }
    f.n_p[n] = np;
    f.n_d[n] = nd;
}

// Per-GPU nodes with every group's role, capacity share floor(C/sz) and remainder C mod sz, and
// a running member count staged in LDS ([Kmax][64] per field, loads of eight slots issued
// together; one division per group, not per GPU), then the GPUs taken in ascending id with their
// group ids loaded sixteen at a time: the k-th member of a group met so far is its rank.  The
// same rows as nodes_kernel's per-GPU branch with ~Kmax/8 + G/16 memory round trips per lane
// instead of two per GPU.  Kmax <= kNodesGpuMaxK (the staging fits 64 KB).
constexpr int kNodesGpuMaxK = 128;
__host__ __device__ inline size_t nodes_gpu_lds(int Kmax) { return (size_t)Kmax * 64 * 7; }

// kValue (hx_score_batch): the kernel also settles the network's value, and writes the node rows
// only of the networks it does not settle (the counts always).  Every KV edge of a per-GPU
// network has its link's capacity (tab: [G][G], computed once per call), so when every edge can
// carry min(a_i, b_j) (a_i the prefill node's source-or-node capacity, b_j the decode node's
// node-or-sink capacity) the maximum flow is min(sum a, sum b), the max-flow kernel's
// dominant-KV closed form, and the KV rows are never needed.  rmin[g], the smallest capacity of
// GPU g's links, decides most networks on the fly: an edge out of prefill node i can be thin
// only if rmin[g_i] < min(a_i, b_max).  The others are checked edge by edge; a network with a
// thin edge gets its KV rows and flow_value -1, and its candidate goes to the list the max-flow
// kernel works through (list_count, cleared by link_table_kernel).  Edges with an end of
// capacity 0 never bind (min(a_i, b_j) = 0); an infeasible replica's GPUs carry 0.
template <int W, bool kValue>
__global__ void __launch_bounds__(64) nodes_gpu_kernel(Problem p, CostOut o, FlowNet f, const int32_t* tab,
                                                       const int32_t* rmin, int32_t* flow_value, int32_t* list,
                                                       int32_t* list_count) {
    extern __shared__ __attribute__((aligned(16))) uint8_t sm[];
    const int lane = threadIdx.x;
    const int Kmax = p.Kmax;
    int32_t* gquo = reinterpret_cast<int32_t*>(sm);        // [Kmax][64] floor(C / sz)
    uint8_t* grole = sm + sizeof(int32_t) * (size_t)Kmax * 64;  // [Kmax][64]
    uint8_t* grem = grole + (size_t)Kmax * 64;               // [Kmax][64] C mod sz (< sz <= 255)
    uint8_t* gseen = grem + (size_t)Kmax * 64;               // [Kmax][64]: members met so far
    const int64_t N = p.N;
    const int64_t n = (int64_t)blockIdx.x * 64 + lane;
    if (n >= N) return;  // no barrier below: every lane stages and reads its own column
    constexpr int kC = 8;
    for (int k0 = 0; k0 < Kmax; k0 += kC) {
        int32_t cp[kC];
        int rl[kC], sz[kC];
        // every load issued (slots past Kmax read slot Kmax - 1 and are replaced), so that the
        // chunk's loads are in flight together
#pragma unroll
        for (int x = 0; x < kC; ++x) {
            const int k = k0 + x < Kmax ? k0 + x : Kmax - 1;
            sz[x] = mask_size<W>(o.members, k, N, (int)n);
            rl[x] = p.role[(int64_t)k * N + n];
            cp[x] = o.cap[(int64_t)k * N + n];
        }
#pragma unroll
        for (int x = 0; x < kC; ++x)
            if (k0 + x >= Kmax) {
                sz[x] = 0;
                rl[x] = HX_UNUSED;
                cp[x] = 0;
            }
#pragma unroll
        for (int x = 0; x < kC; ++x) {
            const int k = k0 + x;
            if (k >= Kmax) break;
            // a slot with no member is never looked up (no GPU names it)
            const int d = sz[x] > 0 ? sz[x] : 1;
            gquo[k * 64 + lane] = cp[x] / d;
            grem[k * 64 + lane] = (uint8_t)(cp[x] % d);
            grole[k * 64 + lane] = (uint8_t)rl[x];
            gseen[k * 64 + lane] = 0;
        }
    }
    int np = 0, nd = 0;
    long long sa = 0, sb = 0;  // kValue
    int32_t bmax = 0, t1 = 0x7fffffff;
    bool any_a = false;
    // One pass over the GPUs in ascending id: node counts, sums for kValue, and the node rows
    // when `rows` (a replayed pass starts from zeroed member counts).
    auto pass = [&](bool rows, bool replay) {
        np = nd = 0;
        sa = sb = 0;
        bmax = 0;
        t1 = 0x7fffffff;
        any_a = false;
        if (replay)
            for (int k = 0; k < Kmax; ++k) gseen[k * 64 + lane] = 0;
        constexpr int kCG = 16;  // GPUs per batch of loads (eight slots per batch above)
        for (int g0 = 0; g0 < p.G; g0 += kCG) {
            // the chunk's loads issued together (rows past G read row G - 1 and are replaced);
            // kValue: the GPUs' smallest link capacities with them
            int kk[kCG];
            int32_t rm[kCG];
#pragma unroll
            for (int x = 0; x < kCG; ++x) {
                const int g = g0 + x < p.G ? g0 + x : p.G - 1;
                kk[x] = p.assign[(int64_t)g * N + n];
                rm[x] = kValue ? rmin[g] : 0;
            }
#pragma unroll
            for (int x = 0; x < kCG; ++x)
                if (g0 + x >= p.G) kk[x] = HX_UNUSED;
#pragma unroll
            for (int x = 0; x < kCG; ++x) {
                const int g = g0 + x, k = kk[x];
                if (g >= p.G || k >= Kmax) continue;
                const int r = grole[k * 64 + lane];
                if (r != HX_PREFILL && r != HX_DECODE) continue;
                const int rk = gseen[k * 64 + lane];
                gseen[k * 64 + lane] = (uint8_t)(rk + 1);
                const int32_t share = gquo[k * 64 + lane] + (rk < grem[k * 64 + lane] ? 1 : 0);
                if (r == HX_PREFILL) {
                    if (rows) {
                        const int64_t e = (int64_t)np * N + n;
                        f.p_slot[e] = g;
                        f.src_cap[e] = p.coord_cap;
                        f.p_cap[e] = share;
                    }
                    ++np;
                    if (kValue) {
                        const int32_t a = p.coord_cap < share ? p.coord_cap : share;
                        sa += a;
                        if (a > 0) {
                            any_a = true;
                            const int32_t m = rm[x];
                            if (m < a && m < t1) t1 = m;
                        }
                    }
                } else {
                    if (rows) {
                        const int64_t e = (int64_t)nd * N + n;
                        f.d_slot[e] = g;
                        f.d_cap[e] = share;
                        f.sink_cap[e] = p.coord_cap;
                    }
                    ++nd;
                    if (kValue) {
                        const int32_t b = share < p.coord_cap ? share : p.coord_cap;
                        sb += b;
                        bmax = b > bmax ? b : bmax;
                    }
                }
            }
        }
    };
    pass(!kValue, false);
    f.n_p[n] = np;
    f.n_d[n] = nd;
    if (!kValue) return;
    if (t1 >= bmax) {  // every KV edge dominant: no row is needed
        // < 2^31: the smaller side has at most 127 nodes of at most 2^24 - 1
        flow_value[n] = (!any_a || bmax <= 0) ? 0 : (int32_t)(sa < sb ? sa : sb);
        return;
    }
    pass(true, true);  // the rows, for the edge-by-edge check and the max-flow
    const int G = p.G;
    bool dominant;
    {  // edge by edge (this lane's own rows, just written)
        bool thin = false;
        for (int i = 0; i < np && !thin; ++i) {
            const int32_t ps = f.src_cap[(int64_t)i * N + n], pc = f.p_cap[(int64_t)i * N + n];
            const int32_t a = ps < pc ? ps : pc;
            if (a <= 0) continue;
            const int g = f.p_slot[(int64_t)i * N + n];
            for (int j = 0; j < nd && !thin; ++j) {
                const int32_t dc = f.d_cap[(int64_t)j * N + n], dt = f.sink_cap[(int64_t)j * N + n];
                const int32_t b = dc < dt ? dc : dt;
                thin = b > 0 && tab[g * G + f.d_slot[(int64_t)j * N + n]] < (a < b ? a : b);
            }
        }
        dominant = !thin;
    }
    if (dominant) {
        // < 2^31: the smaller side has at most 127 nodes of at most 2^24 - 1
        flow_value[n] = (!any_a || bmax <= 0) ? 0 : (int32_t)(sa < sb ? sa : sb);
        return;
    }
    // a thin edge: the max-flow kernel solves this network from its KV rows
    for (int i = 0; i < np; ++i) {
        const int g = f.p_slot[(int64_t)i * N + n];
        const int kg = p.assign[(int64_t)g * N + n];
        const bool okg = o.tp[(int64_t)kg * N + n] > 0;
        for (int j = 0; j < nd; ++j) {
            const int h = f.d_slot[(int64_t)j * N + n];
            const int kh = p.assign[(int64_t)h * N + n];
            const bool okh = o.tp[(int64_t)kh * N + n] > 0;
            f.kv_cap[(int64_t)(i * nd + j) * N + n] = okg && okh ? tab[g * G + h] : 0;
        }
    }
    flow_value[n] = -1;
    list[atomicAdd(list_count, 1)] = (int32_t)n;
}


// Launches the node rows: nodes_gpu_kernel for per-GPU networks of up to kNodesGpuMaxK slots,
// nodes_kernel otherwise.
template <int W>
void launch_nodes(const Problem& p, const CostOut& o, const FlowNet& f, hipStream_t s) {
    if (p.granularity == 1 && p.Kmax <= kNodesGpuMaxK)
        hipLaunchKernelGGL((nodes_gpu_kernel<W, false>), dim3((p.N + 63) / 64), dim3(64), nodes_gpu_lds(p.Kmax), s, p,
                           o, f, nullptr, nullptr, nullptr, nullptr, nullptr);
    else
        hipLaunchKernelGGL(nodes_kernel<W>, dim3((p.N + kNodeBlock - 1) / kNodeBlock), dim3(kNodeBlock), 0, s, p, o, f);
}

// Members of group k in ascending GPU id into out[r * stride]; returns the count.
template <int W>
__device__ __forceinline__ int expand(const uint64_t* gm, int k, int64_t N, int n, uint8_t* out, int stride) {
    int cnt = 0;
#pragma unroll
    for (int i = 0; i < W; ++i) {
        uint64_t m = gm[((int64_t)k * W + i) * N + n];
        while (m) {
            out[(cnt++) * stride] = (uint8_t)(i * 64 + __builtin_ctzll(m));
            m &= m - 1;
        }
    }
    return cnt;
}

// Members of a group given its mask words, in ascending GPU id into out[r * stride]; returns the
// count.
template <int W>
__device__ __forceinline__ int expand_words(const uint64_t* mw, uint8_t* out, int stride) {
    int cnt = 0;
#pragma unroll
    for (int i = 0; i < W; ++i) {
        uint64_t m = mw[i];
        while (m) {
            out[(cnt++) * stride] = (uint8_t)(i * 64 + __builtin_ctzll(m));
            m &= m - 1;
        }
    }
    return cnt;
}

// KV time of one request from a prefill replica (pm, ptp x ppp) to a decode replica
// (dm, dtp x dpp): the slowest of the links that carry a layer range and head slice.  The
// stage layer ranges of the two sides are two partitions of [0, L), and the rank head
// slices (in units of 1/(ptp*dtp)) two partitions of [0, ptp*dtp), so merge walks visit
// exactly the overlapping (stage, stage) and (rank, rank) pairs.
__device__ double kv_time(const Problem& p, const uint8_t* pm, int ptp, int ppp, const uint8_t* dm, int dtp,
                          int dpp, int stride) {
    const double V1 = 2.0 * p.s_in * p.Hkv * p.B;
    const int deni = ptp * dtp;
    const double den = (double)deni;
    // Dividing by a power of two only shifts the exponent, so it equals multiplying by the
    // exact reciprocal: the same binary64 value with one division less per link.
    const bool pow2 = (deni & (deni - 1)) == 0;
    const double inv_den = 1.0 / den;
    const int lqp = p.L / ppp, lrp = p.L % ppp, lqd = p.L / dpp, lrd = p.L % dpp;
    double worst = 0.0;
    int a = 0, bb = 0, a0 = 0, b0 = 0;
    int a1 = lqp + (0 < lrp ? 1 : 0), b1 = lqd + (0 < lrd ? 1 : 0);
    while (a < ppp && bb < dpp) {
        const int nab = (a1 < b1 ? a1 : b1) - (a0 > b0 ? a0 : b0);
        const double Vn = V1 * (double)nab;
        const uint8_t* Sa = pm + (a * ptp) * stride;
        const uint8_t* Sb = dm + (bb * dtp) * stride;
        int r = 0, q = 0;
        while (r < ptp && q < dtp) {
            const int re = (r + 1) * dtp, qe = (q + 1) * ptp;
            const int ov = (re < qe ? re : qe) - (r * dtp > q * ptp ? r * dtp : q * ptp);
            const int g = Sa[r * stride], h = Sb[q * stride];
            const double bytes = pow2 ? (Vn * (double)ov) * inv_den : (Vn * (double)ov) / den;
            const double time = p.alpha[g * p.G + h] + bytes / p.beta[g * p.G + h];
            if (time > worst) worst = time;
            if (re <= qe) ++r;
            if (qe <= re) ++q;
        }
        const bool adv_a = a1 <= b1, adv_b = b1 <= a1;
        if (adv_a) {
            ++a;
            a0 = a1;
            a1 = a0 + lqp + (a < lrp ? 1 : 0);
        }
        if (adv_b) {
            ++bb;
            b0 = b1;
            b1 = b0 + lqd + (bb < lrd ? 1 : 0);
        }
    }
    return worst;
}

// kv_time of every request class in one walk: the links, their member ids and alpha/beta are
// the same for every class, only the bytes differ (V1 from the class's s_in), so the walk keeps
// one running maximum per class and returns sum_k w_k worst_k (class order, left to right).
// Each class's maximum is the binary64 value kv_time returns for that class.
__device__ double kv_time_classes(const Problem& p, const uint8_t* pm, int ptp, int ppp, const uint8_t* dm, int dtp,
                                  int dpp, int stride) {
    const int nc = p.n_cls;
    double V1[HX_MAX_CLASSES], worst[HX_MAX_CLASSES];
#pragma unroll
    for (int k = 0; k < HX_MAX_CLASSES; ++k) {
        V1[k] = 2.0 * p.cls_in[k] * p.Hkv * p.B;
        worst[k] = 0.0;
    }
    const int deni = ptp * dtp;
    const double den = (double)deni;
    const bool pow2 = (deni & (deni - 1)) == 0;
    const double inv_den = 1.0 / den;
    const int lqp = p.L / ppp, lrp = p.L % ppp, lqd = p.L / dpp, lrd = p.L % dpp;
    int a = 0, bb = 0, a0 = 0, b0 = 0;
    int a1 = lqp + (0 < lrp ? 1 : 0), b1 = lqd + (0 < lrd ? 1 : 0);
    while (a < ppp && bb < dpp) {
        const int nab = (a1 < b1 ? a1 : b1) - (a0 > b0 ? a0 : b0);
        const uint8_t* Sa = pm + (a * ptp) * stride;
        const uint8_t* Sb = dm + (bb * dtp) * stride;
        int r = 0, q = 0;
        while (r < ptp && q < dtp) {
            const int re = (r + 1) * dtp, qe = (q + 1) * ptp;
            const int ov = (re < qe ? re : qe) - (r * dtp > q * ptp ? r * dtp : q * ptp);
            const int g = Sa[r * stride], h = Sb[q * stride];
            const double al = p.alpha[g * p.G + h], be = p.beta[g * p.G + h];
#pragma unroll
            for (int k = 0; k < HX_MAX_CLASSES; ++k) {
                if (k >= nc) break;
                const double Vn = V1[k] * (double)nab;
                const double bytes = pow2 ? (Vn * (double)ov) * inv_den : (Vn * (double)ov) / den;
                const double time = al + bytes / be;
                if (time > worst[k]) worst[k] = time;
            }
            if (re <= qe) ++r;
            if (qe <= re) ++q;
        }
        const bool adv_a = a1 <= b1, adv_b = b1 <= a1;
        if (adv_a) {
            ++a;
            a0 = a1;
            a1 = a0 + lqp + (a < lrp ? 1 : 0);
        }
        if (adv_b) {
            ++bb;
            b0 = b1;
            b1 = b0 + lqd + (bb < lrd ? 1 : 0);
        }
    }
    double t = 0.0;
#pragma unroll
    for (int k = 0; k < HX_MAX_CLASSES; ++k)
        if (k < nc) t = t + p.cls_w[k] * worst[k];
    return t;
}

// KV stage-order search (HX_VARIANT_KV_ORDER; Appendix A, edge capacity estimation): the stage
// orders of both replicas are chosen to minimise the KV time, over every pair of orders.
//
// The KV time of an order pair is the largest block time over the pairs of pipeline positions
// that share layers (a block: the slowest link between the two stages serving the positions).
// With the order of one side X fixed, each position y of the other side Y contributes
// C[y][t] = max over the X positions sharing layers with y of the block time when Y's stage t
// serves y, and the KV time is max_y C[y][ord_Y(y)]; the best Y order is a bottleneck
// assignment of C.  So the search runs over the orders of X, the side with fewer stages
// (prefill on ties; at most 8! = 40,320), cutting those that bounds rule out, and solves one
// bottleneck assignment per order left: the smallest threshold T, among C's entries, under which
// a perfect matching of positions to stages exists.  Orders are packed 4 bits per pipeline
// position (position a is served by stage (ord >> 4a) & 15).  Pipelines of up to 8 stages (the
// PP mask is validated).
constexpr int kOrderStages = 8;
constexpr int kBlockPairs = 2 * kOrderStages - 1;  // position pairs sharing layers, at most
__device__ __forceinline__ int nib(uint32_t v, int i) { return (int)((v >> (4 * i)) & 15u); }

// First layer of pipeline position a of a pipeline of pp stages (uniform split, remainder to the
// earlier positions).
__device__ __forceinline__ int pos_first(int L, int pp, int a) { return a * (L / pp) + (a < L % pp ? a : L % pp); }

// Slowest link between prefill stage s and decode stage t when they serve positions sharing nab
// layers: the merge walk of kv_time over the rank pairs whose head slices overlap.
__device__ double kv_block_time(const Problem& p, const uint8_t* pm, int ptp, int s, const uint8_t* dm, int dtp,
                                int t, int nab, int stride) {
    const double Vn = (2.0 * p.s_in * p.Hkv * p.B) * (double)nab;
    const int deni = ptp * dtp;
    const double den = (double)deni;
    const bool pow2 = (deni & (deni - 1)) == 0;
    const double inv_den = 1.0 / den;
    const uint8_t* Sa = pm + (s * ptp) * stride;
    const uint8_t* Sb = dm + (t * dtp) * stride;
    double worst = 0.0;
    int r = 0, q = 0;
    while (r < ptp && q < dtp) {
        const int re = (r + 1) * dtp, qe = (q + 1) * ptp;
        const int ov = (re < qe ? re : qe) - (r * dtp > q * ptp ? r * dtp : q * ptp);
        const int g = Sa[r * stride], h = Sb[q * stride];
        const double bytes = pow2 ? (Vn * (double)ov) * inv_den : (Vn * (double)ov) / den;
        const double time = p.alpha[g * p.G + h] + bytes / p.beta[g * p.G + h];
        if (time > worst) worst = time;
        if (re <= qe) ++r;
        if (qe <= re) ++q;
    }
    return worst;
}

// Whether the bipartite graph with rows 0..n-1 (n <= 8) and row y's columns the bits of byte y
// of rm has a matching covering at least need rows: augmenting paths found by breadth-first
// search from each row in turn (a row with none now never gains one later), with the matching
// and the search's parents packed 4 bits per column / row.
__device__ bool has_matching(uint64_t rm, int n, int need) {
    int missed = 0;
    uint32_t row_of_col = 0xFFFFFFFFu, col_of_row = 0xFFFFFFFFu;  // 15: none
    for (int i = 0; i < n; ++i) {
        uint32_t parent = 0, seen = 0, front = 1u << i;
        int found = -1;
        while (front && found < 0) {
            const int u = __ffs(front) - 1;
            front &= front - 1;
            uint32_t av = (uint32_t)((rm >> (8 * u)) & 0xFFu) & ~seen;
            while (av) {
                const int j = __ffs(av) - 1;
                av &= av - 1;
                seen |= 1u << j;
                parent = (parent & ~(15u << (4 * j))) | ((uint32_t)u << (4 * j));
                const int r = (int)((row_of_col >> (4 * j)) & 15u);
                if (r == 15) {
                    found = j;
                    break;
                }
                front |= 1u << r;
            }
        }
        if (found < 0) {
            if (++missed > n - need) return false;
            continue;
        }
        for (int j = found;;) {  // flip the path: each row on it takes the column it reached
            const int u = (int)((parent >> (4 * j)) & 15u);
            const int prev = (int)((col_of_row >> (4 * u)) & 15u);
            col_of_row = (col_of_row & ~(15u << (4 * u))) | ((uint32_t)j << (4 * u));
            row_of_col = (row_of_col & ~(15u << (4 * j))) | ((uint32_t)u << (4 * j));
            if (u == i) break;
            j = prev;
        }
    }
    return true;
}

// C[y][t] for X order sig: the largest block of the X positions sharing layers with y.
__device__ __forceinline__ double order_cell(const double* blk, const int* px, const int* ystart, uint32_t sig, int y,
                                             int t) {
    double c = 0.0;
    for (int k = ystart[y]; k < ystart[y + 1]; ++k) {
        const double b = blk[(k * kOrderStages + nib(sig, px[k])) * kOrderStages + t];
        c = b > c ? b : c;
    }
    return c;
}

// Rows y in [y0, y1) of C (X order sig): the largest row minimum min_t C[y][t] (every Y order
// takes one entry of each row, so this bounds its KV time from below) into lb, and the entries
// below best into mask bits 8y + t.
__device__ __forceinline__ void rows_scan(const double* blk, const int* px, const int* ystart, uint32_t sig, int y0,
                                          int y1, int ny, double best, double& lb, uint64_t& mask) {
    lb = 0.0;
    mask = 0;
    for (int y = y0; y < y1; ++y) {
        double m = 0.0;
        for (int c = 0; c < ny; ++c) {
            const double v = order_cell(blk, px, ystart, sig, y, c);
            m = (c == 0 || v < m) ? v : m;
            if (v < best) mask |= 1ull << (8 * y + c);
        }
        lb = m > lb ? m : lb;
    }
}

// A complete X order sig whose row bound lb is below the best: the column bound, a test that a
// perfect matching below the best exists at all, then the bottleneck assignment from the bound
// upwards; returns the KV time if below best.
__device__ double order_leaf(const double* blk, const int* px, const int* ystart, uint32_t sig, int ny, double lb,
                             double best) {
    for (int c = 0; c < ny && lb < best; ++c) {
        double m = order_cell(blk, px, ystart, sig, 0, c);
        for (int y = 1; y < ny; ++y) {
            const double v = order_cell(blk, px, ystart, sig, y, c);
            m = v < m ? v : m;
        }
        lb = m > lb ? m : lb;
    }
    if (lb >= best) return best;
    {  // no perfect matching strictly below best: this order cannot improve on it
        uint64_t rm = 0;
        for (int y = 0; y < ny; ++y)
            for (int c = 0; c < ny; ++c)
                if (order_cell(blk, px, ystart, sig, y, c) < best) rm |= 1ull << (8 * y + c);
        if (!has_matching(rm, ny, ny)) return best;
    }
    double T = lb;
    while (T < best) {
        uint64_t rm = 0;
        double next = best;
        for (int y = 0; y < ny; ++y)
            for (int c = 0; c < ny; ++c) {
                const double v = order_cell(blk, px, ystart, sig, y, c);
                if (v <= T) rm |= 1ull << (8 * y + c);
                else if (v < next) next = v;
            }
        if (has_matching(rm, ny, ny)) return T;
        T = next;  // the next entry above T, or best when none is below it
    }
    return best;
}

// A bound below the KV time of every order pair, from the position pairs sharing layers: take
// pairs with no position in common (S: a greedy matching along the merge walk, here among the
// pairs sharing at least pn[k0] layers).  Any order pair serves S by |S| distinct X stages and
// |S| distinct Y stages, and a block time never decreases with the layers shared, so the KV
// time is at least the smallest threshold under which the block times of S's fewest shared
// layers admit a matching of |S| X stages to Y stages.  One wavefront finds it by bisection over
// the entries: lane l holds entry (X stage l / 8, Y stage l % 8), a wavefront minimum picks the
// entry inside (lo, hi) nearest the middle, and the ballot of the entries at most that pivot is
// the matching's bit mask (byte x, bit y).  Every lane returns the bound.
__device__ double pairs_bound(const double* blk, const int* px, const int* py, const int* pn, int npairs, int k0,
                              int nx, int ny, int lane) {
    const int q = pn[k0];
    uint32_t ux = 0, uy = 0;
    int size = 0, kmin = -1;
    for (int k = 0; k < npairs; ++k) {
        if (pn[k] < q || ((ux >> px[k]) & 1u) || ((uy >> py[k]) & 1u)) continue;
        ux |= 1u << px[k];
        uy |= 1u << py[k];
        ++size;
        if (kmin < 0 || pn[k] < pn[kmin]) kmin = k;
    }
    const int xs = lane >> 3, yt = lane & 7;
    const bool ok = xs < nx && yt < ny;
    const double v = ok ? blk[kmin * kOrderStages * kOrderStages + lane] : 0.0;
    double hi = v;  // the largest entry admits a matching of size |S| (times are positive)
    for (int off = 32; off > 0; off >>= 1) {
        const double o = __shfl_xor(hi, off, 64);
        hi = o > hi ? o : hi;
    }
    double lo = 0.0;  // no entry is at most 0: no matching
    for (;;) {
        const double mid = 0.5 * (lo + hi);
        const bool inside = ok && v > lo && v < hi;
        double g = inside ? (v > mid ? v - mid : mid - v) : hi;  // hi - lo bounds every gap inside
        double piv = inside ? v : hi;
        bool any = inside;
        for (int off = 32; off > 0; off >>= 1) {
            const double og = __shfl_xor(g, off, 64), op = __shfl_xor(piv, off, 64);
            const bool oa = __shfl_xor((int)any, off, 64) != 0;
            if (oa && (!any || og < g || (og == g && op < piv))) {
                g = og;
                piv = op;
                any = true;
            }
        }
        if (!any) return hi;
        const uint64_t rm = __ballot(ok && v <= piv);
        if (has_matching(rm, nx, size)) hi = piv;
        else lo = piv;
    }
}

__device__ __forceinline__ uint32_t set_nib(uint32_t v, int i, int x) {
    return (v & ~(15u << (4 * i))) | ((uint32_t)x << (4 * i));
}

constexpr int kOrderThreads = 256;  // kv_order_kernel: wave 0 holds the lanes, all four waves search
constexpr int kOrderLevels = 4;     // search levels below a queued prefix, at most
constexpr int kOrderQueue = 2 * kOrderThreads;  // prefixes handed out per edge, at least (when nx allows)

// LDS of kv_order_kernel before the member lists.
struct OrderShared {
    double blk[kBlockPairs * kOrderStages * kOrderStages];  // [pair][X stage][Y stage]
    double lbsave[kOrderLevels * kOrderThreads];             // [level][thread]: row bound before the level
    uint64_t mksave[kOrderLevels * kOrderThreads];           // [level][thread]: final-row mask before it
    double t[kKvBlock];                                      // lanes' ascending-order times
    double best, glb;
    uint32_t colord[kBlockPairs * kOrderStages];  // [pair][Y stage]: X stages by ascending block time
    int32_t shape[kKvBlock];                      // lanes' ptp | ppp << 8 | dtp << 16 | dpp << 24
    int32_t list[kKvBlock];                       // lanes whose edge is searched
    int32_t px[kBlockPairs], py[kBlockPairs], pn[kBlockPairs];
    int32_t ystart[kOrderStages + 1];  // first pair of each Y position
    int32_t yfin[kOrderStages + 1];    // rows below yfin[d] are final once X positions 0..d-1 are assigned
    int32_t count, queue;
};
constexpr size_t kOrderLds = (sizeof(OrderShared) + 15) & ~(size_t)15;

// Whether an order pair below best can still complete the partial X order sig (positions
// 0..nass-1 assigned, stages used taken): every entry of C is bounded below by taking, at each
// unassigned position sharing layers with its row, the cheapest block over the stages still
// unused (colord lists them by block time), and a perfect matching of the rows to the Y stages
// over entries whose bound is below best must exist.
__device__ bool order_bound_ok(const OrderShared& S, uint32_t sig, int nass, uint32_t used, int ny, double best) {
    uint64_t m = 0;
    for (int y = 0; y < ny; ++y)
        for (int c = 0; c < ny; ++c) {
            double v = 0.0;
            for (int k = S.ystart[y]; k < S.ystart[y + 1]; ++k) {
                int st;
                if (S.px[k] < nass) {
                    st = nib(sig, S.px[k]);
                } else {  // some stage is unused while a position is unassigned
                    const uint32_t ord = S.colord[k * kOrderStages + c];
                    int j = 0;
                    do st = nib(ord, j++);
                    while ((used >> st) & 1u);
                }
                const double b = S.blk[(k * kOrderStages + st) * kOrderStages + c];
                v = b > v ? b : v;
            }
            if (v < best) m |= 1ull << (8 * y + c);
        }
    return has_matching(m, ny, ny);
}

// One thread's part of an edge's search: prefixes of the X order (the first pd positions) are
// taken from a queue in LDS, then searched depth first below the prefix.  A branch is cut when
// the largest final-row minimum reaches the best time found, when the final rows cannot be
// matched to distinct Y stages by entries below it, or (three or more positions left) when
// order_bound_ok fails; a complete order solves its bottleneck assignment.  Returns when the
// queue is empty or the best has reached the edge's global bound.
__device__ __forceinline__ void order_search(OrderShared& S, int nx, int ny, int tid) {
    volatile double* vbest = &S.best;
    const double glb = S.glb;
    int pd = 0, P = 1;  // prefix depth: at least kOrderQueue prefixes, at most kOrderLevels levels below
    while (pd < nx && (P < kOrderQueue || nx - pd > kOrderLevels)) P *= nx - pd++;
    for (;;) {
        if (*vbest <= glb) return;
        int r = atomicAdd(&S.queue, 1);
        if (r >= P) return;
        uint32_t sig = 0, used = 0;
        double lb = 0.0;
        bool cut = false;
        for (int l = 0, f = P; l < pd && !cut; ++l) {  // prefix r: mixed radix nx, nx - 1, ...
            f /= nx - l;
            int k = r / f, st = 0;
            r -= k * f;
            for (;; ++st)
                if (!((used >> st) & 1u) && k-- == 0) break;
            sig = set_nib(sig, l, st);
            used |= 1u << st;
            double b;
            uint64_t unused_mask;
            rows_scan(S.blk, S.px, S.ystart, sig, S.yfin[l], S.yfin[l + 1], ny, 0.0, b, unused_mask);
            lb = b > lb ? b : lb;
            cut = lb >= *vbest;
        }
        if (cut) continue;
        double best = *vbest, b0;
        uint64_t mk;
        rows_scan(S.blk, S.px, S.ystart, sig, 0, S.yfin[pd], ny, best, b0, mk);
        if (!has_matching(mk, S.yfin[pd], S.yfin[pd])) continue;
        if (pd <= nx - 3 && !order_bound_ok(S, sig, pd, used, ny, best)) continue;
        uint32_t next = 0;  // nibble d: the next stage to try at position d
        int d = pd;
        for (;;) {
            best = *vbest;
            if (best <= glb) return;
            if (d == nx) {  // a complete order
                const double v = order_leaf(S.blk, S.px, S.ystart, sig, ny, lb, best);
                if (v < best)
                    atomicMin(reinterpret_cast<unsigned long long*>(&S.best),
                              (unsigned long long)__double_as_longlong(v));
            } else {
                int st = nib(next, d);
                while (st < nx && ((used >> st) & 1u)) ++st;
                if (st < nx) {
                    next = set_nib(next, d, st + 1);
                    sig = set_nib(sig, d, st);
                    double b;
                    uint64_t add;
                    rows_scan(S.blk, S.px, S.ystart, sig, S.yfin[d], S.yfin[d + 1], ny, best, b, add);
                    const double lb2 = b > lb ? b : lb;
                    const uint64_t mk2 = mk | add;
                    if (lb2 >= best) continue;  // cut: the next stage at position d
                    if (S.yfin[d + 1] > S.yfin[d] && !has_matching(mk2, S.yfin[d + 1], S.yfin[d + 1])) continue;
                    if (d + 1 <= nx - 3 && !order_bound_ok(S, sig, d + 1, used | (1u << st), ny, best)) continue;
                    S.lbsave[(d - pd) * kOrderThreads + tid] = lb;
                    S.mksave[(d - pd) * kOrderThreads + tid] = mk;
                    used |= 1u << st;
                    lb = lb2;
                    mk = mk2;
                    ++d;
                    continue;
                }
                next = set_nib(next, d, 0);  // position d exhausted
            }
            if (--d < pd) break;  // back to position d
            used &= ~(1u << nib(sig, d));
            lb = S.lbsave[(d - pd) * kOrderThreads + tid];
            mk = S.mksave[(d - pd) * kOrderThreads + tid];
        }
    }
}

// One lane per (KV edge, candidate), as kv_kernel, with the stage-order search: the lanes (wave 0
// of a 256-thread workgroup) first take their ascending-order times; then all four waves search
// the edge of each lane whose replicas are not both single-stage, one edge at a time.  The block
// table of that edge goes to LDS, and the orders of the side with fewer stages (X) are searched
// position by position: row y of C is final once every X position sharing layers with y is
// assigned, and the bounds of order_search cut branches that cannot beat the best time found
// (shared in LDS, starting from the ascending time).  The search ends once the best reaches a
// bound below every order pair (pairs_bound, the largest over the threads).  The minimum is the
// one the enumeration of every order pair finds.  Per-replica granularity.
template <int W>
__global__ void __launch_bounds__(kOrderThreads) kv_order_kernel(Problem p, CostOut o, FlowNet f) {
    extern __shared__ __attribute__((aligned(16))) uint8_t sm[];
    OrderShared& S = *reinterpret_cast<OrderShared*>(sm);
    uint8_t* mem = sm + kOrderLds;
    const int tid = threadIdx.x;
    const int stride = kKvBlock;
    const int64_t gid = (int64_t)blockIdx.x * kKvBlock + tid;
    const int64_t N = p.N;
    bool live = tid < kKvBlock && gid < (int64_t)f.max_pd * N;
    const int e = live ? (int)(gid / N) : 0;
    const int n = live ? (int)(gid - (int64_t)e * N) : 0;
    const int np = live ? f.n_p[n] : 0, nd = live ? f.n_d[n] : 0;
    live = live && e < np * nd;
    int ptp = 0, ppp = 0, dtp = 0, dpp = 0;
    bool feas = false;
    double t = 0.0;
    if (live) {
        uint8_t* pm = mem + tid;
        uint8_t* dm = mem + p.G * stride + tid;
        const int i = e / nd, j = e - i * nd;
        const int kp = f.p_slot[(int64_t)i * N + n], kd = f.d_slot[(int64_t)j * N + n];
        ptp = o.tp[(int64_t)kp * N + n];
        ppp = o.pp[(int64_t)kp * N + n];
        dtp = o.tp[(int64_t)kd * N + n];
        dpp = o.pp[(int64_t)kd * N + n];
        feas = ptp > 0 && dtp > 0 && ppp <= kOrderStages && dpp <= kOrderStages &&
               expand<W>(o.members, kp, N, n, pm, stride) == ptp * ppp &&
               expand<W>(o.members, kd, N, n, dm, stride) == dtp * dpp;
        if (feas) t = kv_time(p, pm, ptp, ppp, dm, dtp, dpp, stride);
    }
    if (tid == 0) S.count = 0;
    __syncthreads();
    if (tid < kKvBlock) {
        S.t[tid] = t;
        S.shape[tid] = ptp | ppp << 8 | dtp << 16 | dpp << 24;
        if (feas && (ppp > 1 || dpp > 1)) S.list[atomicAdd(&S.count, 1)] = tid;
    }
    __syncthreads();
    const int count = S.count;
    for (int li = 0; li < count; ++li) {
        const int owner = S.list[li];
        const int sh = S.shape[owner];
        const int optp = sh & 255, oppp = (sh >> 8) & 255, odtp = (sh >> 16) & 255, odpp = (sh >> 24) & 255;
        const bool swap = odpp < oppp;  // X = the side with fewer stages, prefill on ties
        const int nx = swap ? odpp : oppp, ny = swap ? oppp : odpp;
        const uint8_t* opm = mem + owner;
        const uint8_t* odm = mem + p.G * stride + owner;
        if (tid == 0) {  // position pairs sharing layers, a merge walk: Y positions nondecreasing
            int a = 0, b = 0, k = 0;
            S.ystart[0] = 0;
            for (int d = 0; d <= nx; ++d) S.yfin[d] = 0;
            while (a < nx && b < ny) {
                const int xl = pos_first(p.L, nx, a), xh = pos_first(p.L, nx, a + 1);
                const int yl = pos_first(p.L, ny, b), yh = pos_first(p.L, ny, b + 1);
                S.px[k] = a;
                S.py[k] = b;
                S.pn[k] = (xh < yh ? xh : yh) - (xl > yl ? xl : yl);
                ++k;
                if (xh <= yh) ++a;
                if (yh <= xh) {
                    // Y position b's last overlapping X position is px[k - 1]: its row is final
                    // once that X position is assigned
                    S.yfin[S.px[k - 1] + 1] = b + 1;
                    S.ystart[++b] = k;
                }
            }
            for (int d = 1; d <= nx; ++d) S.yfin[d] = S.yfin[d] > S.yfin[d - 1] ? S.yfin[d] : S.yfin[d - 1];
            S.best = S.t[owner];
            S.glb = 0.0;
            S.queue = 0;
        }
        __syncthreads();
        const int npairs = S.ystart[ny];
        for (int it = tid; it < npairs * nx * ny; it += kOrderThreads) {
            const int k = it / (nx * ny), rest = it - k * nx * ny;
            const int xs = rest / ny, yt = rest - xs * ny;
            S.blk[(k * kOrderStages + xs) * kOrderStages + yt] =
                swap ? kv_block_time(p, opm, optp, yt, odm, odtp, xs, S.pn[k], stride)
                     : kv_block_time(p, opm, optp, xs, odm, odtp, yt, S.pn[k], stride);
        }
        __syncthreads();
        if (tid < npairs * ny) {  // X stages by ascending block time (ties by index), per pair and Y stage
            const int k = tid / ny, c = tid - k * ny;
            const double* col = S.blk + k * kOrderStages * kOrderStages + c;
            double v[kOrderStages];
#pragma unroll
            for (int st = 0; st < kOrderStages; ++st) v[st] = st < nx ? col[st * kOrderStages] : 0.0;
            uint32_t ord = 0;
#pragma unroll
            for (int st = 0; st < kOrderStages; ++st) {
                int r = 0;  // the stage's rank: smaller times first, then smaller index
#pragma unroll
                for (int s2 = 0; s2 < kOrderStages; ++s2)
                    r += (s2 < nx && (v[s2] < v[st] || (v[s2] == v[st] && s2 < st))) ? 1 : 0;
                if (st < nx) ord |= (uint32_t)st << (4 * r);
            }
            S.colord[k * kOrderStages + c] = ord;
        }
        {  // the global bound: a wavefront per distinct shared-layer count
            const int w = tid >> 6, lane = tid & 63;
            for (int k0 = w; k0 < npairs; k0 += kOrderThreads / 64) {
                bool seen = false;
                for (int k = 0; k < k0; ++k) seen = seen || S.pn[k] == S.pn[k0];
                if (seen) continue;
                const double b = pairs_bound(S.blk, S.px, S.py, S.pn, npairs, k0, nx, ny, lane);
                if (lane == 0)
                    atomicMax(reinterpret_cast<unsigned long long*>(&S.glb),
                              (unsigned long long)__double_as_longlong(b));
            }
        }
        __syncthreads();
        order_search(S, nx, ny, tid);
        __syncthreads();
        if (tid == owner) t = S.best;
        __syncthreads();  // the next edge overwrites the shared state
    }
    if (!live) return;
    f.kv_cap[(int64_t)e * N + n] = feas ? quantize(1000.0 / t) : 0;
}

// FLOP/s of GPU g (0 for an unknown type, as the cost model reads it).
__device__ __forceinline__ double gpu_flops(const Problem& p, int g) {
    const int t = p.gpu_type[g];
    return (t >= 0 && t < p.T) ? p.flops[t] : 0.0;
}

// Slowest FLOP/s among stage j's devices of a member list (gfl: every GPU's FLOP/s, in LDS).
__device__ double stage_flops(const double* gfl, const uint8_t* m, int stride, int j, int tp) {
    double c = gfl[m[(j * tp) * stride]];
    for (int r = 1; r < tp; ++r) c = dmin(c, gfl[m[(j * tp + r) * stride]]);
    return c;
}

// kv_time with each replica's layers following the asymmetric split (HX_VARIANT_ASYM).
__device__ double kv_time_asym(const Problem& p, const double* gfl, const uint8_t* pm, int ptp, int ppp,
                               const uint8_t* dm, int dtp, int dpp, int stride) {
    const double V1 = 2.0 * p.s_in * p.Hkv * p.B;
    const int deni = ptp * dtp;
    const double den = (double)deni;
    const bool pow2 = (deni & (deni - 1)) == 0;
    const double inv_den = 1.0 / den;
    const LayerSplit sp = layer_split<true>(p.L, ppp, [&](int j) { return stage_flops(gfl, pm, stride, j, ptp); });
    const LayerSplit sd = layer_split<true>(p.L, dpp, [&](int j) { return stage_flops(gfl, dm, stride, j, dtp); });
    double worst = 0.0;
    int a = 0, bb = 0, a0 = 0, b0 = 0;
    int a1 = split_layers<true>(sp, 0, stage_flops(gfl, pm, stride, 0, ptp));
    int b1 = split_layers<true>(sd, 0, stage_flops(gfl, dm, stride, 0, dtp));
    while (a < ppp && bb < dpp) {
        const int nab = (a1 < b1 ? a1 : b1) - (a0 > b0 ? a0 : b0);
        const double Vn = V1 * (double)nab;
        const uint8_t* Sa = pm + (a * ptp) * stride;
        const uint8_t* Sb = dm + (bb * dtp) * stride;
        int r = 0, q = 0;
        while (r < ptp && q < dtp) {
            const int re = (r + 1) * dtp, qe = (q + 1) * ptp;
            const int ov = (re < qe ? re : qe) - (r * dtp > q * ptp ? r * dtp : q * ptp);
            const int g = Sa[r * stride], h = Sb[q * stride];
            const double bytes = pow2 ? (Vn * (double)ov) * inv_den : (Vn * (double)ov) / den;
            const double time = p.alpha[g * p.G + h] + bytes / p.beta[g * p.G + h];
            if (time > worst) worst = time;
            if (re <= qe) ++r;
            if (qe <= re) ++q;
        }
        const bool adv_a = a1 <= b1, adv_b = b1 <= a1;
        if (adv_a && ++a < ppp) {
            a0 = a1;
            a1 = a0 + split_layers<true>(sp, a, stage_flops(gfl, pm, stride, a, ptp));
        }
        if (adv_b && ++bb < dpp) {
            b0 = b1;
            b1 = b0 + split_layers<true>(sd, bb, stage_flops(gfl, dm, stride, bb, dtp));
        }
    }
    return worst;
}

// With request classes (kCls) an edge's time is sum_k w_k t_k over the classes (t_k the time
// with s_in = cls_in[k], class order, left to right).
template <bool kCls, class TimeOf>
__device__ __forceinline__ double task_mix(const Problem& p, TimeOf time_of) {
    if (!kCls) return time_of(p);
    double t = 0.0;
    for (int k = 0; k < p.n_cls; ++k) {
        Problem pk = p;
        pk.s_in = p.cls_in[k];
        pk.s_out = p.cls_out[k];
        t = t + p.cls_w[k] * time_of(pk);
    }
    return t;
}

// Capacity of the KV edge from prefill node i to decode node j of candidate n (0 unless both
// replicas have a strategy).  pm, dm: the lane's two member columns in LDS, stride bytes apart.
template <int W, bool kAsym, bool kCls>
__device__ __forceinline__ int32_t kv_edge(const Problem& p, const CostOut& o, const FlowNet& f, const double* gfl,
                                           int i, int j, int64_t n, uint8_t* pm, uint8_t* dm, int stride) {
    const int64_t N = p.N;
    int32_t c = 0;
    const int kp = f.p_slot[(int64_t)i * N + n], kd = f.d_slot[(int64_t)j * N + n];
    // The member masks are loaded with the strategies (not after them), so the lane waits on
    // one memory round for both.
    uint64_t mp[W], md[W];
#pragma unroll
    for (int w = 0; w < W; ++w) {
        mp[w] = o.members[((int64_t)kp * W + w) * N + n];
        md[w] = o.members[((int64_t)kd * W + w) * N + n];
    }
    const int ptp = o.tp[(int64_t)kp * N + n], ppp = o.pp[(int64_t)kp * N + n];
    const int dtp = o.tp[(int64_t)kd * N + n], dpp = o.pp[(int64_t)kd * N + n];
    if (ptp > 0 && dtp > 0) {
        // A strategy whose tp*pp is not the group's size (cost outputs of another batch) is
        // treated as infeasible rather than read past the member list.
        if (expand_words<W>(mp, pm, stride) == ptp * ppp && expand_words<W>(md, dm, stride) == dtp * dpp)
            c = quantize(1000.0 / (kCls    ? kv_time_classes(p, pm, ptp, ppp, dm, dtp, dpp, stride)
                                   : kAsym ? kv_time_asym(p, gfl, pm, ptp, ppp, dm, dtp, dpp, stride)
                                           : kv_time(p, pm, ptp, ppp, dm, dtp, dpp, stride)));
    }
    return c;
}

template <int W, bool kAsym, bool kCls>
__global__ void __launch_bounds__(kKvBlock) kv_kernel(Problem p, CostOut o, FlowNet f) {
    extern __shared__ __attribute__((aligned(16))) uint8_t sm[];
    const int tid = threadIdx.x;
    const int stride = blockDim.x;
    const int64_t N = p.N;
    // asymmetric split: every GPU's FLOP/s staged once per workgroup (the walk's layer ranges
    // read them at every stage it enters)
    double* gfl = reinterpret_cast<double*>(sm + 2 * (size_t)p.G * stride);
    if (kAsym) {
        for (int g = tid; g < p.G; g += blockDim.x) gfl[g] = gpu_flops(p, g);
        __syncthreads();
    }
    // KV row e = blockIdx.y (a grid row per row, so no lane divides by N), candidates along x
    const int e = (int)blockIdx.y;
    const int n = (int)blockIdx.x * kKvBlock + tid;
    if (n >= N) return;
    const int np = f.n_p[n], nd = f.n_d[n];
    if (e >= np * nd) return;
    const int i = e / nd, j = e - i * nd;
    // member columns [G][blockDim] each
    f.kv_cap[(int64_t)e * N + n] = kv_edge<W, kAsym, kCls>(p, o, f, gfl, i, j, n, sm + tid, sm + p.G * stride + tid,
                                                           stride);
}

// The listed KV path, first kernel: a wavefront per piece (64 candidates, blockIdx.y the slice
// of their KV rows), a lane per candidate walking its rows of the slice below n_p n_d in order
// (row e of every lane at once, so the stores coalesce): 0 for an edge with an infeasible end
// (FlowNet::feas), the others listed in the piece's own part of the list (no atomics: a counter
// that every wavefront bumps serialises them).
constexpr int kRowsBlock = 256;

__global__ void __launch_bounds__(kRowsBlock) kv_rows_kernel(FlowNet f) {
    const int64_t N = f.N;
    const int64_t n0 = (int64_t)blockIdx.x * kRowsBlock + threadIdx.x;
    const int64_t seg = n0 >> 6;
    if (seg * 64 >= N) return;  // a wavefront wholly past N owns no piece
    const bool in = n0 < N;
    const int64_t n = in ? n0 : N - 1;  // every lane loads, lanes past N own no row
    const int np = f.n_p[n], nd = f.n_d[n];
    const uint64_t fz = f.feas[n];
    const int lane = threadIdx.x & 63;
    const int r0 = (int)blockIdx.y * f.kv_rows;
    const int pd = in ? np * nd : 0;
    const int hi = pd < r0 + f.kv_rows ? pd : r0 + f.kv_rows;  // this lane's rows: [r0, hi)
    int rows = hi;
    for (int off = 32; off > 0; off >>= 1) {
        const int o2 = __shfl_xor(rows, off, 64);
        rows = o2 > rows ? o2 : rows;
    }
    const int64_t piece = seg * kKvSlices + blockIdx.y;
    uint32_t* list = f.kv_list + piece * (int64_t)(64 * f.kv_rows);
    int i = 0, j = 0;
    if (r0 < hi) {
        i = r0 / nd;
        j = r0 - i * nd;
    }
    const uint32_t dm = (uint32_t)(fz >> 32);
    // The row advance is formed with selects (i <= n_p <= 32, so the shift stays below 64), so
    // that only the two stores are predicated.
    int cnt = 0;
    int32_t* row = f.kv_cap + (int64_t)r0 * N + n;
    for (int e = r0; e < rows; ++e, row += N) {
        const bool live = e < hi;
        const bool walk = live && ((((uint32_t)(fz >> i) & (dm >> j)) & 1) != 0);
        if (live && !walk) *row = 0;
        const uint64_t bal = __ballot(walk);
        if (bal) {
            if (walk)
                list[cnt + __popcll(bal & ((1ull << lane) - 1))] = ((uint32_t)n << 10) | ((uint32_t)i << 5) | (uint32_t)j;
            cnt += __popcll(bal);
        }
        const bool wrap = live && j + 1 == nd;
        i += wrap ? 1 : 0;
        j = wrap ? 0 : (live ? j + 1 : j);
    }
    if (lane == 0) f.kv_count[piece] = cnt;
}

// LDS written by some lanes of a wavefront and then read by others of the same wavefront.
__device__ __forceinline__ void lane_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The listed KV path's packing: one workgroup forms the exclusive prefix sums of the pieces'
// counts (kv_offs, the total last); each thread takes a contiguous run of pieces (a multiple of
// four: the piece count is one), sums it, the workgroup scans the 1024 sums, and the thread
// writes its run's offsets.  A run is read and written in 16-byte words, kScanChunk counts at a
// time with their loads issued together (the run's last word repeated past its end): one CU
// does all of it, so the number of memory requests, not bytes, sets the time.
constexpr int kScanBlock = 1024;
constexpr int kScanChunk = 16;

__global__ void __launch_bounds__(kScanBlock) kv_scan_kernel(FlowNet f) {
    __shared__ int32_t part[kScanBlock / 64];
    constexpr int kWords = kScanChunk / 4;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t P = (f.N + 63) / 64 * kKvSlices;  // a multiple of 4
    const int64_t run = (P + 4 * kScanBlock - 1) / (4 * kScanBlock) * 4;
    const int64_t lo = tid * run < P ? tid * run : P, hi = lo + run < P ? lo + run : P;
    const int4* cw = reinterpret_cast<const int4*>(f.kv_count);
    int4* ow = reinterpret_cast<int4*>(f.kv_offs);
    const int64_t wlo = lo / 4, whi = hi / 4;
    int32_t sum = 0;
    int4 v0[kWords];  // the last chunk read: the whole run when it fits in one
    for (int64_t c0 = wlo; c0 < whi; c0 += kWords) {
#pragma unroll
        for (int k = 0; k < kWords; ++k) v0[k] = cw[c0 + k < whi ? c0 + k : whi - 1];
#pragma unroll
        for (int k = 0; k < kWords; ++k)
            if (c0 + k < whi) sum += v0[k].x + v0[k].y + v0[k].z + v0[k].w;
    }
    int32_t x = sum;  // inclusive scan over the wavefront
    for (int off = 1; off < 64; off <<= 1) {
        const int32_t y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    if (lane == 63) part[wave] = x;
    __syncthreads();
    int32_t before = 0, total = 0;
    for (int w = 0; w < kScanBlock / 64; ++w) {
        const int32_t v = part[w];
        if (w < wave) before += v;
        total += v;
    }
    int32_t off = before + x - sum;
    if (whi - wlo <= kWords) {  // a run of one chunk: its counts are still in v0
#pragma unroll
        for (int k = 0; k < kWords; ++k)
            if (wlo + k < whi) {
                int4 o;
                o.x = off;
                o.y = o.x + v0[k].x;
                o.z = o.y + v0[k].y;
                o.w = o.z + v0[k].z;
                off = o.w + v0[k].w;
                ow[wlo + k] = o;
            }
    } else
    for (int64_t c0 = wlo; c0 < whi; c0 += kWords) {
        int4 v[kWords];
#pragma unroll
        for (int k = 0; k < kWords; ++k) v[k] = cw[c0 + k < whi ? c0 + k : whi - 1];
#pragma unroll
        for (int k = 0; k < kWords; ++k)
            if (c0 + k < whi) {
                int4 o;
                o.x = off;
                o.y = o.x + v[k].x;
                o.z = o.y + v[k].y;
                o.w = o.z + v[k].z;
                off = o.w + v[k].w;
                ow[c0 + k] = o;
            }
    }
    if (tid == 0) f.kv_offs[P] = total;
}

// Then a wavefront per piece copies its listed edges to kv_flat from its offset on.
__global__ void __launch_bounds__(256) kv_compact_kernel(FlowNet f) {
    const int64_t P = (f.N + 63) / 64 * kKvSlices;
    const int64_t s = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (s >= P) return;
    const int lane = threadIdx.x & 63;
    const uint32_t* list = f.kv_list + s * (int64_t)(64 * f.kv_rows);
    // the part's first 64 entries are loaded with its count and offset (a part has room for
    // 64 kv_rows >= 64 entries, so the load stays inside it; entries past the count are unused)
    const uint32_t first = list[lane];
    const int cnt = f.kv_count[s];
    const int32_t off = f.kv_offs[s];
    if (lane < cnt) f.kv_flat[off + lane] = first;
    for (int x = lane + 64; x < cnt; x += 64) f.kv_flat[off + x] = list[x];
}

// The listed KV path's walk: kWalkLanes lanes per listed edge.  An edge's links are every
// overlapping (stage, stage) pair crossed with every overlapping (rank, rank) pair, and the rank
// pairs (head slices of ptp x dtp) are the same for every stage pair, so lane l of the group
// takes the rank pairs l, l + kWalkLanes, ... of the merge walk (there are
// ptp + dtp - gcd(ptp, dtp) <= 15 of them, at most 8 when both degrees are powers of two) and
// walks the stage pairs (at most ppp + dpp - 1) with them; the group's maximum is the edge's KV
// time (with kCls one maximum per request class, then sum_k w_k max_k in class order).  Each
// link's time is the binary64 value kv_time or kv_time_classes forms, and a maximum does not
// depend on the order.  (The asymmetric split stays with kv_kernel: every lane of a group would
// recompute the stages' layer counts, which measured twice as slow.)  The group's lanes expand
// the two member masks together (64 / kWalkLanes bits of each word a lane) into the group's two
// member columns in LDS.  The edges come from the packed list, kGroups per wavefront at a time,
// over a grid of kGroupGrid workgroups (about twice what the chip holds at once, so that
// workgroups that finish early are replaced): the walks run side by side, each starting with a
// chain of dependent loads (its list entry, slots, then masks and strategies).  Alpha and beta are read from memory: staging them in LDS per workgroup measured
// slower.
constexpr int kWalkLanes = 4;
constexpr int kGroupBlock = 256;
constexpr int kGroupGrid = 4096;

__host__ __device__ inline size_t kv_group_lds(int G) { return (size_t)kGroupBlock / kWalkLanes * 2 * G; }

template <int W>
__device__ __forceinline__ int expand_group(const uint64_t* m, uint8_t* col, int sub) {
    constexpr int kBits = 64 / kWalkLanes;
    int below = 0, total = 0;
#pragma unroll
    for (int w = 0; w < W; ++w) total += __popcll(m[w]);
#pragma unroll
    for (int w = 0; w < W; ++w) {
        const int b0 = sub * kBits;
        const uint64_t mine = (m[w] >> b0) & ((1ull << kBits) - 1);
        int idx = below + __popcll(m[w] & ((1ull << b0) - 1));
#pragma unroll
        for (int t = 0; t < kBits; ++t)
            if ((mine >> t) & 1) col[idx++] = (uint8_t)(w * 64 + b0 + t);
        below += __popcll(m[w]);
    }
    return total;
}

template <int W, bool kCls>
__global__ void __launch_bounds__(kGroupBlock) kv_walk_group_kernel(Problem p, CostOut o, FlowNet f) {
    constexpr int kGroups = 64 / kWalkLanes, kWaves = kGroupBlock / 64;
    constexpr int kC = kCls ? HX_MAX_CLASSES : 1;
    static_assert(64 % kWalkLanes == 0 && kWalkLanes <= 64, "lanes of a group split each mask word");
    constexpr int kPairs = (2 * HX_MAX_TP - 1 + kWalkLanes - 1) / kWalkLanes;  // rank pairs a lane
    extern __shared__ __attribute__((aligned(16))) uint8_t sm[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int grp = lane / kWalkLanes, sub = lane % kWalkLanes;
    const int G = p.G;
    const int64_t N = p.N;
    uint8_t* colp = sm + (size_t)(wave * kGroups + grp) * 2 * G;  // [G] prefill member ids
    uint8_t* cold = colp + G;                                     // [G] decode member ids
    const int nc = kCls ? p.n_cls : 1;
    double V1[kC];
#pragma unroll
    for (int k = 0; k < kC; ++k) V1[k] = 2.0 * (kCls ? p.cls_in[k] : p.s_in) * p.Hkv * p.B;
    const int64_t total = f.kv_offs[(N + 63) / 64 * kKvSlices];
    for (int64_t w = (int64_t)blockIdx.x * kWaves + wave; w * kGroups < total; w += (int64_t)gridDim.x * kWaves) {
        const int64_t x = w * kGroups + grp;
        const bool live = x < total;
        const uint32_t v = f.kv_flat[live ? x : w * kGroups];
        const int64_t n = v >> 10;
        const int i = (v >> 5) & 31, j = v & 31;
        const int nd = f.n_d[n];
        const int kp = f.p_slot[(int64_t)i * N + n], kd = f.d_slot[(int64_t)j * N + n];
        uint64_t mp[W], md[W];
#pragma unroll
        for (int ww = 0; ww < W; ++ww) {
            mp[ww] = o.members[((int64_t)kp * W + ww) * N + n];
            md[ww] = o.members[((int64_t)kd * W + ww) * N + n];
        }
        const int ptp = o.tp[(int64_t)kp * N + n], ppp = o.pp[(int64_t)kp * N + n];
        const int dtp = o.tp[(int64_t)kd * N + n], dpp = o.pp[(int64_t)kd * N + n];
        const int cp = expand_group<W>(mp, colp, sub), cd = expand_group<W>(md, cold, sub);
        lane_sync();
        // A strategy whose tp*pp is not the group's size (cost outputs of another batch) is
        // treated as infeasible rather than read past the member list.
        const bool ok = live && ptp > 0 && dtp > 0 && cp == ptp * ppp && cd == dtp * dpp;
        double worst[kC];
#pragma unroll
        for (int k = 0; k < kC; ++k) worst[k] = 0.0;
        if (ok) {
            // this lane's rank pairs: steps sub, sub + kWalkLanes, ... of the merge of the two
            // head partitions (rl < 0: none)
            int rl[kPairs], ql[kPairs], ovl[kPairs];
#pragma unroll
            for (int h = 0; h < kPairs; ++h) {
                rl[h] = -1;
                ql[h] = 0;
                ovl[h] = 0;
            }
            {
                int r = 0, q = 0;
                for (int t = 0; t < kPairs * kWalkLanes && r < ptp && q < dtp; ++t) {
                    const int re = (r + 1) * dtp, qe = (q + 1) * ptp;
                    const int ov = (re < qe ? re : qe) - (r * dtp > q * ptp ? r * dtp : q * ptp);
#pragma unroll
                    for (int h = 0; h < kPairs; ++h)
                        if (t == sub + h * kWalkLanes) {
                            rl[h] = r;
                            ql[h] = q;
                            ovl[h] = ov;
                        }
                    if (re <= qe) ++r;
                    if (qe <= re) ++q;
                }
            }
            const int deni = ptp * dtp;
            const double den = (double)deni;
            const bool pow2 = (deni & (deni - 1)) == 0;
            const double inv_den = 1.0 / den;
            const int lqp = p.L / ppp, lrp = p.L % ppp, lqd = p.L / dpp, lrd = p.L % dpp;
            int a = 0, bb = 0, a0 = 0, b0 = 0;
            int a1 = lqp + (0 < lrp ? 1 : 0), b1 = lqd + (0 < lrd ? 1 : 0);
            while (a < ppp && bb < dpp) {
                const int nab = (a1 < b1 ? a1 : b1) - (a0 > b0 ? a0 : b0);
#pragma unroll
                for (int h = 0; h < kPairs; ++h) {
                    const int rr = rl[h], qq = ql[h], oo = ovl[h];
                    if (rr < 0) continue;
                    const int e = colp[a * ptp + rr] * G + cold[bb * dtp + qq];
                    const double al = p.alpha[e], be = p.beta[e];
#pragma unroll
                    for (int k = 0; k < kC; ++k) {
                        if (k >= nc) break;
                        const double Vn = V1[k] * (double)nab;
                        const double bytes = pow2 ? (Vn * (double)oo) * inv_den : (Vn * (double)oo) / den;
                        const double time = al + bytes / be;
                        if (time > worst[k]) worst[k] = time;
                    }
                }
                const bool adv_a = a1 <= b1, adv_b = b1 <= a1;
                if (adv_a) {
                    ++a;
                    a0 = a1;
                    a1 = a0 + lqp + (a < lrp ? 1 : 0);
                }
                if (adv_b) {
                    ++bb;
                    b0 = b1;
                    b1 = b0 + lqd + (bb < lrd ? 1 : 0);
                }
            }
        }
#pragma unroll
        for (int k = 0; k < kC; ++k)
#pragma unroll
            for (int off = kWalkLanes / 2; off > 0; off >>= 1) {
                const double w2 = __shfl_xor(worst[k], off, 64);
                worst[k] = w2 > worst[k] ? w2 : worst[k];
            }
        double t = worst[0];
        if (kCls) {
            t = 0.0;
#pragma unroll
            for (int k = 0; k < kC; ++k)
                if (k < nc) t = t + p.cls_w[k] * worst[k];
        }
        if (live && sub == 0) f.kv_cap[(int64_t)(i * nd + j) * N + n] = ok ? quantize(1000.0 / t) : 0;
        lane_sync();  // the next edge's expansion overwrites the columns
    }
}

// Per-GPU nodes: one workgroup of kGpuKvWaves wavefronts per 64 candidates (a lane per
// candidate in every wavefront).  Every edge of the per-GPU network counts requests (a GPU node
// carries its share of its replica's requests), so the edge from prefill GPU g to decode GPU h
// carries one request's whole KV cache, V1 L bytes, over the link g -> h: its capacity depends
// only on g and h, and is 0 unless both replicas are feasible.  With kTable (G <= 128) the
// workgroup first tabulates the capacity of every link in LDS ([G][G] int32, at most 64 KB: two
// divisions per link, a few per lane, instead of two per edge); then it stages, per candidate,
// every GPU's feasibility ([G][64] bytes: 1 when its replica kept a strategy) and the node lists'
// GPU ids; then each wavefront takes every kGpuKvWaves-th edge row (coalesced stores across the
// 64 candidates), each edge a table lookup (or, without the table, its two divisions).  One
// lane per (edge, candidate) would repeat the lookups of both endpoints for every edge.
constexpr int kGpuKvWaves = 4;
constexpr int kGpuKvWavesTable = 16;  // the table leaves one workgroup per CU: more wavefronts
constexpr int kGpuTableMaxG = 128;

// Node rows staged per side: a side has at most G per-GPU nodes.
__host__ __device__ inline int kv_gpu_rows(int G, int max_rows) { return max_rows < G ? max_rows : G; }

__host__ __device__ inline size_t kv_gpu_lds(int G, int max_p, int max_d, bool table) {
    return (table ? sizeof(int32_t) * (size_t)G * G : 0) +
           ((size_t)G + (size_t)kv_gpu_rows(G, max_p) + (size_t)kv_gpu_rows(G, max_d)) * 64;
}

// Capacity of the per-GPU KV edge over the link g -> h: one request's whole KV cache (V1 L
// bytes; with request classes the mix's mean time).
template <bool kCls>
__device__ __forceinline__ int32_t kv_gpu_cap(const Problem& p, const double* vl, int g, int h) {
    const double al = p.alpha[g * p.G + h], be = p.beta[g * p.G + h];
    double t;
    if (kCls) {
        t = 0.0;
        for (int k = 0; k < p.n_cls; ++k) t = t + p.cls_w[k] * (al + vl[k] / be);
    } else {
        t = al + vl[0] / be;
    }
    return quantize(1000.0 / t);
}

template <int W, bool kCls, bool kTable>
__global__ void __launch_bounds__(64 * (kTable ? kGpuKvWavesTable : kGpuKvWaves))
    kv_gpu_kernel(Problem p, CostOut o, FlowNet f) {
    constexpr int kWaves = kTable ? kGpuKvWavesTable : kGpuKvWaves;
    extern __shared__ __attribute__((aligned(16))) unsigned char sm[];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t N = p.N;
    const int64_t n = (int64_t)blockIdx.x * 64 + lane;
    const bool in = n < N;
    const int G = p.G;
    int32_t* tab = reinterpret_cast<int32_t*>(sm);                    // [G][G] (kTable)
    uint8_t* ok = sm + (kTable ? sizeof(int32_t) * (size_t)G * G : 0);  // [G][64]: 1 if the GPU's
                                                                      // replica is feasible
    uint8_t* ps = ok + (size_t)G * 64;         // [prow][64]: prefill node -> GPU
    const int prow = kv_gpu_rows(G, f.max_p), drow = kv_gpu_rows(G, f.max_d);
    uint8_t* ds = ps + (size_t)prow * 64;      // [drow][64]: decode node -> GPU
    const int np = in ? f.n_p[n] : 0, nd = in ? f.n_d[n] : 0;
    // one request's KV cache for all L layers, per task
    double vl[HX_MAX_CLASSES];
#pragma unroll
    for (int k = 0; k < HX_MAX_CLASSES; ++k)
        vl[k] = (2.0 * (kCls ? p.cls_in[k] : p.s_in) * p.Hkv * p.B) * (double)p.L;
    if (kTable)
        for (int x = threadIdx.x; x < G * G; x += 64 * kWaves) {
            const int g = x / G, h = x - g * G;
            tab[x] = g == h ? 0 : kv_gpu_cap<kCls>(p, vl, g, h);
        }
    for (int g = wave; g < G; g += kWaves) {
        uint8_t d = 0;
        if (in) {
            const int k = p.assign[(int64_t)g * N + n];
            if (k < p.Kmax && o.tp[(int64_t)k * N + n] > 0) d = 1;
        }
        ok[g * 64 + lane] = d;
    }
    for (int i = wave; i < prow; i += kWaves)
        ps[i * 64 + lane] = i < np ? (uint8_t)f.p_slot[(int64_t)i * N + n] : 0;
    for (int j = wave; j < drow; j += kWaves)
        ds[j * 64 + lane] = j < nd ? (uint8_t)f.d_slot[(int64_t)j * N + n] : 0;
    __syncthreads();
    const int E = np * nd;
    int emax = E;
    for (int off = 32; off > 0; off >>= 1) {
        const int v = __shfl_xor(emax, off, 64);
        emax = v > emax ? v : emax;
    }
    // edge e = i * nd + j of this lane's candidate, rows wave, wave + kWaves, ...
    int i = 0, j = wave;
    while (nd > 0 && j >= nd) {
        j -= nd;
        ++i;
    }
    for (int e = wave; e < emax; e += kWaves) {
        if (e < E) {
            const int g = ps[i * 64 + lane], h = ds[j * 64 + lane];
            int32_t c = 0;
            if (ok[g * 64 + lane] && ok[h * 64 + lane]) c = kTable ? tab[g * G + h] : kv_gpu_cap<kCls>(p, vl, g, h);
            f.kv_cap[(int64_t)e * N + n] = c;
            j += kWaves;
            while (j >= nd) {
                j -= nd;
                ++i;
            }
        }
    }
}

template <int W, bool kCls, bool kTable>
hipError_t launch_kv_gpu(const Problem& p, const FlowNet& f, const CostOut& o, hipStream_t s) {
    constexpr int waves = kTable ? kGpuKvWavesTable : kGpuKvWaves;
    const size_t lds = kv_gpu_lds(p.G, f.max_p, f.max_d, kTable);
    if (lds > 64 * 1024) {  // gfx950 gives a workgroup up to 160 KB once the limit is raised
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kv_gpu_kernel<W, kCls, kTable>),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL((kv_gpu_kernel<W, kCls, kTable>), dim3((p.N + 63) / 64), dim3(64 * waves), lds, s, p, o, f);
    return hipSuccess;
}

// The capacity of every per-GPU KV link (kv_gpu_cap) and each GPU's smallest one, for
// hx_score_batch: a workgroup per GPU row, its minimum by a workgroup reduction; also clears the
// count of the candidates left to the max-flow.
constexpr int kLinkBlock = 256;

template <bool kCls>
__global__ void __launch_bounds__(kLinkBlock) link_table_kernel(Problem p, int32_t* tab, int32_t* rmin,
                                                                int32_t* list_count) {
    __shared__ int32_t red[kLinkBlock / 64];
    const int g = blockIdx.x, G = p.G;
    if (g == 0 && threadIdx.x == 0) *list_count = 0;
    double vl[HX_MAX_CLASSES];
#pragma unroll
    for (int k = 0; k < HX_MAX_CLASSES; ++k)
        vl[k] = (2.0 * (kCls ? p.cls_in[k] : p.s_in) * p.Hkv * p.B) * (double)p.L;
    int32_t m = HX_CAP_MAX;
    for (int h = threadIdx.x; h < G; h += kLinkBlock) {
        const int32_t c = g == h ? 0 : kv_gpu_cap<kCls>(p, vl, g, h);
        tab[(int64_t)g * G + h] = c;
        if (h != g && c < m) m = c;
    }
    for (int off = 32; off > 0; off >>= 1) {
        const int32_t o2 = __shfl_xor(m, off, 64);
        m = o2 < m ? o2 : m;
    }
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kLinkBlock / 64; ++w) m = red[w] < m ? red[w] : m;
        rmin[g] = m;
    }
}

template <int W>
hipError_t launch_w(const Problem& p, const CostOut& o, const FlowNet& f, hipStream_t s) {
    prof_mark(kKNodes, false, s);
    launch_nodes<W>(p, o, f, s);
    prof_mark(kKNodes, true, s);
    const int64_t lanes = (int64_t)f.max_pd * p.N;
    const int blocks = (int)((lanes + kKvBlock - 1) / kKvBlock);
    // kv_kernel: a grid row per KV row a replica network can have (its n_p + n_d <= Kmax nodes
    // give at most floor(Kmax/2) ceil(Kmax/2) <= 16,256 rows, within the grid's y limit)
    const int64_t rows_pd = (int64_t)(p.Kmax / 2) * ((p.Kmax + 1) / 2);
    const dim3 grid_kv((unsigned)((p.N + kKvBlock - 1) / kKvBlock),
                       (unsigned)(f.max_pd < rows_pd ? f.max_pd : rows_pd));
    const size_t lds = 2 * (size_t)p.G * kKvBlock;
    prof_mark(kKKv, false, s);
    if (p.granularity != 0) {
        const bool table = p.G <= kGpuTableMaxG;
        hipError_t e;
        if (p.n_cls > 0)
            e = table ? launch_kv_gpu<W, true, true>(p, f, o, s) : launch_kv_gpu<W, true, false>(p, f, o, s);
        else
            e = table ? launch_kv_gpu<W, false, true>(p, f, o, s) : launch_kv_gpu<W, false, false>(p, f, o, s);
        if (e != hipSuccess) return e;
    } else if (p.variant & HX_VARIANT_KV_ORDER) {
        hipLaunchKernelGGL(kv_order_kernel<W>, dim3(blocks), dim3(kOrderThreads), kOrderLds + lds, s, p, o, f);
    } else if (f.kv_list && !(p.variant & HX_VARIANT_ASYM)) {
        // the listed path: zero rows and the edge list, its packing, then the walks
        const int64_t pieces = (p.N + 63) / 64 * kKvSlices;
        hipLaunchKernelGGL(kv_rows_kernel, dim3((unsigned)((p.N + kRowsBlock - 1) / kRowsBlock), kKvSlices),
                           dim3(kRowsBlock), 0, s, f);
        hipLaunchKernelGGL(kv_scan_kernel, dim3(1), dim3(kScanBlock), 0, s, f);
        hipLaunchKernelGGL(kv_compact_kernel, dim3((unsigned)((pieces + 3) / 4)), dim3(256), 0, s, f);
        const size_t gl = kv_group_lds(p.G);
        if (p.n_cls > 0)
            hipLaunchKernelGGL((kv_walk_group_kernel<W, true>), dim3(kGroupGrid), dim3(kGroupBlock), gl, s, p, o, f);
        else
            hipLaunchKernelGGL((kv_walk_group_kernel<W, false>), dim3(kGroupGrid), dim3(kGroupBlock), gl, s, p, o, f);
    } else if (p.variant & HX_VARIANT_ASYM) {
        hipLaunchKernelGGL((kv_kernel<W, true, false>), grid_kv, dim3(kKvBlock), lds + sizeof(double) * p.G, s, p,
                           o, f);
    } else if (p.n_cls > 0) {
        hipLaunchKernelGGL((kv_kernel<W, false, true>), grid_kv, dim3(kKvBlock), lds, s, p, o, f);
    } else {
        hipLaunchKernelGGL((kv_kernel<W, false, false>), grid_kv, dim3(kKvBlock), lds, s, p, o, f);
    }
    prof_mark(kKKv, true, s);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_flownet(const Problem& p, const CostOut& o, const FlowNet& f, hipStream_t s) {
    switch (mask_words(p.G)) {
        case 1: return launch_w<1>(p, o, f, s);
        case 2: return launch_w<2>(p, o, f, s);
        default: return launch_w<4>(p, o, f, s);
    }
}

}  // namespace hx

namespace hx {

bool flownet_values_direct(const Problem& p) {
    return p.granularity == 1 && p.G <= kGpuTableMaxG && p.Kmax <= kNodesGpuMaxK;
}

// Layout: int32 tab [G][G], rmin [G]; then, 256-byte aligned, the list count and the list [N].
static size_t list_offset(int32_t n_gpus) {
    return (sizeof(int32_t) * ((size_t)n_gpus * n_gpus + n_gpus) + 255) & ~(size_t)255;
}

size_t link_table_bytes(int32_t n_gpus, int32_t n_cand) {
    return list_offset(n_gpus) + sizeof(int32_t) * (16 + (size_t)n_cand);
}

int32_t* flownet_values_list_count(void* table, int32_t n_gpus) {
    return reinterpret_cast<int32_t*>(static_cast<unsigned char*>(table) + list_offset(n_gpus));
}

hipError_t launch_flownet_values(const Problem& p, const CostOut& o, const FlowNet& f, int32_t* flow_value,
                                 void* table, hipStream_t s) {
    int32_t* tab = static_cast<int32_t*>(table);
    int32_t* rmin = tab + (size_t)p.G * p.G;
    int32_t* list_count = reinterpret_cast<int32_t*>(static_cast<unsigned char*>(table) + list_offset(p.G));
    int32_t* list = list_count + 16;
    prof_mark(kKKv, false, s);
    if (p.n_cls > 0)
        hipLaunchKernelGGL(link_table_kernel<true>, dim3(p.G), dim3(kLinkBlock), 0, s, p, tab, rmin, list_count);
    else
        hipLaunchKernelGGL(link_table_kernel<false>, dim3(p.G), dim3(kLinkBlock), 0, s, p, tab, rmin, list_count);
    prof_mark(kKKv, true, s);
    prof_mark(kKNodes, false, s);
    if (mask_words(p.G) == 1)
        hipLaunchKernelGGL((nodes_gpu_kernel<1, true>), dim3((p.N + 63) / 64), dim3(64), nodes_gpu_lds(p.Kmax), s, p,
                           o, f, tab, rmin, flow_value, list, list_count);
    else
        hipLaunchKernelGGL((nodes_gpu_kernel<2, true>), dim3((p.N + 63) / 64), dim3(64), nodes_gpu_lds(p.Kmax), s, p,
                           o, f, tab, rmin, flow_value, list, list_count);
    prof_mark(kKNodes, true, s);
    return hipGetLastError();
}

}  // namespace hx
