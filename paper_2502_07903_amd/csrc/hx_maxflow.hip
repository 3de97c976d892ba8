// hx_maxflow.hip -- maximum flow of every candidate's network (Sec. 3.3) on gfx950.
//
// The paper solves each network with preflow-push.  Here a segment of SEG lanes owns one
// candidate and runs a synchronous push-relabel with the candidate's whole residual graph
// in LDS, one lane per node.  Small networks (SEG <= 64, e.g. <= 16 replicas per side) pack
// 64/SEG candidates into one wavefront, so a wave's rounds serve several candidates at
// once; larger networks (per-GPU nodes) take a workgroup of SEG = 128 or 256 lanes each.
//
// Network.  In the Sec. 3.3 network every replica is an in -> out chain with one edge in
// and the KV edges out (prefill) or the KV edges in and one edge out (decode), so the
// chains contract without changing any s-t cut: prefill node p gets a_p = min(src, p_cap)
// from the source, decode node d sends b_d = min(d_cap, sink) to the sink, and c_pd are the
// KV edges.  The contracted graph is bipartite: s -> P -> D -> t.
//
// Algorithm (Goldberg-Tarjan push-relabel, in synchronous rounds).  The source sits at
// height V = P + D + 2, the sink at 0.  A round has two phases separated by barriers:
//   P-phase: each active prefill node pushes along its admissible arcs (to decode nodes one
//            level lower, then back to the source), then relabels if excess remains;
//   D-phase: each active decode node pushes to the sink and back along its reverse KV arcs,
//            then relabels if excess remains.
// Within a phase the active nodes lie on one side of the bipartition, so their pushes touch
// disjoint arcs and their relabels read only the other side's heights, which that phase never
// changes: the phase equals some sequential order of the same push/relabel operations, and
// the usual termination and optimality arguments apply.  Excess arriving at the other side
// is added with LDS atomics.  Exact heights (BFS distances to the sink, else V + distance to
// the source) are recomputed every few rounds by label-correcting sweeps (global relabel).
// A candidate is done when none of its nodes has excess: the preflow is then a maximum flow.
//
// Shortcuts.  Nodes that can carry nothing (a = 0 or b = 0) leave most networks trivial.
// Single-wavefront plans: if one side has a single node that can, the network is a star and
// its maximum flow has a closed form (with a flow that fills the star's arcs in node order).
// Every plan: if every KV arc can carry min(a_i, b_j), the maximum flow is min(sum a, sum b)
// with the north-west-corner flow (below).  Single-wavefront plans, value only: if the
// smaller side has m <= kEnumMax nodes that can carry flow, the minimum cut is taken over the
// 2^m ways to split that side.  Push-relabel runs for the rest; every path gives the unique
// maximum-flow value.
//
// Outputs: the flow value, the flow on every KV edge, and the canonical minimum cut (nodes of
// the uncontracted network reachable from the source in the residual graph).
#include <limits.h>

#include "hx_internal.h"

namespace hx {
namespace {

constexpr int kGlobalRelabelEvery = 2;  // rounds between exact relabels
// Largest smaller side whose 2^m minimum-cut subsets are enumerated when only the flow value
// is wanted (64 subsets over a candidate's lanes).
constexpr int kEnumMax = 6;
constexpr int kPackedLanes = 64;  // workgroup size for packed segments: one wavefront

struct MfLayout {
    int32_t* cap;   // [P][Ds] KV capacities, row stride Ds = D | 1 (odd: no bank conflicts)
    int32_t* fl;    // [P][Ds] KV flows
    int32_t* a;     // [P] source -> p capacity
    int32_t* fs;    // [P] source -> p flow
    int32_t* ep;    // [P] excess
    int32_t* hp;    // [P] height
    int32_t* b;     // [D] d -> sink capacity
    int32_t* ft;    // [D] d -> sink flow
    int32_t* ed;    // [D] excess
    int32_t* hd;    // [D] height
    int32_t* misc;  // [4] scalars
};

__host__ __device__ inline size_t mf_words(int max_p, int max_d, int max_pd) {
    return 2 * ((size_t)max_pd + max_p) + 4 * (size_t)max_p + 4 * (size_t)max_d + 4;
}

__device__ inline MfLayout carve(int32_t* sm, int max_p, int max_d, int max_pd) {
    MfLayout L;
    const int arc = max_pd + max_p;  // P*(D|1) <= P*D + P
    L.cap = sm;
    L.fl = L.cap + arc;
    L.a = L.fl + arc;
    L.fs = L.a + max_p;
    L.ep = L.fs + max_p;
    L.hp = L.ep + max_p;
    L.b = L.hp + max_p;
    L.ft = L.b + max_d;
    L.ed = L.ft + max_d;
    L.hd = L.ed + max_d;
    L.misc = L.hd + max_d;
    return L;
}

// Exact heights by label-correcting sweeps: hd = 1 where d -> t has residual, hp = V + 1 where
// p -> s has residual (reverse of a used source edge), then relax along residual arcs.  Every
// lane of the workgroup calls it (barriers inside); lane l of a segment owns node l, l+SEG, ...
template <int SEG>
__device__ void global_relabel(const MfLayout& L, int l, int P, int D, int Ds, int V, int INF) {
    for (int i = l; i < P; i += SEG) L.hp[i] = L.fs[i] > 0 ? V + 1 : INF;
    for (int j = l; j < D; j += SEG) L.hd[j] = L.b[j] - L.ft[j] > 0 ? 1 : INF;
    __syncthreads();
    for (;;) {
        bool changed = false;
        for (int i = l; i < P; i += SEG) {
            int h = L.hp[i];
            const int32_t* c = L.cap + i * Ds;
            const int32_t* f = L.fl + i * Ds;
            for (int d = 0; d < D; ++d)
                if (c[d] - f[d] > 0 && L.hd[d] + 1 < h) h = L.hd[d] + 1;
            if (h < L.hp[i]) {
                L.hp[i] = h;
                changed = true;
            }
        }
        __syncthreads();
        for (int j = l; j < D; j += SEG) {
            int h = L.hd[j];
            for (int q = 0; q < P; ++q)
                if (L.fl[q * Ds + j] > 0 && L.hp[q] + 1 < h) h = L.hp[q] + 1;
            if (h < L.hd[j]) {
                L.hd[j] = h;
                changed = true;
            }
        }
        if (!__syncthreads_or(changed)) break;
    }
}

// Dominant KV arcs.  When c_ij >= min(a_i, b_j) on every KV arc, no cut is below
// U = min(sum a, sum b): a cut keeping prefill set A on the source side costs
// sum_{i not in A} a_i + sum_j min(b_j, sum_{i in A} c_ij) >= sum_{i not in A} a_i +
// sum_j min(b_j, S) with S = sum_{i in A} a_i (each term: some a_i >= b_j gives b_j, else
// c_ij >= a_i for all of A), which is >= sum b when S >= every b_j and >= sum a otherwise.
// The maximum flow is then U, and the north-west-corner fill is one: with prefix sums A_i of a
// and B_j of b clamped to U, arc (i, j) carries the overlap of [A_{i-1}, A_i) and
// [B_{j-1}, B_j), at most min(a_i, b_j) <= c_ij; node i sends A_i - A_{i-1}, node j receives
// B_j - B_{j-1}.
__device__ __forceinline__ int32_t nw_overlap(int32_t ae, int32_t ai, int32_t be, int32_t bi) {
    const int32_t hi = ai < bi ? ai : bi, lo = ae > be ? ae : be;
    return hi > lo ? hi - lo : 0;
}

// Value-only pre-pass of the workgroup plans.  Those plans give a workgroup one candidate,
// whose KV rows then sit in as many cache lines as it has arcs; here lanes run over candidates
// (candidate-fastest, so every row load coalesces across the wavefront) in two kernels:
//   bound_kernel  one lane per candidate: writes min(sum a, sum b) as the candidate's flow
//                 value, 0 when no source-side or no sink-side node can carry flow, and -1 for
//                 networks with negative capacities or counts outside the plan;
//   dom_kernel    the dominant-KV condition c_ij >= min(a_i, b_j) on every arc, the arcs of a
//                 candidate split over kDomParts wavefronts (a long serial walk per candidate
//                 would leave the kernel waiting on one memory round per few arcs): an arc
//                 that fails it sets the flow value to -1.  It only ever writes -1, so the
//                 order of its writes does not matter.  c_ij >= a_i already implies the
//                 condition, so b_j is loaded only for arcs below a_i.
// maxflow_kernel then solves only the candidates left at -1.
constexpr int kBoundBlock = 256;
constexpr int kDomParts = 32;
constexpr int kDomUnroll = 8;

__device__ __forceinline__ bool plan_ok(const FlowNet& f, int P, int D) {
    return P >= 0 && D >= 0 && P <= f.max_p && D <= f.max_d && P * D <= f.max_pd;
}

__global__ void __launch_bounds__(kBoundBlock) bound_kernel(FlowNet f, int32_t* flow_value) {
    const int n = blockIdx.x * kBoundBlock + threadIdx.x;
    if (n >= f.N) return;
    const int64_t N = f.N;
    const int P = f.n_p[n], D = f.n_d[n];
    int32_t out = -1;
    if (plan_ok(f, P, D)) {
        long long sa = 0, sb = 0;
        bool neg = false, any_a = false, any_b = false;
        for (int i = 0; i < P; ++i) {
            const int32_t s = f.src_cap[(int64_t)i * N + n], c = f.p_cap[(int64_t)i * N + n];
            const int32_t a = s < c ? s : c;
            sa += a;
            neg |= a < 0;
            any_a |= a > 0;
        }
        for (int j = 0; j < D; ++j) {
            const int32_t c = f.d_cap[(int64_t)j * N + n], t = f.sink_cap[(int64_t)j * N + n];
            const int32_t b = c < t ? c : t;
            sb += b;
            neg |= b < 0;
            any_b |= b > 0;
        }
        if (!neg) out = (!any_a || !any_b) ? 0 : (int32_t)(sa < sb ? sa : sb);
    }
    flow_value[n] = out;
}

// Wavefront (part k, candidate chunk): arcs e in [k R, (k + 1) R) of each lane's candidate,
// R = ceil(max_pd / kDomParts), in ascending e (prefill node i = e / D, decode node j = e mod D).
__global__ void __launch_bounds__(64) dom_kernel(FlowNet f, int32_t* flow_value) {
    const int64_t N = f.N;
    // part-major: consecutive wavefronts take neighbouring candidate chunks of the same rows
    const int chunks = (int)((N + 63) / 64);
    const int part = blockIdx.x / chunks;
    const int64_t n = (int64_t)(blockIdx.x - part * chunks) * 64 + threadIdx.x;
    if (n >= N) return;
    if (flow_value[n] <= 0) return;  // -1: left to maxflow_kernel; 0: no flow either way
    const int P = f.n_p[n], D = f.n_d[n];
    const int R = (f.max_pd + kDomParts - 1) / kDomParts;
    const int E = P * D;
    const int lo = part * R, hi = lo + R < E ? lo + R : E;
    if (lo >= hi) return;
    auto a_of = [&](int i) {
        const int32_t s = f.src_cap[(int64_t)i * N + n], c = f.p_cap[(int64_t)i * N + n];
        return s < c ? s : c;
    };
    auto b_of = [&](int j) {
        const int32_t c = f.d_cap[(int64_t)j * N + n], t = f.sink_cap[(int64_t)j * N + n];
        return c < t ? c : t;
    };
    int i = lo / D, j = lo - i * D;
    int32_t ai = a_of(i);
    bool dom = true;
    for (int e0 = lo; e0 < hi && dom; e0 += kDomUnroll) {
        int32_t c[kDomUnroll];
#pragma unroll
        for (int x = 0; x < kDomUnroll; ++x) c[x] = e0 + x < hi ? f.kv_cap[(int64_t)(e0 + x) * N + n] : INT_MAX;
#pragma unroll
        for (int x = 0; x < kDomUnroll; ++x) {
            if (e0 + x < hi) {
                if (c[x] < ai) {
                    const int32_t bj = b_of(j);
                    dom = dom && c[x] >= (ai < bj ? ai : bj);
                }
                if (++j == D) {
                    j = 0;
                    if (++i < P && e0 + x + 1 < hi) ai = a_of(i);
                }
            }
        }
    }
    if (!dom) flow_value[n] = -1;
}

// SEG lanes per candidate; the workgroup holds max(64, SEG) lanes, i.e. 64/SEG candidates
// when SEG <= 64.  Workgroups are ordered XCD-aware: the hardware deals consecutive
// workgroups to the 8 XCDs in turn, so workgroup w takes tile (w mod 8) * chunk + w / 8 and
// each XCD walks a contiguous candidate range, sharing the L2 lines of the candidate-fastest
// input arrays.
// kStats: the diagnostic instantiation behind hx_maxflow_stats, which also counts into stats
// (HX_MF_STATS words, see hx.h) which path each candidate took and the push-relabel work; the
// production instantiation compiles none of it.
// The work of one tile (64/SEG candidates of a packed plan, or one candidate of a workgroup
// plan); every lane of the workgroup calls it with the same tile.
// kArg: fold the best of each wavefront's candidates (lane 0 of a segment holds its candidate's
// key, argmax_key) into slot blockIdx mod kArgSlots of arg with a 64-bit atomic max; every lane of
// the wavefront calls it.
__device__ __forceinline__ void fold_argmax(unsigned long long key, unsigned long long* arg) {
    for (int off = 32; off > 0; off >>= 1) {
        const unsigned long long o = __shfl_xor(key, off, 64);
        key = o > key ? o : key;
    }
    if ((threadIdx.x & 63) == 0 && key != 0) atomicMax(&arg[blockIdx.x % kArgSlots], key);
}

template <int SEG, bool kStats, bool kArg = false>
__device__ __forceinline__ void maxflow_tile(const FlowNet& f, int32_t* flow_value, int32_t* kv_flow, uint8_t* cut,
                                             int32_t round_budget, unsigned long long* stats, int tile,
                                             unsigned long long* arg = nullptr) {
    constexpr int kLanes = SEG < 64 ? kPackedLanes : SEG;
    constexpr int kPer = kLanes / SEG;
    const int N = f.N;
    const int tiles = (N + kPer - 1) / kPer;
    const int seg = threadIdx.x / SEG, l = threadIdx.x % SEG;
    const int n = tile * kPer + seg;

    extern __shared__ int32_t smem[];
    const MfLayout L = carve(smem + seg * mf_words(f.max_p, f.max_d, f.max_pd), f.max_p, f.max_d, f.max_pd);
    bool valid = tile < tiles && n < N;
    // value-only workgroup plans: bound_kernel has already written the candidates it could
    // (one candidate per workgroup, so the exit is uniform)
    if (SEG > 64 && kv_flow == nullptr && cut == nullptr && valid) {
        const int32_t pre = flow_value[n];
        if (pre >= 0) {
            if (kStats && l == 0) atomicAdd(&stats[HX_MF_PREPASS], 1ull);
            if (kArg) fold_argmax(l == 0 ? argmax_key(pre, n) : 0ull, arg);
            return;
        }
    }
    // kArg: a candidate in range that the checks below reject (HX_EINVAL) ends with valid false
    const bool in_range = valid;

    // Packed segments (SEG <= 64) own at most one node row per side and SEG/4 KV rows per
    // lane, so every global load is issued at once, before the counts that say which rows
    // are used have arrived: one memory round trip instead of three.  Unused rows are read
    // from the caller's [max][N] arrays and ignored.
    constexpr int kKvRows = SEG <= 64 ? (SEG / 4 > 0 ? SEG / 4 : 1) : 1;
    int32_t src0 = 0, pc0 = 0, dc0 = 0, sk0 = 0;
    int32_t kvr[kKvRows];
    int P = 0, D = 0;
    if (valid) {
        P = f.n_p[n];
        D = f.n_d[n];
        if (SEG <= 64) {
            if (l < f.max_p) {
                src0 = f.src_cap[(int64_t)l * N + n];
                pc0 = f.p_cap[(int64_t)l * N + n];
            }
            if (l < f.max_d) {
                dc0 = f.d_cap[(int64_t)l * N + n];
                sk0 = f.sink_cap[(int64_t)l * N + n];
            }
#pragma unroll
            for (int r = 0; r < kKvRows; ++r) {
                const int e = l + r * SEG;
                kvr[r] = e < f.max_pd ? f.kv_cap[(int64_t)e * N + n] : 0;
            }
        }
        // A network larger than the plan it was built for is rejected before any LDS or array
        // index is formed from it.
        if (P < 0 || D < 0 || P > f.max_p || D > f.max_d || P * D > f.max_pd ||
            (SEG <= 64 && (P > SEG || D > SEG || P * D > kKvRows * SEG))) {
            if (l == 0) flow_value[n] = HX_EINVAL;
            valid = false;
        }
    }
    if (!valid) P = D = 0;
    const int Ds = D | 1;

    // Node capacities first: a candidate whose source side or sink side carries nothing has
    // flow 0 and never needs its KV capacities (the cut sweep still sees zero flows).
    if (l == 0) {
        L.misc[0] = 0;
        L.misc[1] = 0;
        L.misc[2] = 0;
        L.misc[3] = 0;
    }
    __syncthreads();
    for (int i = l; i < P; i += SEG) {
        const int32_t s = SEG <= 64 ? src0 : f.src_cap[(int64_t)i * N + n];
        const int32_t c = SEG <= 64 ? pc0 : f.p_cap[(int64_t)i * N + n];
        const int32_t a = s < c ? s : c;
        L.a[i] = a;
        if (a > 0) L.misc[2] = 1;
    }
    for (int j = l; j < D; j += SEG) {
        const int32_t c = SEG <= 64 ? dc0 : f.d_cap[(int64_t)j * N + n];
        const int32_t t = SEG <= 64 ? sk0 : f.sink_cap[(int64_t)j * N + n];
        const int32_t b = c < t ? c : t;
        L.b[j] = b;
        L.ft[j] = 0;
        L.ed[j] = 0;
        if (b > 0) L.misc[3] = 1;
    }
    __syncthreads();
    const bool has_flow = P > 0 && D > 0 && L.misc[2] && L.misc[3];
    int path = has_flow ? HX_MF_PUSH_RELABEL : HX_MF_NO_FLOW;  // kStats: the path this candidate takes
    for (int i = l; i < P; i += SEG) {
        const int32_t a = has_flow ? L.a[i] : 0;
        L.fs[i] = a;  // saturate every source edge
        L.ep[i] = a;
    }
    if (SEG <= 64) {
#pragma unroll
        for (int r = 0; r < kKvRows; ++r) {
            const int e = l + r * SEG;
            if (e < P * D) {
                const int i = e / D, d = e - i * D;
                L.cap[i * Ds + d] = kvr[r];
                L.fl[i * Ds + d] = 0;
            }
        }
    } else {
        const bool need_kv = has_flow || kv_flow != nullptr || cut != nullptr;
        for (int e = l; need_kv && e < P * D; e += SEG) {
            const int i = e / D, d = e - i * D;
            L.cap[i * Ds + d] = f.kv_cap[(int64_t)e * N + n];
            L.fl[i * Ds + d] = 0;
        }
    }
    __syncthreads();

    // One side with a single node that can carry flow (a > 0 on the prefill side, b > 0 on
    // the decode side) makes the network a star: with prefill node i alone the maximum flow
    // is min(a_i, sum_j min(c_ij, b_j)), with decode node j alone min(b_j, sum_i min(a_i,
    // c_ij)).  Such a candidate takes that value and a flow that fills the star's arcs in
    // node order (a prefix sum over the candidate's lanes), and skips push-relabel; the cut
    // sweep below works from any maximum flow.  Only the single-wavefront plans do this.
    // The shuffles below stay inside a candidate's lanes, whose branches agree.
    int32_t cut_value = -1;  // the flow value when a minimum cut was taken directly
    if (SEG <= 64) {
        const uint64_t segmask = SEG == 64 ? ~0ull : ((1ull << SEG) - 1);
        const int sh = (seg * SEG) & 63;
        const uint64_t ba = (__ballot(l < P && L.a[l] > 0) >> sh) & segmask;
        const uint64_t bb = (__ballot(l < D && L.b[l] > 0) >> sh) & segmask;
        const bool one_p = __popcll(ba) == 1, one_d = __popcll(bb) == 1;
        bool thin = false;  // some KV arc below min(a_i, b_j)
#pragma unroll
        for (int r = 0; r < kKvRows; ++r) {
            const int e = l + r * SEG;
            if (e < P * D) {
                const int i = e / D, d = e - i * D;
                const int32_t m = L.a[i] < L.b[d] ? L.a[i] : L.b[d];
                thin |= L.cap[i * Ds + d] < m;
            }
        }
        const bool dominant = ((__ballot(thin) >> sh) & segmask) == 0;
        if (has_flow && (one_p || one_d)) {
            path = HX_MF_STAR;
            const int is = __ffsll((unsigned long long)ba) - 1, js = __ffsll((unsigned long long)bb) - 1;
            int32_t v = 0;
            if (one_p) {
                if (l < D && L.b[l] > 0) {
                    const int32_t c = L.cap[is * Ds + l];
                    v = c < L.b[l] ? c : L.b[l];
                }
            } else if (l < P && L.a[l] > 0) {
                const int32_t c = L.cap[l * Ds + js];
                v = c < L.a[l] ? c : L.a[l];
            }
            int32_t incl = v;
#pragma unroll
            for (int off = 1; off < SEG; off <<= 1) {
                const int32_t u = __shfl_up(incl, off, SEG);
                if (l >= off) incl += u;
            }
            const int32_t total = __shfl(incl, SEG - 1, SEG);
            const int32_t side = one_p ? L.a[is] : L.b[js];
            const int32_t F = total < side ? total : side;
            const int32_t room = F - (incl - v);
            const int32_t fv = room <= 0 ? 0 : (room < v ? room : v);
            if (one_p) {
                if (l < D) {
                    L.fl[is * Ds + l] = fv;
                    L.ft[l] = fv;
                }
                if (l == is) L.fs[is] = F;
            } else {
                if (l < P) {
                    L.fl[l * Ds + js] = fv;
                    L.fs[l] = fv;
                }
                if (l == js) L.ft[js] = F;
            }
            if (l < P) L.ep[l] = 0;
        } else if (has_flow && dominant) {
            path = HX_MF_DOMINANT;
            // lane l holds prefill node l and decode node l (packed plans: P, D <= SEG); the
            // sums stay below 64 * 2^24 < 2^31
            const int32_t av = l < P ? L.a[l] : 0, bv = l < D ? L.b[l] : 0;
            int32_t ia = av, ib = bv;
#pragma unroll
            for (int off = 1; off < SEG; off <<= 1) {
                const int32_t ua = __shfl_up(ia, off, SEG), ub = __shfl_up(ib, off, SEG);
                if (l >= off) {
                    ia += ua;
                    ib += ub;
                }
            }
            const int32_t ta = __shfl(ia, SEG - 1, SEG), tb = __shfl(ib, SEG - 1, SEG);
            const int32_t U = ta < tb ? ta : tb;
            const int32_t ai = ia < U ? ia : U, ae = ia - av < U ? ia - av : U;
            const int32_t bi = ib < U ? ib : U, be = ib - bv < U ? ib - bv : U;
            if (l < P) {
                L.fs[l] = ai - ae;
                L.ep[l] = 0;
            }
            if (l < D) L.ft[l] = bi - be;
#pragma unroll
            for (int r = 0; r < kKvRows; ++r) {
                const int e = l + r * SEG;
                const bool in = e < P * D;
                const int i = in ? e / D : 0, d = in ? e - i * D : 0;
                const int32_t Ai = __shfl(ai, i, SEG), Ae = __shfl(ae, i, SEG);
                const int32_t Bj = __shfl(bi, d, SEG), Be = __shfl(be, d, SEG);
                if (in) L.fl[i * Ds + d] = nw_overlap(Ae, Ai, Be, Bj);
            }
        } else if (has_flow && kv_flow == nullptr && cut == nullptr) {
            // Only the value is wanted: with m = min(P', D') <= kEnumMax nodes that can carry
            // flow on the smaller side, take the minimum cut directly.  Fixing which of those
            // nodes stay on the source side (a subset A of the prefill side, say) leaves every
            // other node one cheapest choice: cut = sum_{i not in A} a_i + sum_j min(b_j,
            // sum_{i in A} c_ij); the maximum flow is the minimum over the 2^m subsets, which
            // the candidate's lanes share.
            const int pe = __popcll(ba), de = __popcll(bb);
            const int m = pe <= de ? pe : de;
            if (m <= kEnumMax) {
                const bool byp = pe <= de;
                const uint64_t side = byp ? ba : bb, other = byp ? bb : ba;
                int32_t best = 0x7fffffff;
                for (int sub = l; sub < (1 << m); sub += SEG) {
                    int32_t cost = 0;
                    uint64_t rest = side;
                    for (int k = 0; rest; ++k, rest &= rest - 1)
                        if (!((sub >> k) & 1)) {
                            const int u = __ffsll((unsigned long long)rest) - 1;
                            cost += byp ? L.a[u] : L.b[u];
                        }
                    for (uint64_t ow = other; ow; ow &= ow - 1) {
                        const int w = __ffsll((unsigned long long)ow) - 1;
                        int32_t arcs = 0;
                        uint64_t in = side;
                        for (int k = 0; in; ++k, in &= in - 1)
                            if ((sub >> k) & 1) {
                                const int u = __ffsll((unsigned long long)in) - 1;
                                arcs += byp ? L.cap[u * Ds + w] : L.cap[w * Ds + u];
                            }
                        const int32_t cw = byp ? L.b[w] : L.a[w];
                        cost += cw < arcs ? cw : arcs;
                    }
                    best = cost < best ? cost : best;
                }
#pragma unroll
                for (int off = SEG / 2; off > 0; off >>= 1) {
                    const int32_t o2 = __shfl_xor(best, off, SEG);
                    best = o2 < best ? o2 : best;
                }
                cut_value = best;
                path = HX_MF_MIN_CUT;
                if (l < P) L.ep[l] = 0;
            }
        }
        __syncthreads();
    } else {
        // Workgroup plans (one candidate per workgroup, so every branch here is uniform).
        __shared__ long long wave_sum[SEG > 64 ? SEG / 64 : 1];
        bool thin = false;
        for (int e = l; has_flow && e < P * D; e += SEG) {
            const int i = e / D, d = e - i * D;
            const int32_t m = L.a[i] < L.b[d] ? L.a[i] : L.b[d];
            thin |= L.cap[i * Ds + d] < m;
        }
        if (!__syncthreads_or(thin) && has_flow) {
            path = HX_MF_DOMINANT;
            // block scan: lane l owns a contiguous run of nodes on each side; clamped inclusive
            // prefix sums go to ep (prefill) and ed (decode), then become the flows
            const int cp = (P + SEG - 1) / SEG, cd = (D + SEG - 1) / SEG;
            const int p0 = l * cp < P ? l * cp : P, p1 = p0 + cp < P ? p0 + cp : P;
            const int d0 = l * cd < D ? l * cd : D, d1 = d0 + cd < D ? d0 + cd : D;
            long long sa = 0, sb = 0;
            for (int i = p0; i < p1; ++i) sa += L.a[i];
            for (int j = d0; j < d1; ++j) sb += L.b[j];
            long long tot[2], excl[2];
            const long long v2[2] = {sa, sb};
            for (int k = 0; k < 2; ++k) {
                long long incl = v2[k];
                for (int off = 1; off < 64; off <<= 1) {
                    const long long u = __shfl_up(incl, off, 64);
                    if ((l & 63) >= off) incl += u;
                }
                if ((l & 63) == 63) wave_sum[l >> 6] = incl;
                __syncthreads();
                long long before = 0, all = 0;
                for (int w = 0; w < SEG / 64; ++w) {
                    if (w < (l >> 6)) before += wave_sum[w];
                    all += wave_sum[w];
                }
                __syncthreads();
                excl[k] = before + incl - v2[k];
                tot[k] = all;
            }
            const long long U = tot[0] < tot[1] ? tot[0] : tot[1];  // < 2^31: min(P, D) <= 127
            long long run = excl[0];
            for (int i = p0; i < p1; ++i) {
                run += L.a[i];
                L.ep[i] = (int32_t)(run < U ? run : U);
            }
            run = excl[1];
            for (int j = d0; j < d1; ++j) {
                run += L.b[j];
                L.ed[j] = (int32_t)(run < U ? run : U);
            }
            __syncthreads();
            for (int e = l; e < P * D; e += SEG) {
                const int i = e / D, d = e - i * D;
                L.fl[i * Ds + d] = nw_overlap(i > 0 ? L.ep[i - 1] : 0, L.ep[i], d > 0 ? L.ed[d - 1] : 0, L.ed[d]);
            }
            for (int i = l; i < P; i += SEG) L.fs[i] = L.ep[i] - (i > 0 ? L.ep[i - 1] : 0);
            for (int j = l; j < D; j += SEG) L.ft[j] = L.ed[j] - (j > 0 ? L.ed[j - 1] : 0);
            __syncthreads();
            for (int i = l; i < P; i += SEG) L.ep[i] = 0;
            for (int j = l; j < D; j += SEG) L.ed[j] = 0;
        }
        __syncthreads();
    }

    const int V = P + D + 2;
    const int INF = 2 * V + 2;
    bool active = false;
    for (int i = l; i < P; i += SEG) active |= L.ep[i] > 0;
    unsigned long long pushes = 0, relabels = 0;  // kStats
    if (kStats && valid && l == 0) atomicAdd(&stats[path], 1ull);
    for (int round = 0; __syncthreads_or(active) && round < round_budget; ++round) {
        if (kStats && threadIdx.x == 0) {
            atomicAdd(&stats[HX_MF_ROUNDS], 1ull);
            if (round % kGlobalRelabelEvery == 0) atomicAdd(&stats[HX_MF_GLOBAL_RELABELS], 1ull);
        }
        if (round % kGlobalRelabelEvery == 0) {
            global_relabel<SEG>(L, l, P, D, Ds, V, INF);
            __syncthreads();
        }
        // P-phase: push along admissible arcs and, in the same pass, track the lowest height
        // across arcs still holding residual capacity, for the relabel if excess remains.
        for (int i = l; i < P; i += SEG) {
            int e = L.ep[i];
            if (e <= 0) continue;
            const int h = L.hp[i];
            const int32_t* c = L.cap + i * Ds;
            int32_t* fr = L.fl + i * Ds;
            int mh = INF;
            for (int d = 0; d < D && e > 0; ++d) {
                int r = c[d] - fr[d];
                if (r <= 0) continue;
                const int hd = L.hd[d];
                if (h == hd + 1) {
                    const int amt = r < e ? r : e;
                    fr[d] += amt;
                    e -= amt;
                    r -= amt;
                    atomicAdd(&L.ed[d], amt);
                    if (kStats) ++pushes;
                }
                if (r > 0 && hd < mh) mh = hd;
            }
            if (e > 0 && h == V + 1) {
                const int amt = L.fs[i] < e ? L.fs[i] : e;
                L.fs[i] -= amt;
                e -= amt;
                if (kStats && amt > 0) ++pushes;
            }
            if (e > 0) {
                if (L.fs[i] > 0 && V < mh) mh = V;
                L.hp[i] = mh + 1 < INF ? mh + 1 : INF;
                if (kStats) ++relabels;
            }
            L.ep[i] = e;
        }
        __syncthreads();
        // D-phase: push to the sink, then back along used KV arcs, tracking the lowest height
        // across arcs left with residual capacity for the relabel.
        for (int j = l; j < D; j += SEG) {
            int e = L.ed[j];
            if (e <= 0) continue;
            const int h = L.hd[j];
            if (h == 1) {
                const int r = L.b[j] - L.ft[j];
                const int amt = r < e ? r : e;
                if (amt > 0) {
                    L.ft[j] += amt;
                    e -= amt;
                    if (kStats) ++pushes;
                }
            }
            int mh = INF;
            for (int q = 0; q < P && e > 0; ++q) {
                int fq = L.fl[q * Ds + j];
                if (fq <= 0) continue;
                const int hq = L.hp[q];
                if (h == hq + 1) {
                    const int amt = fq < e ? fq : e;
                    fq -= amt;
                    L.fl[q * Ds + j] = fq;
                    e -= amt;
                    atomicAdd(&L.ep[q], amt);
                    if (kStats) ++pushes;
                }
                if (fq > 0 && hq < mh) mh = hq;
            }
            if (e > 0) {
                if (L.b[j] - L.ft[j] > 0) mh = 0;
                L.hd[j] = mh + 1 < INF ? mh + 1 : INF;
                if (kStats) ++relabels;
            }
            L.ed[j] = e;
        }
        __syncthreads();
        active = false;
        for (int i = l; i < P; i += SEG) active |= L.ep[i] > 0;
        for (int j = l; j < D; j += SEG) active |= L.ed[j] > 0;
    }
    if (kStats) {
        if (pushes) atomicAdd(&stats[HX_MF_PUSHES], pushes);
        if (relabels) atomicAdd(&stats[HX_MF_RELABELS], relabels);
    }
    // Flow value = total flow into the sink; a candidate still holding excess ran out of rounds.
    for (int j = l; j < D; j += SEG)
        if (L.ft[j] > 0) atomicAdd(&L.misc[0], L.ft[j]);
    if (active) L.misc[1] = 1;
    __syncthreads();
    const int32_t value = cut_value >= 0 ? cut_value : (L.misc[1] ? HX_ENOCONV : L.misc[0]);
    if (valid && l == 0) flow_value[n] = value;
    if (kArg) fold_argmax(l == 0 && in_range ? argmax_key(valid ? value : HX_EINVAL, n) : 0ull, arg);
    if (valid && kv_flow)
        for (int e = l; e < P * D; e += SEG) {
            const int i = e / D, d = e - i * D;
            kv_flow[(int64_t)e * N + n] = L.fl[i * Ds + d];
        }
    if (!cut) return;  // uniform across the workgroup

    // Canonical minimum cut: reachability from s in the residual graph of the uncontracted
    // network, by sweeps until nothing changes.  Reuses a/ep (prefill in/out flags) and
    // b/ed (decode in/out flags); source/node/sink capacities are reloaded.
    int32_t* rin = L.ep;
    int32_t* rout = L.a;
    int32_t* din = L.ed;
    int32_t* dout = L.b;
    __syncthreads();
    for (int i = l; i < P; i += SEG) {
        rin[i] = f.src_cap[(int64_t)i * N + n] - L.fs[i] > 0;
        rout[i] = 0;
    }
    for (int j = l; j < D; j += SEG) {
        din[j] = 0;
        dout[j] = 0;
    }
    __syncthreads();
    for (;;) {
        bool changed = false;
        // prefill replica: phi_out is reached from a reached delta_in over a used KV edge (its
        // reverse arc), and in <-> out inside the chain along whichever arcs have residual.
        for (int i = l; i < P; i += SEG) {
            const int32_t fsi = L.fs[i];
            const int32_t pres = f.p_cap[(int64_t)i * N + n] - fsi;
            int in = rin[i], out = rout[i];
            for (int d = 0; d < D && !out; ++d) out = din[d] && L.fl[i * Ds + d] > 0;
            for (int k = 0; k < 2; ++k) {
                in |= out && fsi > 0;
                out |= in && pres > 0;
            }
            if (in != rin[i] || out != rout[i]) {
                rin[i] = in;
                rout[i] = out;
                changed = true;
            }
        }
        __syncthreads();
        // decode replica: delta_in is reached from a reached phi_out over a KV edge with
        // residual capacity, then in <-> out inside the chain.
        for (int j = l; j < D; j += SEG) {
            const int32_t ftj = L.ft[j];
            const int32_t dres = f.d_cap[(int64_t)j * N + n] - ftj;
            int in = din[j], out = dout[j];
            for (int q = 0; q < P && !in; ++q) in = rout[q] && L.cap[q * Ds + j] - L.fl[q * Ds + j] > 0;
            for (int k = 0; k < 2; ++k) {
                out |= in && dres > 0;
                in |= out && ftj > 0;
            }
            if (in != din[j] || out != dout[j]) {
                din[j] = in;
                dout[j] = out;
                changed = true;
            }
        }
        if (!__syncthreads_or(changed)) break;
    }
    if (!valid) return;
    for (int i = l; i < P; i += SEG) cut[(int64_t)i * N + n] = (uint8_t)(rin[i] | (rout[i] << 1));
    for (int j = l; j < D; j += SEG) cut[(int64_t)(f.max_p + j) * N + n] = (uint8_t)(din[j] | (dout[j] << 1));
}

// kArg (hx_score_batch): each wavefront also takes the best of its candidates' flow values
// (highest value, lowest index) and folds it into slot blockIdx mod kArgSlots of arg, as the key
// argmax_key, with a 64-bit atomic max; the slots must be zero at launch, and best_final_kernel
// reduces them.
template <int SEG, bool kStats, bool kArg = false>
__global__ void __launch_bounds__(SEG < 64 ? kPackedLanes : SEG, SEG <= 64 ? 8 : 1)
    maxflow_kernel(FlowNet f, int32_t* flow_value, int32_t* kv_flow, uint8_t* cut, int32_t round_budget,
                   unsigned long long* stats, unsigned long long* arg) {
    constexpr int kPer = (SEG < 64 ? kPackedLanes : SEG) / SEG;
    const int tiles = (f.N + kPer - 1) / kPer;
    const int chunk = (tiles + 7) / 8;
    const int tile = (int)(blockIdx.x & 7) * chunk + (int)(blockIdx.x >> 3);
    maxflow_tile<SEG, kStats, kArg>(f, flow_value, kv_flow, cut, round_budget, stats, tile, arg);
}

// Value only, workgroup plans: the candidates listed (list[0 .. *count), written by the kernel that
// settled the others), a workgroup taking every gridDim.x-th entry.
template <int SEG>
__global__ void __launch_bounds__(SEG) maxflow_list_kernel(FlowNet f, int32_t* flow_value, int32_t round_budget,
                                                           const int32_t* list, const int32_t* count) {
    const int c = *count;
    for (int idx = blockIdx.x; idx < c; idx += gridDim.x) {
        maxflow_tile<SEG, false>(f, flow_value, nullptr, nullptr, round_budget, nullptr, list[idx]);
        __syncthreads();  // the next candidate reuses the LDS
    }
}

constexpr size_t kMaxLds = 64 * 1024;

// Lanes per candidate: the smallest power of two (at least 8) with one lane per node of the
// widest side and SEG/4 KV rows per lane covering max_pd (SEG^2/4 >= max_pd); beyond 256
// lanes a lane owns several nodes.
int segment_lanes(int max_p, int max_d, int max_pd) {
    const int widest = max_p > max_d ? max_p : max_d;
    int s = 8;
    while (s < 256 && (s < widest || (int64_t)s * s / 4 < max_pd)) s *= 2;
    return s;
}

__global__ void clear_stats_kernel(unsigned long long* stats) {
    if (threadIdx.x < HX_MF_STATS) stats[threadIdx.x] = 0;
}

template <int SEG>
hipError_t launch_seg(const FlowNet& f, int32_t* fv, int32_t* kv, uint8_t* cut, int32_t budget,
                      unsigned long long* stats, unsigned long long* arg, hipStream_t s) {
    constexpr int kLanes = SEG < 64 ? kPackedLanes : SEG;
    constexpr int kPer = kLanes / SEG;
    const size_t lds = kPer * mf_words(f.max_p, f.max_d, f.max_pd) * sizeof(int32_t);
    const int tiles = (f.N + kPer - 1) / kPer;
    const int blocks = 8 * ((tiles + 7) / 8);
    prof_mark(kKMaxflow, false, s);
    if (SEG > 64 && kv == nullptr && cut == nullptr) {
        hipLaunchKernelGGL(bound_kernel, dim3((f.N + kBoundBlock - 1) / kBoundBlock), dim3(kBoundBlock), 0, s, f, fv);
        const int chunks = (f.N + 63) / 64;
        hipLaunchKernelGGL(dom_kernel, dim3(chunks * kDomParts), dim3(64), 0, s, f, fv);
    }
    if (stats) {
        hipLaunchKernelGGL(clear_stats_kernel, dim3(1), dim3(64), 0, s, stats);
        hipLaunchKernelGGL((maxflow_kernel<SEG, true>), dim3(blocks), dim3(kLanes), lds, s, f, fv, kv, cut, budget,
                           stats, nullptr);
    } else if (arg) {
        hipLaunchKernelGGL((maxflow_kernel<SEG, false, true>), dim3(blocks), dim3(kLanes), lds, s, f, fv, kv, cut,
                           budget, nullptr, arg);
    } else {
        hipLaunchKernelGGL((maxflow_kernel<SEG, false>), dim3(blocks), dim3(kLanes), lds, s, f, fv, kv, cut, budget,
                           nullptr, nullptr);
    }
    prof_mark(kKMaxflow, true, s);
    return hipGetLastError();
}

}  // namespace

size_t maxflow_lds_bytes(int32_t max_p, int32_t max_d, int32_t max_pd) {
    const int seg = segment_lanes(max_p, max_d, max_pd);
    const int per = seg < 64 ? kPackedLanes / seg : 1;
    const size_t bytes = per * mf_words(max_p, max_d, max_pd) * sizeof(int32_t);
    return bytes <= kMaxLds ? bytes : 0;
}

bool maxflow_workgroup_plan(int32_t max_p, int32_t max_d, int32_t max_pd) {
    return segment_lanes(max_p, max_d, max_pd) > 64;
}

hipError_t launch_maxflow_listed(const FlowNet& f, int32_t* flow_value, int32_t round_budget, const int32_t* list,
                                 const int32_t* count, hipStream_t s) {
    const int seg = segment_lanes(f.max_p, f.max_d, f.max_pd);
    const size_t lds = mf_words(f.max_p, f.max_d, f.max_pd) * sizeof(int32_t);
    const int blocks = f.N < 2048 ? f.N : 2048;  // eight workgroups per CU at most
    prof_mark(kKMaxflow, false, s);
    if (seg == 128)
        hipLaunchKernelGGL(maxflow_list_kernel<128>, dim3(blocks), dim3(128), lds, s, f, flow_value, round_budget, list,
                           count);
    else
        hipLaunchKernelGGL(maxflow_list_kernel<256>, dim3(blocks), dim3(256), lds, s, f, flow_value, round_budget, list,
                           count);
    prof_mark(kKMaxflow, true, s);
    return hipGetLastError();
}

hipError_t launch_maxflow(const FlowNet& f, int32_t* flow_value, int32_t* kv_flow, uint8_t* cut, int32_t round_budget,
                          unsigned long long* stats, hipStream_t s, unsigned long long* arg) {
    switch (segment_lanes(f.max_p, f.max_d, f.max_pd)) {
        case 8: return launch_seg<8>(f, flow_value, kv_flow, cut, round_budget, stats, arg, s);
        case 16: return launch_seg<16>(f, flow_value, kv_flow, cut, round_budget, stats, arg, s);
        case 32: return launch_seg<32>(f, flow_value, kv_flow, cut, round_budget, stats, arg, s);
        case 64: return launch_seg<64>(f, flow_value, kv_flow, cut, round_budget, stats, arg, s);
        case 128: return launch_seg<128>(f, flow_value, kv_flow, cut, round_budget, stats, arg, s);
        default: return launch_seg<256>(f, flow_value, kv_flow, cut, round_budget, stats, arg, s);
    }
}

}  // namespace hx
