// hx_refine.hip -- max-flow guided refinement (Sec. 3.4) on gfx950.
//
// The refinement step compares every edge's flow with its capacity and moves GPUs between
// groups to relieve bottleneck edges with underutilized ones.  A maximum flow assignment is
// not unique, so the classes are the flow-independent ones (identical for every maximum flow):
//   bottleneck     raising the capacity by one raises the maximum flow: in the residual graph
//                  of a maximum flow, s reaches the edge's tail and its head reaches t;
//   underutilized  capacity >= 1 and lowering it by one keeps the maximum flow: the edge has
//                  spare capacity, or its tail reaches its head in the residual graph.
//
//   classes_kernel  one workgroup per candidate: the residual graph of the flow given by
//                   kv_flow (node flows follow by conservation), its transitive closure as
//                   bitset rows in LDS (one Warshall pass, a lane per row), then the class of
//                   every edge;
//   moves_kernel    one workgroup per (parent, 256 children): the parent's donor GPUs,
//                   receiver groups and flip-eligible groups, listed in ascending id in LDS;
//                   then a lane per child applies one MOVE, SWAP or FLIP chosen by its draw;
//   gather_kernel   copies chosen columns of a batch (the best child) into another batch.
// All three are graph and byte work, not dense contractions: no MFMA.
#include "hx_internal.h"

namespace hx {
namespace {

constexpr int kClsBlock = 256;
constexpr int kClsWords = kClsMaxV / 64;  // bitset words per closure row

__device__ __forceinline__ void drain_barrier() {
    // LDS atomics with unused results must have landed before the workgroup reads their
    // targets: wait for this wave's LDS operations (lgkmcnt(0)), then the barrier.
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __syncthreads();
}

struct ClsArgs {
    FlowNet f;
    const int32_t* flow_value;
    const int32_t* kv_flow;
    uint8_t* node_cls;
    uint8_t* kv_cls;
};

__global__ void __launch_bounds__(kClsBlock) classes_kernel(ClsArgs a) {
    __shared__ uint64_t reach[kClsMaxV * kClsWords];  // row u: the vertices u reaches
    __shared__ int32_t pf[HX_MAX_GPUS + 1], df[HX_MAX_GPUS + 1];
    const FlowNet& f = a.f;
    const int n = blockIdx.x, tid = threadIdx.x;
    const int64_t N = f.N;
    const int P = f.n_p[n], D = f.n_d[n];
    // a network that does not fit its arrays or the closure's LDS rows, or whose max-flow
    // failed, gets no classes
    if (P < 0 || D < 0 || P > f.max_p || D > f.max_d || P * D > f.max_pd || 2 + 2 * (P + D) > kClsMaxV ||
        a.flow_value[n] < 0) {
        for (int r = tid; r < f.max_p + f.max_d; r += kClsBlock) a.node_cls[(int64_t)r * N + n] = 0;
        return;
    }
    const int V = 2 + 2 * (P + D);
    const int W = (V + 63) >> 6;
    auto pin = [](int i) { return 2 + 2 * i; };
    auto pout = [](int i) { return 3 + 2 * i; };
    auto din = [P](int j) { return 2 + 2 * P + 2 * j; };
    auto dout = [P](int j) { return 3 + 2 * P + 2 * j; };
    auto kvf = [&](int i, int j) { return a.kv_flow[(int64_t)(i * D + j) * N + n]; };
    auto kvc = [&](int i, int j) { return f.kv_cap[(int64_t)(i * D + j) * N + n]; };

    // node flows by conservation: prefill i carries its KV row's sum, decode j its column's
    for (int i = tid; i < P; i += kClsBlock) {
        int32_t s = 0;
        for (int j = 0; j < D; ++j) s += kvf(i, j);
        pf[i] = s;
    }
    for (int j = tid; j < D; j += kClsBlock) {
        int32_t s = 0;
        for (int i = 0; i < P; ++i) s += kvf(i, j);
        df[j] = s;
    }
    __syncthreads();

    // residual arcs: u -> v when flow < capacity, v -> u when flow > 0; each lane owns its rows
    for (int u = tid; u < V; u += kClsBlock) {
        uint64_t* row = reach + u * kClsWords;
        for (int w = 0; w < W; ++w) row[w] = 0;
        auto set = [row](int v) { row[v >> 6] |= 1ull << (v & 63); };
        set(u);
        if (u == 0) {
            for (int i = 0; i < P; ++i)
                if (pf[i] < f.src_cap[(int64_t)i * N + n]) set(pin(i));
        } else if (u == 1) {
            for (int j = 0; j < D; ++j)
                if (df[j] > 0) set(dout(j));
        } else if (u < 2 + 2 * P) {
            const int i = (u - 2) >> 1;
            if ((u & 1) == 0) {  // prefill in-node
                if (pf[i] < f.p_cap[(int64_t)i * N + n]) set(pout(i));
                if (pf[i] > 0) set(0);
            } else {             // prefill out-node
                for (int j = 0; j < D; ++j)
                    if (kvf(i, j) < kvc(i, j)) set(din(j));
                if (pf[i] > 0) set(pin(i));
            }
        } else {
            const int j = (u - 2 - 2 * P) >> 1;
            if ((u & 1) == 0) {  // decode in-node
                if (df[j] < f.d_cap[(int64_t)j * N + n]) set(dout(j));
                for (int i = 0; i < P; ++i)
                    if (kvf(i, j) > 0) set(pout(i));
            } else {             // decode out-node
                if (df[j] < f.sink_cap[(int64_t)j * N + n]) set(1);
                if (df[j] > 0) set(din(j));
            }
        }
    }
    // transitive closure (Warshall): after step k every row holds the vertices it reaches
    // through intermediates < k + 1.  Row k does not change in step k, so lanes update their
    // own rows from it concurrently.
    for (int k = 0; k < V; ++k) {
        __syncthreads();
        const uint64_t* rk = reach + k * kClsWords;
        for (int u = tid; u < V; u += kClsBlock) {
            if (u == k) continue;
            uint64_t* ru = reach + u * kClsWords;
            if ((ru[k >> 6] >> (k & 63)) & 1ull)
                for (int w = 0; w < W; ++w) ru[w] |= rk[w];
        }
    }
    __syncthreads();

    auto reaches = [](int u, int v) { return (int)((reach[u * kClsWords + (v >> 6)] >> (v & 63)) & 1ull); };
    auto cls = [&](int u, int v, int32_t fl, int32_t c) {
        int k = reaches(0, u) & reaches(v, 1);
        if (c >= 1 && (fl < c || reaches(u, v))) k |= 2;
        return k;
    };
    for (int i = tid; i < P; i += kClsBlock) {
        const int64_t o = (int64_t)i * N + n;
        int k = cls(pin(i), pout(i), pf[i], f.p_cap[o]) | (cls(0, pin(i), pf[i], f.src_cap[o]) << 2);
        int kvb = 0;
        if (reaches(0, pout(i)))
            for (int j = 0; j < D && !kvb; ++j) kvb = reaches(din(j), 1);
        a.node_cls[o] = (uint8_t)(k | (kvb << 4));
    }
    for (int j = tid; j < D; j += kClsBlock) {
        const int64_t o = (int64_t)j * N + n;
        int k = cls(din(j), dout(j), df[j], f.d_cap[o]) | (cls(dout(j), 1, df[j], f.sink_cap[o]) << 2);
        int kvb = 0;
        if (reaches(din(j), 1))
            for (int i = 0; i < P && !kvb; ++i) kvb = reaches(0, pout(i));
        a.node_cls[(int64_t)(f.max_p + j) * N + n] = (uint8_t)(k | (kvb << 4));
    }
    for (int e = tid; e < P * D; e += kClsBlock) {
        const int i = e / D, j = e - i * D;
        a.kv_cls[(int64_t)e * N + n] = (uint8_t)cls(pout(i), din(j), kvf(i, j), kvc(i, j));
    }
}

// ------------------------------------------------------------------ guided moves

constexpr int kMoveBlock = 256;  // >= HX_MAX_GPUS + 1 and HX_MAX_GROUPS + 1: a lane per GPU / group

struct MoveArgs {
    int32_t G, K, gran, M, n_child, max_p, max_d;
    const uint8_t *p_assign, *p_role;            // [G][M], [K][M]
    const int32_t *n_p, *n_d, *p_slot, *d_slot;  // the parents' network
    const uint8_t* node_cls;                     // [max_p + max_d][M]
    const uint64_t* rnd;                         // [n_child]
    uint8_t *c_assign, *c_role;                  // [G][n_child], [K][n_child]
    int32_t* move;                               // [n_child]
};

// Index into m candidates from a b-bit draw u: floor(u m / 2^b).
__device__ __forceinline__ int pick(uint64_t u, int m, int bits) { return (int)((u * (uint64_t)m) >> bits); }

// Block-wide compaction of lane flags into an ascending list of lane ids; returns the count.
__device__ int compact(bool flag, uint8_t* list, int32_t* wave_cnt) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint64_t b = __ballot(flag);
    if (lane == 0) wave_cnt[wave] = __popcll(b);
    __syncthreads();
    int off = 0, total = 0;
    for (int w = 0; w < kMoveBlock / 64; ++w) {
        if (w < wave) off += wave_cnt[w];
        total += wave_cnt[w];
    }
    if (flag) list[off + __popcll(b & ((1ull << lane) - 1))] = (uint8_t)tid;
    __syncthreads();  // wave_cnt is reused by the next compaction
    return total;
}

__global__ void __launch_bounds__(kMoveBlock) moves_kernel(MoveArgs a) {
    __shared__ uint8_t pa[256], pr[256];
    __shared__ int16_t grp[256];
    __shared__ int32_t node_p[256], node_d[256];  // slot key -> node index (largest on repeats)
    __shared__ int32_t members[256], donors_in[256];
    __shared__ uint8_t donor[256], recv[256];
    __shared__ int32_t recv_role[2];
    __shared__ uint8_t recv_list[256], donor_list[256], rgpu_list[256], flip_list[256];
    __shared__ int32_t wave_cnt[kMoveBlock / 64];
    const int m = blockIdx.y, tid = threadIdx.x;
    const int G = a.G, K = a.K, M = a.M;
    if (tid < G) pa[tid] = a.p_assign[(int64_t)tid * M + m];
    if (tid < K) pr[tid] = a.p_role[(int64_t)tid * M + m];
    members[tid] = 0;
    donors_in[tid] = 0;
    recv[tid] = 0;
    node_p[tid] = -1;
    node_d[tid] = -1;
    if (tid < 2) recv_role[tid] = 0;
    int P = a.n_p[m], D = a.n_d[m];
    if (P < 0 || D < 0 || P > a.max_p || D > a.max_d) P = D = 0;  // no usable network
    __syncthreads();
    // groups and flow-node lookup
    int g_grp = -1;
    if (tid < G) {
        const int as = pa[tid];
        const int r = as < K ? pr[as] : HX_UNUSED;
        g_grp = (as < K && (r == HX_PREFILL || r == HX_DECODE)) ? as : -1;
        grp[tid] = (int16_t)g_grp;
        if (g_grp >= 0) atomicAdd(&members[g_grp], 1);
    }
    for (int i = tid; i < P; i += kMoveBlock) {
        const int key = a.p_slot[(int64_t)i * M + m];
        if (key >= 0 && key < 256) atomicMax(&node_p[key], i);
    }
    for (int j = tid; j < D; j += kMoveBlock) {
        const int key = a.d_slot[(int64_t)j * M + m];
        if (key >= 0 && key < 256) atomicMax(&node_d[key], j);
    }
    drain_barrier();
    // donors (unused, or an underutilized node edge) and receivers (a bottleneck node or KV
    // edge at a member's node)
    bool is_donor = false;
    if (tid < G) {
        is_donor = g_grp < 0;
        if (g_grp >= 0) {
            const int key = a.gran == 0 ? g_grp : tid;
            const int role = pr[g_grp];
            const int row = role == HX_PREFILL ? node_p[key] : (node_d[key] >= 0 ? a.max_p + node_d[key] : -1);
            if (row >= 0) {
                const uint8_t nc = a.node_cls[(int64_t)row * M + m];
                if (nc & 2) is_donor = true;
                if (nc & 17) {
                    recv[g_grp] = 1;
                    recv_role[role] = 1;
                }
            }
            if (is_donor) atomicAdd(&donors_in[g_grp], 1);
        }
        donor[tid] = is_donor;
    }
    drain_barrier();
    bool flip = false;
    if (tid < K && members[tid] > 0 && !recv[tid] && donors_in[tid] == members[tid])
        flip = recv_role[1 - pr[tid]] != 0;
    const int n_recv = compact(tid < K && recv[tid], recv_list, wave_cnt);
    const int n_flip = compact(flip, flip_list, wave_cnt);
    const int n_donor = compact(is_donor, donor_list, wave_cnt);
    const int n_rgpu = compact(tid < G && g_grp >= 0 && recv[g_grp], rgpu_list, wave_cnt);

    // one child per lane: children m, m + M, m + 2M, ... descend from parent m
    const int64_t t = (int64_t)blockIdx.x * kMoveBlock + tid;
    const int64_t c = m + t * M;
    if (c >= a.n_child) return;
    const int64_t Nc = a.n_child;
    int code = 0, g1 = -1, g2 = -1, v1 = 0, v2 = 0, fk = -1;
    if (c >= M) {
        const uint64_t r = a.rnd[c];
        const uint64_t u0 = r & 0xFFFFull, u1 = (r >> 16) & 0xFFFFFFull, u2 = r >> 40;
        const int t0 = pick(u0, 3, 16);
        for (int at = 0; at < 3 && code == 0; ++at) {
            const int ty = (t0 + at) % 3;
            if (ty == 0 && n_recv > 0) {
                const int k = recv_list[pick(u1, n_recv, 24)];
                const int na = n_donor - donors_in[k];
                if (na == 0) continue;
                int want = pick(u2, na, 24), g = -1;
                for (int x = 0; x < n_donor; ++x) {
                    const int d = donor_list[x];
                    if (grp[d] == k) continue;
                    if (want-- == 0) { g = d; break; }
                }
                g1 = g;
                v1 = k;
                code = 1 | (g << 8) | (k << 16);
            } else if (ty == 1 && n_rgpu > 0) {
                const int g = rgpu_list[pick(u1, n_rgpu, 24)];
                const int kg = grp[g];
                const int na = n_donor - donors_in[kg];
                if (na == 0) continue;
                int want = pick(u2, na, 24), h = -1;
                for (int x = 0; x < n_donor; ++x) {
                    const int d = donor_list[x];
                    if (grp[d] == kg) continue;
                    if (want-- == 0) { h = d; break; }
                }
                g1 = g;
                v1 = pa[h];
                g2 = h;
                v2 = pa[g];
                code = 2 | (g << 8) | (h << 16);
            } else if (ty == 2 && n_flip > 0) {
                fk = flip_list[pick(u1, n_flip, 24)];
                code = 3 | (fk << 8);
            }
        }
    }
    for (int g = 0; g < G; ++g)
        a.c_assign[(int64_t)g * Nc + c] = g == g1 ? (uint8_t)v1 : (g == g2 ? (uint8_t)v2 : pa[g]);
    for (int k = 0; k < K; ++k) a.c_role[(int64_t)k * Nc + c] = k == fk ? (uint8_t)(1 - pr[k]) : pr[k];
    a.move[c] = code;
}

// ------------------------------------------------------------------ gather

__global__ void gather_kernel(int G, int K, int Ns, const uint8_t* sa, const uint8_t* sr, const int32_t* index,
                              int count, uint8_t* da, uint8_t* dr) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= (int64_t)(G + K) * count) return;
    const int row = (int)(e / count), m = (int)(e - (int64_t)row * count);
    const int idx = index[m];
    const bool ok = idx >= 0 && idx < Ns;
    if (row < G) da[(int64_t)row * count + m] = ok ? sa[(int64_t)row * Ns + idx] : (uint8_t)HX_UNUSED;
    else dr[(int64_t)(row - G) * count + m] = ok ? sr[(int64_t)(row - G) * Ns + idx] : (uint8_t)HX_UNUSED;
}

}  // namespace

hipError_t launch_classes(const FlowNet& f, const int32_t* flow_value, const int32_t* kv_flow, uint8_t* node_cls,
                          uint8_t* kv_cls, hipStream_t s) {
    prof_mark(kKClasses, false, s);
    hipLaunchKernelGGL(classes_kernel, dim3(f.N), dim3(kClsBlock), 0, s,
                       ClsArgs{f, flow_value, kv_flow, node_cls, kv_cls});
    prof_mark(kKClasses, true, s);
    return hipGetLastError();
}

hipError_t launch_moves(int32_t G, int32_t K, int32_t gran, int32_t M, const uint8_t* p_assign,
                        const uint8_t* p_role, const FlowNet& pn, const uint8_t* node_cls, int32_t n_child,
                        const uint64_t* rnd, uint8_t* c_assign, uint8_t* c_role, int32_t* move, hipStream_t s) {
    const int64_t per = ((int64_t)n_child + M - 1) / M;  // children of parent 0, the most
    const dim3 grid((unsigned)((per + kMoveBlock - 1) / kMoveBlock), (unsigned)M);
    MoveArgs a{G, K, gran, M, n_child, pn.max_p, pn.max_d, p_assign, p_role, pn.n_p, pn.n_d, pn.p_slot, pn.d_slot,
               node_cls, rnd, c_assign, c_role, move};
    prof_mark(kKMoves, false, s);
    hipLaunchKernelGGL(moves_kernel, grid, dim3(kMoveBlock), 0, s, a);
    prof_mark(kKMoves, true, s);
    return hipGetLastError();
}

hipError_t launch_gather(int32_t G, int32_t K, int32_t Ns, const uint8_t* sa, const uint8_t* sr, const int32_t* index,
                         int32_t count, uint8_t* da, uint8_t* dr, hipStream_t s) {
    const int64_t cells = (int64_t)(G + K) * count;
    prof_mark(kKGather, false, s);
    hipLaunchKernelGGL(gather_kernel, dim3((unsigned)((cells + 255) / 256)), dim3(256), 0, s, G, K, Ns, sa, sr, index,
                       count, da, dr);
    prof_mark(kKGather, true, s);
    return hipGetLastError();
}

}  // namespace hx
