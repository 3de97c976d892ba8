// hx_internal.h -- launch interfaces and device helpers shared by libhx's HIP sources.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hx.h"

namespace hx {

constexpr double kBmaxClamp = 1073741824.0;  // 2^30

// Scalars of one scoring problem, copied into every kernel's argument block.
struct Problem {
    int32_t G, T, N, Kmax, L;
    uint32_t tp_mask, pp_mask;
    int32_t granularity;
    uint32_t variant;  // HX_VARIANT_* bits
    double H, Hkv, B, s_in, s_out;
    int32_t n_cls;  // request classes (0: the single task s_in, s_out)
    double cls_in[HX_MAX_CLASSES], cls_out[HX_MAX_CLASSES], cls_w[HX_MAX_CLASSES];
    int32_t coord_cap;
    const int32_t* gpu_type;
    const double *flops, *hbm, *mem, *beta, *alpha;
    const uint8_t *assign, *role;
};

struct CostOut {
    uint8_t *tp, *pp;
    int32_t *bmax, *cap;
    double* lat;
    uint64_t* members;  // [Kmax][W][N] group member bitmasks
};

struct FlowNet {
    int32_t N, max_p, max_d, max_pd;
    int32_t *n_p, *n_d, *p_slot, *d_slot, *src_cap, *p_cap, *kv_cap, *d_cap, *sink_cap;
    // Optional scratch of the listed KV path (replica nodes, kv_list_fits), per piece: 64
    // candidates (s = n / 64) and a slice r of kKvSlices of their KV rows (rows r kv_rows to
    // (r + 1) kv_rows - 1):
    //   feas     [N]: bit i of the low word set when prefill node i's replica has a strategy,
    //            bit j of the high word the same for decode node j (nodes_kernel writes it);
    //   kv_count [ceil(N / 64)][kKvSlices]: how many of the piece's KV edges are listed;
    //   kv_list  [ceil(N / 64)][kKvSlices][64 kv_rows]: the piece's KV edges whose two replicas
    //            have a strategy, (n << 10) | (i << 5) | j, in row order (kv_rows_kernel writes
    //            both, kv_walk_kernel walks them).
    //   kv_offs  [pieces + 1]: exclusive prefix sums of kv_count, the total last;
    //   kv_flat  the listed edges of all pieces, packed in piece order (kv_offs[s] onwards).
    uint64_t* feas = nullptr;
    int32_t* kv_count = nullptr;
    uint32_t* kv_list = nullptr;
    int32_t* kv_offs = nullptr;
    uint32_t* kv_flat = nullptr;
    int32_t kv_rows = 0;  // ceil(floor(Kmax/2) ceil(Kmax/2) / kKvSlices)
};

constexpr int kKvSlices = 4;

// The listed KV path takes networks of up to 32 replica slots (node indices in 5 bits, bits of
// feas) and up to 2^22 candidates (n in the list entry's other 22 bits).
inline bool kv_list_fits(int32_t granularity, int32_t max_groups, int32_t n_cand) {
    return granularity == 0 && max_groups <= 32 && n_cand <= (1 << 22);
}
// Its scratch: the pieces' counts and offsets, feas, then twice room for every KV row of every
// piece (the per-piece lists and the packed list).
inline int32_t kv_slice_rows(int32_t max_groups) {
    return ((max_groups / 2) * ((max_groups + 1) / 2) + kKvSlices - 1) / kKvSlices;
}
inline size_t kv_pieces(int32_t n_cand) { return (size_t)kKvSlices * (((size_t)n_cand + 63) / 64); }
inline size_t kv_round256(size_t x) { return (x + 255) & ~(size_t)255; }
inline size_t kv_list_entries(int32_t max_groups, int32_t n_cand) {
    return kv_pieces(n_cand) * 64 * (size_t)kv_slice_rows(max_groups);
}
inline size_t kv_list_bytes(int32_t max_groups, int32_t n_cand) {
    return kv_round256(sizeof(int32_t) * kv_pieces(n_cand)) + kv_round256(sizeof(int32_t) * (kv_pieces(n_cand) + 1)) +
           kv_round256(sizeof(uint64_t) * (size_t)n_cand) +
           2 * kv_round256(sizeof(uint32_t) * kv_list_entries(max_groups, n_cand));
}
inline void kv_list_carve(FlowNet& f, void* base, int32_t max_groups, int32_t n_cand) {
    unsigned char* b = static_cast<unsigned char*>(base);
    f.kv_count = reinterpret_cast<int32_t*>(b);
    b += kv_round256(sizeof(int32_t) * kv_pieces(n_cand));
    f.kv_offs = reinterpret_cast<int32_t*>(b);
    b += kv_round256(sizeof(int32_t) * (kv_pieces(n_cand) + 1));
    f.feas = reinterpret_cast<uint64_t*>(b);
    b += kv_round256(sizeof(uint64_t) * (size_t)n_cand);
    f.kv_list = reinterpret_cast<uint32_t*>(b);
    b += kv_round256(sizeof(uint32_t) * kv_list_entries(max_groups, n_cand));
    f.kv_flat = reinterpret_cast<uint32_t*>(b);
    f.kv_rows = kv_slice_rows(max_groups);
}

// Capacity in milli-requests/s: floor(x), clamped to [0, HX_CAP_MAX].
__device__ __forceinline__ int32_t quantize(double x) {
    if (!(x >= 0.0)) return 0;
    if (x >= (double)HX_CAP_MAX) return HX_CAP_MAX;
    return (int32_t)floor(x);
}

__device__ __forceinline__ double dmin(double a, double b) { return b < a ? b : a; }
__device__ __forceinline__ double dmax(double a, double b) { return b > a ? b : a; }

// Layers held by stage j of pp: floor(L/pp) + [j < L mod pp].
__device__ __forceinline__ int stage_layers(int L, int pp, int j) { return L / pp + (j < L % pp ? 1 : 0); }

// Layers per pipeline stage.  As written: the uniform split, floor(L/pp) + [j < L mod pp].
// With HX_VARIANT_ASYM (the asymmetric split): every stage first takes one layer and the other
// L - pp are shared in proportion to the stage's compute c_j (its slowest device's FLOP/s),
// f_j = floor(((L - pp) c_j) / sum_k c_k) (summed left to right), the layers left over going one
// each to the first stages: l_j = 1 + f_j + [j < L - pp - sum_k f_k].  Stages of one device
// type get the uniform split; a zero compute sum falls back to it.
struct LayerSplit {
    int lq, lr, base, rem;
    double csum;  // > 0: the asymmetric split applies
};

// stage_c(j): c_j of stage j.
template <bool kAsym, class StageC>
__device__ __forceinline__ LayerSplit layer_split(int L, int pp, StageC stage_c) {
    LayerSplit s{L / pp, L % pp, L - pp, 0, 0.0};
    if (kAsym) {
        for (int j = 0; j < pp; ++j) s.csum = s.csum + stage_c(j);
        if (s.csum > 0.0) {
            int F = 0;
            for (int j = 0; j < pp; ++j) F += (int)floor(((double)s.base * stage_c(j)) / s.csum);
            s.rem = s.base - F;
        }
    }
    return s;
}

// Layers of stage j whose slowest device has cj FLOP/s.
template <bool kAsym>
__device__ __forceinline__ int split_layers(const LayerSplit& s, int j, double cj) {
    if (kAsym && s.csum > 0.0) return 1 + (int)floor(((double)s.base * cj) / s.csum) + (j < s.rem ? 1 : 0);
    return s.lq + (j < s.lr ? 1 : 0);
}

// Kernels of libhx, for the diagnostic per-kernel timing behind hx_profile.
enum KernelId {
    kKSetup, kKDecode, kKScatter, kKEval, kKNodes, kKKv, kKMaxflow, kKBest, kKClasses, kKMoves, kKGather,
    kKSpectral, kKPartition, kKShared, kKCount
};
// While profiling is enabled, records a HIP event on s before (end = false) or after
// (end = true) a launch of kernel k; does nothing otherwise.
void prof_mark(int k, bool end, hipStream_t s);

// 64-bit words of a GPU bitmask: 1 up to 64 GPUs, 2 up to 128, 4 up to 255.
int mask_words(int32_t n_gpus);
size_t cost_workspace_bytes(int32_t n_gpus, int32_t max_groups, int32_t n_cand);
// The word after the histogram and cursors of a cost workspace: zero once launch_cost's first
// kernel has run, untouched by the cost kernels.
int32_t* cost_workspace_counter(void* workspace, int32_t n_gpus);
// clear / n_clear: more 64-bit words for the cost model's first kernel to zero (the fused
// argmax's slots in hx_score_batch).
hipError_t launch_cost(const Problem& p, const CostOut& o, void* workspace, hipStream_t s,
                       unsigned long long* clear = nullptr, int n_clear = 0);
hipError_t launch_flownet(const Problem& p, const CostOut& o, const FlowNet& f, hipStream_t s);
// LDS bytes the max-flow kernel needs for a network plan; 0 if it does not fit.
size_t maxflow_lds_bytes(int32_t max_p, int32_t max_d, int32_t max_pd);
// arg (hx_score_batch, replica networks): kArgSlots zeroed slots that the max-flow kernel folds
// each wavefront's best candidate into (argmax_key); launch_best_final then reduces them.
hipError_t launch_maxflow(const FlowNet& f, int32_t* flow_value, int32_t* kv_flow, uint8_t* cut, int32_t round_budget,
                          unsigned long long* stats, hipStream_t s, unsigned long long* arg = nullptr);
hipError_t launch_best(const int32_t* flow_value, int32_t n, int32_t* best, hipStream_t s);
// The same argmax over several workgroups: each writes its winner to part, and the last to
// finish (counted in *counter, which must be zero at launch and is zero again after it) reduces
// them.  part holds best_parts_bytes().
size_t best_parts_bytes();
// The fused argmax: slots of 64-bit keys, ordered as (value, then lower index) so that a larger key
// is a better candidate; 0 is no candidate (below every value a flow or an error code takes).
constexpr int kArgSlots = 4096;
__host__ __device__ inline unsigned long long argmax_key(int32_t value, int32_t n) {
    return ((unsigned long long)((uint32_t)value ^ 0x80000000u) << 32) | (unsigned long long)(0xFFFFFFFFu - (uint32_t)n);
}
hipError_t launch_best_final(const unsigned long long* slots, int32_t* best, hipStream_t s);
hipError_t launch_best_parts(const int32_t* flow_value, int32_t n, int32_t* best, int32_t* counter, uint64_t* part,
                             hipStream_t s);
// hx_score_batch: per-GPU networks of up to 128 GPUs and 128 slots are settled from a table of
// link capacities (flownet_values_direct): node rows written, flow_value the closed form where
// every KV edge is dominant, else -1 with the KV rows written and the candidate appended to a
// list; launch_maxflow_listed then solves the listed networks (workgroup plans only:
// maxflow_workgroup_plan).
bool flownet_values_direct(const Problem& p);
// Bytes of its scratch: the link table (int32 [G][G] capacities, [G] row minima), then the count
// and list of the candidates left to the max-flow (int32 [1 + N]).
size_t link_table_bytes(int32_t n_gpus, int32_t n_cand);
// The list count inside that scratch (the list follows it at +16 words).
int32_t* flownet_values_list_count(void* table, int32_t n_gpus);
hipError_t launch_flownet_values(const Problem& p, const CostOut& o, const FlowNet& f, int32_t* flow_value,
                                 void* table, hipStream_t s);
bool maxflow_workgroup_plan(int32_t max_p, int32_t max_d, int32_t max_pd);
hipError_t launch_maxflow_listed(const FlowNet& f, int32_t* flow_value, int32_t round_budget, const int32_t* list,
                                 const int32_t* count, hipStream_t s);

// Refinement (Sec. 3.4): edge classes of networks of at most kClsMaxV vertices, guided moves,
// and the column gather.
constexpr int kClsMaxV = 512;
hipError_t launch_classes(const FlowNet& f, const int32_t* flow_value, const int32_t* kv_flow, uint8_t* node_cls,
                          uint8_t* kv_cls, hipStream_t s);
hipError_t launch_moves(int32_t G, int32_t K, int32_t gran, int32_t M, const uint8_t* p_assign,
                        const uint8_t* p_role, const FlowNet& pn, const uint8_t* node_cls, int32_t n_child,
                        const uint64_t* rnd, uint8_t* c_assign, uint8_t* c_role, int32_t* move, hipStream_t s);
// Graph partition (Sec. 3.2): w is an [G][G] int64 scratch both calls fill first.
hipError_t launch_spectral(int32_t G, const double* beta, int64_t* w, int32_t iters, int32_t* order, double* fiedler,
                           hipStream_t s);
hipError_t launch_partition(const Problem& p, int64_t* w, const int32_t* order, const uint64_t* rnd, uint8_t* assign,
                            uint8_t* role, hipStream_t s);
hipError_t launch_gather(int32_t G, int32_t K, int32_t Ns, const uint8_t* sa, const uint8_t* sr, const int32_t* index,
                         int32_t count, uint8_t* da, uint8_t* dr, hipStream_t s);

}  // namespace hx
