/*
 * hx.h -- C-ABI of libhx: batched scoring of HexGen-2 model placements on one MI355X.
 *
 * HexGen-2 (arXiv 2502.07903) schedules LLM serving on a heterogeneous GPU cluster by
 * searching over "model placement strategies" (Sec. 3.1): a partition of the GPUs into
 * groups, a role per group (prefill or decode replica), a TP x PP strategy per group and
 * a KV-cache routing between replicas.  The inner loop of that search (Sec. 3.3, run again
 * after every refinement step of Sec. 3.4) scores a placement: the Table 1 cost model gives
 * each replica's capacity, the placement becomes a flow network, and its maximum flow is
 * the placement's serving throughput.  libhx runs that loop for many thousands of candidate
 * placements at once:
 *
 *   hx_cost_eval       Table 1 + Appendix A node capacities     (one lane per group, sorted by shape)
 *   hx_build_flownet   the Sec. 3.3 network and its KV edges     (one lane per candidate / KV edge)
 *   hx_maxflow_batch   maximum flow, flow assignment, min cut    (one lane per node, LDS-resident)
 *   hx_best_candidate  the best candidate                        (one workgroup)
 *   hx_score_batch     the four above in one call, value only     (per-GPU networks settled from a
 *                                                                   table of link capacities)
 *
 * and the max-flow guided refinement step of Sec. 3.4 that feeds the next batch:
 *
 *   hx_edge_classes       bottleneck / underutilized edges        (one workgroup per candidate)
 *   hx_guided_moves       children of the best placements          (one lane per child)
 *   hx_gather_candidates  the chosen candidates into a new batch   (one lane per byte)
 *
 * and the graph-partition phase of Sec. 3.2 that generates candidates in the first place:
 *
 *   hx_spectral_order        the Fiedler order of the device graph  (one workgroup)
 *   hx_partition_candidates  partition, swaps, role split per draw  (one workgroup per candidate)
 *
 * Conventions
 *   - Every array pointer is a DEVICE pointer unless marked [host].  The caller owns every
 *     buffer; libhx allocates no device memory and keeps no state between calls.
 *   - Per-candidate arrays are candidate-fastest ("structure of arrays"): element (row, n)
 *     of an array with R rows lives at [row * n_cand + n].
 *   - Every call validates its arguments on the host (no device access, no sync), enqueues
 *     its kernels on `stream` and returns.  The return code reports validation and launch
 *     errors; results are ready when the stream reaches the enqueued work.
 *   - Capacities and flows are int32 milli-requests per second (1000 x requests/s),
 *     clamped to HX_CAP_MAX so that any cut of <= 128 edges fits in int32.
 *   - Floating point is IEEE binary64 with no contraction into fused multiply-add and
 *     correctly rounded division, each expression evaluated in the order documented at
 *     the function, so results do not depend on the launch shape.
 */
#ifndef HX_H
#define HX_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HX_ABI_VERSION 3
#define HX_CAP_MAX 16777215      /* 2^24 - 1 */
#define HX_MAX_GPUS 255
#define HX_MAX_GROUPS 255
#define HX_MAX_TP 8              /* tp_mask bits 0..7 */
#define HX_MAX_PP 32             /* pp_mask bits 0..31 */
#define HX_UNUSED 0xFF
#define HX_PREFILL 0
#define HX_DECODE 1

/* Return codes.  HX_ENOCONV is never returned: it marks a candidate's flow_value on the device. */
enum {
    HX_OK = 0,
    HX_EINVAL = -1,   /* invalid argument (null pointer, size or mask out of range) */
    HX_ETOOBIG = -2,  /* a flow network exceeds the max-flow kernel's LDS plan */
    HX_EHIP = -3,     /* a HIP launch failed; hx_last_error() keeps the runtime's message */
    HX_ENOCONV = -4   /* max-flow did not finish within its operation budget (per candidate) */
};

/* The device graph G = (D, E) of Sec. 3.2 with the per-GPU parameters of Table 1's legend. */
typedef struct hx_cluster {
    int32_t n_gpus;             /* G, 1..255 */
    int32_t n_types;            /* T >= 1 */
    const int32_t *gpu_type;    /* [G], each in [0, T) */
    const double *type_flops;   /* [T] c_d, tensor FLOP/s */
    const double *type_hbm_bw;  /* [T] m_d as memory bandwidth, bytes/s (decode weight scan) */
    const double *type_mem;     /* [T] m_d as memory limit, bytes (memory-limit row) */
    const double *beta;         /* [G*G] beta_{d,d'} bytes/s, row d = sender; diagonal unused, > 0 elsewhere */
    const double *alpha;        /* [G*G] alpha_{d,d'} seconds, row d = sender; diagonal unused */
    double coord_bw;            /* [host] coordinator link bytes/s; 0 = source/sink edges unbounded */
    double req_bytes;           /* [host] bytes per request on coordinator links */
} hx_cluster;

/* Model shape (Table 1 legend): L layers, hidden size H, B bytes per element.  KV-cache
 * terms use H_kv = H * n_kv_heads / n_heads (grouped-query attention); H*n_kv_heads must be
 * divisible by n_heads. */
typedef struct hx_model { int32_t n_layers, hidden, n_heads, n_kv_heads, bytes_per_elem; } hx_model;

/* Inference task t of Table 1: prompt length s_in and output length s_out (> 0, may be means).
 *
 * Request classes (per-bucket workloads): with n_classes in 1..HX_MAX_CLASSES the requests are
 * costed as n_classes length classes instead of the single task (s_in, s_out), class k with
 * prompt length cls_in[k], output length cls_out[k] (> 0) and weight cls_w[k] (> 0, its share of
 * the requests; used as given, not normalised).  A strategy must then fit every class in
 * memory: b_max is the smallest per-class b_max; the latency is the mix's mean sum_k w_k lat_k;
 * a replica's capacity is x = 1 / tau with tau = sum_k w_k / x_k (x_k its capacity on class k
 * alone; sums left to right in class order), so prefill keeps the strategy of lowest mix
 * latency and decode the one of highest x; a KV edge's time is sum_k w_k t_k.  The graph
 * partition still reads the single task (s_in, s_out).  Classes are refused (HX_EINVAL) with
 * HX_VARIANT_KV_ORDER or HX_VARIANT_ASYM.  n_classes 0: the single task; entries past
 * n_classes are ignored. */
#define HX_MAX_CLASSES 4
typedef struct hx_workload {
    double s_in, s_out;
    int32_t n_classes;
    double cls_in[HX_MAX_CLASSES], cls_out[HX_MAX_CLASSES], cls_w[HX_MAX_CLASSES];
} hx_workload;

/* Strategy space: bit k of tp_mask admits TP degree k+1 (<= 8), bit k of pp_mask PP degree
 * k+1 (<= 32).  granularity 0: one flow node per replica; 1: one flow node per GPU.
 * variant: cost-model variant bits, 0 for the model as written (see hx_cost_eval). */
typedef struct hx_space { uint32_t tp_mask, pp_mask; int32_t granularity; uint32_t variant; } hx_space;

/* Pipelined decode capacity: a decode replica's batches leave at the pace of its slowest
 * stage (an alternative reading of Appendix A's decode capacity). */
#define HX_VARIANT_PIPELINED 1u
/* KV stage-order search (Appendix A, edge capacity estimation): each KV edge's time is
 * minimised over the stage orders of both replicas, pipelines of up to 8 stages (see
 * hx_build_flownet). */
#define HX_VARIANT_KV_ORDER 2u
/* Asymmetric layer split (HexGen's asymmetric parallelism; Table 1 leaves l_j open): every
 * stage holds one layer plus its compute's share of the other L - pp (see hx_cost_eval).  Not
 * combinable with HX_VARIANT_KV_ORDER. */
#define HX_VARIANT_ASYM 4u
/* A hint in hx_space.variant, not a variant of the model: the batch's candidates share most of
 * their groups with candidate 0 (refinement rounds, whose candidates are single-step moves of
 * one placement).  hx_cost_eval then costs candidate 0's groups first, and a group of another
 * candidate with the same member set and role as candidate 0's group in the same slot, or in
 * one of the two slots next to it, takes that group's outputs instead of being costed again.
 * The outputs are the same with or without the hint. */
#define HX_HINT_SHARED_GROUPS (1u << 16)

/* Candidate placements (Sec. 3.1).  assign[g][n] = group of GPU g in candidate n (HX_UNUSED
 * or >= max_groups: GPU unused); role[k][n] = HX_PREFILL, HX_DECODE, or anything else (no
 * group).  A group exists when it has a member and a valid role. */
typedef struct hx_candidates {
    int32_t n_cand;             /* N >= 1 */
    int32_t max_groups;         /* Kmax, 1..255 */
    const uint8_t *assign;      /* [G][N] */
    const uint8_t *role;        /* [Kmax][N] */
} hx_candidates;

/* Per (group slot k, candidate n): the kept strategy and its node capacity.  Absent groups
 * and groups with no feasible strategy: every field 0.  members[k][w][n] is the group's
 * member set as a GPU bitmask (bit g of word w = GPU 64w + g), hx_member_words(n_gpus) words
 * per group; hx_build_flownet reads it. */
typedef struct hx_cost_out {
    uint8_t *tp, *pp;           /* [Kmax][N] */
    int32_t *bmax;              /* [Kmax][N] largest batch the memory limit admits */
    int32_t *cap;               /* [Kmax][N] node capacity, milli-requests/s */
    double *lat;                /* [Kmax][N] latency of one batch, seconds */
    uint64_t *members;          /* [Kmax][W][N] group member bitmasks, W = hx_member_words(n_gpus) */
} hx_cost_out;

/* The Sec. 3.3 network of every candidate.  Prefill nodes i < n_p and decode nodes j < n_d
 * (replicas in ascending group id, or GPUs in ascending GPU id at granularity 1); the edges
 * are source->phi_in (src_cap), phi_in->phi_out (p_cap), phi_out(i)->delta_in(j) (kv_cap row
 * i*n_d + j), delta_in->delta_out (d_cap), delta_out->sink (sink_cap).  Rows past n_p, n_d
 * and n_p*n_d are not written.  max_p, max_d >= max_groups (granularity 0) or n_gpus
 * (granularity 1), and max_pd >= floor(B/2)*ceil(B/2) for that bound B. */
typedef struct hx_flownet {
    int32_t n_cand, max_p, max_d, max_pd;
    int32_t *n_p, *n_d;         /* [N] */
    int32_t *p_slot, *d_slot;   /* [max_p][N], [max_d][N]: group id (or GPU id) of each node */
    int32_t *src_cap, *p_cap;   /* [max_p][N] */
    int32_t *kv_cap;            /* [max_pd][N] */
    int32_t *d_cap, *sink_cap;  /* [max_d][N] */
} hx_flownet;

/* Host-only check of everything the calls below validate (no HIP call, no device access).
 * cost / net may be NULL to skip their checks.  Returns HX_OK, HX_EINVAL or HX_ETOOBIG. */
int hx_validate(const hx_cluster *cluster, hx_model model, hx_workload wl, hx_space space,
                const hx_candidates *cand, const hx_cost_out *cost, const hx_flownet *net);

/* Table 1 cost model and Appendix A node capacities.  For every group of every candidate,
 * every admissible strategy (tp*pp = group size, tp and pp in the masks, pp <= L; stage j =
 * the members ranked j*tp .. j*tp+tp-1 in ascending GPU id, holding floor(L/pp) + [j < L mod
 * pp] layers) is costed:
 *   b_max   = min over stages and their devices of floor((M_d - A)/K) (clamped to 2^30),
 *             A = ((12*H*H*B)/tp)*l, K = ((2*(s_in+s_out)*H_kv*B)/tp)*l + 4*(s_in+s_out)*H*B;
 *             b_max < 1 makes the strategy infeasible.  Prefill runs at b = 1, decode at b_max.
 *   latency = sum_j (comp_j + tp_j) + sum_{j<pp-1} pp_j with, for stage j (t = tp, l = l_j):
 *     prefill comp = max_d((24*b*s_in*H*H)/(t*c_d))*l
 *     decode  comp = max_d((12*H*H*B*s_out)/(t*m_d))*l + max_d((24*b*s_out*H*H)/(t*c_d))*l
 *     TP: max_d sum_{d' != d, ascending} (alpha_{dd'} + X/(t*beta_{dd'})), times 4 then
 *         (decode) s_out then l; X = b*s_in*H*B (prefill) or b*H*B (decode)
 *     PP: min over d in stage j, d' in stage j+1 of (alpha_{dd'} + X/beta_{dd'}), decode
 *         times s_out
 *   x = (1000*b)/latency milli-requests/s; cap = min(HX_CAP_MAX, floor(x)).
 * A prefill group keeps its lowest-latency strategy, a decode group its highest-x one (Sec.
 * 3.3 "Compute nodes"); ties keep the smaller tp.
 * With space.variant & HX_VARIANT_PIPELINED, a decode strategy's x is (1000*b)/max_j T_j,
 * T_j = (comp_j + tp_j) + pp_j (pp_j: the PP term of the link into stage j+1 as in the
 * latency, none for the last stage); latencies and prefill are unchanged.
 * With space.variant & HX_VARIANT_ASYM, stage j holds l_j = 1 + f_j + [j < L - pp - sum_k f_k]
 * layers instead, f_j = floor(((L - pp) * c_j) / sum_k c_k) with c_j the slowest FLOP/s of the
 * stage's devices (the sum left to right; the uniform split when it is 0), in the memory row,
 * the computation and the TP term alike, and each replica's KV layer ranges follow its split.
 * With request classes (wl.n_classes > 0) every strategy is costed per class and mixed as
 * described at hx_workload; tp, pp, bmax, cap and lat are then the mix's. */
int hx_cost_eval(const hx_cluster *cluster, hx_model model, hx_workload wl, hx_space space,
                 const hx_candidates *cand, const hx_cost_out *out, void *workspace,
                 size_t workspace_bytes, hipStream_t stream);

/* Device scratch hx_cost_eval needs (it sorts the batch's groups by role and size so that
 * a wavefront costs groups of one shape): caller-owned, >= this many bytes, 256-byte
 * aligned, contents ignored on entry.  Calls that share a workspace must not overlap. */
size_t hx_cost_workspace_bytes(int32_t n_gpus, int32_t max_groups, int32_t n_cand);

/* For callers that cannot allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid hipMalloc): hx_cost_eval without the workspace argument.  Its scratch is
 * a static device array of HX_STATIC_SCRATCH_BYTES in libhx, one per GPU, resident from the
 * first call on that GPU until the process ends; the call allocates nothing.  Same arguments
 * (but the workspace), results and errors as hx_cost_eval, plus HX_ETOOBIG when the batch needs
 * more scratch than that (hx_cost_workspace_bytes(n_gpus, max_groups, n_cand) >
 * HX_STATIC_SCRATCH_BYTES; 18 bytes per group slot, n_cand * min(max_groups, n_gpus), at up to
 * 64 GPUs, so about 1.8 million slots: 65,536 candidates of 32 GPUs and 16 groups take 19.2 MB,
 * and 262,144 candidates of 64 GPUs and 32 groups are refused).  Every call on a GPU uses that GPU's one array: calls
 * that overlap on one GPU (two streams, two host threads) race and must be serialised by the
 * caller.  The scratch needs no clearing between calls.  The caller's device must be current. */
#define HX_STATIC_SCRATCH_BYTES (32u << 20)
int hx_cost_eval_static(const hx_cluster *cluster, hx_model model, hx_workload wl, hx_space space,
                        const hx_candidates *cand, const hx_cost_out *out, hipStream_t stream);
size_t hx_static_scratch_bytes(void);

/* 64-bit words per GPU bitmask: 1 for n_gpus <= 64, 2 for <= 128, 4 for <= 255. */
int hx_member_words(int32_t n_gpus);

/* Sec. 3.3 network and Appendix A edge capacities.  Node capacities come from cost->cap
 * (granularity 1: GPU k of a group of n GPUs with capacity C gets floor(C/n) + [k < C mod n],
 * k its rank by GPU id).  Source and sink edges carry floor(1000*coord_bw/req_bytes), or
 * HX_CAP_MAX when either is 0.  KV edge (connection type 3) of a prefill replica (tp_p x
 * pp_p) and a decode replica (tp_d x pp_d): over every pair of a prefill stage and a decode
 * stage sharing n > 0 layers and every rank pair (r, q) whose KV-head slices overlap by
 * ov = min((r+1)tp_d, (q+1)tp_p) - max(r tp_d, q tp_p) > 0, the link g -> h carries
 * bytes = ((V1*n)*ov)/(tp_p*tp_d) with V1 = (2*s_in)*H_kv*B, in alpha_{gh} + bytes/beta_{gh};
 * the KV time is the largest of these, and the edge capacity floor(1000/time) clamped to
 * HX_CAP_MAX, or 0 when either replica is infeasible.  Granularity 1: every edge counts
 * requests, so the edge from prefill GPU g to decode GPU h carries one request's whole KV cache
 * over the link g -> h: time alpha_{gh} + (V1*L)/beta_{gh} (the KV edge of two one-GPU
 * replicas on that link), whatever the replicas' sizes; 0 when either replica is infeasible.
 * With space.variant & HX_VARIANT_KV_ORDER (granularity 0), pipeline position a of a replica
 * may be served by any of its stages (stage s = the members ranked s*tp .. s*tp+tp-1): the
 * KV time is the minimum over every pair of stage orders of the two replicas (exact for
 * pipelines of up to 8 stages; with this variant a pp_mask bit past 8 is HX_EINVAL).  With request
 * classes (wl.n_classes > 0) the KV time is sum_k w_k t_k, t_k the time above with s_in =
 * cls_in[k] (left to right in class order), at either granularity. */
int hx_build_flownet(const hx_cluster *cluster, hx_model model, hx_workload wl, hx_space space,
                     const hx_candidates *cand, const hx_cost_out *cost, const hx_flownet *net,
                     hipStream_t stream);

/* Maximum source-sink flow of every candidate's network (Sec. 3.3, solved there by
 * preflow-push), by a synchronous push-relabel on the network with each replica's
 * in -> out chain contracted, one workgroup per candidate with the residual graph in LDS.
 * Closed forms skip push-relabel: networks where one side has a single node that can carry
 * flow (a star), and networks whose every KV edge can carry min(a_i, b_j) (a_i = min(source,
 * prefill node) and b_j = min(decode node, sink) capacities), whose maximum flow is
 * min(sum a, sum b) with the north-west-corner flow; when kv_flow and cut are both null,
 * networks whose smaller side has at most 6 nodes that can carry flow take the minimum cut
 * directly.  Every path gives the same (unique) flow value.
 *   flow_value [N]       the maximum flow (or HX_ENOCONV)
 *   kv_flow    [max_pd][N] nullable: one maximum flow's value on every KV edge (not unique)
 *   cut        [max_p + max_d][N] nullable: the canonical minimum cut, the nodes reachable from
 *              the source in the residual graph; row i < max_p is prefill node i, row max_p + j
 *              decode node j; bit 0 = its in-node, bit 1 = its out-node.  Unique for every max flow.
 * Returns HX_ETOOBIG when max_p, max_d or max_pd exceed the kernel's LDS plan. */
int hx_maxflow_batch(const hx_flownet *net, int32_t *flow_value, int32_t *kv_flow, uint8_t *cut,
                     hipStream_t stream);

/* Diagnostic (no counterpart in the paper): hx_maxflow_batch with the same arguments and
 * results, which also counts how each candidate was solved and the push-relabel work.
 * stats: device, 8-byte aligned, HX_MF_STATS uint64 words, cleared by the call then filled:
 *   [HX_MF_NO_FLOW .. HX_MF_PUSH_RELABEL]  candidates by path: no source- or sink-side node can
 *       carry flow; star closed form; dominant-KV closed form; direct minimum cut; push-relabel;
 *   [HX_MF_PREPASS]  value-only calls on the per-workgroup plans: candidates the lane-per-
 *       candidate pre-pass settled (they skip the kernel above);
 *   [HX_MF_PUSHES], [HX_MF_RELABELS]  pushes (KV, sink and return-to-source) and node relabels
 *       summed over all candidates;
 *   [HX_MF_GLOBAL_RELABELS], [HX_MF_ROUNDS]  global-relabel passes and synchronous rounds,
 *       counted once per workgroup (a packed plan's workgroup holds 64/SEG candidates).
 * Networks rejected with HX_EINVAL in flow_value are not counted.  Slower than
 * hx_maxflow_batch (global atomics); not for the search loop. */
#define HX_MF_NO_FLOW 0
#define HX_MF_STAR 1
#define HX_MF_DOMINANT 2
#define HX_MF_MIN_CUT 3
#define HX_MF_PUSH_RELABEL 4
#define HX_MF_PREPASS 5
#define HX_MF_PUSHES 6
#define HX_MF_RELABELS 7
#define HX_MF_GLOBAL_RELABELS 8
#define HX_MF_ROUNDS 9
#define HX_MF_STATS 10
int hx_maxflow_stats(const hx_flownet *net, int32_t *flow_value, int32_t *kv_flow, uint8_t *cut, uint64_t *stats,
                     hipStream_t stream);

/* The candidate with the highest flow_value (Sec. 3.1 objective), lowest index on ties.
 * best = device int32[2]: {index, value}.  n_cand >= 1. */
int hx_best_candidate(const int32_t *flow_value, int32_t n_cand, int32_t *best, hipStream_t stream);

/* The whole scoring path for a search loop that needs each candidate's flow value and the best
 * candidate but not a flow assignment (Sec. 3.1 objective, Sec. 3.3 network, Appendix A
 * capacities): hx_cost_eval, hx_build_flownet, hx_maxflow_batch with kv_flow and cut null, and
 * hx_best_candidate, enqueued by one call with the same arguments and errors, a workspace of
 * hx_score_workspace_bytes (the cost model's scratch; then a table of link capacities and a list
 * of candidates, or, for up to 32 group slots, the KV edge lists: a word per candidate marking
 * its nodes with a strategy and, twice, 4 bytes for each of its possible KV edges; then the
 * argmax's partial winners (one per workgroup, or one per slot that the max-flow kernel's
 * workgroups fold into); 256-byte aligned, contents ignored on entry), and the same results: every cost
 * output, the network's node counts (n_p, n_d), flow_value and best, bit for bit.  At
 * granularity 0, and beyond 128 GPUs or 128 group slots, every row of the network is written as
 * by hx_build_flownet (with up to 32 group slots the KV edges whose two replicas both have a
 * strategy are listed and walked apart from the others, which are written 0).  At
 * granularity 1 on clusters of up to 128 GPUs a KV edge's capacity depends only on its link,
 * so a network whose every KV edge can carry min(a_i, b_j) (the dominant-KV closed form: maximum flow min(sum a, sum b)) is settled from a table of link
 * capacities while its nodes are counted, and only the other networks get their node and KV rows
 * written and are solved by push-relabel; the rows of the settled networks are left as they
 * were. */
size_t hx_score_workspace_bytes(int32_t n_gpus, int32_t max_groups, int32_t n_cand);
int hx_score_batch(const hx_cluster *cluster, hx_model model, hx_workload wl, hx_space space,
                   const hx_candidates *cand, const hx_cost_out *cost, const hx_flownet *net, int32_t *flow_value,
                   int32_t *best, void *workspace, size_t workspace_bytes, hipStream_t stream);

/* ---------------------------------------------------------------- refinement (Sec. 3.4)
 * The refinement step compares each edge's flow with its capacity and swaps GPUs between groups
 * so that underutilized capacity relieves bottlenecks, then scores the new partitions again;
 * it stops when no new partition scores higher.  A flow assignment is not unique, so the edge
 * classes are taken in the form every maximum flow agrees on:
 *   bottleneck     raising the edge's capacity by one raises the maximum flow;
 *   underutilized  its capacity is >= 1 and lowering it by one keeps the maximum flow. */

/* Edge classes of every candidate's network, from one maximum flow of it (flow_value and
 * kv_flow as written by hx_maxflow_batch with kv_flow requested; node flows follow by
 * conservation).  One workgroup per candidate.
 *   node_cls [max_p + max_d][N]: row i < max_p prefill node i, row max_p + j decode node j;
 *            bit 0 / 1 = its node edge (in -> out) is a bottleneck / underutilized, bit 2 / 3 =
 *            the same for its coordinator edge (source -> in, out -> sink), bit 4 = a KV edge at
 *            the node is a bottleneck.
 *   kv_cls   [max_pd][N]: row i*n_d + j, bit 0 / 1 for the KV edge of prefill i and decode j.
 * Rows past a network's counts are not written.  A candidate with flow_value < 0, counts
 * outside the plan, or more than 255 nodes (n_p + n_d > 255: the closure's LDS rows) gets
 * node_cls 0 in every row and no kv_cls. */
int hx_edge_classes(const hx_flownet *net, const int32_t *flow_value, const int32_t *kv_flow, uint8_t *node_cls,
                    uint8_t *kv_cls, hipStream_t stream);

/* Guided moves: n_child children of the M = parents->n_cand (<= 65535) parent placements, whose network
 * (parent_net, built for this batch of M) and node classes (hx_edge_classes) are given.  Child c
 * descends from parent c mod M; children 0 .. M-1 are the parents unchanged (move 0), so a
 * scored batch's best is never worse than its parent.  Every other child applies one move:
 *   a GPU is a donor when it is unused, or the node edge of its flow node is underutilized
 *   (its flow node: its group's replica node, or its own node at granularity 1);
 *   a group is a receiver when a member's flow node has a bottleneck node edge or KV edge;
 *   a group may flip when it is no receiver, every member is a donor, and a receiver has the
 *   other role.
 *   MOVE (1)  a donor GPU outside the receiver joins a receiver group;
 *   SWAP (2)  a GPU of a receiver group and a donor GPU of another group (or unused) exchange
 *             their assign entries;
 *   FLIP (3)  a flip-eligible group takes the other role.
 * rnd[c] (uniform 64-bit draws, [n_child]) chooses: bits 0-15 the first type tried (u*3/2^16;
 * the next types in turn when it has no choice), bits 16-39 the receiver (MOVE: a receiver group,
 * SWAP: a GPU of a receiver group, FLIP: a flip-eligible group), bits 40-63 the donor GPU among
 * those allowed; each choice is entry floor(u*m/2^b) of the m candidates in ascending id.
 * A child with no possible move copies its parent (move 0).
 *   child_assign [n_gpus][n_child], child_role [max_groups][n_child]: written;
 *   move [n_child]: type | a << 8 | b << 16 (MOVE: GPU a, group b; SWAP: GPUs a, b; FLIP: group a). */
int hx_guided_moves(int32_t n_gpus, int32_t granularity, const hx_candidates *parents, const hx_flownet *parent_net,
                    const uint8_t *node_cls, int32_t n_child, const uint64_t *rnd, uint8_t *child_assign,
                    uint8_t *child_role, int32_t *move, hipStream_t stream);

/* dst column m = src column index[m] for m < count (index: device int32[count], e.g. the best
 * index of hx_best_candidate); an index outside [0, src->n_cand) gives a column of HX_UNUSED.
 *   dst_assign [n_gpus][count], dst_role [src->max_groups][count]. */
int hx_gather_candidates(int32_t n_gpus, const hx_candidates *src, const int32_t *index, int32_t count,
                         uint8_t *dst_assign, uint8_t *dst_role, hipStream_t stream);

/* ---------------------------------------------------------------- graph partition (Sec. 3.2)
 * The first phase of the scheduler as a candidate generator: the device graph (GPUs weighted by
 * memory, links by bandwidth) is partitioned into K groups (spectral order, then Kernighan-Lin
 * swaps), the groups are coarsened into super nodes and split into prefill and decode replicas
 * by a cut of maximum weight, and the partition is projected back onto the GPUs.  Edge weights
 * are w_de = floor(((beta_de + beta_ed) * 0.5) / 1e6) clamped to [0, 2^47] (whole MB/s; the
 * bound keeps every cut of up to 255 GPUs below 2^62), node weights the memory limits in whole
 * bytes, so cuts, gains and their sums are exact 64-bit integer sums. */

/* Device scratch both calls need (an [n_gpus][n_gpus] int64 weight table they fill first);
 * 0 for n_gpus outside [2, 255]. */
size_t hx_partition_workspace_bytes(int32_t n_gpus);

/* Spectral order: the GPUs sorted by (x_d, d), x the Fiedler direction of the Laplacian
 * Deg - w by `iters` power iterations on (c I - Lap), c = 2 max_d Deg_d, from x_d = d - (G-1)/2,
 * each iteration taking out the mean and normalising.  Every sum (a row's product, the mean,
 * the squared norm) runs in ascending index order.  One workgroup.
 *   order [n_gpus] device int32 out; fiedler [n_gpus] device double out, nullable. */
int hx_spectral_order(const hx_cluster *cluster, int32_t iters, void *workspace, size_t workspace_bytes,
                      int32_t *order, double *fiedler, hipStream_t stream);

/* n_cand candidates of the first phase, one per 64-bit draw rnd[n]:
 *   K = floor(total memory / (12 H^2 B L + 32 * (2 (s_in + s_out) H_kv B L))) (a replica holds the
 *       weights and the KV caches of 32 requests, Appendix A), plus (bits 0-2 mod 5) - 2,
 *       clamped to [2, min(n_gpus, max_groups, 32)];
 *   step (i): the spectral order rotated by (bits 3-10 mod n_gpus); the i-th GPU d of it goes to
 *       group min(K-1, floor(K (2 C_i + m_d) / (2 M))), C_i the memory before it, M the total;
 *       then Kernighan-Lin passes: with every GPU unlocked, repeatedly the swap of two unlocked
 *       GPUs of different groups that does not widen the memory gap between the two groups and
 *       has the largest cut reduction, negative or not (lowest (u, v) on ties), is made and both
 *       GPUs locked, until no such pair is left; the pass keeps its first k swaps, k the
 *       smallest with the largest summed reduction, when that sum is positive, and undoes the
 *       rest; passes repeat while one lowers the cut, at most 64;
 *   groups are numbered by smallest member;
 *   step (ii): super node k starts on side bit (11 + k) of the draw (the last one flipped if all
 *       agree); while flipping one super node raises the coarse cut with both sides occupied,
 *       the flip with the largest gain (lowest k on ties) is applied; side 0 = prefill;
 *   step (iii): assign[g][n] = the group of GPU g, role[k][n] = its side for k below the group
 *       count, HX_UNUSED beyond.
 *   order: the spectral order (hx_spectral_order).  One workgroup per candidate. */
int hx_partition_candidates(const hx_cluster *cluster, hx_model model, hx_workload wl, int32_t max_groups,
                            void *workspace, size_t workspace_bytes, const int32_t *order, int32_t n_cand,
                            const uint64_t *rnd, uint8_t *assign, uint8_t *role, hipStream_t stream);

/* Diagnostic per-kernel timing (not part of the scoring path; process-global, for one host
 * thread).  hx_profile(1) clears earlier records and makes every later launch by libhx record a
 * HIP event on the call's stream before and after each of its kernels; hx_profile(0) stops
 * recording.  hx_profile_read waits for the recorded events and fills ms[k] (total
 * milliseconds) and launches[k] for kernel k = 0 .. n-1 since the last hx_profile call, then
 * clears the records; n >= HX_KERNELS.  Returns HX_KERNELS or a negative error.  hx_kernel_name
 * gives kernel k's name: setup, decode, scatter, eval (hx_cost_eval), nodes, kv
 * (hx_build_flownet), maxflow, best, classes (hx_edge_classes), moves (hx_guided_moves),
 * gather (hx_gather_candidates), spectral (hx_spectral_order), partition
 * (hx_partition_candidates), shared (candidate 0's groups under HX_HINT_SHARED_GROUPS). */
#define HX_KERNELS 14
int hx_profile(int32_t enable);
int hx_profile_read(double *ms, int32_t *launches, int32_t n);
const char *hx_kernel_name(int32_t k);

/* Human-readable text of a return code, and the last HIP error message kept by HX_EHIP. */
const char *hx_strerror(int code);
const char *hx_last_error(void);
int hx_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* HX_H */
