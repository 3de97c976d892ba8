/*
 * hxo.c -- CPU oracle for batched placement scoring (HexGen-2, arXiv 2502.07903).
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow, obviously-correct reference
 * the HIP path is checked against.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg load it; the product path never does.  It shares
 * no code, header, table or helper with the HIP path.
 *
 * Per candidate placement it computes, in the paper's order:
 *   1. the Table 1 cost model of every admissible TP x PP strategy of every group
 *      (computation, TP and PP communication, memory limit), and the node
 *      capacity of Appendix A ("Node capacity estimation"): prefill T/latency at
 *      batch 1, decode b_max*T/latency; prefill keeps its latency-optimal
 *      strategy, decode its throughput-optimal one (Sec. 3.3, "Compute nodes");
 *   2. the KV-cache edge capacities (Table 1 last row; Sec. 3.3 "Network
 *      connections", connection type 3; Appendix A "Edge capacity estimation");
 *   3. the directed flow network of Sec. 3.3 with split in/out compute nodes;
 *   4. its maximum s-t flow.  The paper runs preflow-push; any exact algorithm
 *      reaches the same value (max-flow = min-cut), and this oracle uses
 *      Edmonds-Karp (shortest augmenting paths found by BFS);
 *   5. the best candidate (highest flow, lowest index on ties; Sec. 3.1, 3.4).
 *
 * Readings where the paper is silent or ambiguous (all listed in the design notes):
 *   - m_d is two inputs: memory bandwidth (decode weight scan) and memory limit.
 *   - KV-cache terms use the KV hidden size H*n_kv_heads/n_heads (grouped-query
 *     attention); every other term uses H.
 *   - Stage j of a (tp, pp) strategy holds the group's members ranked j*tp ..
 *     j*tp+tp-1 in ascending GPU id, and floor(L/pp) + [j < L mod pp] layers.
 *   - Prefill is evaluated at batch 1, decode at b_max, the largest batch the
 *     memory limit admits on every device: floor((M - A)/K) with A the weight term
 *     and K the per-request term of the memory row, clamped to 2^30.
 *   - Latency = sum over stages of (computation + TP) + sum of the PP terms.
 *   - Capacities are int32 milli-requests per second: x = 1000*b/latency,
 *     cap = min(2^24 - 1, floor(x)).
 *   - KV edge: for every pair of (prefill stage, decode stage) sharing n layers and
 *     every pair of ranks whose KV-head slices overlap by a fraction f, a link
 *     carries 2*s_in*H_kv*B*n*f bytes in alpha + bytes/beta; links run in
 *     parallel, so the KV time is the slowest link.  Per-GPU flow nodes use the
 *     per-GPU rule of hxo_kv_gpu_time(): a whole request's KV cache per unit of flow.
 *   - Source and sink edges are unbounded (2^24 - 1) unless a coordinator
 *     bandwidth and request size are given.
 *   - Request classes (length buckets, at most four, in place of the single mean
 *     task): a strategy must fit every class; a replica's latency is the mix's
 *     weighted mean, its capacity 1/(sum_k w_k/x_k) (the mix's time per request),
 *     its b_max the smallest; a KV edge's time is the weighted mean of the class
 *     times.  Not combined with the stage-order search or the asymmetric split.
 *
 * Floating point: IEEE-754 binary64, round to nearest, no contraction into FMA
 * (built with -ffp-contract=off, no fast-math), correctly rounded division, and
 * every expression evaluated left to right as written here.
 *
 * Parity pins: the cost model against hand-derived worked values and closed
 * forms, the memory limit against exact rational arithmetic, the max-flow against
 * brute-force min-cut enumeration and library solvers, and flow validity
 * (conservation, capacity, cut capacity) on every result.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define HXO_CAP_MAX 16777215          /* 2^24 - 1 milli-requests/s */
#define HXO_BMAX_CLAMP 1073741824.0   /* 2^30 */
#define HXO_UNUSED 0xFF
#define HXO_PREFILL 0
#define HXO_DECODE 1
#define HXO_MAX_TP 8
#define HXO_MAX_PP 32

typedef struct {
    int32_t n_gpus, n_types;
    const int32_t *gpu_type;
    const double *type_flops, *type_hbm_bw, *type_mem;
    const double *beta, *alpha;
    double coord_bw, req_bytes;
} hxo_cluster;

typedef struct { int32_t n_layers, hidden, n_heads, n_kv_heads, bytes_per_elem; } hxo_model;
/* The inference task t of Table 1: mean prompt and output lengths.  n_classes > 0: the requests
 * form classes (length buckets), class k with lengths cls_in[k], cls_out[k] and weight cls_w[k]
 * (its share of the requests); see hxo_group_select. */
#define HXO_MAX_CLASSES 4
typedef struct {
    double s_in, s_out;
    int32_t n_classes;
    double cls_in[HXO_MAX_CLASSES], cls_out[HXO_MAX_CLASSES], cls_w[HXO_MAX_CLASSES];
} hxo_workload;

/* the single task of class k */
static hxo_workload class_task(const hxo_workload *w, int k)
{
    hxo_workload t = *w;
    t.s_in = w->cls_in[k];
    t.s_out = w->cls_out[k];
    t.n_classes = 0;
    return t;
}
/* variant bit 0: pipelined decode capacity; bit 1: KV stage-order search; bit 2: asymmetric
 * layer split (all below) */
typedef struct { uint32_t tp_mask, pp_mask; int32_t granularity; uint32_t variant; } hxo_space;
#define HXO_VARIANT_PIPELINED 1u
#define HXO_VARIANT_KV_ORDER 2u  /* bit 1: KV stage-order search (hxo_kv_time_best) */
#define HXO_VARIANT_ASYM 4u      /* bit 2: asymmetric layer split (layer_split) */

/* Request classes are read with the as-written stage layout only: with the stage-order search
 * or the asymmetric split a class mix is refused (-1). */
static int classes_ok(const hxo_workload *w, uint32_t variant)
{
    if (w->n_classes < 0 || w->n_classes > HXO_MAX_CLASSES) return 0;
    if (w->n_classes > 0 && (variant & (HXO_VARIANT_KV_ORDER | HXO_VARIANT_ASYM))) return 0;
    return 1;
}

/* Variants the oracle reads: request classes as above, and the stage-order search on pipelines of
 * up to 8 stages (the PP mask past 8 is refused with it). */
static int space_ok(const hxo_workload *w, const hxo_space *sp)
{
    if (!classes_ok(w, sp->variant)) return 0;
    if ((sp->variant & HXO_VARIANT_KV_ORDER) && (sp->pp_mask >> 8)) return 0;
    return 1;
}

/* ------------------------------------------------------------------ helpers */

static double flops_of(const hxo_cluster *c, int d) { return c->type_flops[c->gpu_type[d]]; }
static double hbm_of(const hxo_cluster *c, int d) { return c->type_hbm_bw[c->gpu_type[d]]; }
static double memlim_of(const hxo_cluster *c, int d) { return c->type_mem[c->gpu_type[d]]; }
static double beta_of(const hxo_cluster *c, int d, int e) { return c->beta[(int64_t)d * c->n_gpus + e]; }
static double alpha_of(const hxo_cluster *c, int d, int e) { return c->alpha[(int64_t)d * c->n_gpus + e]; }

static double kv_hidden(const hxo_model *m)
{
    return (double)((int64_t)m->hidden * m->n_kv_heads / m->n_heads);
}

/* layers held by stage j of pp stages: uniform split, remainder to earlier stages */
static int stage_layers(int L, int pp, int j) { return L / pp + (j < L % pp ? 1 : 0); }

int32_t hxo_quantize(double x)
{
    if (!(x >= 0.0)) return 0;
    if (x >= (double)HXO_CAP_MAX) return HXO_CAP_MAX;
    return (int32_t)floor(x);
}

int32_t hxo_coord_cap(const hxo_cluster *c)
{
    if (c->coord_bw > 0.0 && c->req_bytes > 0.0) return hxo_quantize((1000.0 * c->coord_bw) / c->req_bytes);
    return HXO_CAP_MAX;
}

/* Layers of every stage of a (tp, pp) strategy of a group (members ascending).  As written: the
 * uniform split.  Variant HXO_VARIANT_ASYM (the asymmetric split of HexGen, whose cost model the
 * paper adopts; Table 1 leaves l_j open): every stage first takes one layer, the other L - pp
 * are shared in proportion to the stage's compute c_j (its slowest device's FLOP/s), each share
 * rounded down, f_j = floor(((L - pp) * c_j) / sum_k c_k) (the sum left to right), and the
 * layers left over go one each to the first stages: l_j = 1 + f_j + [j < L - pp - sum_k f_k].
 * Stages of one device type get the uniform split; no compute at all falls back to it. */
static void layer_split(const hxo_cluster *c, int L, const int32_t *members, int tp, int pp, uint32_t variant,
                        int *l)
{
    double cs[HXO_MAX_PP], C = 0.0;
    if (variant & HXO_VARIANT_ASYM) {
        for (int j = 0; j < pp; j++) {
            double mn = flops_of(c, members[j * tp]);
            for (int r = 1; r < tp; r++)
                if (flops_of(c, members[j * tp + r]) < mn) mn = flops_of(c, members[j * tp + r]);
            cs[j] = mn;
            C = C + mn;
        }
    }
    if (!(variant & HXO_VARIANT_ASYM) || !(C > 0.0)) {
        for (int j = 0; j < pp; j++) l[j] = stage_layers(L, pp, j);
        return;
    }
    const int base = L - pp;
    int F = 0;
    for (int j = 0; j < pp; j++) {
        l[j] = (int)floor(((double)base * cs[j]) / C);
        F += l[j];
    }
    for (int j = 0; j < pp; j++) l[j] = 1 + l[j] + (j < base - F ? 1 : 0);
}

int hxo_layer_split(const hxo_cluster *c, int32_t L, const int32_t *members, int32_t tp, int32_t pp,
                    uint32_t variant, int32_t *l)
{
    int tmp[HXO_MAX_PP];
    if (pp < 1 || pp > HXO_MAX_PP || pp > L) return -1;
    layer_split(c, L, members, tp, pp, variant, tmp);
    for (int j = 0; j < pp; j++) l[j] = tmp[j];
    return 0;
}

/* ------------------------------------------------------------------ Table 1 */

/* Memory limit row of Table 1 for the stage devices S (tp of them, l layers):
 * the largest batch b with (12H^2B/t + 2b(s_in+s_out)H_kv B/t) l + 4b(s_in+s_out)HB <= M_d
 * on every device d of the stage, written as floor((M_d - A)/K). */
static double stage_batch_limit(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w,
                                const int32_t *S, int tp, int l)
{
    const double H = m->hidden, Hkv = kv_hidden(m), B = m->bytes_per_elem;
    const double t = tp, ld = l;
    const double A = ((12.0 * H * H * B) / t) * ld;
    const double K = ((2.0 * (w->s_in + w->s_out) * Hkv * B) / t) * ld + 4.0 * (w->s_in + w->s_out) * H * B;
    double best = HXO_BMAX_CLAMP;
    for (int r = 0; r < tp; r++) {
        double q = (memlim_of(c, S[r]) - A) / K;
        double b = q >= HXO_BMAX_CLAMP ? HXO_BMAX_CLAMP : (q <= -HXO_BMAX_CLAMP ? -HXO_BMAX_CLAMP : floor(q));
        if (b < best) best = b;
    }
    return best;
}

/* Computation cost of one stage (Table 1 row 1). */
static double stage_compute(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w,
                            const int32_t *S, int tp, int l, int role, double b)
{
    const double H = m->hidden, B = m->bytes_per_elem, t = tp, ld = l;
    if (role == HXO_PREFILL) {
        double mx = 0.0;
        for (int r = 0; r < tp; r++) {
            double v = (24.0 * b * w->s_in * H * H) / (t * flops_of(c, S[r]));
            if (r == 0 || v > mx) mx = v;
        }
        return mx * ld;
    }
    double scan = 0.0, fl = 0.0;
    for (int r = 0; r < tp; r++) {
        double v = (12.0 * H * H * B * w->s_out) / (t * hbm_of(c, S[r]));
        if (r == 0 || v > scan) scan = v;
    }
    for (int r = 0; r < tp; r++) {
        double v = (24.0 * b * w->s_out * H * H) / (t * flops_of(c, S[r]));
        if (r == 0 || v > fl) fl = v;
    }
    return scan * ld + fl * ld;
}

/* TP communication cost of one stage (Table 1 row 2): the slowest device's sum over its peers. */
static double stage_tp_comm(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w,
                            const int32_t *S, int tp, int l, int role, double b)
{
    const double H = m->hidden, B = m->bytes_per_elem, t = tp, ld = l;
    const double X = role == HXO_PREFILL ? b * w->s_in * H * B : b * H * B;
    double mx = 0.0;
    for (int r = 0; r < tp; r++) {
        double sum = 0.0;
        for (int q = 0; q < tp; q++) {
            if (q == r) continue;
            sum = sum + (alpha_of(c, S[r], S[q]) + X / (t * beta_of(c, S[r], S[q])));
        }
        if (r == 0 || sum > mx) mx = sum;
    }
    if (role == HXO_PREFILL) return (mx * 4.0) * ld;
    return ((mx * 4.0) * w->s_out) * ld;
}

/* PP communication cost between consecutive stages S -> S2 (Table 1 row 3): the fastest pair. */
static double stage_pp_comm(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w,
                            const int32_t *S, const int32_t *S2, int tp, int role, double b)
{
    const double H = m->hidden, B = m->bytes_per_elem;
    const double X = role == HXO_PREFILL ? b * w->s_in * H * B : b * H * B;
    double mn = 0.0;
    int first = 1;
    for (int r = 0; r < tp; r++)
        for (int q = 0; q < tp; q++) {
            double v = alpha_of(c, S[r], S2[q]) + X / beta_of(c, S[r], S2[q]);
            if (first || v < mn) mn = v;
            first = 0;
        }
    if (role == HXO_PREFILL) return mn;
    return mn * w->s_out;
}

/* One strategy (tp, pp) of one group (members ascending, n = tp*pp of them).
 * Returns 1 if the memory limit admits a batch of at least 1, else 0.
 * Outputs b_max, the latency of one batch, and x = 1000*b/latency milli-requests/s.
 *
 * Variant HXO_VARIANT_PIPELINED (an alternative reading of Appendix A): the latency stays the
 * sum over stages, but a decode replica runs its stages as a pipeline, so batches leave it at
 * the pace of its slowest stage: x = 1000*b / max_j T_j with T_j = (comp_j + tp_j) + pp_j, the
 * PP term of the link into stage j+1 counted with stage j (none after the last stage).
 * Prefill capacity is unchanged (one request's latency). */
int hxo_strategy_cost_v(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w,
                        const int32_t *members, int32_t n, int32_t tp, int32_t pp, int32_t role, uint32_t variant,
                        int32_t *bmax_out, double *lat_out, double *x_out)
{
    const int L = m->n_layers;
    *bmax_out = 0; *lat_out = 0.0; *x_out = 0.0;
    if (tp < 1 || pp < 1 || tp * pp != n || pp > L) return 0;
    int lay[HXO_MAX_PP];
    layer_split(c, L, members, tp, pp, variant, lay);
    double bmax = HXO_BMAX_CLAMP;
    for (int j = 0; j < pp; j++) {
        double bj = stage_batch_limit(c, m, w, members + j * tp, tp, lay[j]);
        if (bj < bmax) bmax = bj;
    }
    *bmax_out = (int32_t)bmax;
    if (bmax < 1.0) return 0;
    const double b = role == HXO_PREFILL ? 1.0 : bmax;
    double s1 = 0.0, s2 = 0.0;
    for (int j = 0; j < pp; j++) {
        const int32_t *S = members + j * tp;
        const int l = lay[j];
        s1 = s1 + (stage_compute(c, m, w, S, tp, l, role, b) + stage_tp_comm(c, m, w, S, tp, l, role, b));
    }
    for (int j = 0; j + 1 < pp; j++)
        s2 = s2 + stage_pp_comm(c, m, w, members + j * tp, members + (j + 1) * tp, tp, role, b);
    const double lat = s1 + s2;
    *lat_out = lat;
    *x_out = (1000.0 * b) / lat;
    if ((variant & HXO_VARIANT_PIPELINED) && role == HXO_DECODE) {
        double slowest = 0.0;
        for (int j = 0; j < pp; j++) {
            const int32_t *S = members + j * tp;
            const int l = lay[j];
            double T = stage_compute(c, m, w, S, tp, l, role, b) + stage_tp_comm(c, m, w, S, tp, l, role, b);
            if (j + 1 < pp) T = T + stage_pp_comm(c, m, w, S, members + (j + 1) * tp, tp, role, b);
            if (T > slowest) slowest = T;
        }
        *x_out = (1000.0 * b) / slowest;
    }
    return 1;
}

int hxo_strategy_cost(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w,
                      const int32_t *members, int32_t n, int32_t tp, int32_t pp, int32_t role,
                      int32_t *bmax_out, double *lat_out, double *x_out)
{
    return hxo_strategy_cost_v(c, m, w, members, n, tp, pp, role, 0u, bmax_out, lat_out, x_out);
}

/* Try every admissible TP x PP of a group and keep prefill's latency-optimal and decode's
 * throughput-optimal strategy (ties keep the smaller tp).  No feasible strategy: all zero.
 *
 * Request classes (w->n_classes > 0; per-bucket workloads, an alternative to the single mean
 * task): a strategy is feasible when it is for every class; a replica serving the mix spends
 * tau = sum_k w_k / x_k per request (x_k its capacity on class k alone, the sum in class
 * order), so its capacity is x = 1 / tau; its latency is the mix's mean sum_k w_k lat_k and its
 * b_max the smallest over the classes.  Prefill keeps the lowest mix latency, decode the highest
 * x. */
int hxo_group_select(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w, const hxo_space *sp,
                     const int32_t *members, int32_t n, int32_t role,
                     int32_t *tp_out, int32_t *pp_out, int32_t *bmax_out, int32_t *cap_out, double *lat_out)
{
    int have = 0;
    double best_lat = 0.0, best_x = 0.0;
    *tp_out = 0; *pp_out = 0; *bmax_out = 0; *cap_out = 0; *lat_out = 0.0;
    for (int tp = 1; tp <= HXO_MAX_TP; tp++) {
        if (!((sp->tp_mask >> (tp - 1)) & 1u)) continue;
        if (n % tp != 0) continue;
        int pp = n / tp;
        if (pp > HXO_MAX_PP || !((sp->pp_mask >> (pp - 1)) & 1u) || pp > m->n_layers) continue;
        int32_t bmax;
        double lat, x;
        if (w->n_classes > 0) {
            int ok = 1;
            double tau = 0.0;
            lat = 0.0;
            bmax = 0;
            for (int k = 0; k < w->n_classes && ok; k++) {
                const hxo_workload tk = class_task(w, k);
                int32_t bk;
                double lk, xk;
                ok = hxo_strategy_cost_v(c, m, &tk, members, n, tp, pp, role, sp->variant, &bk, &lk, &xk);
                if (!ok) break;
                lat = lat + w->cls_w[k] * lk;
                tau = tau + w->cls_w[k] / xk;
                if (k == 0 || bk < bmax) bmax = bk;
            }
            if (!ok) continue;
            x = 1.0 / tau;
        } else if (!hxo_strategy_cost_v(c, m, w, members, n, tp, pp, role, sp->variant, &bmax, &lat, &x)) {
            continue;
        }
        int better = !have || (role == HXO_PREFILL ? lat < best_lat : x > best_x);
        if (better) {
            have = 1; best_lat = lat; best_x = x;
            *tp_out = tp; *pp_out = pp; *bmax_out = bmax; *cap_out = hxo_quantize(x); *lat_out = lat;
        }
    }
    return have;
}

/* KV-cache transfer time of one request from a prefill replica (members pm, ptp x ppp) to a
 * decode replica (dm, dtp x dpp): every GPU holding layer j's KV heads sends them to the
 * GPUs holding the same layer and heads on the decode side; the slowest link decides. */
/* The same with an explicit stage order: the prefill replica's stage ord_p[a] (its members
 * ranked ord_p[a]*ptp .. +ptp-1) serves pipeline position a, which holds the layers of position
 * a; likewise ord_d on the decode side. */
/* lp / ld (nullable): the layers held by each pipeline position; the uniform split when null. */
static double kv_time_ordered(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w,
                              const int32_t *pm, int ptp, int ppp, const int *ord_p,
                              const int32_t *dm, int dtp, int dpp, const int *ord_d, const int *lp, const int *ld)
{
    const int L = m->n_layers;
    const double V1 = 2.0 * w->s_in * kv_hidden(m) * (double)m->bytes_per_elem;
    double worst = 0.0;
    int a0 = 0;
    for (int a = 0; a < ppp; a++) {
        const int a1 = a0 + (lp ? lp[a] : stage_layers(L, ppp, a));
        int b0 = 0;
        for (int bb = 0; bb < dpp; bb++) {
            const int b1 = b0 + (ld ? ld[bb] : stage_layers(L, dpp, bb));
            const int nab = (a1 < b1 ? a1 : b1) - (a0 > b0 ? a0 : b0);
            for (int r = 0; r < ptp && nab > 0; r++)
                for (int q = 0; q < dtp; q++) {
                    int hi = (r + 1) * dtp < (q + 1) * ptp ? (r + 1) * dtp : (q + 1) * ptp;
                    int lo = r * dtp > q * ptp ? r * dtp : q * ptp;
                    int ov = hi - lo;
                    if (ov <= 0) continue;
                    int g = pm[ord_p[a] * ptp + r], h = dm[ord_d[bb] * dtp + q];
                    double bytes = ((V1 * (double)nab) * (double)ov) / (double)(ptp * dtp);
                    double time = alpha_of(c, g, h) + bytes / beta_of(c, g, h);
                    if (time > worst) worst = time;
                }
            b0 = b1;
        }
        a0 = a1;
    }
    return worst;
}

double hxo_kv_time(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w,
                   const int32_t *pm, int32_t ptp, int32_t ppp, const int32_t *dm, int32_t dtp, int32_t dpp)
{
    int op[HXO_MAX_PP], od[HXO_MAX_PP];
    for (int a = 0; a < ppp; a++) op[a] = a;
    for (int b = 0; b < dpp; b++) od[b] = b;
    return kv_time_ordered(c, m, w, pm, ptp, ppp, op, dm, dtp, dpp, od, NULL, NULL);
}

/* next permutation of v[0..n) in lexicographic order; returns 0 after the last one */
static int next_order(int *v, int n)
{
    int i = n - 2;
    while (i >= 0 && v[i] >= v[i + 1]) i--;
    if (i < 0) return 0;
    int j = n - 1;
    while (v[j] <= v[i]) j--;
    int t = v[i]; v[i] = v[j]; v[j] = t;
    for (int a = i + 1, b = n - 1; a < b; a++, b--) { t = v[a]; v[a] = v[b]; v[b] = t; }
    return 1;
}

/* KV time with explicit stage orders (ord_p[a]: the prefill stage serving pipeline position a;
 * ord_d likewise), the uniform layer split. */
double hxo_kv_time_orders(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w,
                          const int32_t *pm, int32_t ptp, int32_t ppp, const int32_t *ord_p,
                          const int32_t *dm, int32_t dtp, int32_t dpp, const int32_t *ord_d)
{
    int op[HXO_MAX_PP], od[HXO_MAX_PP];
    for (int a = 0; a < ppp; a++) op[a] = ord_p[a];
    for (int b = 0; b < dpp; b++) od[b] = ord_d[b];
    return kv_time_ordered(c, m, w, pm, ptp, ppp, op, dm, dtp, dpp, od, NULL, NULL);
}

/* Slowest link between prefill stage s and decode stage t when they serve pipeline positions
 * sharing nab > 0 layers: the link times kv_time_ordered visits for that pair of positions. */
static double kv_block_time(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w,
                            const int32_t *pm, int ptp, int s, const int32_t *dm, int dtp, int t, int nab)
{
    const double V1 = 2.0 * w->s_in * kv_hidden(m) * (double)m->bytes_per_elem;
    double worst = 0.0;
    for (int r = 0; r < ptp; r++)
        for (int q = 0; q < dtp; q++) {
            int hi = (r + 1) * dtp < (q + 1) * ptp ? (r + 1) * dtp : (q + 1) * ptp;
            int lo = r * dtp > q * ptp ? r * dtp : q * ptp;
            int ov = hi - lo;
            if (ov <= 0) continue;
            int g = pm[s * ptp + r], h = dm[t * dtp + q];
            double bytes = ((V1 * (double)nab) * (double)ov) / (double)(ptp * dtp);
            double time = alpha_of(c, g, h) + bytes / beta_of(c, g, h);
            if (time > worst) worst = time;
        }
    return worst;
}

/* Kuhn's augmenting path from row i over the entries of C (n x n) that are <= T. */
static int kuhn_augment(const double *C, int n, double T, int i, int *row_of_col, int *seen)
{
    for (int j = 0; j < n; j++) {
        if (C[i * n + j] > T || seen[j]) continue;
        seen[j] = 1;
        if (row_of_col[j] < 0 || kuhn_augment(C, n, T, row_of_col[j], row_of_col, seen)) {
            row_of_col[j] = i;
            return 1;
        }
    }
    return 0;
}

static int perfect_matching_below(const double *C, int n, double T)
{
    int row_of_col[HXO_MAX_PP], seen[HXO_MAX_PP];
    for (int j = 0; j < n; j++) row_of_col[j] = -1;
    for (int i = 0; i < n; i++) {
        for (int j = 0; j < n; j++) seen[j] = 0;
        if (!kuhn_augment(C, n, T, i, row_of_col, seen)) return 0;
    }
    return 1;
}

/* Linear bottleneck assignment: the smallest over permutations pi of max_i C[i][pi(i)].  The
 * value is one of C's entries, so the entries are tried in ascending order and the first one
 * whose entries <= it admit a perfect matching is the answer. */
static double bottleneck_assignment(const double *C, int n)
{
    double v[HXO_MAX_PP * HXO_MAX_PP];
    const int k = n * n;
    for (int i = 0; i < k; i++) v[i] = C[i];
    for (int i = 1; i < k; i++) {  /* insertion sort */
        double x = v[i];
        int j = i - 1;
        while (j >= 0 && v[j] > x) { v[j + 1] = v[j]; j--; }
        v[j + 1] = x;
    }
    for (int i = 0; i < k; i++) {
        if (i > 0 && v[i] == v[i - 1]) continue;
        if (perfect_matching_below(C, n, v[i])) return v[i];
    }
    return v[k - 1];
}

/* Stage-order search (Appendix A, "Edge capacity estimation": the pipeline stage order of both
 * replicas is adjusted to minimise the KV cache communication cost, which sets the edge
 * capacity): the smallest KV time over every pair of stage orders.  Node capacities keep the
 * ascending order.
 *
 * The KV time of an order pair is the largest block time over the pairs of pipeline positions
 * that share layers (a block: the slowest link between the stages serving the two positions).
 * Fix the order of one side X; each position y of the other side Y then contributes
 * C[y][t] = max over the X positions sharing layers with y of the block time, when Y's stage t
 * serves y, and the KV time is max_y C[y][ord_Y(y)].  So the best Y order for a fixed X order
 * is a bottleneck assignment of C, and the minimum over both orders is the minimum over the X
 * orders of that assignment's value: every order pair is covered, none is visited one by one.
 * X is the pipeline with fewer stages (prefill on ties); its orders are enumerated in
 * lexicographic order (at most 8! = 40,320). */
double hxo_kv_time_best(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w,
                        const int32_t *pm, int32_t ptp, int32_t ppp, const int32_t *dm, int32_t dtp, int32_t dpp)
{
    const int L = m->n_layers;
    const int swap = dpp < ppp;  /* X = decode when it has fewer stages */
    const int nx = swap ? dpp : ppp, ny = swap ? ppp : dpp;
    int xb[HXO_MAX_PP + 1], yb[HXO_MAX_PP + 1];  /* layer boundaries of the positions */
    xb[0] = yb[0] = 0;
    for (int a = 0; a < nx; a++) xb[a + 1] = xb[a] + stage_layers(L, nx, a);
    for (int b = 0; b < ny; b++) yb[b + 1] = yb[b] + stage_layers(L, ny, b);
    /* blk[((xa * nx + xs) * ny + y) * ny + yt]: X position xa served by X stage xs, Y position y by
     * Y stage yt; -1 where the two positions share no layer */
    double *blk = (double *)malloc(sizeof(double) * nx * nx * ny * ny);
    for (int xa = 0; xa < nx; xa++)
        for (int y = 0; y < ny; y++) {
            const int lo = xb[xa] > yb[y] ? xb[xa] : yb[y];
            const int hi = xb[xa + 1] < yb[y + 1] ? xb[xa + 1] : yb[y + 1];
            for (int xs = 0; xs < nx; xs++)
                for (int yt = 0; yt < ny; yt++) {
                    double v = -1.0;
                    if (hi > lo)
                        v = swap ? kv_block_time(c, m, w, pm, ptp, yt, dm, dtp, xs, hi - lo)
                                 : kv_block_time(c, m, w, pm, ptp, xs, dm, dtp, yt, hi - lo);
                    blk[((xa * nx + xs) * ny + y) * ny + yt] = v;
                }
        }
    int ord[HXO_MAX_PP];
    double C[HXO_MAX_PP * HXO_MAX_PP];
    for (int a = 0; a < nx; a++) ord[a] = a;
    double best = -1.0;
    do {
        for (int y = 0; y < ny; y++)
            for (int yt = 0; yt < ny; yt++) {
                double v = 0.0;
                for (int xa = 0; xa < nx; xa++) {
                    const double b = blk[((xa * nx + ord[xa]) * ny + y) * ny + yt];
                    if (b > v) v = b;
                }
                C[y * ny + yt] = v;
            }
        const double t = bottleneck_assignment(C, ny);
        if (best < 0.0 || t < best) best = t;
    } while (next_order(ord, nx));
    free(blk);
    return best;
}

/* Per-GPU flow nodes (a refinement of the Sec. 3.3 network that the paper does not draw): every
 * edge of the network counts requests, and a GPU node carries its share of its replica's
 * requests, so a unit of flow on the KV edge from prefill GPU g to decode GPU h is one request
 * whose whole KV cache (2 s_in H_kv B bytes per layer, all L layers) crosses the link g -> h.
 * The time is that of a KV edge between two one-GPU replicas on the same link (one stage pair
 * sharing all L layers, one rank pair overlapping fully), whatever the replicas' sizes. */
double hxo_kv_gpu_time(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w, int32_t g, int32_t h)
{
    const double V1 = 2.0 * w->s_in * kv_hidden(m) * (double)m->bytes_per_elem;
    const double bytes = V1 * (double)m->n_layers;
    return alpha_of(c, g, h) + bytes / beta_of(c, g, h);
}

/* ------------------------------------------------------------------ batch cost model */

typedef struct {
    const hxo_cluster *c; const hxo_model *m; const hxo_workload *w; const hxo_space *sp;
    int32_t n_cand, max_groups;
    const uint8_t *assign, *role;
} hxo_batch;

/* members of group k of candidate n, ascending GPU id; returns the count */
static int group_members(const hxo_batch *bt, int n, int k, int32_t *out)
{
    int cnt = 0;
    for (int g = 0; g < bt->c->n_gpus; g++)
        if (bt->assign[(int64_t)g * bt->n_cand + n] == k) out[cnt++] = g;
    return cnt;
}

static int group_role(const hxo_batch *bt, int n, int k)
{
    return bt->role[(int64_t)k * bt->n_cand + n];
}

static void cost_range(const hxo_batch *bt, int n0, int n1, uint8_t *tp, uint8_t *pp, int32_t *bmax,
                       int32_t *cap, double *lat)
{
    int32_t *mem = (int32_t *)malloc(sizeof(int32_t) * (bt->c->n_gpus + 1));
    for (int n = n0; n < n1; n++)
        for (int k = 0; k < bt->max_groups; k++) {
            int64_t o = (int64_t)k * bt->n_cand + n;
            int r = group_role(bt, n, k);
            int cnt = group_members(bt, n, k, mem);
            int32_t t = 0, p = 0, b = 0, cp = 0;
            double l = 0.0;
            if (cnt > 0 && (r == HXO_PREFILL || r == HXO_DECODE))
                hxo_group_select(bt->c, bt->m, bt->w, bt->sp, mem, cnt, r, &t, &p, &b, &cp, &l);
            tp[o] = (uint8_t)t; pp[o] = (uint8_t)p; bmax[o] = b; cap[o] = cp; lat[o] = l;
        }
    free(mem);
}

int hxo_cost_eval(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w, const hxo_space *sp,
                  int32_t n_cand, int32_t max_groups, const uint8_t *assign, const uint8_t *role,
                  uint8_t *tp, uint8_t *pp, int32_t *bmax, int32_t *cap, double *lat)
{
    if (!space_ok(w, sp)) return -1;
    hxo_batch bt = {c, m, w, sp, n_cand, max_groups, assign, role};
    cost_range(&bt, 0, n_cand, tp, pp, bmax, cap, lat);
    return 0;
}

/* ------------------------------------------------------------------ flow network */

typedef struct {
    int32_t max_p, max_d, max_pd;
    int32_t *n_p, *n_d, *p_slot, *d_slot, *src_cap, *p_cap, *kv_cap, *d_cap, *sink_cap;
} hxo_flownet;

static void flownet_range(const hxo_batch *bt, int n0, int n1, const uint8_t *tp, const uint8_t *pp,
                          const int32_t *cap, const hxo_flownet *f)
{
    const hxo_cluster *c = bt->c;
    const int N = bt->n_cand, G = c->n_gpus, Kmax = bt->max_groups;
    int32_t *pm = (int32_t *)malloc(sizeof(int32_t) * (G + 1));
    int32_t *dm = (int32_t *)malloc(sizeof(int32_t) * (G + 1));
    int32_t *pnode = (int32_t *)malloc(sizeof(int32_t) * (G + Kmax + 1));
    int32_t *dnode = (int32_t *)malloc(sizeof(int32_t) * (G + Kmax + 1));
    const int32_t cc = hxo_coord_cap(c);
    for (int n = n0; n < n1; n++) {
        int np = 0, nd = 0;
        if (bt->sp->granularity == 0) {
            for (int k = 0; k < Kmax; k++) {
                int r = group_role(bt, n, k);
                if (group_members(bt, n, k, pm) == 0) continue;
                if (r == HXO_PREFILL) pnode[np++] = k;
                else if (r == HXO_DECODE) dnode[nd++] = k;
            }
        } else {
            for (int g = 0; g < G; g++) {
                int k = bt->assign[(int64_t)g * N + n];
                if (k >= Kmax) continue;
                int r = group_role(bt, n, k);
                if (r == HXO_PREFILL) pnode[np++] = g;
                else if (r == HXO_DECODE) dnode[nd++] = g;
            }
        }
        f->n_p[n] = np; f->n_d[n] = nd;
        for (int i = 0; i < f->max_p; i++) {
            int64_t o = (int64_t)i * N + n;
            f->p_slot[o] = -1; f->src_cap[o] = 0; f->p_cap[o] = 0;
        }
        for (int j = 0; j < f->max_d; j++) {
            int64_t o = (int64_t)j * N + n;
            f->d_slot[o] = -1; f->d_cap[o] = 0; f->sink_cap[o] = 0;
        }
        for (int e = 0; e < f->max_pd; e++) f->kv_cap[(int64_t)e * N + n] = 0;

        if (bt->sp->granularity == 0) {
            for (int i = 0; i < np; i++) {
                int64_t o = (int64_t)i * N + n, go = (int64_t)pnode[i] * N + n;
                f->p_slot[o] = pnode[i]; f->src_cap[o] = cc; f->p_cap[o] = cap[go];
            }
            for (int j = 0; j < nd; j++) {
                int64_t o = (int64_t)j * N + n, go = (int64_t)dnode[j] * N + n;
                f->d_slot[o] = dnode[j]; f->d_cap[o] = cap[go]; f->sink_cap[o] = cc;
            }
            for (int i = 0; i < np; i++) {
                int64_t gp = (int64_t)pnode[i] * N + n;
                int pn = group_members(bt, n, pnode[i], pm);
                for (int j = 0; j < nd; j++) {
                    int64_t gd = (int64_t)dnode[j] * N + n;
                    int dn = group_members(bt, n, dnode[j], dm);
                    int32_t kv = 0;
                    (void)pn; (void)dn;
                    if (tp[gp] > 0 && tp[gd] > 0) {
                        double t;
                        if (bt->w->n_classes > 0) {
                            /* request classes: the mix's mean KV time (weights in class order) */
                            t = 0.0;
                            for (int k = 0; k < bt->w->n_classes; k++) {
                                const hxo_workload tk = class_task(bt->w, k);
                                t = t + bt->w->cls_w[k] * hxo_kv_time(c, bt->m, &tk, pm, tp[gp], pp[gp], dm, tp[gd], pp[gd]);
                            }
                        } else if (bt->sp->variant & HXO_VARIANT_ASYM) {
                            /* each replica's layers follow its own (asymmetric) split */
                            int lp[HXO_MAX_PP], ld[HXO_MAX_PP], op[HXO_MAX_PP], od[HXO_MAX_PP];
                            layer_split(c, bt->m->n_layers, pm, tp[gp], pp[gp], bt->sp->variant, lp);
                            layer_split(c, bt->m->n_layers, dm, tp[gd], pp[gd], bt->sp->variant, ld);
                            for (int x = 0; x < pp[gp]; x++) op[x] = x;
                            for (int x = 0; x < pp[gd]; x++) od[x] = x;
                            t = kv_time_ordered(c, bt->m, bt->w, pm, tp[gp], pp[gp], op, dm, tp[gd], pp[gd], od, lp, ld);
                        } else if (bt->sp->variant & HXO_VARIANT_KV_ORDER) {
                            t = hxo_kv_time_best(c, bt->m, bt->w, pm, tp[gp], pp[gp], dm, tp[gd], pp[gd]);
                        } else {
                            t = hxo_kv_time(c, bt->m, bt->w, pm, tp[gp], pp[gp], dm, tp[gd], pp[gd]);
                        }
                        kv = hxo_quantize(1000.0 / t);
                    }
                    f->kv_cap[(int64_t)(i * nd + j) * N + n] = kv;
                }
            }
        } else {
            /* per-GPU nodes: a GPU's node capacity is its equal share of its replica's capacity */
            for (int side = 0; side < 2; side++) {
                int cnt = side == 0 ? np : nd;
                int32_t *node = side == 0 ? pnode : dnode;
                for (int i = 0; i < cnt; i++) {
                    int g = node[i];
                    int k = bt->assign[(int64_t)g * N + n];
                    int64_t go = (int64_t)k * N + n;
                    int sz = group_members(bt, n, k, pm);
                    int rank = 0;
                    while (pm[rank] != g) rank++;
                    int32_t C = cap[go];
                    int32_t share = C / sz + (rank < C % sz ? 1 : 0);
                    int64_t o = (int64_t)i * N + n;
                    if (side == 0) { f->p_slot[o] = g; f->src_cap[o] = cc; f->p_cap[o] = share; }
                    else { f->d_slot[o] = g; f->d_cap[o] = share; f->sink_cap[o] = cc; }
                }
            }
            for (int i = 0; i < np; i++) {
                int g = pnode[i];
                int kp = bt->assign[(int64_t)g * N + n];
                for (int j = 0; j < nd; j++) {
                    int h = dnode[j];
                    int kd = bt->assign[(int64_t)h * N + n];
                    int32_t kv = 0;
                    if (tp[(int64_t)kp * N + n] > 0 && tp[(int64_t)kd * N + n] > 0) {
                        double t;
                        if (bt->w->n_classes > 0) {
                            t = 0.0;
                            for (int k = 0; k < bt->w->n_classes; k++) {
                                const hxo_workload tk = class_task(bt->w, k);
                                t = t + bt->w->cls_w[k] * hxo_kv_gpu_time(c, bt->m, &tk, g, h);
                            }
                        } else {
                            t = hxo_kv_gpu_time(c, bt->m, bt->w, g, h);
                        }
                        kv = hxo_quantize(1000.0 / t);
                    }
                    f->kv_cap[(int64_t)(i * nd + j) * N + n] = kv;
                }
            }
        }
    }
    free(pm); free(dm); free(pnode); free(dnode);
}

int hxo_build_flownet(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w, const hxo_space *sp,
                      int32_t n_cand, int32_t max_groups, const uint8_t *assign, const uint8_t *role,
                      const uint8_t *tp, const uint8_t *pp, const int32_t *cap,
                      int32_t max_p, int32_t max_d, int32_t max_pd,
                      int32_t *n_p, int32_t *n_d, int32_t *p_slot, int32_t *d_slot,
                      int32_t *src_cap, int32_t *p_cap, int32_t *kv_cap, int32_t *d_cap, int32_t *sink_cap)
{
    if (!space_ok(w, sp)) return -1;
    hxo_batch bt = {c, m, w, sp, n_cand, max_groups, assign, role};
    hxo_flownet f = {max_p, max_d, max_pd, n_p, n_d, p_slot, d_slot, src_cap, p_cap, kv_cap, d_cap, sink_cap};
    flownet_range(&bt, 0, n_cand, tp, pp, cap, &f);
    return 0;
}

/* ------------------------------------------------------------------ max-flow (Edmonds-Karp) */

typedef struct {
    int nv, na;
    int *head, *next, *to;
    int64_t *res;
    int *parent_arc, *queue;
} ek_graph;

static void ek_init(ek_graph *g, int nv, int max_edges)
{
    g->nv = nv; g->na = 0;
    g->head = (int *)malloc(sizeof(int) * nv);
    g->next = (int *)malloc(sizeof(int) * 2 * max_edges);
    g->to = (int *)malloc(sizeof(int) * 2 * max_edges);
    g->res = (int64_t *)malloc(sizeof(int64_t) * 2 * max_edges);
    g->parent_arc = (int *)malloc(sizeof(int) * nv);
    g->queue = (int *)malloc(sizeof(int) * nv);
    for (int v = 0; v < nv; v++) g->head[v] = -1;
}

static void ek_free(ek_graph *g)
{
    free(g->head); free(g->next); free(g->to); free(g->res); free(g->parent_arc); free(g->queue);
}

/* adds edge u->v with capacity cap as arc pair (2e forward, 2e+1 reverse); returns e */
static int ek_add(ek_graph *g, int u, int v, int64_t cap)
{
    int a = g->na;
    g->to[a] = v; g->res[a] = cap; g->next[a] = g->head[u]; g->head[u] = a;
    g->to[a + 1] = u; g->res[a + 1] = 0; g->next[a + 1] = g->head[v]; g->head[v] = a + 1;
    g->na += 2;
    return a / 2;
}

/* BFS over arcs with residual > 0 from s; fills parent_arc (-1 unreached, -2 for s) */
static void ek_bfs(ek_graph *g, int s)
{
    for (int v = 0; v < g->nv; v++) g->parent_arc[v] = -1;
    g->parent_arc[s] = -2;
    int qh = 0, qt = 0;
    g->queue[qt++] = s;
    while (qh < qt) {
        int u = g->queue[qh++];
        for (int a = g->head[u]; a >= 0; a = g->next[a])
            if (g->res[a] > 0 && g->parent_arc[g->to[a]] == -1) {
                g->parent_arc[g->to[a]] = a;
                g->queue[qt++] = g->to[a];
            }
    }
}

static int64_t ek_run(ek_graph *g, int s, int t)
{
    int64_t total = 0;
    for (;;) {
        ek_bfs(g, s);
        if (g->parent_arc[t] == -1) break;
        int64_t aug = INT64_MAX;
        for (int v = t; v != s; v = g->to[g->parent_arc[v] ^ 1])
            if (g->res[g->parent_arc[v]] < aug) aug = g->res[g->parent_arc[v]];
        for (int v = t; v != s; v = g->to[g->parent_arc[v] ^ 1]) {
            g->res[g->parent_arc[v]] -= aug;
            g->res[g->parent_arc[v] ^ 1] += aug;
        }
        total += aug;
    }
    return total;
}

/* Max s-t flow of an explicit edge list; flow[e] receives edge e's flow, reach[v] (nullable)
 * is 1 for the vertices reachable from s in the final residual graph. */
int64_t hxo_maxflow_edges(int32_t nv, int32_t ne, const int32_t *from, const int32_t *to, const int64_t *cap,
                          int32_t s, int32_t t, int64_t *flow, uint8_t *reach)
{
    ek_graph g;
    ek_init(&g, nv, ne > 0 ? ne : 1);
    for (int e = 0; e < ne; e++) ek_add(&g, from[e], to[e], cap[e]);
    int64_t v = ek_run(&g, s, t);
    for (int e = 0; e < ne; e++) flow[e] = g.res[2 * e + 1];
    if (reach) {
        ek_bfs(&g, s);
        for (int u = 0; u < nv; u++) reach[u] = g.parent_arc[u] != -1;
    }
    ek_free(&g);
    return v;
}

typedef struct {
    int32_t n_cand, max_p, max_d, max_pd;
    const int32_t *n_p, *n_d, *src_cap, *p_cap, *kv_cap, *d_cap, *sink_cap;
    int32_t *flow_value, *kv_flow;
    uint8_t *cut;
} hxo_mf;

/* The Sec. 3.3 network of candidate n: s=0, t=1, prefill replica i as in 2+2i -> out 3+2i,
 * decode replica j as in 2+2P+2j -> out 3+2P+2j; edges s->phi_in, phi_in->phi_out,
 * phi_out->delta_in (every pair), delta_in->delta_out, delta_out->t. */
static void maxflow_range(const hxo_mf *q, int n0, int n1)
{
    const int N = q->n_cand;
    const int maxv = 2 + 2 * (q->max_p + q->max_d);
    const int maxe = q->max_p * 2 + q->max_d * 2 + q->max_pd;
    int32_t *from = (int32_t *)malloc(sizeof(int32_t) * (maxe + 1));
    int32_t *to = (int32_t *)malloc(sizeof(int32_t) * (maxe + 1));
    int64_t *cp = (int64_t *)malloc(sizeof(int64_t) * (maxe + 1));
    int64_t *fl = (int64_t *)malloc(sizeof(int64_t) * (maxe + 1));
    uint8_t *reach = (uint8_t *)malloc(maxv);
    for (int n = n0; n < n1; n++) {
        const int P = q->n_p[n], D = q->n_d[n];
        int ne = 0;
        for (int i = 0; i < P; i++) {
            int64_t o = (int64_t)i * N + n;
            from[ne] = 0; to[ne] = 2 + 2 * i; cp[ne++] = q->src_cap[o];
            from[ne] = 2 + 2 * i; to[ne] = 3 + 2 * i; cp[ne++] = q->p_cap[o];
        }
        const int kv0 = ne;
        for (int i = 0; i < P; i++)
            for (int j = 0; j < D; j++) {
                from[ne] = 3 + 2 * i; to[ne] = 2 + 2 * P + 2 * j;
                cp[ne++] = q->kv_cap[(int64_t)(i * D + j) * N + n];
            }
        for (int j = 0; j < D; j++) {
            int64_t o = (int64_t)j * N + n;
            from[ne] = 2 + 2 * P + 2 * j; to[ne] = 3 + 2 * P + 2 * j; cp[ne++] = q->d_cap[o];
            from[ne] = 3 + 2 * P + 2 * j; to[ne] = 1; cp[ne++] = q->sink_cap[o];
        }
        int64_t v = hxo_maxflow_edges(2 + 2 * (P + D), ne, from, to, cp, 0, 1, fl, reach);
        q->flow_value[n] = (int32_t)v;
        if (q->kv_flow) {
            for (int e = 0; e < q->max_pd; e++) q->kv_flow[(int64_t)e * N + n] = 0;
            for (int e = 0; e < P * D; e++) q->kv_flow[(int64_t)e * N + n] = (int32_t)fl[kv0 + e];
        }
        if (q->cut) {
            for (int i = 0; i < q->max_p + q->max_d; i++) q->cut[(int64_t)i * N + n] = 0;
            for (int i = 0; i < P; i++)
                q->cut[(int64_t)i * N + n] = (uint8_t)(reach[2 + 2 * i] | (reach[3 + 2 * i] << 1));
            for (int j = 0; j < D; j++)
                q->cut[(int64_t)(q->max_p + j) * N + n] =
                    (uint8_t)(reach[2 + 2 * P + 2 * j] | (reach[3 + 2 * P + 2 * j] << 1));
        }
    }
    free(from); free(to); free(cp); free(fl); free(reach);
}

int hxo_maxflow_batch(int32_t n_cand, int32_t max_p, int32_t max_d, int32_t max_pd,
                      const int32_t *n_p, const int32_t *n_d, const int32_t *src_cap, const int32_t *p_cap,
                      const int32_t *kv_cap, const int32_t *d_cap, const int32_t *sink_cap,
                      int32_t *flow_value, int32_t *kv_flow, uint8_t *cut)
{
    hxo_mf q = {n_cand, max_p, max_d, max_pd, n_p, n_d, src_cap, p_cap, kv_cap, d_cap, sink_cap,
                flow_value, kv_flow, cut};
    maxflow_range(&q, 0, n_cand);
    return 0;
}

/* ------------------------------------------------------------------ argmax */

int hxo_best_candidate(const int32_t *flow_value, int32_t n_cand, int32_t *best)
{
    if (n_cand <= 0) return -1;
    int32_t bi = 0, bv = flow_value[0];
    for (int32_t n = 1; n < n_cand; n++)
        if (flow_value[n] > bv) { bv = flow_value[n]; bi = n; }
    best[0] = bi; best[1] = bv;
    return 0;
}

/* ------------------------------------------------------------------ whole batch, threaded */

typedef struct {
    const hxo_batch *bt;
    hxo_flownet f;
    uint8_t *tp, *pp;
    int32_t *bmax, *cap;
    double *lat;
    int32_t *flow_value;
    int n0, n1;
} hxo_job;

static void *score_worker(void *arg)
{
    hxo_job *j = (hxo_job *)arg;
    cost_range(j->bt, j->n0, j->n1, j->tp, j->pp, j->bmax, j->cap, j->lat);
    flownet_range(j->bt, j->n0, j->n1, j->tp, j->pp, j->cap, &j->f);
    hxo_mf q = {j->bt->n_cand, j->f.max_p, j->f.max_d, j->f.max_pd, j->f.n_p, j->f.n_d, j->f.src_cap,
                j->f.p_cap, j->f.kv_cap, j->f.d_cap, j->f.sink_cap, j->flow_value, NULL, NULL};
    maxflow_range(&q, j->n0, j->n1);
    return NULL;
}

/* Scores candidates [0, n_cand) end to end on n_threads host threads (all buffers caller
 * owned, same layouts as the individual calls) and writes the best (index, value). */
int hxo_score_batch(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w, const hxo_space *sp,
                    int32_t n_cand, int32_t max_groups, const uint8_t *assign, const uint8_t *role,
                    uint8_t *tp, uint8_t *pp, int32_t *bmax, int32_t *cap, double *lat,
                    int32_t max_p, int32_t max_d, int32_t max_pd,
                    int32_t *n_p, int32_t *n_d, int32_t *p_slot, int32_t *d_slot,
                    int32_t *src_cap, int32_t *p_cap, int32_t *kv_cap, int32_t *d_cap, int32_t *sink_cap,
                    int32_t *flow_value, int32_t *best, int32_t n_threads)
{
    if (!space_ok(w, sp)) return -1;
    hxo_batch bt = {c, m, w, sp, n_cand, max_groups, assign, role};
    hxo_flownet f = {max_p, max_d, max_pd, n_p, n_d, p_slot, d_slot, src_cap, p_cap, kv_cap, d_cap, sink_cap};
    if (n_threads < 1) n_threads = 1;
    if (n_threads > n_cand) n_threads = n_cand > 0 ? n_cand : 1;
    hxo_job *jobs = (hxo_job *)calloc(n_threads, sizeof(hxo_job));
    pthread_t *th = (pthread_t *)calloc(n_threads, sizeof(pthread_t));
    for (int i = 0; i < n_threads; i++) {
        jobs[i].bt = &bt; jobs[i].f = f;
        jobs[i].tp = tp; jobs[i].pp = pp; jobs[i].bmax = bmax; jobs[i].cap = cap; jobs[i].lat = lat;
        jobs[i].flow_value = flow_value;
        jobs[i].n0 = (int)((int64_t)n_cand * i / n_threads);
        jobs[i].n1 = (int)((int64_t)n_cand * (i + 1) / n_threads);
    }
    for (int i = 1; i < n_threads; i++) pthread_create(&th[i], NULL, score_worker, &jobs[i]);
    score_worker(&jobs[0]);
    for (int i = 1; i < n_threads; i++) pthread_join(th[i], NULL);
    free(jobs); free(th);
    return hxo_best_candidate(flow_value, n_cand, best);
}

/* ------------------------------------------------------------------ refinement (Sec. 3.4) */

/*
 * Max-flow guided refinement (Sec. 3.4).  The paper compares every edge's flow with its
 * capacity: a bottleneck edge carries flow at its capacity and holds the total back, an
 * underutilized edge carries less than it could; GPUs are then swapped between groups to
 * relieve the one with the other, the new partition is scored again, and the loop stops when
 * nothing improves.  A maximum flow assignment is not unique, so the two properties are taken
 * here in the form every maximum flow agrees on (the same for any solver):
 *   bottleneck     raising the edge's capacity by one raises the maximum flow;
 *   underutilized  the capacity is >= 1 and lowering it by one keeps the maximum flow.
 * For an edge u -> v with flow f of capacity c in one maximum flow, in that flow's residual
 * graph (arc u -> v when f < c, arc v -> u when f > 0):
 *   bottleneck     iff s reaches u and v reaches t (the extra unit is the only way through);
 *   underutilized  iff c >= 1 and (f < c, or u reaches v: the residual cycle through v -> u
 *                  moves one unit off the edge without changing the value).
 */

/* reach[u * nv + v] = 1 when v is reachable from u in the residual graph of the flow fl on
 * the edge list (from, to, cp); every vertex reaches itself. */
static void residual_reach(int nv, int ne, const int32_t *from, const int32_t *to, const int64_t *cp,
                           const int64_t *fl, uint8_t *reach)
{
    int *queue = (int *)malloc(sizeof(int) * nv);
    memset(reach, 0, (size_t)nv * nv);
    for (int src = 0; src < nv; src++) {
        uint8_t *seen = reach + (size_t)src * nv;
        int qh = 0, qt = 0;
        seen[src] = 1;
        queue[qt++] = src;
        while (qh < qt) {
            int u = queue[qh++];
            for (int e = 0; e < ne; e++) {
                int w = -1;
                if (from[e] == u && fl[e] < cp[e]) w = to[e];
                else if (to[e] == u && fl[e] > 0) w = from[e];
                if (w >= 0 && !seen[w]) { seen[w] = 1; queue[qt++] = w; }
            }
        }
    }
    free(queue);
}

static uint8_t edge_class(int nv, const uint8_t *reach, int s, int t, int u, int v, int64_t f, int64_t c)
{
    uint8_t k = 0;
    if (reach[(size_t)s * nv + u] && reach[(size_t)v * nv + t]) k |= 1;
    if (c >= 1 && (f < c || reach[(size_t)u * nv + v])) k |= 2;
    return k;
}

/* Edge classes of every candidate's Sec. 3.3 network (same layout as hxo_maxflow_batch's
 * inputs).  node_cls[i][n] for prefill node i, node_cls[max_p + j][n] for decode node j:
 * bit 0 / bit 1 = the node edge (in -> out) is a bottleneck / underutilized, bit 2 / bit 3 =
 * the same for its coordinator edge (source -> in, resp. out -> sink), bit 4 = a KV edge at the
 * node is a bottleneck.  kv_cls[i*n_d + j][n]: bit 0 / bit 1 for the KV edge of prefill i and
 * decode j.  Rows past the counts are left. */
int hxo_edge_classes(int32_t n_cand, int32_t max_p, int32_t max_d, int32_t max_pd,
                     const int32_t *n_p, const int32_t *n_d, const int32_t *src_cap, const int32_t *p_cap,
                     const int32_t *kv_cap, const int32_t *d_cap, const int32_t *sink_cap,
                     uint8_t *node_cls, uint8_t *kv_cls)
{
    const int N = n_cand;
    const int maxv = 2 + 2 * (max_p + max_d);
    const int maxe = max_p * 2 + max_d * 2 + max_pd;
    int32_t *from = (int32_t *)malloc(sizeof(int32_t) * (maxe + 1));
    int32_t *to = (int32_t *)malloc(sizeof(int32_t) * (maxe + 1));
    int64_t *cp = (int64_t *)malloc(sizeof(int64_t) * (maxe + 1));
    int64_t *fl = (int64_t *)malloc(sizeof(int64_t) * (maxe + 1));
    uint8_t *reach = (uint8_t *)malloc((size_t)maxv * maxv);
    for (int n = 0; n < N; n++) {
        const int P = n_p[n], D = n_d[n];
        const int nv = 2 + 2 * (P + D);
        int ne = 0;
        /* the same vertex and edge numbering as the max-flow above */
        for (int i = 0; i < P; i++) {
            int64_t o = (int64_t)i * N + n;
            from[ne] = 0; to[ne] = 2 + 2 * i; cp[ne++] = src_cap[o];
            from[ne] = 2 + 2 * i; to[ne] = 3 + 2 * i; cp[ne++] = p_cap[o];
        }
        const int kv0 = ne;
        for (int i = 0; i < P; i++)
            for (int j = 0; j < D; j++) {
                from[ne] = 3 + 2 * i; to[ne] = 2 + 2 * P + 2 * j;
                cp[ne++] = kv_cap[(int64_t)(i * D + j) * N + n];
            }
        const int d0 = ne;
        for (int j = 0; j < D; j++) {
            int64_t o = (int64_t)j * N + n;
            from[ne] = 2 + 2 * P + 2 * j; to[ne] = 3 + 2 * P + 2 * j; cp[ne++] = d_cap[o];
            from[ne] = 3 + 2 * P + 2 * j; to[ne] = 1; cp[ne++] = sink_cap[o];
        }
        hxo_maxflow_edges(nv, ne, from, to, cp, 0, 1, fl, NULL);
        residual_reach(nv, ne, from, to, cp, fl, reach);
        for (int i = 0; i < P; i++) {
            const int es = 2 * i, en = 2 * i + 1;
            uint8_t k = edge_class(nv, reach, 0, 1, from[en], to[en], fl[en], cp[en]);
            k |= (uint8_t)(edge_class(nv, reach, 0, 1, from[es], to[es], fl[es], cp[es]) << 2);
            node_cls[(int64_t)i * N + n] = k;
        }
        for (int j = 0; j < D; j++) {
            const int en = d0 + 2 * j, et = d0 + 2 * j + 1;
            uint8_t k = edge_class(nv, reach, 0, 1, from[en], to[en], fl[en], cp[en]);
            k |= (uint8_t)(edge_class(nv, reach, 0, 1, from[et], to[et], fl[et], cp[et]) << 2);
            node_cls[(int64_t)(max_p + j) * N + n] = k;
        }
        for (int e = 0; e < P * D; e++) {
            const uint8_t k = edge_class(nv, reach, 0, 1, from[kv0 + e], to[kv0 + e], fl[kv0 + e], cp[kv0 + e]);
            kv_cls[(int64_t)e * N + n] = k;
            if (k & 1) {
                node_cls[(int64_t)(e / D) * N + n] |= 16;
                node_cls[(int64_t)(max_p + e % D) * N + n] |= 16;
            }
        }
    }
    free(from); free(to); free(cp); free(fl); free(reach);
    return 0;
}

/* Index into a list of m entries from a b-bit uniform draw u: floor(u * m / 2^b). */
static int pick_index(uint64_t u, int m, int bits) { return (int)((u * (uint64_t)m) >> bits); }

/*
 * Guided moves (Sec. 3.4): the children of a batch of parent placements.  Child c descends
 * from parent c mod n_par; children 0 .. n_par-1 are the parents themselves, so the best
 * child of a batch is never worse than its parent and a batch whose best is a parent has
 * found no improvement.  Every other child applies one move, read from the parent's edge
 * classes (hxo_edge_classes of the parent's own network):
 *   a GPU is a donor when it is unused or the node edge of its flow node is underutilized;
 *   a group is a receiver when the node edge of one of its members' flow nodes, or a KV
 *   edge at one of them, is a bottleneck;
 *   a group may flip its role when it is no receiver, all its members are donors, and some
 *   receiver has the other role.
 * (A member's flow node is its group's replica node, or at per-GPU granularity its own.)
 *   MOVE  a donor GPU outside the receiver joins a receiver group;
 *   SWAP  a GPU of a receiver group and a donor GPU of another group (or unused) trade places;
 *   FLIP  a flip-eligible group takes the other role.
 * Random draws come from rnd[c]: bits 0-15 choose the first move type tried (MOVE, SWAP,
 * FLIP in turn after it, the first that has a choice is applied), bits 16-39 the receiver
 * (MOVE: a receiver group; SWAP: a GPU of any receiver group; FLIP: a flip-eligible group),
 * bits 40-63 the donor GPU among those allowed; each choice is the floor(u*m/2^b)-th of the
 * m candidates in ascending id.  move[c] = type | a << 8 | b << 16: 0 none, 1 MOVE (a GPU,
 * b group), 2 SWAP (a, b GPUs), 3 FLIP (a group).
 */
int hxo_guided_moves(int32_t n_gpus, int32_t max_groups, int32_t granularity,
                     int32_t n_par, const uint8_t *p_assign, const uint8_t *p_role,
                     int32_t max_p, const int32_t *n_p, const int32_t *n_d,
                     const int32_t *p_slot, const int32_t *d_slot, const uint8_t *node_cls, const uint8_t *kv_cls,
                     int32_t n_child, const uint64_t *rnd, uint8_t *c_assign, uint8_t *c_role, int32_t *move)
{
    const int G = n_gpus, K = max_groups, M = n_par;
    int grp[256], node_row[256], donor[256], recv_grp[256], flip_ok[256], members[256];
    int recv_list[256], donor_list[256], recv_gpu_list[256], flip_list[256];
    for (int c = 0; c < n_child; c++) {
        const int m = c % M;
        for (int g = 0; g < G; g++) c_assign[(int64_t)g * n_child + c] = p_assign[(int64_t)g * M + m];
        for (int k = 0; k < K; k++) c_role[(int64_t)k * n_child + c] = p_role[(int64_t)k * M + m];
        move[c] = 0;
        if (c < M) continue;

        /* the parent's groups: a GPU belongs to group a = assign when a < K has a valid role */
        for (int k = 0; k < K; k++) members[k] = 0;
        for (int g = 0; g < G; g++) {
            const int a = p_assign[(int64_t)g * M + m];
            const int r = a < K ? p_role[(int64_t)a * M + m] : HXO_UNUSED;
            grp[g] = (a < K && (r == HXO_PREFILL || r == HXO_DECODE)) ? a : -1;
            if (grp[g] >= 0) members[grp[g]]++;
        }
        /* flow node of each GPU: the row of its node in the parent's network (prefill i ->
         * row i, decode j -> row max_p + j), or -1 */
        const int P = n_p[m], D = n_d[m];
        for (int g = 0; g < G; g++) {
            node_row[g] = -1;
            if (grp[g] < 0) continue;
            const int key = granularity == 0 ? grp[g] : g;
            const int r = p_role[(int64_t)grp[g] * M + m];
            if (r == HXO_PREFILL) {
                for (int i = 0; i < P; i++)
                    if (p_slot[(int64_t)i * M + m] == key) node_row[g] = i;
            } else {
                for (int j = 0; j < D; j++)
                    if (d_slot[(int64_t)j * M + m] == key) node_row[g] = max_p + j;
            }
        }
        /* donors and receivers */
        for (int k = 0; k < K; k++) recv_grp[k] = 0;
        for (int g = 0; g < G; g++) {
            donor[g] = grp[g] < 0;
            if (node_row[g] < 0) continue;
            const int row = node_row[g];
            const uint8_t nc = node_cls[(int64_t)row * M + m];
            if (nc & 2) donor[g] = 1;
            int bott = nc & 1;
            if (row < max_p) {
                for (int j = 0; j < D; j++)
                    if (kv_cls[(int64_t)(row * D + j) * M + m] & 1) bott = 1;
            } else {
                for (int i = 0; i < P; i++)
                    if (kv_cls[(int64_t)(i * D + (row - max_p)) * M + m] & 1) bott = 1;
            }
            if (bott) recv_grp[grp[g]] = 1;
        }
        int recv_role_seen[2] = {0, 0};
        for (int k = 0; k < K; k++)
            if (recv_grp[k]) recv_role_seen[p_role[(int64_t)k * M + m]] = 1;
        for (int k = 0; k < K; k++) flip_ok[k] = members[k] > 0 && !recv_grp[k];
        for (int g = 0; g < G; g++)
            if (grp[g] >= 0 && !donor[g]) flip_ok[grp[g]] = 0;
        for (int k = 0; k < K; k++)
            if (flip_ok[k] && !recv_role_seen[1 - p_role[(int64_t)k * M + m]]) flip_ok[k] = 0;
        int n_recv = 0, n_donor = 0, n_rg = 0, n_flip = 0;
        for (int k = 0; k < K; k++) {
            if (recv_grp[k]) recv_list[n_recv++] = k;
            if (flip_ok[k]) flip_list[n_flip++] = k;
        }
        for (int g = 0; g < G; g++) {
            if (donor[g]) donor_list[n_donor++] = g;
            if (grp[g] >= 0 && recv_grp[grp[g]]) recv_gpu_list[n_rg++] = g;
        }

        const uint64_t r = rnd[c];
        const uint64_t u0 = r & 0xFFFF, u1 = (r >> 16) & 0xFFFFFF, u2 = r >> 40;
        const int t0 = pick_index(u0, 3, 16);
        for (int attempt = 0; attempt < 3 && move[c] == 0; attempt++) {
            const int t = (t0 + attempt) % 3;
            if (t == 0 && n_recv > 0) {
                const int k = recv_list[pick_index(u1, n_recv, 24)];
                int allowed[256], na = 0;
                for (int x = 0; x < n_donor; x++)
                    if (grp[donor_list[x]] != k) allowed[na++] = donor_list[x];
                if (na == 0) continue;
                const int g = allowed[pick_index(u2, na, 24)];
                c_assign[(int64_t)g * n_child + c] = (uint8_t)k;
                move[c] = 1 | (g << 8) | (k << 16);
            } else if (t == 1 && n_rg > 0) {
                const int g = recv_gpu_list[pick_index(u1, n_rg, 24)];
                int allowed[256], na = 0;
                for (int x = 0; x < n_donor; x++)
                    if (grp[donor_list[x]] != grp[g]) allowed[na++] = donor_list[x];
                if (na == 0) continue;
                const int h = allowed[pick_index(u2, na, 24)];
                const uint8_t ag = p_assign[(int64_t)g * M + m], ah = p_assign[(int64_t)h * M + m];
                c_assign[(int64_t)g * n_child + c] = ah;
                c_assign[(int64_t)h * n_child + c] = ag;
                move[c] = 2 | (g << 8) | (h << 16);
            } else if (t == 2 && n_flip > 0) {
                const int k = flip_list[pick_index(u1, n_flip, 24)];
                c_role[(int64_t)k * n_child + c] = (uint8_t)(1 - p_role[(int64_t)k * M + m]);
                move[c] = 3 | (k << 8);
            }
        }
    }
    return 0;
}

/* ------------------------------------------------------------------ graph partition (Sec. 3.2) */

/*
 * The first phase of the scheduler (Sec. 3.2) as a candidate generator.  The device graph has
 * the GPUs as nodes, weighted by their memory limits, and the links as edges, weighted by
 * bandwidth.  Readings (the paper names the methods, not their parameters):
 *   - edge weight w_de = floor(((beta_de + beta_ed) * 0.5) / 1e6), clamped to [0, 2^47]: the
 *     symmetrised bandwidth in whole MB/s, so that every cut and gain below is an exact integer
 *     sum; the bound (1.4e20 bytes/s, far beyond any link) keeps every cut of a graph of up to
 *     255 GPUs below 2^62, so cuts, gains and sums of gains are exact 64-bit integers; node
 *     weight = the memory limit in whole bytes;
 *   - Step (i), initial partition: spectral order by the Fiedler direction of the Laplacian
 *     Deg - w (power iteration, hxo_spectral_order), cut into K contiguous groups of balanced
 *     memory; K = floor(total memory / replica memory), a replica holding the weights and the
 *     KV caches of 32 requests (Appendix A: 12 H^2 B L + 32 * 2 (s_in + s_out) H_kv B L);
 *     then Kernighan-Lin passes (hxo_kl_refine): tentative pair swaps on unlocked GPUs, each
 *     the admissible swap of largest cut reduction even when it is negative, then the best
 *     prefix of the pass kept; passes repeat while one lowers the cut;
 *   - Step (ii), coarsen and secondary partition: groups become super nodes joined by the
 *     summed weights of their links; a local search for a maximum cut splits them into
 *     prefill and decode replicas (single flips with the largest gain, both sides kept);
 *   - Step (iii), projection: every GPU takes its group; groups are numbered by smallest member.
 * Candidates of one batch differ by a 64-bit draw each: bits 0-2 shift K by (v mod 5) - 2,
 * bits 3-10 rotate the spectral order by (v mod G), bits 11-42 set the initial side of super
 * node k (bit 11 + k).
 */

/* whole MB/s of the symmetrised bandwidth, clamped to [0, 2^47] */
#define HXO_PG_WEIGHT_MAX 140737488355328.0  /* 2^47 */
static int64_t pg_weight(const hxo_cluster *c, int d, int e)
{
    if (d == e) return 0;
    double v = floor(((beta_of(c, d, e) + beta_of(c, e, d)) * 0.5) / 1.0e6);
    if (!(v >= 0.0)) v = 0.0;
    if (v > HXO_PG_WEIGHT_MAX) v = HXO_PG_WEIGHT_MAX;
    return (int64_t)v;
}

/* Spectral order: iters power iterations on (cap I - Lap), Lap = Deg - w, cap = 2 max_d Deg_d,
 * from x_d = d - (G-1)/2, each iteration removing the mean (the constant eigenvector) and
 * normalising; every sum (a row's product, the mean, the squared norm) runs in ascending index
 * order.  order = GPUs sorted by (x_d, d); fiedler (nullable) receives x. */
int hxo_spectral_order(const hxo_cluster *c, int32_t iters, int32_t *order, double *fiedler)
{
    const int G = c->n_gpus;
    double *x = (double *)malloc(sizeof(double) * G), *y = (double *)malloc(sizeof(double) * G);
    double *deg = (double *)malloc(sizeof(double) * G), *sq = (double *)malloc(sizeof(double) * G);
    double cap = 0.0;
    for (int d = 0; d < G; d++) {
        int64_t s = 0;
        for (int e = 0; e < G; e++) s += pg_weight(c, d, e);
        deg[d] = (double)s;
        if (2.0 * deg[d] > cap) cap = 2.0 * deg[d];
    }
    for (int d = 0; d < G; d++) x[d] = (double)d - (double)(G - 1) * 0.5;
    for (int it = 0; it < iters; it++) {
        for (int d = 0; d < G; d++) {
            double s = 0.0;
            for (int e = 0; e < G; e++) s = s + (double)pg_weight(c, d, e) * x[e];
            y[d] = (cap - deg[d]) * x[d] + s;
        }
        double tot = 0.0;
        for (int d = 0; d < G; d++) tot = tot + y[d];
        const double mean = tot / (double)G;
        for (int d = 0; d < G; d++) {
            y[d] = y[d] - mean;
            sq[d] = y[d] * y[d];
        }
        double ss = 0.0;
        for (int d = 0; d < G; d++) ss = ss + sq[d];
        const double nrm = sqrt(ss);
        if (!(nrm > 0.0)) break;
        for (int d = 0; d < G; d++) x[d] = y[d] / nrm;
    }
    for (int d = 0; d < G; d++) order[d] = d;
    for (int i = 1; i < G; i++) {  /* insertion sort by (x, id) */
        int v = order[i], j = i - 1;
        while (j >= 0 && (x[order[j]] > x[v] || (x[order[j]] == x[v] && order[j] > v))) {
            order[j + 1] = order[j];
            j--;
        }
        order[j + 1] = v;
    }
    if (fiedler)
        for (int d = 0; d < G; d++) fiedler[d] = x[d];
    free(x); free(y); free(deg); free(sq);
    return 0;
}

/* K of the initial partition before the per-candidate shift. */
int32_t hxo_partition_groups(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w)
{
    const double H = m->hidden, Hkv = kv_hidden(m), B = m->bytes_per_elem, L = m->n_layers;
    double total = 0.0;
    for (int d = 0; d < c->n_gpus; d++) total = total + (double)(int64_t)memlim_of(c, d);
    const double rep = 12.0 * H * H * B * L + 32.0 * (2.0 * (w->s_in + w->s_out) * Hkv * B * L);
    return (int32_t)floor(total / rep);
}

static int64_t iabs64(int64_t v) { return v < 0 ? -v : v; }

/* Cut reduction of exchanging GPUs u and v of different groups: u's links into v's group and
 * v's links into u's group stop being cut, their links into their own groups start being cut,
 * and the link u-v stays cut. */
static int64_t kl_swap_gain(const hxo_cluster *c, const int *grp, int u, int v)
{
    const int A = grp[u], B = grp[v];
    int64_t gain = 0;
    for (int x = 0; x < c->n_gpus; x++) {
        if (x == u || x == v) continue;
        if (grp[x] == B) gain += pg_weight(c, u, x);
        if (grp[x] == A) gain -= pg_weight(c, u, x);
        if (grp[x] == A) gain += pg_weight(c, v, x);
        if (grp[x] == B) gain -= pg_weight(c, v, x);
    }
    return gain;
}

/* A swap may not widen the memory gap between the two groups ("balances node weights"). */
static int kl_balanced(const int64_t *gmem, const int64_t *mem, int A, int B, int u, int v)
{
    const int64_t gap0 = iabs64(gmem[A] - gmem[B]);
    const int64_t gap1 = iabs64((gmem[A] - mem[u] + mem[v]) - (gmem[B] - mem[v] + mem[u]));
    return gap1 <= gap0;
}

static void kl_exchange(int *grp, int64_t *gmem, const int64_t *mem, int u, int v)
{
    const int A = grp[u], B = grp[v];
    gmem[A] += mem[v] - mem[u];
    gmem[B] += mem[u] - mem[v];
    grp[u] = B;
    grp[v] = A;
}

/* Kernighan-Lin refinement of a partition of the GPUs into groups 0..K-1 (Sec. 3.2 step (i);
 * Kernighan and Lin's pass structure, with the pair swaps taken between any two groups).
 * A pass unlocks every GPU, then repeatedly takes, among the pairs of unlocked GPUs in
 * different groups whose swap keeps the memory balance, the one with the largest cut reduction
 * (possibly negative; lowest (u, v) on ties), exchanges them tentatively and locks both, until
 * no pair is left.  With S_k the summed reduction of the first k swaps, the pass keeps the
 * first k* swaps, k* the smallest k with the largest S_k, when S_k* > 0, and undoes the rest;
 * otherwise it undoes every swap and the refinement stops.  At most HXO_KL_PASSES passes.
 * Returns the number of passes that lowered the cut. */
#define HXO_KL_PASSES 64
int hxo_kl_refine(const hxo_cluster *c, int32_t *grp32)
{
    const int G = c->n_gpus;
    int *grp = (int *)malloc(sizeof(int) * G), *locked = (int *)malloc(sizeof(int) * G);
    int *su = (int *)malloc(sizeof(int) * G), *sv = (int *)malloc(sizeof(int) * G);
    int64_t *mem = (int64_t *)malloc(sizeof(int64_t) * G), *gmem = (int64_t *)malloc(sizeof(int64_t) * 256);
    int passes = 0;
    for (int d = 0; d < G; d++) {
        grp[d] = grp32[d];
        mem[d] = (int64_t)memlim_of(c, d);
    }
    for (int k = 0; k < 256; k++) gmem[k] = 0;
    for (int d = 0; d < G; d++) gmem[grp[d]] += mem[d];
    for (; passes < HXO_KL_PASSES; passes++) {
        for (int d = 0; d < G; d++) locked[d] = 0;
        int n_swaps = 0, kbest = 0;
        int64_t run = 0, best = 0;
        for (;;) {
            int bu = -1, bv = -1;
            int64_t bg = 0;
            for (int u = 0; u < G; u++)
                for (int v = u + 1; v < G; v++) {
                    if (locked[u] || locked[v] || grp[u] == grp[v]) continue;
                    if (!kl_balanced(gmem, mem, grp[u], grp[v], u, v)) continue;
                    const int64_t g = kl_swap_gain(c, grp, u, v);
                    if (bu < 0 || g > bg) { bg = g; bu = u; bv = v; }
                }
            if (bu < 0) break;
            kl_exchange(grp, gmem, mem, bu, bv);
            locked[bu] = locked[bv] = 1;
            su[n_swaps] = bu; sv[n_swaps] = bv; n_swaps++;
            run += bg;
            if (run > best) { best = run; kbest = n_swaps; }
        }
        /* undo the swaps past the best prefix, last first */
        for (int i = n_swaps - 1; i >= kbest; i--) kl_exchange(grp, gmem, mem, su[i], sv[i]);
        if (kbest == 0) break;
    }
    for (int d = 0; d < G; d++) grp32[d] = grp[d];
    free(grp); free(locked); free(su); free(sv); free(mem); free(gmem);
    return passes;
}

int hxo_partition_candidates(const hxo_cluster *c, const hxo_model *m, const hxo_workload *w,
                             const int32_t *order, int32_t max_groups, int32_t n_cand, const uint64_t *rnd,
                             uint8_t *assign, uint8_t *role)
{
    const int G = c->n_gpus;
    int kmax = max_groups < G ? max_groups : G;
    if (kmax > 32) kmax = 32;
    const int32_t k_est = hxo_partition_groups(c, m, w);
    int64_t *mem = (int64_t *)malloc(sizeof(int64_t) * G);
    int64_t total = 0;
    for (int d = 0; d < G; d++) {
        mem[d] = (int64_t)memlim_of(c, d);
        total += mem[d];
    }
    if (total <= 0) total = 1;  /* no memory anywhere: every GPU falls in group 0 */
    int32_t *grp = (int32_t *)malloc(sizeof(int32_t) * G);
    int64_t *sw = (int64_t *)malloc(sizeof(int64_t) * 32 * 32);
    for (int n = 0; n < n_cand; n++) {
        const uint64_t r = rnd[n];
        int K = k_est + (int)((r & 7) % 5) - 2;
        if (K > kmax) K = kmax;
        if (K < 2) K = 2;
        const int rot = (int)(((r >> 3) & 0xFF) % (uint64_t)G);
        /* step (i): balanced contiguous cut of the rotated spectral order, by memory midpoints */
        int64_t cum = 0;
        for (int i = 0; i < G; i++) {
            const int d = order[(i + rot) % G];
            int k = (int)(((int64_t)K * (2 * cum + mem[d])) / (2 * total));
            grp[d] = k < K - 1 ? k : K - 1;
            cum += mem[d];
        }
        hxo_kl_refine(c, grp);
        /* step (iii) numbering: groups by smallest member */
        int map[256], used = 0;
        for (int k = 0; k < 256; k++) map[k] = -1;
        for (int d = 0; d < G; d++)
            if (map[grp[d]] < 0) map[grp[d]] = used++;
        for (int d = 0; d < G; d++) grp[d] = map[grp[d]];
        /* step (ii): coarsened weights and the max-cut split */
        for (int k = 0; k < used * used; k++) sw[k] = 0;
        for (int d = 0; d < G; d++)
            for (int e = 0; e < G; e++)
                if (grp[d] != grp[e]) sw[grp[d] * used + grp[e]] += pg_weight(c, d, e);
        int side[32], n1 = 0;
        for (int k = 0; k < used; k++) {
            side[k] = (int)((r >> (11 + k)) & 1);
            n1 += side[k];
        }
        if (n1 == 0 || n1 == used) { side[used - 1] ^= 1; n1 += side[used - 1] ? 1 : -1; }
        for (int step = 0; step < used * used; step++) {
            int64_t best = 0;
            int bk = -1;
            for (int k = 0; k < used; k++) {
                if ((side[k] && n1 == 1) || (!side[k] && n1 == used - 1)) continue;  /* keep both sides */
                int64_t gain = 0;
                for (int l = 0; l < used; l++) {
                    if (l == k) continue;
                    gain += side[l] == side[k] ? sw[k * used + l] : -sw[k * used + l];
                }
                if (gain > best) { best = gain; bk = k; }
            }
            if (bk < 0) break;
            n1 += side[bk] ? -1 : 1;
            side[bk] ^= 1;
        }
        for (int d = 0; d < G; d++) assign[(int64_t)d * n_cand + n] = (uint8_t)grp[d];
        for (int k = 0; k < max_groups; k++)
            role[(int64_t)k * n_cand + n] = k < used ? (uint8_t)(side[k] ? HXO_DECODE : HXO_PREFILL) : (uint8_t)HXO_UNUSED;
    }
    free(mem); free(grp); free(sw);
    return 0;
}
