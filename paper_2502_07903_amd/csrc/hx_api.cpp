// hx_api.cpp -- the C-ABI of libhx: host-side validation, launch geometry and error codes.
// Every entry point checks its arguments without touching device memory, enqueues its
// kernels on the caller's stream and returns; see include/hx.h for the contract.
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>

#include "hx_internal.h"

// The scratch of hx_cost_eval_static: one copy per GPU, held until the process ends.  In host
// code this name is only a stand-in for the symbol; its device address comes from
// hipGetSymbolAddress (scratch_address below), and only that address is passed to kernels.
static __device__ __align__(256) unsigned char scratch[HX_STATIC_SCRATCH_BYTES];

namespace {

thread_local char g_last_error[256] = "";

int hip_error(hipError_t e) {
    snprintf(g_last_error, sizeof g_last_error, "%s: %s", hipGetErrorName(e), hipGetErrorString(e));
    return HX_EHIP;
}

bool finite_pos(double x) { return isfinite(x) && x > 0.0; }

int check_problem(const hx_cluster* c, const hx_model& m, const hx_workload& w, const hx_space& s,
                  const hx_candidates* k) {
    if (!c || !k) return HX_EINVAL;
    if (c->n_gpus < 1 || c->n_gpus > HX_MAX_GPUS || c->n_types < 1) return HX_EINVAL;
    if (!c->gpu_type || !c->type_flops || !c->type_hbm_bw || !c->type_mem || !c->beta || !c->alpha)
        return HX_EINVAL;
    if (!(c->coord_bw >= 0.0) || !(c->req_bytes >= 0.0) || !isfinite(c->coord_bw) || !isfinite(c->req_bytes))
        return HX_EINVAL;
    if (m.n_layers < 1 || m.hidden < 1 || m.n_heads < 1 || m.n_kv_heads < 1 || m.n_kv_heads > m.n_heads ||
        m.bytes_per_elem < 1)
        return HX_EINVAL;
    if (((int64_t)m.hidden * m.n_kv_heads) % m.n_heads != 0) return HX_EINVAL;
    if (!finite_pos(w.s_in) || !finite_pos(w.s_out)) return HX_EINVAL;
    if (w.n_classes < 0 || w.n_classes > HX_MAX_CLASSES) return HX_EINVAL;
    for (int k = 0; k < w.n_classes; ++k)
        if (!finite_pos(w.cls_in[k]) || !finite_pos(w.cls_out[k]) || !finite_pos(w.cls_w[k])) return HX_EINVAL;
    if (w.n_classes > 0 && (s.variant & (HX_VARIANT_KV_ORDER | HX_VARIANT_ASYM))) return HX_EINVAL;
    if (s.tp_mask == 0 || s.tp_mask >= (1u << HX_MAX_TP) || s.pp_mask == 0) return HX_EINVAL;
    if (s.granularity != 0 && s.granularity != 1) return HX_EINVAL;
    if (s.variant & ~(uint32_t)(HX_VARIANT_PIPELINED | HX_VARIANT_KV_ORDER | HX_VARIANT_ASYM | HX_HINT_SHARED_GROUPS))
        return HX_EINVAL;
    if ((s.variant & HX_VARIANT_KV_ORDER) && (s.variant & HX_VARIANT_ASYM)) return HX_EINVAL;
    // the stage-order search covers pipelines of up to 8 stages
    if ((s.variant & HX_VARIANT_KV_ORDER) && (s.pp_mask >> 8)) return HX_EINVAL;
    if (k->n_cand < 1 || k->max_groups < 1 || k->max_groups > HX_MAX_GROUPS || !k->assign || !k->role)
        return HX_EINVAL;
    return HX_OK;
}

int check_cost(const hx_cost_out* o) {
    if (!o || !o->tp || !o->pp || !o->bmax || !o->cap || !o->lat || !o->members) return HX_EINVAL;
    return HX_OK;
}

// Room every network of the batch needs: nodes per side and KV edges.
int check_net_shape(const hx_flownet* f) {
    if (!f || f->n_cand < 1 || f->max_p < 1 || f->max_d < 1 || f->max_pd < 1) return HX_EINVAL;
    if (!f->n_p || !f->n_d || !f->src_cap || !f->p_cap || !f->kv_cap || !f->d_cap || !f->sink_cap)
        return HX_EINVAL;
    return HX_OK;
}

int check_net_for(const hx_cluster* c, const hx_space& s, const hx_candidates* k, const hx_flownet* f) {
    int rc = check_net_shape(f);
    if (rc) return rc;
    if (!f->p_slot || !f->d_slot || f->n_cand != k->n_cand) return HX_EINVAL;
    const int64_t bound = s.granularity == 0 ? k->max_groups : c->n_gpus;
    if (f->max_p < bound || f->max_d < bound || f->max_pd < (bound / 2) * ((bound + 1) / 2)) return HX_EINVAL;
    return HX_OK;
}

int32_t coord_cap(const hx_cluster* c) {
    if (c->coord_bw > 0.0 && c->req_bytes > 0.0) {
        const double x = (1000.0 * c->coord_bw) / c->req_bytes;
        if (!(x >= 0.0)) return 0;
        return x >= (double)HX_CAP_MAX ? HX_CAP_MAX : (int32_t)floor(x);
    }
    return HX_CAP_MAX;
}

hx::Problem make_problem(const hx_cluster* c, const hx_model& m, const hx_workload& w, const hx_space& s,
                         const hx_candidates* k) {
    hx::Problem p;
    p.G = c->n_gpus;
    p.T = c->n_types;
    p.N = k->n_cand;
    p.Kmax = k->max_groups;
    p.L = m.n_layers;
    p.tp_mask = s.tp_mask;
    p.pp_mask = s.pp_mask;
    p.granularity = s.granularity;
    p.variant = s.variant;
    p.H = (double)m.hidden;
    p.Hkv = (double)((int64_t)m.hidden * m.n_kv_heads / m.n_heads);
    p.B = (double)m.bytes_per_elem;
    p.s_in = w.s_in;
    p.s_out = w.s_out;
    p.n_cls = w.n_classes;
    for (int k = 0; k < HX_MAX_CLASSES; ++k) {
        const bool in = k < w.n_classes;
        p.cls_in[k] = in ? w.cls_in[k] : 0.0;
        p.cls_out[k] = in ? w.cls_out[k] : 0.0;
        p.cls_w[k] = in ? w.cls_w[k] : 0.0;
    }
    p.coord_cap = coord_cap(c);
    p.gpu_type = c->gpu_type;
    p.flops = c->type_flops;
    p.hbm = c->type_hbm_bw;
    p.mem = c->type_mem;
    p.beta = c->beta;
    p.alpha = c->alpha;
    p.assign = k->assign;
    p.role = k->role;
    return p;
}

hx::CostOut make_cost(const hx_cost_out* o) { return hx::CostOut{o->tp, o->pp, o->bmax, o->cap, o->lat, o->members}; }

hx::FlowNet make_net(const hx_flownet* f) {
    return hx::FlowNet{f->n_cand, f->max_p,   f->max_d,  f->max_pd, f->n_p,   f->n_d,    f->p_slot,
                       f->d_slot, f->src_cap, f->p_cap, f->kv_cap, f->d_cap, f->sink_cap};
}

// Rounds of push-relabel allowed per candidate; HX_MAXFLOW_ROUND_BUDGET overrides it so that
// tests can force the non-convergence path from the host.
int32_t round_budget() {
    const char* e = getenv("HX_MAXFLOW_ROUND_BUDGET");
    if (e && *e) {
        long v = strtol(e, nullptr, 10);
        if (v >= 1 && v <= (1L << 30)) return (int32_t)v;
    }
    return 1 << 22;
}

static_assert(hx::kKCount == HX_KERNELS, "kernel ids and HX_KERNELS disagree");

// Diagnostic per-kernel timing (hx_profile): HIP event pairs recorded around every launch
// while enabled, from a pool that grows as needed.  Process-global, for one host thread.
struct Profile {
    bool on = false;
    hipEvent_t open[hx::kKCount] = {};
    struct Pair {
        int k;
        hipEvent_t b, e;
    };
    Pair* pairs = nullptr;
    size_t n = 0, cap = 0;
    hipEvent_t* pool = nullptr;
    size_t npool = 0, cappool = 0;
};
Profile g_prof;

// Timing-only events: no system-scope fence when they are recorded, so that recording one
// does not write back and invalidate caches between the kernels it brackets.
hipEvent_t prof_event() {
    if (g_prof.npool) return g_prof.pool[--g_prof.npool];
    hipEvent_t e = nullptr;
    return hipEventCreateWithFlags(&e, hipEventDisableSystemFence) == hipSuccess ? e : nullptr;
}

void prof_release(hipEvent_t e) {
    if (!e) return;
    if (g_prof.npool == g_prof.cappool) {
        const size_t c = g_prof.cappool ? 2 * g_prof.cappool : 64;
        hipEvent_t* q = static_cast<hipEvent_t*>(realloc(g_prof.pool, c * sizeof(hipEvent_t)));
        if (!q) {
            (void)hipEventDestroy(e);
            return;
        }
        g_prof.pool = q;
        g_prof.cappool = c;
    }
    g_prof.pool[g_prof.npool++] = e;
}

void prof_clear() {
    for (size_t i = 0; i < g_prof.n; ++i) {
        prof_release(g_prof.pairs[i].b);
        prof_release(g_prof.pairs[i].e);
    }
    g_prof.n = 0;
    for (int k = 0; k < hx::kKCount; ++k) {
        prof_release(g_prof.open[k]);
        g_prof.open[k] = nullptr;
    }
}

}  // namespace

namespace hx {

void prof_mark(int k, bool end, hipStream_t s) {
    if (!g_prof.on || k < 0 || k >= kKCount) return;
    hipEvent_t e = prof_event();
    if (!e || hipEventRecord(e, s) != hipSuccess) {
        prof_release(e);
        return;
    }
    if (!end) {
        prof_release(g_prof.open[k]);
        g_prof.open[k] = e;
        return;
    }
    if (!g_prof.open[k]) {
        prof_release(e);
        return;
    }
    if (g_prof.n == g_prof.cap) {
        const size_t c = g_prof.cap ? 2 * g_prof.cap : 256;
        auto* q = static_cast<Profile::Pair*>(realloc(g_prof.pairs, c * sizeof(Profile::Pair)));
        if (!q) {
            prof_release(e);
            return;
        }
        g_prof.pairs = q;
        g_prof.cap = c;
    }
    g_prof.pairs[g_prof.n++] = Profile::Pair{k, g_prof.open[k], e};
    g_prof.open[k] = nullptr;
}

}  // namespace hx

extern "C" {

int hx_profile(int32_t enable) {
    prof_clear();
    g_prof.on = enable != 0;
    return HX_OK;
}

int hx_profile_read(double* ms, int32_t* launches, int32_t n) {
    if (!ms || !launches || n < hx::kKCount) return HX_EINVAL;
    for (int k = 0; k < hx::kKCount; ++k) {
        ms[k] = 0.0;
        launches[k] = 0;
    }
    // The events carry no fence, so wait for the device before reading their timestamps.
    if (g_prof.n) {
        hipError_t e = hipDeviceSynchronize();
        if (e != hipSuccess) return hip_error(e);
    }
    for (size_t i = 0; i < g_prof.n; ++i) {
        const auto& q = g_prof.pairs[i];
        float t = 0.0f;
        hipError_t e = hipEventSynchronize(q.e);
        if (e == hipSuccess) e = hipEventElapsedTime(&t, q.b, q.e);
        if (e != hipSuccess) return hip_error(e);
        ms[q.k] += t;
        launches[q.k] += 1;
    }
    prof_clear();
    return hx::kKCount;
}

const char* hx_kernel_name(int32_t k) {
    static const char* names[hx::kKCount] = {"setup", "decode",  "scatter", "eval",     "nodes",
                                             "kv",    "maxflow", "best",    "classes",  "moves",
                                             "gather", "spectral", "partition", "shared"};
    return k >= 0 && k < hx::kKCount ? names[k] : "";
}


int hx_abi_version(void) { return HX_ABI_VERSION; }

const char* hx_strerror(int code) {
    switch (code) {
        case HX_OK: return "ok";
        case HX_EINVAL: return "invalid argument";
        case HX_ETOOBIG: return "problem exceeds the max-flow kernel's LDS plan or the static scratch";
        case HX_EHIP: return "HIP launch error (see hx_last_error)";
        case HX_ENOCONV: return "max-flow did not converge within its round budget";
        default: return "unknown error";
    }
}

const char* hx_last_error(void) { return g_last_error; }

int hx_validate(const hx_cluster* cluster, hx_model model, hx_workload wl, hx_space space, const hx_candidates* cand,
                const hx_cost_out* cost, const hx_flownet* net) {
    int rc = check_problem(cluster, model, wl, space, cand);
    if (rc) return rc;
    if (cost && (rc = check_cost(cost))) return rc;
    if (net) {
        if ((rc = check_net_for(cluster, space, cand, net))) return rc;
        if (hx::maxflow_lds_bytes(net->max_p, net->max_d, net->max_pd) == 0) return HX_ETOOBIG;
    }
    return HX_OK;
}

size_t hx_cost_workspace_bytes(int32_t n_gpus, int32_t max_groups, int32_t n_cand) {
    if (n_gpus < 1 || n_gpus > HX_MAX_GPUS || max_groups < 1 || max_groups > HX_MAX_GROUPS || n_cand < 1) return 0;
    return hx::cost_workspace_bytes(n_gpus, max_groups, n_cand);
}

int hx_member_words(int32_t n_gpus) { return n_gpus < 1 || n_gpus > HX_MAX_GPUS ? 0 : hx::mask_words(n_gpus); }

int hx_cost_eval(const hx_cluster* cluster, hx_model model, hx_workload wl, hx_space space, const hx_candidates* cand,
                 const hx_cost_out* out, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    int rc = check_problem(cluster, model, wl, space, cand);
    if (rc || (rc = check_cost(out))) return rc;
    if (!workspace || ((uintptr_t)workspace & 255) ||
        workspace_bytes < hx::cost_workspace_bytes(cluster->n_gpus, cand->max_groups, cand->n_cand))
        return HX_EINVAL;
    hipError_t e = hx::launch_cost(make_problem(cluster, model, wl, space, cand), make_cost(out), workspace, stream);
    return e == hipSuccess ? HX_OK : hip_error(e);
}

namespace {

// Device address of `scratch` on each device, looked up once per device (with that device
// current) on the first hx_cost_eval_static call there.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

int scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_error(e);
    if (dev < 0 || dev >= kMaxDevices) return HX_EINVAL;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_error(e);
        if (!p) return HX_EINVAL;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return HX_OK;
}

}  // namespace

size_t hx_static_scratch_bytes(void) { return HX_STATIC_SCRATCH_BYTES; }

int hx_cost_eval_static(const hx_cluster* cluster, hx_model model, hx_workload wl, hx_space space,
                        const hx_candidates* cand, const hx_cost_out* out, hipStream_t stream) {
    int rc = check_problem(cluster, model, wl, space, cand);
    if (rc || (rc = check_cost(out))) return rc;
    if (hx::cost_workspace_bytes(cluster->n_gpus, cand->max_groups, cand->n_cand) > HX_STATIC_SCRATCH_BYTES)
        return HX_ETOOBIG;
    void* ws = nullptr;
    if ((rc = scratch_address(&ws))) return rc;
    hipError_t e = hx::launch_cost(make_problem(cluster, model, wl, space, cand), make_cost(out), ws, stream);
    return e == hipSuccess ? HX_OK : hip_error(e);
}

int hx_build_flownet(const hx_cluster* cluster, hx_model model, hx_workload wl, hx_space space,
                     const hx_candidates* cand, const hx_cost_out* cost, const hx_flownet* net, hipStream_t stream) {
    int rc = check_problem(cluster, model, wl, space, cand);
    if (rc || (rc = check_cost(cost)) || (rc = check_net_for(cluster, space, cand, net))) return rc;
    hipError_t e = hx::launch_flownet(make_problem(cluster, model, wl, space, cand), make_cost(cost), make_net(net),
                                      stream);
    return e == hipSuccess ? HX_OK : hip_error(e);
}

int hx_maxflow_batch(const hx_flownet* net, int32_t* flow_value, int32_t* kv_flow, uint8_t* cut, hipStream_t stream) {
    int rc = check_net_shape(net);
    if (rc) return rc;
    if (!flow_value) return HX_EINVAL;
    if (hx::maxflow_lds_bytes(net->max_p, net->max_d, net->max_pd) == 0) return HX_ETOOBIG;
    hipError_t e = hx::launch_maxflow(make_net(net), flow_value, kv_flow, cut, round_budget(), nullptr, stream);
    return e == hipSuccess ? HX_OK : hip_error(e);
}

int hx_maxflow_stats(const hx_flownet* net, int32_t* flow_value, int32_t* kv_flow, uint8_t* cut, uint64_t* stats,
                     hipStream_t stream) {
    int rc = check_net_shape(net);
    if (rc) return rc;
    if (!flow_value || !stats || ((uintptr_t)stats & 7)) return HX_EINVAL;
    if (hx::maxflow_lds_bytes(net->max_p, net->max_d, net->max_pd) == 0) return HX_ETOOBIG;
    hipError_t e = hx::launch_maxflow(make_net(net), flow_value, kv_flow, cut, round_budget(),
                                      reinterpret_cast<unsigned long long*>(stats), stream);
    return e == hipSuccess ? HX_OK : hip_error(e);
}

int hx_best_candidate(const int32_t* flow_value, int32_t n_cand, int32_t* best, hipStream_t stream) {
    if (!flow_value || !best || n_cand < 1) return HX_EINVAL;
    hipError_t e = hx::launch_best(flow_value, n_cand, best, stream);
    return e == hipSuccess ? HX_OK : hip_error(e);
}

// hx_score_batch's scratch after the cost model's: the link table and list (per-GPU path) or the
// listed KV path's feasibility words and edge list (replica path), whichever is larger, then the
// argmax's area.
static size_t score_mid_bytes(int32_t n_gpus, int32_t max_groups, int32_t n_cand) {
    const size_t t = hx::link_table_bytes(n_gpus, n_cand);
    const size_t f = max_groups <= 32 && n_cand <= (1 << 22) ? hx::kv_list_bytes(max_groups, n_cand) : 0;
    return ((t > f ? t : f) + 255) & ~(size_t)255;
}

size_t hx_score_workspace_bytes(int32_t n_gpus, int32_t max_groups, int32_t n_cand) {
    const size_t c = hx_cost_workspace_bytes(n_gpus, max_groups, n_cand);
    if (c == 0) return 0;
    return ((c + 255) & ~(size_t)255) + score_mid_bytes(n_gpus, max_groups, n_cand) + ((hx::best_parts_bytes() + 255) & ~(size_t)255);
}

int hx_score_batch(const hx_cluster* cluster, hx_model model, hx_workload wl, hx_space space,
                   const hx_candidates* cand, const hx_cost_out* cost, const hx_flownet* net, int32_t* flow_value,
                   int32_t* best, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    int rc = check_problem(cluster, model, wl, space, cand);
    if (rc || (rc = check_cost(cost)) || (rc = check_net_for(cluster, space, cand, net))) return rc;
    if (!flow_value || !best) return HX_EINVAL;
    if (!workspace || ((uintptr_t)workspace & 255) ||
        workspace_bytes < hx_score_workspace_bytes(cluster->n_gpus, cand->max_groups, cand->n_cand))
        return HX_EINVAL;
    if (hx::maxflow_lds_bytes(net->max_p, net->max_d, net->max_pd) == 0) return HX_ETOOBIG;
    const hx::Problem p = make_problem(cluster, model, wl, space, cand);
    hx::FlowNet f = make_net(net);
    // the link table (or the feasibility words) follows the cost model's scratch, the argmax's
    // area follows them: per-workgroup winners for the per-GPU path, the fused argmax's slots
    // (zeroed by the cost model's first kernel) otherwise
    const size_t off_mid =
        (hx::cost_workspace_bytes(cluster->n_gpus, cand->max_groups, cand->n_cand) + 255) & ~(size_t)255;
    const size_t off_part = off_mid + score_mid_bytes(cluster->n_gpus, cand->max_groups, cand->n_cand);
    unsigned char* part = static_cast<unsigned char*>(workspace) + off_part;
    const bool direct = hx::flownet_values_direct(p) && hx::maxflow_workgroup_plan(net->max_p, net->max_d, net->max_pd);
    unsigned long long* slots = direct ? nullptr : reinterpret_cast<unsigned long long*>(part);
    hipError_t e = hx::launch_cost(p, make_cost(cost), workspace, stream, slots, direct ? 0 : hx::kArgSlots);
    if (e == hipSuccess) {
        if (direct) {
            void* table = static_cast<unsigned char*>(workspace) + off_mid;
            e = hx::launch_flownet_values(p, make_cost(cost), f, flow_value, table, stream);
            int32_t* count = hx::flownet_values_list_count(table, cluster->n_gpus);
            if (e == hipSuccess) e = hx::launch_maxflow_listed(f, flow_value, round_budget(), count + 16, count, stream);
        } else {
            if (hx::kv_list_fits(p.granularity, cand->max_groups, cand->n_cand))
                hx::kv_list_carve(f, static_cast<unsigned char*>(workspace) + off_mid, cand->max_groups, cand->n_cand);
            e = hx::launch_flownet(p, make_cost(cost), f, stream);
            if (e == hipSuccess)
                e = hx::launch_maxflow(f, flow_value, nullptr, nullptr, round_budget(), nullptr, stream, slots);
        }
    }
    if (e == hipSuccess) {
        // per-GPU path: the argmax's counter is the cost workspace's word that the cost model's
        // first kernel cleared
        if (direct)
            e = hx::launch_best_parts(flow_value, cand->n_cand, best,
                                      hx::cost_workspace_counter(workspace, cluster->n_gpus),
                                      reinterpret_cast<uint64_t*>(part), stream);
        else
            e = hx::launch_best_final(slots, best, stream);
    }
    return e == hipSuccess ? HX_OK : hip_error(e);
}

int hx_edge_classes(const hx_flownet* net, const int32_t* flow_value, const int32_t* kv_flow, uint8_t* node_cls,
                    uint8_t* kv_cls, hipStream_t stream) {
    int rc = check_net_shape(net);
    if (rc) return rc;
    if (!flow_value || !kv_flow || !node_cls || !kv_cls) return HX_EINVAL;
    hipError_t e = hx::launch_classes(make_net(net), flow_value, kv_flow, node_cls, kv_cls, stream);
    return e == hipSuccess ? HX_OK : hip_error(e);
}

int hx_guided_moves(int32_t n_gpus, int32_t granularity, const hx_candidates* parents, const hx_flownet* parent_net,
                    const uint8_t* node_cls, int32_t n_child, const uint64_t* rnd, uint8_t* child_assign,
                    uint8_t* child_role, int32_t* move, hipStream_t stream) {
    if (n_gpus < 1 || n_gpus > HX_MAX_GPUS || (granularity != 0 && granularity != 1)) return HX_EINVAL;
    if (!parents || parents->n_cand < 1 || parents->max_groups < 1 || parents->max_groups > HX_MAX_GROUPS ||
        !parents->assign || !parents->role)
        return HX_EINVAL;
    int rc = check_net_shape(parent_net);
    if (rc) return rc;
    if (!parent_net->p_slot || !parent_net->d_slot || parent_net->n_cand != parents->n_cand) return HX_EINVAL;
    if (parents->n_cand > 65535) return HX_EINVAL;  // one grid row per parent
    if (!node_cls || !rnd || !child_assign || !child_role || !move || n_child < 1) return HX_EINVAL;
    hipError_t e = hx::launch_moves(n_gpus, parents->max_groups, granularity, parents->n_cand, parents->assign,
                                    parents->role, make_net(parent_net), node_cls, n_child, rnd, child_assign,
                                    child_role, move, stream);
    return e == hipSuccess ? HX_OK : hip_error(e);
}

size_t hx_partition_workspace_bytes(int32_t n_gpus) {
    if (n_gpus < 2 || n_gpus > HX_MAX_GPUS) return 0;
    return ((size_t)n_gpus * n_gpus * sizeof(int64_t) + 255) & ~(size_t)255;
}

int hx_spectral_order(const hx_cluster* cluster, int32_t iters, void* workspace, size_t workspace_bytes,
                      int32_t* order, double* fiedler, hipStream_t stream) {
    if (!cluster || cluster->n_gpus < 2 || cluster->n_gpus > HX_MAX_GPUS || !cluster->beta || !order) return HX_EINVAL;
    if (iters < 0 || !workspace || workspace_bytes < hx_partition_workspace_bytes(cluster->n_gpus)) return HX_EINVAL;
    hipError_t e = hx::launch_spectral(cluster->n_gpus, cluster->beta, static_cast<int64_t*>(workspace), iters, order,
                                       fiedler, stream);
    return e == hipSuccess ? HX_OK : hip_error(e);
}

int hx_partition_candidates(const hx_cluster* cluster, hx_model model, hx_workload wl, int32_t max_groups,
                            void* workspace, size_t workspace_bytes, const int32_t* order, int32_t n_cand,
                            const uint64_t* rnd, uint8_t* assign, uint8_t* role, hipStream_t stream) {
    const hx_space sp{1u, 1u, 0, 0u};
    const hx_candidates cand{n_cand, max_groups, assign, role};
    int rc = check_problem(cluster, model, wl, sp, &cand);
    if (rc) return rc;
    if (cluster->n_gpus < 2 || !order || !rnd || !workspace ||
        workspace_bytes < hx_partition_workspace_bytes(cluster->n_gpus))
        return HX_EINVAL;
    hipError_t e = hx::launch_partition(make_problem(cluster, model, wl, sp, &cand), static_cast<int64_t*>(workspace),
                                        order, rnd, assign, role, stream);
    return e == hipSuccess ? HX_OK : hip_error(e);
}

int hx_gather_candidates(int32_t n_gpus, const hx_candidates* src, const int32_t* index, int32_t count,
                         uint8_t* dst_assign, uint8_t* dst_role, hipStream_t stream) {
    if (n_gpus < 1 || n_gpus > HX_MAX_GPUS || !src || src->n_cand < 1 || src->max_groups < 1 ||
        src->max_groups > HX_MAX_GROUPS || !src->assign || !src->role)
        return HX_EINVAL;
    if (!index || count < 1 || !dst_assign || !dst_role) return HX_EINVAL;
    hipError_t e = hx::launch_gather(n_gpus, src->max_groups, src->n_cand, src->assign, src->role, index, count,
                                     dst_assign, dst_role, stream);
    return e == hipSuccess ? HX_OK : hip_error(e);
}

}  // extern "C"
