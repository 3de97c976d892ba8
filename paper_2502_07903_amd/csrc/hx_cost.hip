// hx_cost.hip -- Table 1 cost model and Appendix A node capacities on gfx950.
//
// One lane per (group slot k, candidate n), candidate-fastest, so every load of the
// candidate arrays (assign[g][n], role[k][n]) and every store of the outputs ([k][n]) is
// coalesced across the wavefront.  A lane decodes its group's members (ascending GPU id)
// into an LDS column of its own, then costs every admissible TP x PP strategy and keeps
// prefill's latency-optimal / decode's throughput-optimal one (Sec. 3.3, "Compute nodes").
// The work is FP64 scalar arithmetic: no dense contraction, so no MFMA.
//
// Per-GPU parameters (c_d, memory bandwidth, memory limit) are gathered once per block into
// LDS.  Every expression follows the evaluation order documented in hx.h; a stage's max over
// devices of X/(t*c_d) is taken as X/(t*min c_d), which is the same binary64 value because
// rounding is monotone.
#include "hx_internal.h"

namespace hx {
namespace {

constexpr int kCostBlock = 128;

struct StrategyCost {
    double bmax, lat, x;
};

// Costs strategy (tp, pp) of a group whose r-th member (ascending id) is mem[r * stride].
// Returns false when the memory limit admits no batch of 1.
__device__ bool cost_strategy(const Problem& p, const double* gfl, const double* ghb, const double* gme,
                              const uint8_t* mem, int stride, int tp, int pp, int role, StrategyCost& out) {
    const double t = (double)tp;
    const double H = p.H, B = p.B;
    const double W12 = 12.0 * H * H * B;
    const double Kkv = 2.0 * (p.s_in + p.s_out) * p.Hkv * B;
    const double Kact = 4.0 * (p.s_in + p.s_out) * H * B;

    // Memory-limit row: b_j = floor((M_j - A_j)/K_j) on the stage's smallest memory.
    double bmin = kBmaxClamp;
    for (int j = 0; j < pp; ++j) {
        const double l = (double)stage_layers(p.L, pp, j);
        const double A = (W12 / t) * l;
        const double K = (Kkv / t) * l + Kact;
        const uint8_t* S = mem + (j * tp) * stride;
        double Mmin = gme[S[0]];
        for (int r = 1; r < tp; ++r) Mmin = dmin(Mmin, gme[S[r * stride]]);
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

    double s1 = 0.0;
    for (int j = 0; j < pp; ++j) {
        const double l = (double)stage_layers(p.L, pp, j);
        const uint8_t* S = mem + (j * tp) * stride;
        double cmin = gfl[S[0]], hmin = ghb[S[0]];
        for (int r = 1; r < tp; ++r) {
            cmin = dmin(cmin, gfl[S[r * stride]]);
            hmin = dmin(hmin, ghb[S[r * stride]]);
        }
        const double comp = prefill ? (Xcomp_p / (t * cmin)) * l
                                    : (Xscan_d / (t * hmin)) * l + (Xcomp_d / (t * cmin)) * l;
        // TP row: the device with the largest sum over its peers (ascending peer order).
        double mx = 0.0;
        for (int r = 0; r < tp; ++r) {
            const int d = S[r * stride];
            const double* arow = p.alpha + d * p.G;
            const double* brow = p.beta + d * p.G;
            double sum = 0.0;
            for (int q = 0; q < tp; ++q) {
                if (q == r) continue;
                const int e = S[q * stride];
                sum = sum + (arow[e] + X / (t * brow[e]));
            }
            if (r == 0 || sum > mx) mx = sum;
        }
        const double tpc = prefill ? (mx * 4.0) * l : ((mx * 4.0) * p.s_out) * l;
        s1 = s1 + (comp + tpc);
    }
    // PP row: the fastest link between consecutive stages.
    double s2 = 0.0;
    for (int j = 0; j + 1 < pp; ++j) {
        const uint8_t* S = mem + (j * tp) * stride;
        const uint8_t* S2 = mem + ((j + 1) * tp) * stride;
        double mn = 0.0;
        for (int r = 0; r < tp; ++r) {
            const int d = S[r * stride];
            for (int q = 0; q < tp; ++q) {
                const int e = S2[q * stride];
                const double v = p.alpha[d * p.G + e] + X / p.beta[d * p.G + e];
                if ((r == 0 && q == 0) || v < mn) mn = v;
            }
        }
        s2 = s2 + (prefill ? mn : mn * p.s_out);
    }
    out.lat = s1 + s2;
    out.x = (1000.0 * b) / out.lat;
    return true;
}

__global__ void __launch_bounds__(kCostBlock) cost_kernel(Problem p, CostOut o) {
    extern __shared__ double smem[];
    double* gfl = smem;
    double* ghb = gfl + p.G;
    double* gme = ghb + p.G;
    uint8_t* lists = reinterpret_cast<uint8_t*>(gme + p.G);  // [G][blockDim]
    const int tid = threadIdx.x;
    for (int g = tid; g < p.G; g += blockDim.x) {
        const int t = p.gpu_type[g];
        const bool ok = t >= 0 && t < p.T;  // an unknown type can hold nothing: infeasible
        gfl[g] = ok ? p.flops[t] : 0.0;
        ghb[g] = ok ? p.hbm[t] : 0.0;
        gme[g] = ok ? p.mem[t] : 0.0;
    }
    __syncthreads();

    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + tid;
    if (gid >= (int64_t)p.Kmax * p.N) return;
    const int k = (int)(gid / p.N);
    const int n = (int)(gid - (int64_t)k * p.N);
    const int stride = blockDim.x;
    uint8_t* mem = lists + tid;

    int cnt = 0;
    for (int g = 0; g < p.G; ++g)
        if (p.assign[(int64_t)g * p.N + n] == k) mem[(cnt++) * stride] = (uint8_t)g;
    const int role = p.role[gid];

    int best_tp = 0, best_pp = 0;
    int32_t best_b = 0, best_cap = 0;
    double best_lat = 0.0, best_x = 0.0;
    if (cnt > 0 && (role == HX_PREFILL || role == HX_DECODE)) {
        bool have = false;
        for (int tp = 1; tp <= HX_MAX_TP; ++tp) {
            if (!((p.tp_mask >> (tp - 1)) & 1u) || cnt % tp != 0) continue;
            const int pp = cnt / tp;
            if (pp > HX_MAX_PP || !((p.pp_mask >> (pp - 1)) & 1u) || pp > p.L) continue;
            StrategyCost c;
            if (!cost_strategy(p, gfl, ghb, gme, mem, stride, tp, pp, role, c)) continue;
            const bool better = !have || (role == HX_PREFILL ? c.lat < best_lat : c.x > best_x);
            if (better) {
                have = true;
                best_tp = tp;
                best_pp = pp;
                best_b = (int32_t)c.bmax;
                best_cap = quantize(c.x);
                best_lat = c.lat;
                best_x = c.x;
            }
        }
    }
    o.tp[gid] = (uint8_t)best_tp;
    o.pp[gid] = (uint8_t)best_pp;
    o.bmax[gid] = best_b;
    o.cap[gid] = best_cap;
    o.lat[gid] = best_lat;
}

}  // namespace

hipError_t launch_cost(const Problem& p, const CostOut& o, hipStream_t s) {
    const int64_t lanes = (int64_t)p.Kmax * p.N;
    const int blocks = (int)((lanes + kCostBlock - 1) / kCostBlock);
    const size_t lds = 3 * sizeof(double) * p.G + (size_t)p.G * kCostBlock;
    hipLaunchKernelGGL(cost_kernel, dim3(blocks), dim3(kCostBlock), lds, s, p, o);
    return hipGetLastError();
}

}  // namespace hx
