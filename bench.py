"""Benchmark: candidate placements scored per second on one MI355X.

A step is one pass of the whole hot path over one batch of candidate placements with the
inputs already resident in HBM: cost model (hx_cost_eval) -> flow network
(hx_build_flownet) -> max-flow (hx_maxflow_batch) -> best candidate (hx_best_candidate).
The default workload is the 32-GPU / 8-node / 4-type cluster serving a Llama-2-70B-shaped
model with lognormal request lengths, 65,536 seeded random candidates of 2-16 groups.

    python bench.py [--gpus 1] [--steps 50] [--warmup 5] [--workload 3] [--no-cpu-baseline]
    python bench.py --refine [--steps 10] [--warmup 2] [--children 131072]

--refine times rounds of the max-flow guided refinement of Sec. 3.4 instead (the 128-GPU
workload with per-GPU flow nodes): each round scores the parent placement with a flow
assignment, classifies its edges, emits the children by guided moves, scores them and keeps
the best; value = children per second.

Prints ONE JSON line.  Per-call durations come from HIP events recorded around every call
inside the timed region, on the stream the kernels run on; per-kernel durations from a second
pass of the same steps with libhx's diagnostic per-kernel events (hx_profile).  The roofline
object reports the kernel with the largest share.  The CPU baseline times the oracle (test
infrastructure, not the product) on the same batch on the host's cores.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "candidate placements scored/sec (cost model + max-flow) at 1 GPU; % HBM/LDS roofline"

# MI355X (gfx950) peaks: 256 CUs at 2.4 GHz.
HBM_PEAK_GBS = 8000.0
# LDS reads: 256 B/clk/CU on gfx950 (twice CDNA3's 128) -> 157,286 GB/s (datasheet figure).
LDS_PEAK_GBS = 256 * 256 * 2.4
# FP64 vector operations that are not fused multiply-adds: 256 CUs x 4 SIMDs x 16 lanes x
# 2.4 GHz = 39,322 G op/s (the 78.6 TFLOP/s headline counts an FMA as two).
FP64_VALU_PEAK_GOPS = 256 * 4 * 16 * 2.4

# HBM bytes per launch from rocprofv3 FETCH_SIZE and WRITE_SIZE passes (workload 3:
# profiles/all_kernels_workload3.md; workload 5: profiles/chain_workload5.md), each scaled by what the counter reads for a 256 MiB
# device copy (FETCH_SIZE x 2.0, WRITE_SIZE x 1.0).  Valid only for the kernel source they were
# taken on (first 16 hex digits of the source file's SHA-256); otherwise traffic is null.
COUNTER_SCALE = {"fetch": 2.0, "write": 1.0}
KERNEL_TRAFFIC = {
    # workload 3 (profiles/all_kernels_workload3.md); kv the listed path's four kernels (rows,
    # scan, packing, walks), maxflow the instantiation with the folded argmax, best the final
    # reduction of its slots
    3: {
        "setup": {"source_sha256_16": "cfe308a8f566cbcf", "fetch_kib": 70.55, "write_kib": 57.43},
        "decode": {"source_sha256_16": "cfe308a8f566cbcf", "fetch_kib": 1714, "write_kib": 2.884e+04},
        "scatter": {"source_sha256_16": "cfe308a8f566cbcf", "fetch_kib": 5425, "write_kib": 1482},
        "eval": {"source_sha256_16": "cfe308a8f566cbcf", "fetch_kib": 1110, "write_kib": 1.204e+04},
        "nodes": {"source_sha256_16": "5fbb928bf73c535c", "fetch_kib": 7215, "write_kib": 1.654e+04},
        "kv": {"source_sha256_16": "5fbb928bf73c535c", "fetch_kib": 4536, "write_kib": 1.423e+04},
        "maxflow": {"source_sha256_16": "b931fad73ca81326", "fetch_kib": 1.674e+04, "write_kib": 768},
        "best": {"source_sha256_16": "89724c3a7f9a387f", "fetch_kib": 18.1, "write_kib": 0.03125},
    },
    # workload 5, one chain round through hx_score_batch with the shared-groups hint
    # (profiles/chain_workload5.md): nodes is the settling nodes kernel, kv the link table,
    # maxflow the list-driven kernel, shared candidate 0's groups, best the split argmax
    5: {
        "setup": {"source_sha256_16": "cfe308a8f566cbcf", "fetch_kib": 184.2, "write_kib": 516.1},
        "shared": {"source_sha256_16": "cfe308a8f566cbcf", "fetch_kib": 179.9, "write_kib": 2},
        "decode": {"source_sha256_16": "cfe308a8f566cbcf", "fetch_kib": 1.047e+04, "write_kib": 1.471e+05},
        "scatter": {"source_sha256_16": "cfe308a8f566cbcf", "fetch_kib": 3.967e+04, "write_kib": 7565},
        "eval": {"source_sha256_16": "cfe308a8f566cbcf", "fetch_kib": 9326, "write_kib": 3.268e+04},
        "nodes": {"source_sha256_16": "5fbb928bf73c535c", "fetch_kib": 6.153e+04, "write_kib": 1536},
        "kv": {"source_sha256_16": "5fbb928bf73c535c", "fetch_kib": 138.3, "write_kib": 68.03},
        "maxflow": {"source_sha256_16": "b931fad73ca81326", "fetch_kib": 18.21, "write_kib": 0},
        "best": {"source_sha256_16": "89724c3a7f9a387f", "fetch_kib": 297.3, "write_kib": 8.062},
    },
}
# The guided-moves kernel at the refinement workload (profiles/refine_workload5.md), per launch of
# 131,072 children, same scaling.
MOVES_TRAFFIC = {"source_sha256_16": "2902f3b847ca3ebd", "children": 131072, "fetch_kib": 561.0,
                 "write_kib": 20990.0}
# The partition kernel at workload 3 (profiles/partition_workload3.md), per launch of 16,384
# candidates, same scaling.
PARTITION_TRAFFIC = {"source_sha256_16": "72b4245b3df4f290", "candidates": 16384, "fetch_kib": 1158.0,
                     "write_kib": 6144.0}
KERNEL_SOURCE = {"setup": "hx_cost.hip", "decode": "hx_cost.hip", "scatter": "hx_cost.hip", "eval": "hx_cost.hip",
                 "nodes": "hx_flownet.hip", "kv": "hx_flownet.hip", "maxflow": "hx_maxflow.hip",
                 "best": "hx_best.hip", "shared": "hx_cost.hip"}


# hx_space.variant bits: 1 pipelined decode capacity, 2 KV stage-order search, 4 asymmetric
# layer split
VARIANTS = {"as-written": 0, "pipelined": 1, "kv-order": 2, "pipelined+kv-order": 3, "asym": 4,
            "pipelined+asym": 5}


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=3, choices=[1, 2, 3, 4, 5],
                    help="5: the refinement chain (--rounds rounds of 131,072 perturbations of the previous "
                         "round's best, per-GPU flow nodes)")
    ap.add_argument("--rounds", type=int, default=0, help="--workload 5: rounds of the chain (default: 16)")
    ap.add_argument("--round-repeats", type=int, default=3,
                    help="--workload 5: each round's batch is scored this many times; its time is the median")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--variant", choices=list(VARIANTS), default="as-written",
                    help="cost-model variant: the model as written, pipelined decode capacity, KV stage-order "
                         "search, asymmetric layer split, or combinations")
    ap.add_argument("--classes", type=int, default=0, choices=[0, 1, 2, 3, 4],
                    help="request classes: cost the requests as this many prompt-length buckets (0: the mean task)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU-baseline wall time")
    ap.add_argument("--refine", action="store_true",
                    help="time max-flow guided refinement rounds on the 128-GPU per-GPU-network workload instead")
    ap.add_argument("--partition", action="store_true",
                    help="time the graph-partition candidate generator (spectral order, partition, scoring) instead")
    ap.add_argument("--pushrelabel", choices=["workload3", "workload5"], default=None,
                    help="time the max-flow alone on networks that need push-relabel, at the network shapes of "
                         "that workload (both sides of at least two nodes, KV arcs below min(a_i, b_j))")
    ap.add_argument("--children", type=int, default=131072, help="children per refinement round (--refine)")
    ap.add_argument("--partition-candidates", type=int, default=16384, help="candidates per step (--partition)")
    ap.add_argument("--spectral-iters", type=int, default=1000, help="power iterations (--partition)")
    ap.add_argument("--quality-rounds", type=int, default=8,
                    help="--refine: also run this many guided and random-perturbation rounds and report the best")
    ap.add_argument("--candidates", type=int, default=0,
                    help="score batches of this many candidates of the workload instead of its own count "
                         "(a scaling study; the headline uses the workload's count)")
    ap.add_argument("--streams", type=int, default=1,
                    help="independent steps in flight in the timed region, each on its own HIP stream with its "
                         "own workspace and outputs (a search loop scoring independently drawn batches); 1 runs "
                         "the steps one after another")
    ap.add_argument("--concurrent-streams", type=int, default=3,
                    help="also report the rate with this many independent steps in flight (a short extra pass; "
                         "0 or 1: none)")
    ap.add_argument("--no-shared-groups-hint", action="store_true",
                    help="--workload 5 and --refine: score without the hint that the batch's candidates share "
                         "candidate 0's groups")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="first run one device-to-device copy of this many MiB (calibrates HBM byte counters)")
    return ap.parse_args()


def lds_floor_bytes(n_p: np.ndarray, n_d: np.ndarray) -> np.ndarray:
    """Algorithmic LDS bytes of one candidate's max-flow: its residual graph written once and
    every arc read once (8 B capacity + 8 B flow state per arc, both directions), plus 12 B of
    per-node state, on the contracted network s -> P -> D -> t."""
    P = n_p.astype(np.int64)
    D = n_d.astype(np.int64)
    arcs = 2 * (P + D + P * D)
    V = P + D + 2
    return 2 * 8 * arcs + 12 * V


def hbm_bytes_per_step(prob, dims, n_p, n_d) -> dict:
    """Algorithmic HBM bytes of one step through the four-call ABI (each intermediate written
    once and read once), by kernel."""
    G, K, N = prob.n_gpus, prob.max_groups, prob.n_cand
    used_pd = int((n_p.astype(np.int64) * n_d).sum())
    used_nodes = int(n_p.sum() + n_d.sum())
    cost = N * (G + K) + N * K * (1 + 1 + 4 + 4 + 8)
    flownet = N * (G + K) + N * K * (1 + 1 + 4) + N * 8 + used_nodes * 4 * 3 + used_pd * 4
    maxflow = N * 8 + used_nodes * 4 * 2 + used_pd * 4 + N * 4
    best = N * 4 + 8
    return dict(cost=cost, flownet=flownet, maxflow=maxflow, best=best)


def kernel_bytes(prob, n_p, n_d, settled_per_gpu: bool = False) -> dict:
    """Algorithmic HBM bytes of one launch of each streaming kernel (every input read once,
    every output written once):
      decode   assign and role of each candidate in, the group member masks out;
      scatter  the member masks in, one unit record (8 B + the mask) per present group out;
      nodes    each slot's mask, role and capacity (and per GPU its assign entry at granularity
               1) in, the counts and 12 B per node out;
      kv       replica networks: per used KV row the two slots, the two strategies and masks in,
               4 B out; per-GPU networks settled from the link table: the node rows in (12 B per
               node and the counts), the flow value out;
      maxflow  the network in (node rows, KV rows), the flow value out;
      best     4 B per candidate."""
    G, K, N = prob.n_gpus, prob.max_groups, prob.n_cand
    W = 1 if G <= 64 else (2 if G <= 128 else 4)
    groups = 0
    for n0 in range(0, N, 65536):
        a = prob.assign[:, n0:n0 + 65536]
        groups += int(sum(((a == k).any(axis=0)).sum() for k in range(K)))
    nodes = int(n_p.astype(np.int64).sum() + n_d.astype(np.int64).sum())
    pd = int((n_p.astype(np.int64) * n_d).sum())
    gran1 = prob.granularity == 1
    out = {
        "decode": N * (G + K) + N * K * 8 * W,
        "scatter": N * K * 8 * W + groups * 8 * (1 + W),
        "nodes": N * K * (8 * W + 1 + 4) + (N * G if gran1 else 0) + N * 8 + nodes * 12,
        "kv": (N * 8 + nodes * 12 + N * 4) if settled_per_gpu else (N * 8 + pd * (8 + 4 + 16 * W + 4)),
        "maxflow": N * 8 + nodes * 16 + pd * 4 + N * 4,
        "best": N * 4 + 8,
    }
    return out


def cpu_model() -> str:
    """The host CPU: model name, vendor, family / model / stepping (first processor in
    /proc/cpuinfo) and the logical CPU count, or "unknown"."""
    info = {}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if not line.strip():
                    break
                k, _, v = line.partition(":")
                info[k.strip()] = v.strip()
    except OSError:
        return "unknown"
    return (f"{info.get('model name', 'unknown')} ({info.get('vendor_id', '?')}, family {info.get('cpu family', '?')} "
            f"model {info.get('model', '?')} stepping {info.get('stepping', '?')}; {os.cpu_count()} logical CPUs)")


def measured_copy_gbs(torch, mib: int = 1024, reps: int = 10) -> float:
    """Device-to-device copy bandwidth (bytes read + written per second) of a mib MiB buffer,
    the measured counterpart of the HBM datasheet peak."""
    src = torch.ones(mib * (1 << 18), dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    t = time.perf_counter()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t) / reps
    del src, dst
    return 2.0 * mib * (1 << 20) / dt / 1e9



def kernel_traffic(kernel: str, workload: int, prob=None):
    """Counter-measured HBM bytes per launch of a kernel, or None when they do not apply (the
    counters were taken on workloads 3 and 5 with the cost model as written, on the sources whose
    hashes they carry)."""
    import hashlib
    t = KERNEL_TRAFFIC.get(workload, {}).get(kernel)
    if t is None:
        return None
    if prob is not None and (getattr(prob, "variant", 0) or getattr(prob, "classes", None) is not None):
        return None
    src = os.path.join(ROOT, "paper_2502_07903_amd", "csrc", KERNEL_SOURCE[kernel])
    if hashlib.sha256(open(src, "rb").read()).hexdigest()[:16] != t["source_sha256_16"]:
        return None
    return 1024.0 * (t["fetch_kib"] * COUNTER_SCALE["fetch"] + t["write_kib"] * COUNTER_SCALE["write"])


def shared_with_first(prob) -> np.ndarray:
    """[max_groups][N] bool: group slot k of candidate n is handed candidate 0's outputs under the
    shared-groups hint, i.e. it has a role (prefill or decode) and candidate 0's slot k - 1, k or
    k + 1 holds the same member set with the same role (candidate 0's own groups included: the
    hint costs them in their own kernel)."""
    G, K, N = prob.n_gpus, prob.max_groups, prob.n_cand
    words = (G + 63) // 64
    m = np.zeros((words, K + 1, N), np.uint64)  # row K collects unused GPUs
    cols = np.arange(N)
    for g in range(G):
        k = np.minimum(prob.assign[g].astype(np.int64), K)
        m[g // 64, k, cols] |= np.uint64(1) << np.uint64(g % 64)
    m = m[:, :K]
    role = prob.role.astype(np.int64)
    present = (m != 0).any(axis=0) & ((role == 0) | (role == 1))
    out = np.zeros((K, N), bool)
    for d in (-1, 0, 1):
        for k in range(K):
            e = k + d
            if e < 0 or e >= K or not present[e, 0]:
                continue
            same = present[k] & (role[k] == role[e, 0])
            for w in range(words):
                same &= m[w, k] == m[w, e, 0]
            out[k] |= same
    return out


def group_members(prob, exclude=None):
    """(members [U][size] ascending GPU ids, role [U]) of every present group, listed by size;
    exclude ([max_groups][N] bool): slots to leave out."""
    G, K, N = prob.n_gpus, prob.max_groups, prob.n_cand
    g, n = np.nonzero(prob.assign < K)
    k = prob.assign[g, n].astype(np.int64)
    order = np.lexsort((g, k, n))
    g, n, k = g[order], n[order], k[order]
    key = n * K + k
    starts = np.flatnonzero(np.concatenate([[True], key[1:] != key[:-1]]))
    sizes = np.diff(np.concatenate([starts, [len(key)]]))
    role = prob.role[k[starts], n[starts]]
    keep = (role == 0) | (role == 1)
    if exclude is not None:
        keep &= ~exclude[k[starts], n[starts]]
    out = {}
    for sz in np.unique(sizes[keep]):
        sel = starts[keep & (sizes == sz)]
        mem = g[sel[:, None] + np.arange(sz)[None, :]]
        out[int(sz)] = (mem, role[keep & (sizes == sz)])
    return out


def eval_fp64_ops(prob) -> float:
    return eval_fp64_counts(prob)[0]


def eval_fp64_counts(prob, exclude=None):
    """Algorithmic FP64 operations of the strategy-evaluation kernel (Table 1 rows as written,
    each add, multiply, divide, min or max one operation; prefill link terms, which do not
    depend on the candidate, count one add each).  The kernel costs the groups that the decode
    pass's memory-row screen leaves (a group holding a GPU that fails the memory row of every
    strategy of its size is settled there, its outputs all zero; no screen with the asymmetric
    split).  For a costed group every admissible strategy costs its memory row, and a strategy
    whose memory row admits a batch of 1 costs the full latency sum.  With request classes a
    strategy is costed class by class until a class does not fit, and each costed class adds 4
    operations to the mix.  Under the shared-groups hint the groups handed candidate 0's outputs
    are not the kernel's (exclude, from shared_with_first).  Returns (operations, divisions among
    them): a binary64 division is about ten VALU instructions on gfx9, so it is reported apart."""
    m = prob.model
    L = m["n_layers"]
    H = float(m["hidden"])
    Hkv = float(m["hidden"] * m["n_kv_heads"] // m["n_heads"])
    B = float(m["bytes_per_elem"])
    W12 = 12.0 * H * H * B
    classes = getattr(prob, "classes", None)
    tasks = [(prob.s_in, prob.s_out)] if classes is None else [(float(i), float(o)) for i, o, _ in classes]
    mix_ops = 0 if classes is None else 4
    screened_variant = not (getattr(prob, "variant", 0) & 4)
    cl = prob.cluster
    gt = np.asarray(cl.gpu_type)
    ok_t = (gt >= 0) & (gt < len(cl.type_mem))
    gmem = np.where(ok_t, np.asarray(cl.type_mem, np.float64)[np.clip(gt, 0, len(cl.type_mem) - 1)], 0.0)
    wild = np.isnan(gmem)
    tps = [t for t in range(1, 9) if (prob.tp_mask >> (t - 1)) & 1]
    total = divs = 0.0
    for sz, (mem, role) in group_members(prob, exclude).items():
        dec = role == 1
        strats = [(tp, sz // tp) for tp in tps if sz % tp == 0 and sz // tp <= 8
                  and (prob.pp_mask >> (sz // tp - 1)) & 1 and sz // tp <= L]
        # the screen: GPUs failing every strategy's memory row at floor(L/pp) layers
        fail_all = np.ones(len(gmem), bool)
        for tp, pp in strats:
            l = L // pp
            fails = np.zeros(len(gmem), bool)
            for s_in, s_out in tasks:
                K = (2.0 * (s_in + s_out) * Hkv * B / tp) * l + 4.0 * (s_in + s_out) * H * B
                fails |= np.floor((gmem - (W12 / tp) * l) / K) < 1.0
            fail_all &= fails
        costed = np.ones(len(mem), bool)
        if screened_variant:
            costed = ~(fail_all[mem].any(axis=1) & ~wild[mem].any(axis=1))
        for tp, pp in strats:
            alive = costed.copy()
            for s_in, s_out in tasks:
                Kkv = 2.0 * (s_in + s_out) * Hkv * B
                Kact = 4.0 * (s_in + s_out) * H * B
                bmin = np.full(len(mem), 2.0 ** 30)
                for j in range(pp):
                    l = L // pp + (1 if j < L % pp else 0)
                    A = (W12 / tp) * l
                    Kj = (Kkv / tp) * l + Kact
                    mm = gmem[mem[:, j * tp:(j + 1) * tp]].min(axis=1)
                    bmin = np.minimum(bmin, np.floor((mm - A) / Kj))
                feas = alive & (bmin >= 1.0)
                total += int(alive.sum()) * pp * (tp + 8)
                divs += int(alive.sum()) * (2 + pp)  # W12 / t, K_kv / t, one per stage
                nf_d = int((feas & dec).sum())
                nf_p = int((feas & ~dec).sum())
                common = 4 + 4 + pp * (2 + (tp - 1) + 2) + 3
                pre = common + pp * (3 + tp * (tp - 1) + 2) + (pp - 1) * (tp * tp + 1)
                dcd = common + pp * ((tp - 1) + 7 + 4 * tp * (tp - 1) + 3) + (pp - 1) * (3 * tp * tp + 2)
                total += nf_p * (pre + mix_ops) + nf_d * (dcd + mix_ops)
                # prefill: computation per stage and x (link terms from tables); decode: two
                # computation terms per stage, X / (t beta) per ordered TP pair, X / beta per PP
                # pair, and x; a class mix adds w / x
                mix_div = 1 if mix_ops else 0
                divs += nf_p * (pp + 1 + mix_div) + nf_d * (2 * pp + tp * (tp - 1) * pp + tp * tp * (pp - 1) + 1 + mix_div)
                alive = feas
    return float(total), float(divs)


def roofline_for(dominant, kernel_us, prob, hbm, n_p, n_d, workload, kbytes=None, exclude=None):
    """Roofline object of one kernel: FP64 ALU for the strategy evaluation, LDS for the
    max-flow, HBM for the streaming kernels.  exclude: the slots the shared-groups hint takes
    out of the evaluation kernel."""
    t_dom = kernel_us[dominant] * 1e-6
    if dominant == "eval":
        ops, divs = eval_fp64_counts(prob, exclude)
        achieved = ops / t_dom / 1e9
        # the same work weighted by issue cost: a division as ten operations
        weighted = (ops + 9.0 * divs) / t_dom / 1e9
        roof = {"kernel": "eval (hx_cost_eval)", "bound": "alu", "achieved": achieved, "peak": FP64_VALU_PEAK_GOPS,
                "unit": "GFLOP/s", "frac": achieved / FP64_VALU_PEAK_GOPS,
                "traffic": kernel_traffic("eval", workload, prob), "algorithmic_flops_per_launch": ops,
                "fp64_divisions_per_launch": divs, "division_weighted_gops": weighted,
                "division_weighted_frac": weighted / FP64_VALU_PEAK_GOPS}
    elif dominant == "maxflow":
        alg = float(lds_floor_bytes(n_p, n_d).sum())
        achieved = alg / t_dom / 1e9
        roof = {"kernel": "maxflow (hx_maxflow_batch)", "bound": "lds", "achieved": achieved,
                "peak": LDS_PEAK_GBS, "unit": "GB/s", "frac": achieved / LDS_PEAK_GBS,
                "traffic": kernel_traffic("maxflow", workload, prob), "algorithmic_bytes_per_launch": alg}
    else:
        if kbytes is not None and dominant in kbytes:
            alg = float(kbytes[dominant])
        else:
            call = {"setup": "cost", "decode": "cost", "scatter": "cost", "nodes": "flownet", "kv": "flownet"}.get(
                dominant, dominant)
            alg = float(hbm[call])
        achieved = alg / t_dom / 1e9
        roof = {"kernel": dominant, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS, "traffic": kernel_traffic(dominant, workload, prob),
                "algorithmic_bytes_per_launch": alg}
    roof["avg_launch_us"] = kernel_us[dominant]
    return roof


def moves_hbm_bytes(G: int, K: int, n_child: int) -> int:
    """Algorithmic HBM bytes of one guided-moves launch: every child's assign and role column
    and move word written, its 8-byte draw read (the parent's few hundred bytes are cached)."""
    return n_child * (G + K + 4 + 8)


def refine_main(args, torch, hx, I):
    """Max-flow guided refinement rounds (Sec. 3.4) on the 128-GPU workload with per-GPU flow
    nodes: each round scores the parent with a flow assignment, classifies its edges, emits
    --children guided children (child 0 = the parent), scores them and keeps the best."""
    cfg = 5
    wl = I.WORKLOADS[cfg]
    base = I.base_placement(wl)
    prob0 = dataclasses.replace(I.make_problem(cfg, n_cand=1), assign=np.ascontiguousarray(base[0].reshape(-1, 1)),
                                role=np.ascontiguousarray(base[1].reshape(-1, 1)))
    n_child = args.children
    rounds_total = args.warmup + args.steps
    draws = [torch.as_tensor(I.move_draws(cfg, r, n_child).view(np.int64)).to("cuda") for r in range(rounds_total)]
    dp = hx.DeviceProblem.upload(prob0)
    hint = not args.no_shared_groups_hint
    ref = hx.Refiner.create(dp, 0, n_child, shared_groups_hint=hint)
    trace = []
    for r in range(args.warmup):
        ref.round(draws[r])
        trace.append(int(ref.child_ws.best[1].item()))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for r in range(args.warmup, rounds_total):
        ref.round(draws[r])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_round = (t1 - t0) * 1000.0 / args.steps
    value = n_child / (ms_per_round / 1000.0)
    final = [int(x) for x in ref.child_ws.best.cpu().numpy()]

    # per-kernel durations over a replay of the same rounds from the same start
    ref2 = hx.Refiner.create(dp, 0, n_child, shared_groups_hint=hint)
    hx.profile(True)
    for r in range(rounds_total):
        ref2.round(draws[r])
    torch.cuda.synchronize()
    prof = hx.profile_read()
    hx.profile(False)
    kernel_us = {k: 1000.0 * ms / n for k, (ms, n) in prof.items() if n > 0}
    kernel_ms_per_round = {k: ms / rounds_total for k, (ms, n) in prof.items() if n > 0}
    child = ref.children
    cp = dataclasses.replace(prob0, assign=child.tensors["assign"].cpu().numpy(),
                             role=child.tensors["role"].cpu().numpy())
    n_p = ref.child_ws.net.n_p.cpu().numpy()
    n_d = ref.child_ws.net.n_d.cpu().numpy()
    hbm = hbm_bytes_per_step(cp, ref.child_ws.net.dims, n_p, n_d)
    hbm["moves"] = moves_hbm_bytes(cp.n_gpus, cp.max_groups, n_child)
    # the children's scoring kernels run once per round on the full batch; the parent's on one
    # candidate: the dominant kernel by time per round
    dominant = max(kernel_ms_per_round, key=kernel_ms_per_round.get)
    scoring = {"setup", "decode", "scatter", "eval", "nodes", "kv", "maxflow", "best"}
    if dominant in scoring:
        # a round launches each scoring kernel twice, on the parent (one candidate) and on the
        # children; the roofline charges the children's work with both launches' time
        kb = kernel_bytes(cp, n_p, n_d, settled_per_gpu=cp.n_gpus <= 128)
        roof = roofline_for(dominant, {dominant: 1000.0 * kernel_ms_per_round[dominant]}, cp, hbm, n_p, n_d, cfg, kb,
                            exclude=shared_with_first(cp) if hint else None)
    else:
        alg = float(hbm.get(dominant, 0))
        t = kernel_ms_per_round[dominant] * 1e-3
        roof = {"kernel": dominant, "bound": "hbm", "achieved": alg / t / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": alg / t / 1e9 / HBM_PEAK_GBS, "traffic": None, "algorithmic_bytes_per_launch": alg,
                "avg_launch_us": 1000.0 * kernel_ms_per_round[dominant]}
    t_mv = kernel_us["moves"] * 1e-6
    import hashlib
    mt = None
    src = os.path.join(ROOT, "paper_2502_07903_amd", "csrc", "hx_refine.hip")
    if (hashlib.sha256(open(src, "rb").read()).hexdigest()[:16] == MOVES_TRAFFIC["source_sha256_16"]
            and n_child == MOVES_TRAFFIC["children"]):
        mt = 1024.0 * (MOVES_TRAFFIC["fetch_kib"] * COUNTER_SCALE["fetch"] + MOVES_TRAFFIC["write_kib"] * COUNTER_SCALE["write"])
    moves_roof = {"kernel": "moves (hx_guided_moves)", "bound": "hbm", "achieved": hbm["moves"] / t_mv / 1e9,
                  "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": hbm["moves"] / t_mv / 1e9 / HBM_PEAK_GBS,
                  "traffic": mt, "algorithmic_bytes_per_launch": hbm["moves"], "avg_launch_us": kernel_us["moves"]}

    # quality beside it: random single-step perturbations (the same move kinds, drawn without
    # the max-flow classes) for the same number of rounds, scored on the GPU
    rand_best = None
    if args.quality_rounds > 0:
        cur = (base[0].copy(), base[1].copy())
        ws_r = None
        rand_best = []
        for r in range(args.quality_rounds):
            pr = I.make_problem(cfg, n_cand=n_child, rnd=r, base=cur)
            dpr = hx.DeviceProblem.upload(pr)
            if ws_r is None:
                ws_r = hx.Workspace.for_problem(dpr)
            hx.score(dpr, ws_r)
            bi, bv = (int(x) for x in ws_r.best.cpu().numpy())
            rand_best.append(bv)
            cur = (pr.assign[:, bi].copy(), pr.role[:, bi].copy())
        ref3 = hx.Refiner.create(dp, 0, n_child, shared_groups_hint=hint)
        guided_best = []
        for r in range(args.quality_rounds):
            ref3.round(draws[r] if r < rounds_total else
                       torch.as_tensor(I.move_draws(cfg, r, n_child).view(np.int64)).to("cuda"))
            guided_best.append(int(ref3.child_ws.best[1].item()))

    out = {
        "metric": "guided refinement children generated and scored/sec (Sec. 3.4 round) at 1 GPU",
        "value": value,
        "unit": "children/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_round,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64+i32",
        "data": "synthetic",
        "config": {"workload": f"workload{cfg}: {wl.name}, max-flow guided rounds from the one-group-per-node base",
                   "children_per_round": n_child, "cluster_gpus": cp.n_gpus, "max_groups": cp.max_groups,
                   "granularity": cp.granularity, "shared_groups_hint": hint},
        "kernel_ms_per_round": kernel_ms_per_round,
        "best_after_warmup_rounds": trace,
        "best": final,
        "roofline": roof,
        "moves_roofline": moves_roof,
    }
    if rand_best is not None:
        out["quality"] = {"rounds": args.quality_rounds, "guided_best_per_round": guided_best,
                          "random_best_per_round": rand_best,
                          "random_best_so_far": [int(x) for x in np.maximum.accumulate(rand_best)]}

    if not args.no_cpu_baseline:
        from oracle import hxo  # test infrastructure: only this baseline leg uses it
        cores = max(1, min(len(os.sched_getaffinity(0)), 64))
        t = time.perf_counter()
        r = hxo.score_batch(cp, n_threads=cores)
        first = time.perf_counter() - t
        reps = max(1, min(50, int(args.cpu_seconds / max(first, 1e-3))))
        times = [first]
        for _ in range(reps - 1):
            t = time.perf_counter()
            hxo.score_batch(cp, n_threads=cores)
            times.append(time.perf_counter() - t)
        med = float(np.median(times))
        # one thread on a bounded sample (about a tenth of the all-core time budget)
        m1 = int(min(cp.n_cand, max(256, cp.n_cand * (args.cpu_seconds / 10.0) / (med * cores))))
        t = time.perf_counter()
        hxo.score_batch(cp.subset(np.arange(m1)), n_threads=1)
        one = m1 / (time.perf_counter() - t)
        gpu_fv = ref.child_ws.flow_value.cpu().numpy()
        out["cpu_baseline"] = {"value": cp.n_cand / med, "unit": "children/s", "cores": cores, "kind": "oracle",
                               "sample": f"the last round's {cp.n_cand} children scored, {len(times)} runs, median; "
                                         f"1 thread: the first {m1} children",
                               "single_thread": {"value": one, "unit": "children/s", "cores": 1},
                               "agrees": bool(np.array_equal(r["flow_value"], gpu_fv)) and list(r["best"]) == final,
                               "cpu": cpu_model()}
    print(json.dumps(out))


def partition_main(args, torch, hx, I):
    """The first phase of Sec. 3.2 as a candidate generator on the headline workload: one
    spectral order, then --partition-candidates candidates (one draw each), each scored by the
    hot path.  value = candidates generated and scored per second."""
    cfg = args.workload
    wl = I.WORKLOADS[cfg]
    n = args.partition_candidates
    prob = I.make_problem(cfg, n_cand=1)
    dp = hx.DeviceProblem.upload(prob)
    ws = hx.partition_workspace(dp)
    order = torch.empty(prob.n_gpus, dtype=torch.int32, device="cuda")
    rnd = torch.as_tensor(I.partition_draws(cfg, n).view(np.int64)).to("cuda")
    assign = torch.empty((prob.n_gpus, n), dtype=torch.uint8, device="cuda")
    role = torch.empty((prob.max_groups, n), dtype=torch.uint8, device="cuda")
    cand = dp.with_candidates(assign, role)
    wsc = hx.Workspace.for_problem(cand)

    def step():
        hx.spectral_order(dp, ws, order, iters=args.spectral_iters)
        hx.partition_candidates(dp, ws, order, rnd, assign, role)
        hx.score(cand, wsc)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1000.0 / args.steps
    hx.profile(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    prof = hx.profile_read()
    hx.profile(False)
    kernel_us = {k: 1000.0 * v / c for k, (v, c) in prof.items() if c > 0}
    best = [int(x) for x in wsc.best.cpu().numpy()]
    # the partition kernel against HBM: its algorithmic bytes are the candidates it writes (the
    # weight table and order stay in cache); its time goes to Kernighan-Lin steps, each a
    # workgroup-wide scan of the GPU pairs and two barriers, so the fraction is small
    t_part = kernel_us["partition"] * 1e-6
    out_bytes = n * (prob.n_gpus + prob.max_groups)
    import hashlib
    src = os.path.join(ROOT, "paper_2502_07903_amd", "csrc", "hx_partition.hip")
    ptraffic = None
    if (hashlib.sha256(open(src, "rb").read()).hexdigest()[:16] == PARTITION_TRAFFIC["source_sha256_16"]
            and n == PARTITION_TRAFFIC["candidates"] and cfg == 3):
        ptraffic = 1024.0 * (PARTITION_TRAFFIC["fetch_kib"] * COUNTER_SCALE["fetch"]
                             + PARTITION_TRAFFIC["write_kib"] * COUNTER_SCALE["write"])
    out = {
        "metric": "graph-partition candidates generated and scored/sec (Sec. 3.2 first phase + hot path) at 1 GPU",
        "value": n / (ms / 1000.0),
        "unit": "candidates/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64+i64", "data": "synthetic",
        "config": {"workload": f"workload{wl.cfg}: {wl.name}, graph-partition candidates", "candidates": n,
                   "cluster_gpus": prob.n_gpus, "max_groups": prob.max_groups, "spectral_iters": args.spectral_iters},
        "kernel_us": kernel_us,
        "best": best,
        "partition_roofline": {"kernel": "partition (hx_partition_candidates)", "bound": "hbm",
                               "achieved": out_bytes / t_part / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                               "frac": out_bytes / t_part / 1e9 / HBM_PEAK_GBS, "traffic": ptraffic,
                               "algorithmic_bytes_per_launch": out_bytes, "avg_launch_us": kernel_us["partition"]},
    }
    if not args.no_cpu_baseline:
        from oracle import hxo  # test infrastructure: only this baseline leg uses it
        t = time.perf_counter()
        o_order, _ = hxo.spectral_order(prob, args.spectral_iters)
        m = 64
        hxo.partition_candidates(prob, o_order, I.partition_draws(cfg, m))
        dt = time.perf_counter() - t
        out["cpu_baseline"] = {"value": m / dt, "unit": "candidates/s (generation only)", "cores": 1,
                               "kind": "oracle", "sample": f"spectral order + {m} candidates, one thread"}
    print(json.dumps(out))


def chain_main(args, torch, hx, I):
    """Workload 5 as defined: rounds of 131,072 single-step perturbations (45% move one GPU, 45%
    swap two GPUs, 10% merge two groups) of the previous round's best placement, the GPU argmax,
    from the one-group-per-node base; per-GPU flow nodes (up to 258 nodes, ~4,000 KV edges).
    Each round's batch is generated on the host (timed apart), copied to the GPU (timed apart),
    then scored --round-repeats times (each a whole scoring, host launch to synchronize; the
    round's time is their median, which drops one-off host stalls); value = all rounds'
    candidates / their summed scoring time, inputs resident."""
    cfg = 5
    wl = I.WORKLOADS[cfg]
    n = args.candidates or wl.n_cand
    rounds = args.rounds or wl.rounds
    G = wl.n_gpus
    cur = I.base_placement(wl)
    prob = I.make_problem(cfg, n_cand=n, rnd=0, base=cur)
    # every candidate is one move away from the same placement: candidate 0's groups are costed
    # once and shared (HX_HINT_SHARED_GROUPS; the outputs are the same without it)
    dp = hx.DeviceProblem.upload(prob).with_hint(not args.no_shared_groups_hint)
    ws = hx.Workspace.for_problem(dp, flows=False)
    h_assign = torch.empty((G, n), dtype=torch.uint8).pin_memory()
    h_role = torch.empty((prob.max_groups, n), dtype=torch.uint8).pin_memory()
    d_assign, d_role = dp.tensors["assign"], dp.tensors["role"]
    for _ in range(args.warmup):
        hx.score_batch(dp, ws)
    torch.cuda.synchronize()
    per_round, probs = [], []
    for r in range(rounds):
        t = time.perf_counter()
        pr = prob if r == 0 else I.make_problem(cfg, n_cand=n, rnd=r, base=cur)
        gen_s = time.perf_counter() - t
        h_assign.copy_(torch.from_numpy(pr.assign))
        h_role.copy_(torch.from_numpy(pr.role))
        torch.cuda.synchronize()
        t = time.perf_counter()
        d_assign.copy_(h_assign, non_blocking=True)
        d_role.copy_(h_role, non_blocking=True)
        torch.cuda.synchronize()
        h2d_ms = (time.perf_counter() - t) * 1000.0
        times = []
        for _ in range(max(1, args.round_repeats)):
            t = time.perf_counter()
            hx.score_batch(dp, ws)
            torch.cuda.synchronize()
            times.append((time.perf_counter() - t) * 1000.0)
        score_ms = float(np.median(times))
        bi, bv = (int(x) for x in ws.best.cpu().numpy())
        per_round.append({"round": r, "score_ms": score_ms, "first_pass_ms": times[0], "h2d_ms": h2d_ms,
                          "host_generation_s": gen_s, "best_index": bi, "best_flow": bv})
        probs.append((pr, bi, bv))
        cur = (pr.assign[:, bi].copy(), pr.role[:, bi].copy())
        print(f"[chain] round {r}: {score_ms:.3f} ms, best {bv} at {bi}", file=sys.stderr, flush=True)
    total_ms = sum(x["score_ms"] for x in per_round)
    value = rounds * n / (total_ms / 1000.0)

    # per-kernel durations: the last round's batch scored again with libhx's kernel events
    hx.profile(True)
    for _ in range(args.steps):
        hx.score_batch(dp, ws)
    torch.cuda.synchronize()
    prof = hx.profile_read()
    hx.profile(False)
    kernel_us = {k: 1000.0 * ms / c for k, (ms, c) in prof.items() if c > 0}
    # the counters need every network in full: hx_score_batch leaves the KV rows of the networks
    # it settled from the link table unwritten, so the network is built again by the two calls
    hx.cost_eval(dp, ws.cost)
    hx.build_flownet(dp, ws.cost, ws.net)
    mf = hx.maxflow_stats(ws.net, torch.empty_like(ws.flow_value))
    last = probs[-1][0]
    n_p = ws.net.n_p.cpu().numpy()
    n_d = ws.net.n_d.cpu().numpy()
    hbm = hbm_bytes_per_step(last, ws.net.dims, n_p, n_d)
    kb = kernel_bytes(last, n_p, n_d, settled_per_gpu=last.granularity == 1 and last.n_gpus <= 128)
    dominant = max(kernel_us, key=kernel_us.get)
    roof = roofline_for(dominant, kernel_us, last, hbm, n_p, n_d, cfg, kb,
                        exclude=None if args.no_shared_groups_hint else shared_with_first(last))
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": rounds,
        "warmup": args.warmup,
        "ms_per_step": total_ms / rounds,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64+i32",
        "data": "synthetic",
        "config": {"workload": f"workload5: {wl.name}; {rounds} chained rounds of {n:,}, each perturbing "
                               "the previous round's GPU best",
                   "candidates": rounds * n, "cluster_gpus": G, "max_groups": prob.max_groups,
                   "granularity": prob.granularity, "shared_groups_hint": not args.no_shared_groups_hint,
                   "round_repeats": max(1, args.round_repeats)},
        "rounds": per_round,
        "host_generation_s": sum(x["host_generation_s"] for x in per_round),
        "first_pass": {"value": rounds * n / (sum(x["first_pass_ms"] for x in per_round) / 1000.0),
                       "unit": "candidates/s",
                       "note": "each round's first scoring only (right after its batch is copied in)"},
        "with_h2d_copy": {"value": rounds * n / ((total_ms + sum(x["h2d_ms"] for x in per_round)) / 1000.0),
                          "unit": "candidates/s", "note": "each round's assign and role copied from pinned host memory"},
        "kernel_us": kernel_us,
        "maxflow_paths": mf,
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        from oracle import hxo  # test infrastructure: only this baseline leg uses it
        # the oracle on a bounded sample of the last round (plus every round's GPU best, which
        # it must score the same)
        m = min(n, 2048)
        sub = last.subset(np.arange(m))
        cores = max(1, min(len(os.sched_getaffinity(0)), 64))
        t = time.perf_counter()
        ra = hxo.score_batch(sub, n_threads=cores)
        all_cores = m / (time.perf_counter() - t)
        m1 = min(m, 256)
        t = time.perf_counter()
        hxo.score_batch(last.subset(np.arange(m1)), n_threads=1)
        one = m1 / (time.perf_counter() - t)
        gpu_fv = ws.flow_value.cpu().numpy()
        agrees = bool(np.array_equal(ra["flow_value"], gpu_fv[:m]))
        for pr, bi, bv in probs:
            agrees = agrees and int(hxo.score_batch(pr.subset(np.array([bi])))["flow_value"][0]) == bv
        out["cpu_baseline"] = {"value": all_cores, "unit": "candidates/s", "cores": cores, "kind": "oracle",
                               "sample": f"the first {m} candidates of the last round on {cores} threads; "
                                         f"1 thread: the first {m1}",
                               "single_thread": {"value": one, "unit": "candidates/s", "cores": 1},
                               "agrees": agrees, "cpu": cpu_model()}
    print(json.dumps(out))


# Network shapes of the push-relabel leg: (max_p, max_d, max_pd, nodes per side (lo, hi), N).
PR_SHAPES = {"workload3": (16, 16, 64, (2, 8), 65536), "workload5": (128, 128, 4096, (16, 64), 4096)}


def pushrelabel_networks(shape: str, seed: int = 7903):
    """Seeded networks of a workload's shape that need push-relabel: P, D nodes per side drawn in
    the shape's range (P * D within its KV rows), node capacities a_i, b_j uniform in [1, 10^4]
    (the per-GPU and replica capacities of the workloads are of that order), source and sink edges
    unbounded, and every KV arc a uniform draw in [0, min(a_i, b_j) - 1]: below what it would
    need to carry for the closed form, so the flow must be found by pushes and relabels."""
    mp, md, mpd, (lo, hi), N = PR_SHAPES[shape]
    rng = np.random.default_rng(seed)
    n_p = rng.integers(lo, hi + 1, N)
    n_d = np.minimum(rng.integers(lo, hi + 1, N), mpd // n_p)
    fn = {"n_p": n_p.astype(np.int32), "n_d": n_d.astype(np.int32), "dims": (mp, md, mpd)}
    for k, rows in (("src_cap", mp), ("p_cap", mp), ("d_cap", md), ("sink_cap", md), ("kv_cap", mpd),
                    ("p_slot", mp), ("d_slot", md)):
        fn[k] = np.zeros((rows, N), np.int32)
    a = rng.integers(1, 10001, (mp, N)) * (np.arange(mp)[:, None] < n_p[None, :])
    b = rng.integers(1, 10001, (md, N)) * (np.arange(md)[:, None] < n_d[None, :])
    fn["p_cap"][:] = a
    fn["d_cap"][:] = b
    fn["src_cap"][:] = np.where(a > 0, 16777215, 0)
    fn["sink_cap"][:] = np.where(b > 0, 16777215, 0)
    fn["p_slot"][:] = np.arange(mp)[:, None]
    fn["d_slot"][:] = np.arange(md)[:, None]
    e = np.arange(mpd)[:, None]
    row_i, row_j = e // n_d[None, :], e % n_d[None, :]
    live = e < (n_p * n_d)[None, :]
    amin = np.minimum(np.take_along_axis(a, np.minimum(row_i, mp - 1), 0),
                      np.take_along_axis(b, np.minimum(row_j, md - 1), 0))
    fn["kv_cap"][:] = np.where(live, np.floor(rng.random((mpd, N)) * amin), 0).astype(np.int32)
    return fn


def pushrelabel_main(args, torch, hx):
    """The max-flow kernel alone on networks that need push-relabel (with flows and the canonical
    cut requested, as the refinement step asks), at a workload's network shapes."""
    fn = pushrelabel_networks(args.pushrelabel)
    net = hx.FlowNetBuffers.from_host(fn)
    N = int(fn["n_p"].shape[0])
    mp, md, mpd = fn["dims"]
    fv = torch.empty(N, dtype=torch.int32, device="cuda")
    kv = torch.empty((mpd, N), dtype=torch.int32, device="cuda")
    cut = torch.empty((mp + md, N), dtype=torch.uint8, device="cuda")
    for _ in range(args.warmup):
        hx.maxflow_batch(net, fv, kv, cut)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        hx.maxflow_batch(net, fv, kv, cut)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1000.0 / args.steps
    hx.profile(True)
    for _ in range(args.steps):
        hx.maxflow_batch(net, fv, kv, cut)
    torch.cuda.synchronize()
    prof = hx.profile_read()
    hx.profile(False)
    kernel_us = {k: 1000.0 * t / c for k, (t, c) in prof.items() if c > 0}
    st = hx.maxflow_stats(net, torch.empty_like(fv), torch.empty_like(kv), torch.empty_like(cut))
    pr = max(1, st["push_relabel"])
    alg = float(lds_floor_bytes(fn["n_p"], fn["n_d"]).sum())
    t_mf = kernel_us["maxflow"] * 1e-6
    out = {
        "metric": "push-relabel networks solved/sec (max-flow with flows and cut) at 1 GPU",
        "value": N / (ms / 1000.0), "unit": "networks/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "i32",
        "data": "synthetic",
        "config": {"workload": f"push-relabel networks at {args.pushrelabel} shapes", "networks": N,
                   "max_p": mp, "max_d": md, "max_pd": mpd},
        "kernel_us": kernel_us,
        "maxflow_paths": st,
        "per_push_relabel_network": {"pushes": st["pushes"] / pr, "relabels": st["relabels"] / pr},
        "per_workgroup": {"global_relabels": st["global_relabels"], "rounds": st["rounds"]},
        "roofline": {"kernel": "maxflow (hx_maxflow_batch)", "bound": "lds", "achieved": alg / t_mf / 1e9,
                     "peak": LDS_PEAK_GBS, "unit": "GB/s", "frac": alg / t_mf / 1e9 / LDS_PEAK_GBS, "traffic": None,
                     "algorithmic_bytes_per_launch": alg, "avg_launch_us": kernel_us["maxflow"],
                     "note": "algorithmic bytes = the residual graph written once and every arc read once; "
                             "push-relabel reads arcs many times per network (pushes, relabels above)"},
    }
    if not args.no_cpu_baseline:
        from oracle import hxo  # test infrastructure: only this baseline leg uses it
        m = N if args.pushrelabel == "workload3" else min(N, 2048)
        sub = {k: (np.ascontiguousarray(v[..., :m]) if isinstance(v, np.ndarray) else v) for k, v in fn.items()}
        t = time.perf_counter()
        want = hxo.maxflow_batch(sub, want_flows=True)
        rate = m / (time.perf_counter() - t)
        out["cpu_baseline"] = {"value": rate, "unit": "networks/s", "cores": 1, "kind": "oracle",
                               "sample": f"the first {m} networks, Edmonds-Karp on one thread",
                               "agrees": bool(np.array_equal(want["flow_value"], fv.cpu().numpy()[:m])),
                               "cpu": cpu_model()}
    print(json.dumps(out))


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark measures one GPU: candidates are independent, so the path "
                                   "shards by candidate range with one 8-byte argmax exchange; run with --gpus 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch
    from paper_2502_07903_amd import hx
    from paper_2502_07903_amd import inputs as I

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    hx.lib()
    if args.copy_mib > 0:
        src = torch.ones(args.copy_mib * (1 << 18), dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.refine:
        refine_main(args, torch, hx, I)
        return
    if args.partition:
        partition_main(args, torch, hx, I)
        return
    if args.workload == 5:
        chain_main(args, torch, hx, I)
        return
    if args.pushrelabel:
        pushrelabel_main(args, torch, hx)
        return
    wl = I.WORKLOADS[args.workload]
    prob = I.make_problem(args.workload, n_cand=args.candidates or None)
    if VARIANTS[args.variant]:
        prob = dataclasses.replace(prob, variant=VARIANTS[args.variant])
    if args.classes:
        prob = dataclasses.replace(prob, classes=I.length_classes(wl, args.classes))
    dp = hx.DeviceProblem.upload(prob)
    ws = hx.Workspace.for_problem(dp, flows=False)
    stream = torch.cuda.current_stream()
    # Independent steps in flight: step s runs on stream s mod S with workspace s mod S (every
    # kernel of a step is bound by the latency of its longest chains, so steps on other streams
    # fill the chip meanwhile).  Inputs are shared and only read; all streams at default priority.
    n_str = max(1, args.streams)
    streams = [stream] + [torch.cuda.Stream() for _ in range(n_str - 1)]
    wss = [ws] + [hx.Workspace.for_problem(dp, flows=False) for _ in range(n_str - 1)]

    for _ in range(args.warmup):
        for i in range(n_str):
            hx.score_batch(dp, wss[i], stream=streams[i])
    torch.cuda.synchronize()

    # Timed region: K steps and nothing else (event markers between the calls cost the GPU a
    # few microseconds each, so the per-call durations come from a separate pass below).
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for st in range(args.steps):
        hx.score_batch(dp, wss[st % n_str], stream=streams[st % n_str])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1000.0 / args.steps
    value = prob.n_cand / (ms_per_step / 1000.0)
    stream_bests = [[int(x) for x in w.best.cpu().numpy()] for w in wss]

    # With several streams in the timed region: up to 10 steps one after another on one stream,
    # the latency of one step.  Without: a short pass with --concurrent-streams steps in flight.
    # (Short, so that a kernel trace of the run averages over dispatches made like the passes
    # below, which keep the timed region's streams.)
    extra = None
    if n_str > 1:
        k1 = min(args.steps, 10)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(k1):
            hx.score_batch(dp, ws)
        torch.cuda.synchronize()
        ms1 = (time.perf_counter() - t0) * 1000.0 / k1
        extra = ("single_stream", {"value": prob.n_cand / (ms1 / 1000.0), "unit": "candidates/s", "ms_per_step": ms1,
                                   "note": "steps one after another on one stream (one step's latency)"})
    elif args.concurrent_streams > 1:
        nc = args.concurrent_streams
        cst = [stream] + [torch.cuda.Stream() for _ in range(nc - 1)]
        cws = [ws] + [hx.Workspace.for_problem(dp, flows=False) for _ in range(nc - 1)]
        for i in range(nc):
            hx.score_batch(dp, cws[i], stream=cst[i])
        kc = min(args.steps, 20)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for st in range(kc):
            hx.score_batch(dp, cws[st % nc], stream=cst[st % nc])
        torch.cuda.synchronize()
        msc = (time.perf_counter() - t0) * 1000.0 / kc
        cb = [[int(x) for x in w.best.cpu().numpy()] for w in cws]
        extra = ("concurrent_streams", {"streams": nc, "steps": kc, "value": prob.n_cand / (msc / 1000.0),
                                        "unit": "candidates/s", "ms_per_step": msc,
                                        "agree": all(b == stream_bests[0] for b in cb),
                                        "note": "independent steps in flight, each on its own stream with its own "
                                                "workspace and outputs (inputs shared, read only)"})

    # The same steps with the host-to-device copy of the candidate arrays (assign, role) from
    # pinned host memory in each step: the rate a caller holding its candidates on the host sees.
    # Each stream copies into its own input buffers, then scores them.
    h_assign = torch.from_numpy(prob.assign).pin_memory()
    h_role = torch.from_numpy(prob.role).pin_memory()
    dps = [dp] + [hx.DeviceProblem.upload(prob) for _ in range(n_str - 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for st in range(args.steps):
        i = st % n_str
        with torch.cuda.stream(streams[i]):
            dps[i].tensors["assign"].copy_(h_assign, non_blocking=True)
            dps[i].tensors["role"].copy_(h_role, non_blocking=True)
        hx.score_batch(dps[i], wss[i], stream=streams[i])
    torch.cuda.synchronize()
    ms_h2d = (time.perf_counter() - t0) * 1000.0 / args.steps

    # Per-call durations: the same steps again through the four calls, HIP events recorded
    # between the calls on the stream each step runs on (kept out of the timed region).
    names = ("cost", "flownet", "maxflow", "best")
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    for st in range(args.steps):
        e, i = ev[st], st % n_str
        sx, w = streams[i], wss[i]
        e[0].record(sx)
        hx.cost_eval(dp, w.cost, stream=sx)
        e[1].record(sx)
        hx.build_flownet(dp, w.cost, w.net, stream=sx)
        e[2].record(sx)
        hx.maxflow_batch(w.net, w.flow_value, stream=sx)
        e[3].record(sx)
        hx.best_candidate(w.flow_value, w.best, dp.n_cand, stream=sx)
        e[4].record(sx)
    torch.cuda.synchronize()
    per_kernel = {k: float(np.mean([ev[s][i].elapsed_time(ev[s][i + 1]) for s in range(args.steps)]))
                  for i, k in enumerate(names)}

    # Per-kernel durations: the same steps again, with the timed region's streams in flight, with
    # libhx recording HIP events around each of its kernels on the stream it runs on (kept out
    # of the timed region above).
    hx.profile(True)
    for st in range(args.steps):
        hx.score_batch(dp, wss[st % n_str], stream=streams[st % n_str])
    torch.cuda.synchronize()
    prof = hx.profile_read()
    hx.profile(False)
    kernel_us = {k: 1000.0 * ms / n for k, (ms, n) in prof.items() if n > 0}

    # How the max-flow solved the batch (diagnostic counters, one extra untimed call).
    mf = hx.maxflow_stats(ws.net, torch.empty_like(ws.flow_value))
    pr = mf["push_relabel"]
    mf["pushes_per_push_relabel_candidate"] = mf["pushes"] / pr if pr else 0.0
    mf["relabels_per_push_relabel_candidate"] = mf["relabels"] / pr if pr else 0.0

    # Roofline of the kernel with the largest share of the step.
    n_p = ws.net.n_p.cpu().numpy()
    n_d = ws.net.n_d.cpu().numpy()
    dims = ws.net.dims
    best = [int(x) for x in ws.best.cpu().numpy()]
    dominant = max(kernel_us, key=kernel_us.get)
    hbm = hbm_bytes_per_step(prob, dims, n_p, n_d)
    kb = kernel_bytes(prob, n_p, n_d, settled_per_gpu=prob.granularity == 1 and prob.n_gpus <= 128)
    roof = roofline_for(dominant, kernel_us, prob, hbm, n_p, n_d, args.workload, kb)
    roof["measured_hbm_copy_gbs"] = measured_copy_gbs(torch)

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64+i32",
        "data": "synthetic",
        "config": {"workload": f"workload{wl.cfg}: {wl.name}" +
                               (f", scored in batches of {prob.n_cand:,}" if args.candidates else ""),
                   "candidates": prob.n_cand,
                   "cluster_gpus": prob.n_gpus, "max_groups": prob.max_groups, "granularity": prob.granularity,
                   "cost_model": args.variant, "request_classes": args.classes, "streams": n_str},
        "streams_agree": all(b == stream_bests[0] for b in stream_bests),
        "with_h2d_copy": {"value": prob.n_cand / (ms_h2d / 1000.0), "unit": "candidates/s",
                          "ms_per_step": ms_h2d,
                          "note": "assign and role copied from pinned host memory in every step"},
        "kernel_ms": per_kernel,
        "kernel_us": kernel_us,
        "maxflow_paths": mf,
        "hbm_bytes_per_step": hbm,
        "best": best,
        "roofline": roof,
    }
    if extra is not None:
        out[extra[0]] = extra[1]
    if dominant != "maxflow" and "maxflow" in kernel_us and mf["push_relabel"] > 0:
        # the LDS-resident max-flow beside the dominant kernel, against the LDS peak, when some
        # candidate needed push-relabel (closed forms touch their arcs once, so an LDS fraction
        # of those would credit work the kernel never did)
        out["maxflow_roofline"] = roofline_for("maxflow", kernel_us, prob, hbm, n_p, n_d, args.workload)

    if not args.no_cpu_baseline:
        from oracle import hxo  # test infrastructure: only this baseline leg uses it
        cores = max(1, min(len(os.sched_getaffinity(0)), 64))
        t = time.perf_counter()
        r = hxo.score_batch(prob, n_threads=cores)
        first = time.perf_counter() - t
        reps = max(1, min(50, int(args.cpu_seconds / max(first, 1e-3))))
        times = [first]
        for _ in range(reps - 1):
            t = time.perf_counter()
            hxo.score_batch(prob, n_threads=cores)
            times.append(time.perf_counter() - t)
        med = float(np.median(times))
        # one thread on a bounded sample (about a tenth of the all-core time budget)
        m1 = int(min(prob.n_cand, max(256, prob.n_cand * (args.cpu_seconds / 10.0) / (med * cores))))
        t = time.perf_counter()
        hxo.score_batch(prob.subset(np.arange(m1)), n_threads=1)
        one = m1 / (time.perf_counter() - t)
        gpu_fv = ws.flow_value.cpu().numpy()
        out["cpu_baseline"] = {"value": prob.n_cand / med, "unit": "candidates/s", "cores": cores, "kind": "oracle",
                               "sample": f"the full {prob.n_cand}-candidate batch, {len(times)} runs, median; "
                                         f"1 thread: the first {m1} candidates",
                               "single_thread": {"value": one, "unit": "candidates/s", "cores": 1},
                               "agrees": bool(np.array_equal(r["flow_value"], gpu_fv)) and list(r["best"]) == best,
                               "cpu": cpu_model()}
    print(json.dumps(out))


if __name__ == "__main__":
    main()
