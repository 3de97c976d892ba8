"""Benchmark: candidate placements scored per second on one MI355X.

A step is one pass of the whole hot path over one batch of candidate placements with the
inputs already resident in HBM: cost model (hx_cost_eval) -> flow network
(hx_build_flownet) -> max-flow (hx_maxflow_batch) -> best candidate (hx_best_candidate).
The default workload is the 32-GPU / 8-node / 4-type cluster serving a Llama-2-70B-shaped
model with lognormal request lengths, 65,536 seeded random candidates of 2-16 groups.

    python bench.py [--gpus 1] [--steps 50] [--warmup 5] [--workload 3] [--no-cpu-baseline]

Prints ONE JSON line.  Per-call durations come from HIP events recorded around every call
inside the timed region, on the stream the kernels run on; per-kernel durations from a second
pass of the same steps with libhx's diagnostic per-kernel events (hx_profile).  The roofline
object reports the kernel with the largest share.  The CPU baseline times the oracle (test
infrastructure, not the product) on the same batch on the host's cores.
"""
from __future__ import annotations

import argparse
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
LDS_PEAK_GBS = 128 * 256 * 2.4          # 128 B/clk/CU -> 78,643 GB/s
# FP64 vector operations that are not fused multiply-adds: 256 CUs x 4 SIMDs x 16 lanes x
# 2.4 GHz = 39,322 G op/s (the 78.6 TFLOP/s headline counts an FMA as two).
FP64_VALU_PEAK_GOPS = 256 * 4 * 16 * 2.4

# HBM bytes per launch at workload 3 from rocprofv3 FETCH_SIZE and WRITE_SIZE passes
# (profiles/all_kernels_workload3.md), each scaled by what the counter reads for a 256 MiB
# device copy (FETCH_SIZE x 2.0, WRITE_SIZE x 1.0).  Valid only for the kernel source they were
# taken on (first 16 hex digits of the source file's SHA-256); otherwise traffic is null.
COUNTER_SCALE = {"fetch": 2.0, "write": 1.0}
KERNEL_TRAFFIC = {
    "setup": {"source_sha256_16": "2fe02144148e6483", "fetch_kib": 37.7, "write_kib": 32.5},
    "decode": {"source_sha256_16": "2fe02144148e6483", "fetch_kib": 1635.8, "write_kib": 22443.6},
    "scatter": {"source_sha256_16": "2fe02144148e6483", "fetch_kib": 4679.0, "write_kib": 9337.1},
    "eval": {"source_sha256_16": "2fe02144148e6483", "fetch_kib": 5310.8, "write_kib": 65706.0},
    "nodes": {"source_sha256_16": "5fbd4e7404ecfaea", "fetch_kib": 6697.6, "write_kib": 20441.6},
    "kv": {"source_sha256_16": "5fbd4e7404ecfaea", "fetch_kib": 5895.5, "write_kib": 13399.1},
    "maxflow": {"source_sha256_16": "092d98a1f13d354c", "fetch_kib": 16706.6, "write_kib": 256.0},
    "best": {"source_sha256_16": "c5dd3bcb6e1178fe", "fetch_kib": 134.3, "write_kib": 0.0},
}
KERNEL_SOURCE = {"setup": "hx_cost.hip", "decode": "hx_cost.hip", "scatter": "hx_cost.hip", "eval": "hx_cost.hip",
                 "nodes": "hx_flownet.hip", "kv": "hx_flownet.hip", "maxflow": "hx_maxflow.hip",
                 "best": "hx_best.hip"}


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=3, choices=[1, 2, 3, 4])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU-baseline wall time")
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


def kernel_traffic(kernel: str, workload: int):
    """Counter-measured HBM bytes per launch of a kernel, or None when they do not apply."""
    import hashlib
    t = KERNEL_TRAFFIC.get(kernel)
    if t is None or workload != 3:
        return None
    src = os.path.join(ROOT, "paper_2502_07903_amd", "csrc", KERNEL_SOURCE[kernel])
    if hashlib.sha256(open(src, "rb").read()).hexdigest()[:16] != t["source_sha256_16"]:
        return None
    return 1024.0 * (t["fetch_kib"] * COUNTER_SCALE["fetch"] + t["write_kib"] * COUNTER_SCALE["write"])


def group_members(prob):
    """(members [U][size] ascending GPU ids, role [U]) of every present group, listed by size."""
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
    out = {}
    for sz in np.unique(sizes[keep]):
        sel = starts[keep & (sizes == sz)]
        mem = g[sel[:, None] + np.arange(sz)[None, :]]
        out[int(sz)] = (mem, role[keep & (sizes == sz)])
    return out


def eval_fp64_ops(prob) -> float:
    """Algorithmic FP64 operations of the strategy-evaluation kernel (Table 1 rows as written,
    each add, multiply, divide, min or max one operation; prefill link terms, which do not
    depend on the candidate, count one add each).  Every admissible strategy costs its memory
    row; a strategy whose memory row admits a batch of 1 costs the full latency sum."""
    m = prob.model
    L = m["n_layers"]
    H = float(m["hidden"])
    Hkv = float(m["hidden"] * m["n_kv_heads"] // m["n_heads"])
    B = float(m["bytes_per_elem"])
    W12 = 12.0 * H * H * B
    Kkv = 2.0 * (prob.s_in + prob.s_out) * Hkv * B
    Kact = 4.0 * (prob.s_in + prob.s_out) * H * B
    cl = prob.cluster
    gmem = np.asarray(cl.type_mem, np.float64)[np.asarray(cl.gpu_type)]
    tps = [t for t in range(1, 9) if (prob.tp_mask >> (t - 1)) & 1]
    total = 0.0
    for sz, (mem, role) in group_members(prob).items():
        dec = role == 1
        for tp in tps:
            if sz % tp:
                continue
            pp = sz // tp
            if pp > 8 or not (prob.pp_mask >> (pp - 1)) & 1 or pp > L:
                continue
            bmin = np.full(len(mem), 2.0 ** 30)
            for j in range(pp):
                l = L // pp + (1 if j < L % pp else 0)
                A = (W12 / tp) * l
                Kj = (Kkv / tp) * l + Kact
                mm = gmem[mem[:, j * tp:(j + 1) * tp]].min(axis=1)
                bmin = np.minimum(bmin, np.floor((mm - A) / Kj))
            feas = bmin >= 1.0
            total += len(mem) * pp * (tp + 8)
            nf_d = int((feas & dec).sum())
            nf_p = int((feas & ~dec).sum())
            common = 4 + 4 + pp * (2 + (tp - 1) + 2) + 3
            pre = common + pp * (3 + tp * (tp - 1) + 2) + (pp - 1) * (tp * tp + 1)
            dcd = common + pp * ((tp - 1) + 7 + 4 * tp * (tp - 1) + 3) + (pp - 1) * (3 * tp * tp + 2)
            total += nf_p * pre + nf_d * dcd
    return float(total)


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
    wl = I.WORKLOADS[args.workload]
    prob = I.make_problem(args.workload)
    dp = hx.DeviceProblem.upload(prob)
    ws = hx.Workspace.for_problem(dp, flows=False)
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        hx.score(dp, ws)
    torch.cuda.synchronize()

    names = ("cost", "flownet", "maxflow", "best")
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        e = ev[s]
        e[0].record(stream)
        hx.cost_eval(dp, ws.cost)
        e[1].record(stream)
        hx.build_flownet(dp, ws.cost, ws.net)
        e[2].record(stream)
        hx.maxflow_batch(ws.net, ws.flow_value)
        e[3].record(stream)
        hx.best_candidate(ws.flow_value, ws.best, dp.n_cand)
        e[4].record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1000.0 / args.steps
    per_kernel = {k: float(np.mean([ev[s][i].elapsed_time(ev[s][i + 1]) for s in range(args.steps)]))
                  for i, k in enumerate(names)}
    value = prob.n_cand / (ms_per_step / 1000.0)

    # Per-kernel durations: the same steps again with libhx recording HIP events around each of
    # its kernels on this stream (kept out of the timed region above).
    hx.profile(True)
    for _ in range(args.steps):
        hx.score(dp, ws)
    torch.cuda.synchronize()
    prof = hx.profile_read()
    hx.profile(False)
    kernel_us = {k: 1000.0 * ms / n for k, (ms, n) in prof.items() if n > 0}

    # Roofline of the kernel with the largest share of the step.
    n_p = ws.net.n_p.cpu().numpy()
    n_d = ws.net.n_d.cpu().numpy()
    dims = ws.net.dims
    best = [int(x) for x in ws.best.cpu().numpy()]
    dominant = max(kernel_us, key=kernel_us.get)
    t_dom = kernel_us[dominant] * 1e-6
    hbm = hbm_bytes_per_step(prob, dims, n_p, n_d)
    if dominant == "eval":
        ops = eval_fp64_ops(prob)
        achieved = ops / t_dom / 1e9
        roof = {"kernel": "eval (hx_cost_eval)", "bound": "alu", "achieved": achieved, "peak": FP64_VALU_PEAK_GOPS,
                "unit": "GFLOP/s", "frac": achieved / FP64_VALU_PEAK_GOPS, "traffic": kernel_traffic("eval", args.workload),
                "algorithmic_flops_per_launch": ops}
    elif dominant == "maxflow":
        alg = float(lds_floor_bytes(n_p, n_d).sum())
        achieved = alg / t_dom / 1e9
        roof = {"kernel": "maxflow (hx_maxflow_batch)", "bound": "lds", "achieved": achieved,
                "peak": LDS_PEAK_GBS, "unit": "GB/s", "frac": achieved / LDS_PEAK_GBS,
                "traffic": kernel_traffic("maxflow", args.workload), "algorithmic_bytes_per_launch": alg}
    else:
        call = {"setup": "cost", "decode": "cost", "scatter": "cost", "nodes": "flownet", "kv": "flownet"}.get(dominant,
                                                                                                          dominant)
        alg = float(hbm[call])
        achieved = alg / t_dom / 1e9
        roof = {"kernel": dominant, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS, "traffic": kernel_traffic(dominant, args.workload),
                "algorithmic_bytes_per_launch": alg}
    roof["avg_launch_us"] = kernel_us[dominant]

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
        "config": {"workload": f"workload{wl.cfg}: {wl.name}", "candidates": prob.n_cand,
                   "cluster_gpus": prob.n_gpus, "max_groups": prob.max_groups, "granularity": prob.granularity},
        "kernel_ms": per_kernel,
        "kernel_us": kernel_us,
        "hbm_bytes_per_step": hbm,
        "best": best,
        "roofline": roof,
    }

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
        out["cpu_baseline"] = {"value": prob.n_cand / med, "unit": "candidates/s", "cores": cores, "kind": "oracle",
                               "sample": f"the full {prob.n_cand}-candidate batch, {len(times)} runs, median",
                               "agrees": list(r["best"]) == best}
    print(json.dumps(out))


if __name__ == "__main__":
    main()
