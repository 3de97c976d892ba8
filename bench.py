"""Benchmark: candidate placements scored per second on one MI355X.

A step is one pass of the whole hot path over one batch of candidate placements with the
inputs already resident in HBM: cost model (hx_cost_eval) -> flow network
(hx_build_flownet) -> max-flow (hx_maxflow_batch) -> best candidate (hx_best_candidate).
The default workload is the 32-GPU / 8-node / 4-type cluster serving a Llama-2-70B-shaped
model with lognormal request lengths, 65,536 seeded random candidates of 2-16 groups.

    python bench.py [--gpus 1] [--steps 50] [--warmup 5] [--workload 3] [--no-cpu-baseline]

Prints ONE JSON line.  Per-kernel durations come from HIP events recorded around every call
inside the timed region, on the stream the kernels run on; the roofline object reports the
kernel with the largest share.  The CPU baseline times the oracle (test infrastructure, not
the product) on the same batch on the host's cores.
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
FP64_VALU_PEAK_TFLOPS = 78.6

# HBM bytes per launch of the max-flow kernel at workload 3, from rocprofv3 FETCH_SIZE and
# WRITE_SIZE passes (profiles/all_kernels_workload3.md), each scaled by what the counter reads
# for a 256 MiB device copy (FETCH_SIZE x 2.0, WRITE_SIZE x 1.0).  Valid only for the kernel
# source they were taken on (first 16 hex digits of its SHA-256); otherwise traffic is null.
MAXFLOW_TRAFFIC = {"source_sha256_16": "68896aad8bb1c1e6", "fetch_kib": 13355.0, "write_kib": 256.4,
                   "fetch_scale": 2.0, "write_scale": 1.0}


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


def maxflow_traffic(workload: int):
    """Counter-measured HBM bytes per max-flow launch, or None when they do not apply."""
    import hashlib
    src = os.path.join(ROOT, "paper_2502_07903_amd", "csrc", "hx_maxflow.hip")
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    t = MAXFLOW_TRAFFIC
    if workload != 3 or sha != t["source_sha256_16"]:
        return None
    return 1024.0 * (t["fetch_kib"] * t["fetch_scale"] + t["write_kib"] * t["write_scale"])


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

    # Roofline of the kernel with the largest share of the step.
    n_p = ws.net.n_p.cpu().numpy()
    n_d = ws.net.n_d.cpu().numpy()
    dims = ws.net.dims
    best = [int(x) for x in ws.best.cpu().numpy()]
    dominant = max(per_kernel, key=per_kernel.get)
    hbm = hbm_bytes_per_step(prob, dims, n_p, n_d)
    if dominant == "maxflow":
        alg = float(lds_floor_bytes(n_p, n_d).sum())
        achieved = alg / (per_kernel["maxflow"] / 1000.0) / 1e9
        roof = {"kernel": "hx_maxflow_batch (maxflow_kernel)", "bound": "lds", "achieved": achieved,
                "peak": LDS_PEAK_GBS, "unit": "GB/s", "frac": achieved / LDS_PEAK_GBS,
                "traffic": maxflow_traffic(args.workload), "algorithmic_bytes_per_launch": alg}
    else:
        alg = float(hbm[dominant])
        achieved = alg / (per_kernel[dominant] / 1000.0) / 1e9
        roof = {"kernel": dominant, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS, "traffic": None, "algorithmic_bytes_per_launch": alg}

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
