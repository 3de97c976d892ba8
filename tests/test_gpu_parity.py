"""GPU parity: the HIP path (through the C-ABI) against the CPU oracle, element by element,
on the same seeded inputs.  Integers (strategies, batch limits, capacities, flow values, the
minimum cut, the argmax) must be bit-exact; latencies must agree to 1e-5 relative (they are
expected bit-identical: both sides evaluate the same binary64 expressions without FMA);
KV flow assignments are not unique, so they are checked for validity instead."""
import dataclasses
import os
import sys

import numpy as np
import pytest

from oracle import hxo
from paper_2502_07903_amd import hx
from paper_2502_07903_amd import inputs as I
from tests import helpers as Hh

pytestmark = pytest.mark.gpu
N_THREADS = max(1, min(16, os.cpu_count() or 1))


def say(msg: str) -> None:
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch():
    import torch as T
    if not T.cuda.is_available():
        pytest.fail("GPU tests need a ROCm GPU (torch.cuda.is_available() is False)")
    hx.lib()
    return T


def run_gpu(torch, prob, flows: bool = True):
    dp = hx.DeviceProblem.upload(prob)
    ws = hx.Workspace.for_problem(dp, flows=flows)
    hx.score(dp, ws)
    torch.cuda.synchronize()
    out = dict(cost={k: getattr(ws.cost, k).cpu().numpy() for k in ("tp", "pp", "bmax", "cap", "lat", "members")},
               flownet=ws.net.host(), flow_value=ws.flow_value.cpu().numpy(),
               best=tuple(int(x) for x in ws.best.cpu().numpy()))
    if flows:
        out["kv_flow"] = ws.kv_flow.cpu().numpy()
        out["cut"] = ws.cut.cpu().numpy()
    return out


def oracle_all(prob):
    res = hxo.score_batch(prob, n_threads=N_THREADS)
    mf = hxo.maxflow_batch(res["flownet"], want_flows=True)
    assert np.array_equal(mf["flow_value"], res["flow_value"])
    res["cut"] = mf["cut"]
    return res


def compare_cost(got, want):
    for k in ("tp", "pp", "bmax", "cap"):
        bad = got[k] != want[k]
        assert not bad.any(), f"cost {k} differs at (group, candidate) {np.argwhere(bad)[:5].tolist()}"
    g, w = got["lat"], want["lat"]
    rel = np.abs(g - w) / np.maximum(np.abs(w), 1e-300)
    assert (rel <= 1e-5).all(), f"latency rel. error {rel.max():.3g}"
    assert np.array_equal(g, w), f"latencies not bit-identical ({int((g != w).sum())} differ)"


def expected_members(prob) -> np.ndarray:
    """Group member bitmasks straight from assign: [Kmax * W][N] uint64, bit g of word w = GPU 64w + g."""
    G, N, K = prob.n_gpus, prob.n_cand, prob.max_groups
    W = 1 if G <= 64 else (2 if G <= 128 else 4)
    m = np.zeros((K * W, N), np.uint64)
    cols = np.arange(N)
    for g in range(G):
        k = prob.assign[g].astype(np.int64)
        ok = k < K
        np.bitwise_or.at(m, (k[ok] * W + g // 64, cols[ok]), np.uint64(1) << np.uint64(g % 64))
    return m


def full_parity(torch, prob, label):
    say(f"{label}: N={prob.n_cand} G={prob.n_gpus} Kmax={prob.max_groups} gran={prob.granularity}")
    got = run_gpu(torch, prob)
    want = oracle_all(prob)
    compare_cost(got["cost"], want["cost"])
    assert np.array_equal(got["cost"]["members"].view(np.uint64), expected_members(prob)), "member bitmasks differ"
    Hh.compare_flownet(got["flownet"], want["flownet"])
    assert np.array_equal(got["flow_value"], want["flow_value"]), \
        f"flow values differ at {np.flatnonzero(got['flow_value'] != want['flow_value'])[:8].tolist()}"
    Hh.check_flow_batch(got["flownet"], got["flow_value"], got["kv_flow"])
    Hh.compare_cut(got["cut"], want["cut"], want["flownet"])
    assert got["best"] == want["best"]
    return got, want


# ------------------------------------------------------------------ hand-derived candidates

def test_golden_candidates(torch):
    cases = Hh.parse_golden("candidates_worked.txt")
    cands = []
    for case in cases:
        groups = [[int(g) for g in grp.split("/")] for grp in case["groups"].split(";")]
        roles = [Hh.ROLE[r] for r in case["roles"].split(",")]
        cands.append(I.placement_from_groups(groups, roles, 8, 4))
    a, r = I.stack_candidates(cands)
    prob = Hh.problem(Hh.cluster_c1(), Hh.MODELS["opt30b"], a, r)
    say("golden candidates")
    got = run_gpu(torch, prob)
    assert got["flow_value"].tolist() == [int(c["flow"]) for c in cases]
    assert got["best"] == (0, int(cases[0]["flow"]))


# ------------------------------------------------------------------ workloads

_WORKLOAD_ORACLE = {}


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_workload_parity(torch, cfg):
    _, want = full_parity(torch, I.make_problem(cfg), f"workload {cfg}")
    _WORKLOAD_ORACLE[cfg] = (want["flow_value"], want["best"])


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_workload_parity_value_only(torch, cfg):
    """The path the benchmark times: no flow assignment or cut requested, so the max-flow may
    take its value-only shortcuts (the pre-passes of the workgroup plans, the direct minimum
    cut); every flow value of the full batch and the best equal the oracle's."""
    prob = I.make_problem(cfg)
    say(f"workload {cfg} value only: N={prob.n_cand}")
    got = run_gpu(torch, prob, flows=False)
    if cfg not in _WORKLOAD_ORACLE:
        res = hxo.score_batch(prob, n_threads=N_THREADS)
        _WORKLOAD_ORACLE[cfg] = (res["flow_value"], res["best"])
    want_fv, want_best = _WORKLOAD_ORACLE[cfg]
    assert np.array_equal(got["flow_value"], want_fv), \
        f"flow values differ at {np.flatnonzero(got['flow_value'] != want_fv)[:8].tolist()}"
    assert got["best"] == want_best


@pytest.mark.parametrize("cfg,n", [(1, 1), (2, 7), (3, 1000), (4, 777), (3, 4097)])
def test_ragged_batches(torch, cfg, n):
    full_parity(torch, I.make_problem(cfg, n_cand=n), f"workload {cfg} ragged")


def max_cluster_problem(max_groups: int, n_cand: int, k_hi: int, granularity: int = 0):
    """255 GPUs (the ABI's maximum: four mask words per group), 4 per node (the last node
    holds 3), the five node types of the 64-GPU workload in turn, seeded inter-node links of
    3-25 GB/s, Llama-2-70B shape and the 64-GPU workload's lengths and strategy space."""
    G = 255
    wl = dataclasses.replace(I.WORKLOADS[4], n_gpus=G, n_cand=n_cand, k_range=(2, k_hi), max_groups=max_groups)
    node = np.arange(G) // I.GPUS_PER_NODE
    n_nodes = int(node[-1]) + 1
    gpu_type = (node % 5).astype(np.int32)
    table = np.array([I.GPU_TYPES[c] for c in "ABCDE"], np.float64)
    rng = np.random.default_rng([2502, 7903, 255])
    inter = rng.uniform(3.0, 25.0, (n_nodes, n_nodes)) * 1e9
    inter = np.triu(inter, 1) + np.triu(inter, 1).T
    cl = I.cluster_from_nodes(gpu_type, table, inter)
    a, r = I.random_candidates(wl)
    s_in, s_out = I.mean_lengths(wl)
    return I.Problem(cl, dict(wl.model), s_in, s_out, wl.tp_mask, wl.pp_mask, granularity, max_groups, a, r)


def test_maximum_cluster(torch):
    """255 GPUs and up to 64 groups per candidate: the whole path against the oracle."""
    full_parity(torch, max_cluster_problem(64, 96, 64), "255 GPUs")


def test_maximum_group_slots(torch):
    """255 GPUs and 255 group slots (both the ABI's maxima): cost model and network against the
    oracle; the max-flow refuses networks beyond its LDS plan with HX_ETOOBIG."""
    prob = max_cluster_problem(255, 24, 255)
    say(f"255 GPUs, 255 slots: N={prob.n_cand}")
    dp = hx.DeviceProblem.upload(prob)
    ws = hx.Workspace.for_problem(dp, flows=False)
    hx.cost_eval(dp, ws.cost)
    hx.build_flownet(dp, ws.cost, ws.net)
    torch.cuda.synchronize()
    want = hxo.score_batch(prob, n_threads=N_THREADS)
    compare_cost({k: getattr(ws.cost, k).cpu().numpy() for k in ("tp", "pp", "bmax", "cap", "lat")}, want["cost"])
    assert np.array_equal(ws.cost.members.cpu().numpy().view(np.uint64), expected_members(prob))
    Hh.compare_flownet(ws.net.host(), want["flownet"])
    with pytest.raises(hx.HxError) as err:
        hx.maxflow_batch(ws.net, ws.flow_value)
    assert err.value.code == hx.HX_ETOOBIG


def test_maximum_cluster_per_gpu_nodes(torch):
    """255 GPUs with a flow node per GPU: cost model and network (up to 255 nodes a side and
    their per-GPU KV edges) against the oracle; the max-flow refuses such networks (HX_ETOOBIG)."""
    prob = max_cluster_problem(32, 16, 32, granularity=1)
    say(f"255 GPUs, per-GPU nodes: N={prob.n_cand}")
    dp = hx.DeviceProblem.upload(prob)
    ws = hx.Workspace.for_problem(dp, flows=False)
    hx.cost_eval(dp, ws.cost)
    hx.build_flownet(dp, ws.cost, ws.net)
    torch.cuda.synchronize()
    want = hxo.score_batch(prob, n_threads=N_THREADS)
    compare_cost({k: getattr(ws.cost, k).cpu().numpy() for k in ("tp", "pp", "bmax", "cap", "lat")}, want["cost"])
    Hh.compare_flownet(ws.net.host(), want["flownet"])
    with pytest.raises(hx.HxError) as err:
        hx.maxflow_batch(ws.net, ws.flow_value)
    assert err.value.code == hx.HX_ETOOBIG


@pytest.mark.parametrize("cfg,frac", [(2, 1.0), (3, 0.5), (3, 0.02)])
def test_asymmetric_links(torch, cfg, frac):
    """Links whose two directions differ (beta_gh != beta_hg, alpha too) on a seeded fraction of
    the GPU pairs: every direction-dependent term, and the decode TP row's reuse of a quotient
    for both directions only where the two betas are the same, against the oracle."""
    prob = I.make_problem(cfg, n_cand=4096)
    G = prob.n_gpus
    rng = np.random.default_rng(7000 + cfg)
    beta = np.asarray(prob.cluster.beta, np.float64).reshape(G, G).copy()
    alpha = np.asarray(prob.cluster.alpha, np.float64).reshape(G, G).copy()
    pick = np.triu(rng.random((G, G)) < frac, 1)
    beta[pick] *= rng.uniform(0.5, 1.5, int(pick.sum()))
    alpha[pick] *= rng.uniform(0.5, 1.5, int(pick.sum()))
    cl = dataclasses.replace(prob.cluster, beta=np.ascontiguousarray(beta.reshape(-1)),
                             alpha=np.ascontiguousarray(alpha.reshape(-1)))
    assert (beta != beta.T).any()
    full_parity(torch, dataclasses.replace(prob, cluster=cl), f"workload {cfg} asymmetric links ({frac})")


def test_refinement_round0_sample(torch):
    """Per-GPU networks (up to 130 nodes, 4,096 KV edges): a full round-0 batch on the GPU,
    checked against the oracle on a seeded sample plus the GPU's best candidate."""
    prob = I.make_problem(5)
    say(f"refinement round 0: N={prob.n_cand} (full batch on GPU)")
    got = run_gpu(torch, prob, flows=False)
    rng = np.random.default_rng(55)
    idx = np.unique(np.concatenate([rng.choice(prob.n_cand, 1536, replace=False), [got["best"][0]]]))
    sub = prob.subset(idx)
    say(f"refinement round 0: oracle on {len(idx)} sampled candidates")
    want = oracle_all(sub)
    for k in ("tp", "pp", "bmax", "cap", "lat"):
        assert np.array_equal(got["cost"][k][:, idx], want["cost"][k]), f"cost {k} differs"
    assert np.array_equal(got["cost"]["members"].view(np.uint64)[:, idx], expected_members(sub))
    gfn = {k: (v[..., idx] if isinstance(v, np.ndarray) else v) for k, v in got["flownet"].items()}
    Hh.compare_flownet(gfn, want["flownet"])
    assert np.array_equal(got["flow_value"][idx], want["flow_value"])
    # the GPU's best is the true maximum: no candidate's upper bound min(sum a, sum b) exceeds it
    fn = got["flownet"]
    up, ud, _ = Hh.used_rows(fn)
    a = np.where(up, np.minimum(fn["src_cap"], fn["p_cap"]), 0).astype(np.int64).sum(0)
    b = np.where(ud, np.minimum(fn["d_cap"], fn["sink_cap"]), 0).astype(np.int64).sum(0)
    ub = np.minimum(a, b)
    assert (got["flow_value"] <= ub).all()
    best_i, best_v = got["best"]
    contenders = np.flatnonzero(ub >= best_v)
    say(f"refinement round 0: certifying the argmax over {len(contenders)} contenders")
    want_c = oracle_all(prob.subset(contenders))
    vals = want_c["flow_value"]
    assert vals.max() == best_v
    assert contenders[np.flatnonzero(vals == best_v)[0]] == best_i


def test_refinement_round1(torch):
    """Round 1 perturbs round 0's best candidate (taken from the oracle's own argmax)."""
    wl = I.WORKLOADS[5]
    base_prob = I.make_problem(5, n_cand=1024)
    want0 = oracle_all(base_prob)
    bi = want0["best"][0]
    base = (base_prob.assign[:, bi].copy(), base_prob.role[:, bi].copy())
    prob = I.make_problem(5, n_cand=1024, rnd=1, base=base)
    full_parity(torch, prob, "refinement round 1")


# ------------------------------------------------------------------ max-flow alone

def _maxflow_on(torch, fn):
    """Max-flow of host networks twice: with the flow assignment and cut, and value only (the
    value-only call may take minimum cuts directly); both values must agree."""
    nb = hx.FlowNetBuffers.from_host(fn)
    N = fn["n_p"].shape[0]
    mp, md, mpd = fn["dims"]
    fv = torch.empty(N, dtype=torch.int32, device="cuda")
    kv = torch.zeros((mpd, N), dtype=torch.int32, device="cuda")
    cut = torch.zeros((mp + md, N), dtype=torch.uint8, device="cuda")
    hx.maxflow_batch(nb, fv, kv, cut)
    fv_only = torch.full((N,), -12345, dtype=torch.int32, device="cuda")
    hx.maxflow_batch(nb, fv_only)
    torch.cuda.synchronize()
    fv_h = fv.cpu().numpy()
    assert np.array_equal(fv_only.cpu().numpy(), fv_h), "value-only max-flow differs"
    return fv_h, kv.cpu().numpy(), cut.cpu().numpy()


def _adversarial_networks(rng):
    """Networks chosen to stress the max-flow kernel: every shape is given as (P, D, caps)."""
    nets = []
    C = Hh.CAP_MAX
    nets.append((4, 4, dict(a=np.zeros(4), b=np.zeros(4), c=np.zeros(16))))                  # all zero
    nets.append((8, 8, dict(a=np.full(8, C), b=np.full(8, C), c=np.full(64, C))))             # all max
    c = np.zeros(16); c[5] = 7
    nets.append((4, 4, dict(a=np.full(4, 100), b=np.full(4, 100), c=c)))                    # single path
    nets.append((1, 31, dict(a=[10 ** 6], b=rng.integers(0, 50000, 31), c=rng.integers(0, 60000, 31))))
    nets.append((31, 1, dict(a=rng.integers(0, 50000, 31), b=[10 ** 6], c=rng.integers(0, 60000, 31))))
    # zig-zag: each prefill node reaches two neighbouring decode nodes; augmenting paths must
    # undo earlier greedy choices along a chain of reverse KV arcs
    P = D = 16
    c = np.zeros(P * D)
    for i in range(P):
        c[i * D + i] = 10
        if i + 1 < D:
            c[i * D + i + 1] = 10
    nets.append((P, D, dict(a=np.full(P, 10), b=np.concatenate([np.full(D - 1, 10), [0]]), c=c)))
    for _ in range(6):                                                                      # dense 64 x 64
        nets.append((64, 64, dict(a=rng.integers(0, 2 ** 20, 64), b=rng.integers(0, 2 ** 20, 64),
                                  c=rng.integers(0, 2 ** 16, 4096))))
    return nets


def test_maxflow_adversarial(torch):
    rng = np.random.default_rng(77)
    nets = _adversarial_networks(rng)
    mp = md = 64
    mpd = 4096
    N = len(nets)
    fn = dict(n_p=np.zeros(N, np.int32), n_d=np.zeros(N, np.int32), dims=(mp, md, mpd))
    for k, rows in (("src_cap", mp), ("p_cap", mp), ("d_cap", md), ("sink_cap", md), ("kv_cap", mpd),
                    ("p_slot", mp), ("d_slot", md)):
        fn[k] = np.zeros((rows, N), np.int32)
    for n, (P, D, caps) in enumerate(nets):
        fn["n_p"][n], fn["n_d"][n] = P, D
        fn["src_cap"][:P, n] = Hh.CAP_MAX
        fn["p_cap"][:P, n] = caps["a"]
        fn["d_cap"][:D, n] = caps["b"]
        fn["sink_cap"][:D, n] = Hh.CAP_MAX
        fn["kv_cap"][:P * D, n] = caps["c"]
    want = hxo.maxflow_batch(fn)
    say(f"adversarial networks: {N}")
    fv, kv, cut = _maxflow_on(torch, fn)
    assert np.array_equal(fv, want["flow_value"])
    Hh.check_flow_batch(fn, fv, kv)
    Hh.compare_cut(cut, want["cut"], fn)


@pytest.mark.parametrize("mp,md,total,N", [(16, 16, 32, 3000), (40, 40, 40, 800), (6, 6, 12, 2000)])
def test_maxflow_random_networks(torch, mp, md, total, N):
    """Random capacities (not from the cost model) over every shape with P + D <= total; the
    plans select 32-, 64- and 8-lane segments."""
    rng = np.random.default_rng(78 + mp)
    n_p = rng.integers(0, mp + 1, N)
    n_d = np.minimum(rng.integers(0, md + 1, N), total - n_p)
    mpd = (total // 2) * ((total + 1) // 2)
    fn = dict(n_p=n_p.astype(np.int32), n_d=n_d.astype(np.int32), dims=(mp, md, mpd))
    for k, rows in (("src_cap", mp), ("p_cap", mp), ("d_cap", md), ("sink_cap", md), ("kv_cap", mpd),
                    ("p_slot", mp), ("d_slot", md)):
        hi = rng.choice([2, 100, 10 ** 5, Hh.CAP_MAX], size=N)
        fn[k] = (rng.random((rows, N)) * (hi[None, :] + 1)).astype(np.int32)
    want = hxo.maxflow_batch(fn)
    say(f"random networks: {N} with P + D <= {total}")
    fv, kv, cut = _maxflow_on(torch, fn)
    assert np.array_equal(fv, want["flow_value"])
    Hh.check_flow_batch(fn, fv, kv)
    Hh.compare_cut(cut, want["cut"], fn)


@pytest.mark.parametrize("mp,md,mpd,N", [(8, 8, 16, 3000), (16, 16, 64, 3000), (16, 16, 256, 2000),
                                          (64, 64, 1024, 600), (128, 128, 4096, 150), (200, 50, 4096, 60)])
def test_maxflow_dominant_kv(torch, mp, md, mpd, N):
    """Networks whose KV arcs can each carry min(a_i, b_j), most of them exactly that much
    (the north-west-corner closed form), plus a few arcs one unit short (push-relabel); the
    plans select 8-, 16-, 32- and 64-lane segments and 128- and 256-lane workgroups."""
    rng = np.random.default_rng(90 + mp + mpd)
    n_p = rng.integers(1, mp + 1, N)
    n_d = rng.integers(1, md + 1, N)
    n_d = np.minimum(n_d, mpd // n_p)
    fn = dict(n_p=n_p.astype(np.int32), n_d=n_d.astype(np.int32), dims=(mp, md, mpd))
    for k, rows in (("src_cap", mp), ("p_cap", mp), ("d_cap", md), ("sink_cap", md), ("kv_cap", mpd),
                    ("p_slot", mp), ("d_slot", md)):
        fn[k] = np.zeros((rows, N), np.int32)
    for n in range(N):
        P, D = int(n_p[n]), int(n_d[n])
        hi = int(rng.choice([5, 1000, 2 ** 20]))
        a = rng.integers(0, hi + 1, P)
        b = rng.integers(0, hi + 1, D)
        fn["src_cap"][:P, n] = Hh.CAP_MAX
        fn["p_cap"][:P, n] = a
        fn["d_cap"][:D, n] = b
        fn["sink_cap"][:D, n] = Hh.CAP_MAX
        c = np.minimum(a[:, None], b[None, :]) + rng.integers(0, 3, (P, D)) * (rng.random((P, D)) < 0.5)
        if n % 5 == 4:                                   # one arc short of the bound: no closed form
            i, j = rng.integers(0, P), rng.integers(0, D)
            c[i, j] = max(0, min(a[i], b[j]) - 1)
        fn["kv_cap"][:P * D, n] = c.reshape(-1)
    want = hxo.maxflow_batch(fn)
    say(f"dominant-KV networks: {N} with P <= {mp}, D <= {md}")
    fv, kv, cut = _maxflow_on(torch, fn)
    assert np.array_equal(fv, want["flow_value"])
    Hh.check_flow_batch(fn, fv, kv)
    Hh.compare_cut(cut, want["cut"], fn)


def test_maxflow_round_budget_reports_noconv(torch, monkeypatch):
    """A round budget of 1 (set from the host) stops every candidate that needs more
    push-relabel rounds with HX_ENOCONV; every workgroup still exits normally.  Random
    capacities (KV arcs often below min(a_i, b_j), several nodes per side) leave many networks
    to push-relabel; flows are requested, so no minimum cut is taken directly."""
    rng = np.random.default_rng(61)
    N, mp, md = 1500, 16, 16
    mpd = mp * md
    n_p = rng.integers(2, mp + 1, N)
    n_d = rng.integers(2, md + 1, N)
    fn = dict(n_p=n_p.astype(np.int32), n_d=n_d.astype(np.int32), dims=(mp, md, mpd))
    for k, rows in (("src_cap", mp), ("p_cap", mp), ("d_cap", md), ("sink_cap", md), ("kv_cap", mpd),
                    ("p_slot", mp), ("d_slot", md)):
        fn[k] = rng.integers(1, 1000, (rows, N)).astype(np.int32)
    want = hxo.maxflow_batch(fn)
    monkeypatch.setenv("HX_MAXFLOW_ROUND_BUDGET", "1")
    say("round budget 1")
    nb = hx.FlowNetBuffers.from_host(fn)
    fv_d = torch.empty(N, dtype=torch.int32, device="cuda")
    kv = torch.zeros((mpd, N), dtype=torch.int32, device="cuda")
    cut = torch.zeros((mp + md, N), dtype=torch.uint8, device="cuda")
    hx.maxflow_batch(nb, fv_d, kv, cut)
    torch.cuda.synchronize()
    fv = fv_d.cpu().numpy()
    assert (fv == hx.HX_ENOCONV).any()
    ok = fv != hx.HX_ENOCONV
    assert np.array_equal(fv[ok], want["flow_value"][ok])


def test_deterministic(torch):
    prob = I.make_problem(3, n_cand=4096)
    say("determinism")
    g1 = run_gpu(torch, prob)
    g2 = run_gpu(torch, prob)
    assert np.array_equal(g1["flow_value"], g2["flow_value"])
    assert np.array_equal(g1["kv_flow"], g2["kv_flow"])
    assert np.array_equal(g1["cut"], g2["cut"])
    for k in g1["cost"]:
        assert np.array_equal(g1["cost"][k], g2["cost"][k])


@pytest.mark.parametrize("cfg", [3, 5])
def test_every_output_written_repeatedly(torch, cfg):
    """Repeated full-size passes with every output and scratch buffer pre-filled with a garbage
    pattern: every present group's cost outputs and every candidate's flow value must be
    written on every call, identically.  This catches a unit the sort loses, or a value left
    over from an earlier call, which a single call on fresh, zeroed memory can hide.  Sizes 32
    GPUs (one mask word) and 128 GPUs (two)."""
    prob = I.make_problem(cfg)
    say(f"workload {cfg}: 12 repeated passes over dirty buffers, N={prob.n_cand}")
    dp = hx.DeviceProblem.upload(prob)
    ws = hx.Workspace.for_problem(dp, flows=False)
    net_rows = ("n_p", "n_d", "p_slot", "d_slot", "src_cap", "p_cap", "kv_cap", "d_cap", "sink_cap")
    ref = None
    for it in range(12):
        ws.cost.tp.fill_(0xAB)
        ws.cost.pp.fill_(0xAB)
        ws.cost.bmax.fill_(-12345)
        ws.cost.cap.fill_(-12345)
        ws.cost.lat.fill_(float("nan"))
        ws.cost.members.fill_(-1)
        ws.cost.workspace.fill_(0x5A)
        for k in net_rows:
            getattr(ws.net, k).fill_(0x7F7F7F7F if k not in ("n_p", "n_d") else 0)
        ws.flow_value.fill_(-12345)
        ws.best.fill_(-12345)
        hx.score(dp, ws)
        torch.cuda.synchronize()
        got = {k: getattr(ws.cost, k).cpu().numpy() for k in ("tp", "pp", "bmax", "cap", "lat")}
        got["flow_value"] = ws.flow_value.cpu().numpy()
        got["best"] = ws.best.cpu().numpy()
        assert not np.isnan(got["lat"]).any(), f"call {it}: unwritten latencies"
        assert not (got["cap"] == -12345).any(), f"call {it}: unwritten capacities"
        if ref is None:
            ref = got
            rng = np.random.default_rng(cfg)
            idx = np.sort(rng.choice(prob.n_cand, 512, replace=False))
            res = hxo.score_batch(prob.subset(idx), n_threads=N_THREADS)
            for k in ("tp", "pp", "bmax", "cap", "lat"):
                assert np.array_equal(got[k][:, idx], res["cost"][k]), f"cost {k} differs from the oracle"
            assert np.array_equal(got["flow_value"][idx], res["flow_value"])
        else:
            for k in got:
                bad = np.argwhere(got[k] != ref[k])
                assert len(bad) == 0, f"call {it}: {k} differs from call 0 at (group, candidate) {bad[:5].tolist()}"


# ------------------------------------------------------------------ argmax

@pytest.mark.parametrize("n", [1, 2, 63, 64, 1025, 100003])
def test_best_candidate(torch, n):
    rng = np.random.default_rng(n)
    v = rng.integers(-4, 40, n).astype(np.int32)
    t = torch.as_tensor(v).cuda()
    best = torch.empty(2, dtype=torch.int32, device="cuda")
    say(f"best of {n}")
    hx.best_candidate(t, best)
    torch.cuda.synchronize()
    assert tuple(best.cpu().tolist()) == hxo.best_candidate(v)
    for off in (1, 2, 3):                      # inputs that do not start on a 16-byte boundary
        if n - off < 1:
            continue
        hx.best_candidate(t[off:], best)
        torch.cuda.synchronize()
        assert tuple(best.cpu().tolist()) == hxo.best_candidate(v[off:])


# ------------------------------------------------------------------ exhaustive search

def _set_partitions(items, max_blocks):
    if not items:
        yield []
        return
    first, rest = items[0], items[1:]
    for part in _set_partitions(rest, max_blocks):
        for i in range(len(part)):
            yield part[:i] + [[first] + part[i]] + part[i + 1:]
        if len(part) < max_blocks:
            yield [[first]] + part


def test_exhaustive_search_best():
    """Every placement of the 8-GPU cluster into at most 4 groups with every role assignment:
    the batch argmax on the GPU equals the oracle's best over the same exhaustive batch (the
    case study's exhaustive-search comparison, on a cluster of its size)."""
    import torch as T
    if not T.cuda.is_available():
        pytest.fail("GPU tests need a ROCm GPU")
    cands = []
    for part in _set_partitions(list(range(8)), 4):
        part = sorted([sorted(b) for b in part])
        k = len(part)
        for roles in range(1, (1 << k) - 1):
            cands.append(I.placement_from_groups(part, [(roles >> i) & 1 for i in range(k)], 8, 4))
    a, r = I.stack_candidates(cands)
    prob = Hh.problem(Hh.cluster_c1(), Hh.MODELS["opt30b"], a, r)
    say(f"exhaustive: {prob.n_cand} placements")
    got = run_gpu(T, prob, flows=False)
    want = hxo.score_batch(prob, n_threads=N_THREADS)
    assert np.array_equal(got["flow_value"], want["flow_value"])
    assert got["best"] == want["best"]


def test_profile_counts_each_kernel(torch):
    """The diagnostic per-kernel timing sees every kernel of one pass exactly once, with a
    positive duration, and records nothing once disabled."""
    prob = I.make_problem(2, n_cand=1000)
    dp = hx.DeviceProblem.upload(prob)
    ws = hx.Workspace.for_problem(dp)
    hx.profile(True)
    hx.score(dp, ws)
    prof = hx.profile_read()
    hx.profile(False)
    scoring = {"setup", "decode", "scatter", "eval", "nodes", "kv", "maxflow", "best"}
    assert set(prof) == scoring | {"classes", "moves", "gather", "spectral", "partition", "shared"}
    for name, (ms, n) in prof.items():
        if name in scoring:
            assert n == 1 and ms > 0.0, (name, ms, n)
        else:
            assert n == 0, (name, ms, n)
    hx.score(dp, ws)
    torch.cuda.synchronize()
    assert all(n == 0 for _, n in hx.profile_read().values())
