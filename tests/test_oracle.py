"""Pins of the CPU oracle against what the paper and the mathematics fix (no GPU).

Cost model: hand-derived Table 1 values (tests/golden/cost_worked.txt), closed forms of the
single-GPU case, the memory limit against exact rational arithmetic, monotonicity.
Max-flow: brute-force min-cut enumeration, the bipartite min-cut closed form, library
solvers (scipy, networkx), flow validity with a certifying cut, special cases.
Argmax: first maximum.  Whole candidates: tests/golden/candidates_worked.txt.
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import hxo
from paper_2502_07903_amd import inputs as I
from tests import helpers as Hh

COST_CASES = Hh.parse_golden("cost_worked.txt")


@pytest.mark.parametrize("case", [c for c in COST_CASES if c["kind"] == "strategy"], ids=lambda c: c["name"])
def test_strategy_golden(case):
    members = Hh.ints(case["members"])
    prob = Hh.single_group_problem(case["cluster"], case["model"], members)
    ok, bmax, lat, x = hxo.strategy_cost(prob, members, int(case["tp"]), int(case["pp"]), Hh.ROLE[case["role"]])
    assert bmax == int(case["bmax"])
    want_lat = float(case["lat"])
    if want_lat == 0:
        assert not ok
        assert int(case["cap"]) == 0
        return
    assert ok
    assert lat == pytest.approx(want_lat, rel=1e-12, abs=0)
    assert hxo.quantize(x) == int(case["cap"])


@pytest.mark.parametrize("case", [c for c in COST_CASES if c["kind"] == "select"], ids=lambda c: c["name"])
def test_select_golden(case):
    members = Hh.ints(case["members"])
    prob = Hh.single_group_problem(case["cluster"], case["model"], members)
    tp, pp, bmax, cap, lat = hxo.group_select(prob, members, Hh.ROLE[case["role"]])
    assert (tp, pp, cap) == (int(case["tp"]), int(case["pp"]), int(case["cap"]))


@pytest.mark.parametrize("case", [c for c in COST_CASES if c["kind"] == "kv"], ids=lambda c: c["name"])
def test_kv_golden(case):
    pm, dm = Hh.ints(case["pm"]), Hh.ints(case["dm"])
    prob = Hh.single_group_problem(case["cluster"], case["model"], pm)
    t = hxo.kv_time(prob, pm, int(case["ptp"]), int(case["ppp"]), dm, int(case["dtp"]), int(case["dpp"]))
    assert t == pytest.approx(float(case["time"]), rel=1e-12, abs=0)
    assert hxo.quantize(1000.0 / t) == int(case["cap"])


@pytest.mark.parametrize("case", Hh.parse_golden("candidates_worked.txt"), ids=lambda c: c["name"])
def test_candidate_golden(case):
    groups = [[int(g) for g in grp.split("/")] for grp in case["groups"].split(";")]
    roles = [Hh.ROLE[r] for r in case["roles"].split(",")]
    cl = Hh.cluster_c1()
    a, r = I.placement_from_groups(groups, roles, 8, 4)
    prob = Hh.problem(cl, Hh.MODELS["opt30b"], a, r)
    res = hxo.score_batch(prob)
    assert int(res["flow_value"][0]) == int(case["flow"])


# ------------------------------------------------------------------ closed forms (single GPU)

def _random_single_gpu(rng):
    flops = rng.uniform(50e12, 1000e12)
    hbm = rng.uniform(0.5e12, 4e12)
    mem = rng.uniform(40e9, 200e9)
    cl = I.cluster_from_nodes(np.zeros(4, np.int32), np.array([[flops, hbm, mem]]), np.zeros((1, 1)))
    heads = int(rng.choice([32, 40, 56, 64]))
    kv = int(rng.choice([h for h in (1, 2, 4, 8, heads) if heads % h == 0]))
    model = dict(n_layers=int(rng.integers(8, 81)), hidden=heads * 128, n_heads=heads, n_kv_heads=kv,
                 bytes_per_elem=2)
    s_in = float(rng.integers(64, 4096))
    s_out = float(rng.integers(16, 1024))
    a, r = I.placement_from_groups([[0]], [0], 4, 1)
    return Hh.problem(cl, model, a, r, s_in=s_in, s_out=s_out), flops, hbm, mem


def test_single_gpu_closed_forms():
    """One GPU, TP = PP = 1: no communication term, so
    lat_P = 24 s_in H^2 L / c,  lat_D = L (12 H^2 B s_out / m + 24 b s_out H^2 / c),
    b_max = floor((M - 12 H^2 B L) / (2 (s_in+s_out) H_kv B L + 4 (s_in+s_out) H B))."""
    rng = np.random.default_rng(7)
    checked = 0
    for _ in range(300):
        prob, c, m, M = _random_single_gpu(rng)
        md = prob.model
        H, L, B = md["hidden"], md["n_layers"], md["bytes_per_elem"]
        Hkv = H * md["n_kv_heads"] // md["n_heads"]
        si, so = prob.s_in, prob.s_out
        want_b = (M - 12.0 * H * H * B * L) / (2 * (si + so) * Hkv * B * L + 4 * (si + so) * H * B)
        okp, bp, latp, xp = hxo.strategy_cost(prob, [0], 1, 1, 0)
        okd, bd, latd, xd = hxo.strategy_cost(prob, [0], 1, 1, 1)
        if abs(want_b - round(want_b)) < 1e-6:
            continue
        assert bp == bd == int(np.floor(want_b))
        if want_b < 1:
            assert not okp and not okd
            continue
        checked += 1
        assert latp == pytest.approx(24.0 * si * H * H * L / c, rel=1e-13)
        assert xp == pytest.approx(1000.0 / latp, rel=1e-15)
        b = bd
        assert latd == pytest.approx(L * (12.0 * H * H * B * so / m + 24.0 * b * so * H * H / c), rel=1e-13)
        assert xd == pytest.approx(1000.0 * b / latd, rel=1e-15)
    assert checked > 100


def test_memory_limit_exact():
    """b_max is the largest integer batch whose Table 1 memory footprint fits every device of every
    stage, checked in exact rational arithmetic on random groups of the four-type cluster."""
    prob3 = I.make_problem(3, n_cand=8)
    cl = prob3.cluster
    rng = np.random.default_rng(11)
    md = prob3.model
    H, L, B = md["hidden"], md["n_layers"], md["bytes_per_elem"]
    Hkv = H * md["n_kv_heads"] // md["n_heads"]
    si, so = Fraction(prob3.s_in), Fraction(prob3.s_out)
    checked = 0
    for _ in range(200):
        tp = int(rng.choice([1, 2, 4, 8]))
        pp = int(rng.integers(1, min(8, cl.n_gpus // tp) + 1))
        members = sorted(rng.choice(cl.n_gpus, tp * pp, replace=False).tolist())
        ok, bmax, lat, x = hxo.strategy_cost(prob3, members, tp, pp, 1)

        def fits(b):
            for j in range(pp):
                l = L // pp + (1 if j < L % pp else 0)
                need = (Fraction(12 * H * H * B, tp) + Fraction(2 * b, tp) * (si + so) * Hkv * B) * l \
                    + 4 * b * (si + so) * H * B
                for d in members[j * tp:(j + 1) * tp]:
                    if need > Fraction(cl.type_mem[cl.gpu_type[d]]):
                        return False
            return True
        if bmax >= 1:
            assert fits(bmax) and not fits(bmax + 1)
            assert ok
            checked += 1
        else:
            assert not fits(1) and not ok
    assert checked > 20


def test_tp_and_pp_terms_vanish():
    """TP = 1 has no TP term and PP = 1 no PP term: with alpha = 0 and beta -> inf the latency of
    a strategy equals its computation alone, for any tp, pp."""
    prob = I.make_problem(2, n_cand=4)
    cl = prob.cluster
    huge = I.Cluster(cl.gpu_type, cl.type_flops, cl.type_hbm_bw, cl.type_mem,
                     np.full_like(cl.beta, 1e300), np.zeros_like(cl.alpha))
    p2 = I.Problem(huge, prob.model, prob.s_in, prob.s_out, prob.tp_mask, prob.pp_mask, 0, prob.max_groups,
                   prob.assign, prob.role)
    H, L = prob.model["hidden"], prob.model["n_layers"]
    # four A GPUs of node 0: per stage compute is (24 s_in H^2 / (tp c)) l, summed: 24 s_in H^2 L / (tp c)
    for tp, pp in [(1, 4), (2, 2), (4, 1)]:
        ok, b, lat, x = hxo.strategy_cost(p2, [0, 1, 2, 3], tp, pp, 0)
        assert ok
        assert lat == pytest.approx(24.0 * prob.s_in * H * H * L / (tp * 312e12), rel=1e-13)


def test_monotone_capacity():
    """A group's capacity never drops when any GPU gets more FLOP/s, bandwidth or memory, or a
    link gets faster (each Table 1 term is monotone and so is the max over strategies)."""
    rng = np.random.default_rng(3)
    base = I.make_problem(3, n_cand=64)
    ref = hxo.cost_eval(base)
    for trial in range(6):
        cl = base.cluster
        kind = trial % 4
        f, h, m = cl.type_flops.copy(), cl.type_hbm_bw.copy(), cl.type_mem.copy()
        beta = cl.beta.copy()
        t = int(rng.integers(0, cl.n_types))
        if kind == 0:
            f[t] *= 1.5
        elif kind == 1:
            h[t] *= 1.5
        elif kind == 2:
            m[t] *= 1.3
        else:
            beta *= rng.uniform(1.0, 2.0, beta.shape)
        cl2 = I.Cluster(cl.gpu_type, f, h, m, beta, cl.alpha)
        p2 = I.Problem(cl2, base.model, base.s_in, base.s_out, base.tp_mask, base.pp_mask, 0, base.max_groups,
                       base.assign, base.role)
        out = hxo.cost_eval(p2)
        assert (out["cap"] >= ref["cap"]).all(), f"capacity dropped after raising parameter kind {kind}"


def test_batch_matches_single_group():
    """The batch cost call equals per-group selection on the decoded member lists."""
    prob = I.make_problem(2, n_cand=40)
    out = hxo.cost_eval(prob)
    for n in range(prob.n_cand):
        for k in range(prob.max_groups):
            members = [g for g in range(prob.n_gpus) if prob.assign[g, n] == k]
            r = int(prob.role[k, n])
            if not members or r > 1:
                assert out["tp"][k, n] == 0 and out["cap"][k, n] == 0
                continue
            tp, pp, bmax, cap, lat = hxo.group_select(prob, members, r)
            assert (out["tp"][k, n], out["pp"][k, n], out["bmax"][k, n], out["cap"][k, n]) == (tp, pp, bmax, cap)
            assert out["lat"][k, n] == lat


# ------------------------------------------------------------------ max-flow

def _random_network(rng, nv, p_edge, cmax):
    E = []
    for u in range(nv):
        for v in range(nv):
            if u != v and v != 0 and u != 1 and rng.random() < p_edge:
                E.append((u, v, int(rng.integers(0, cmax + 1))))
    return E


def test_maxflow_edges_brute_force():
    """Edmonds-Karp value = brute-force minimum cut over all vertex subsets (max-flow min-cut)."""
    rng = np.random.default_rng(5)
    for trial in range(150):
        nv = int(rng.integers(2, 11))
        E = _random_network(rng, nv, float(rng.uniform(0.15, 0.7)), int(rng.choice([1, 5, 1000, Hh.CAP_MAX])))
        v, fl, reach = hxo.maxflow_edges(nv, E, 0, 1)
        assert v == Hh.brute_force_min_cut(nv, E)
        # validity: capacity, conservation, and the residual-reachable set certifies the cut
        net = np.zeros(nv, np.int64)
        for (a, b, c), f in zip(E, fl):
            assert 0 <= f <= c
            net[a] -= f
            net[b] += f
        assert all(net[x] == 0 for x in range(2, nv))
        assert net[1] == v
        assert not reach[1]
        assert sum(c for (a, b, c) in E if reach[a] and not reach[b]) == v


def test_maxflow_edges_libraries():
    """Edmonds-Karp value = scipy's and networkx's maximum flow on random graphs."""
    nx = pytest.importorskip("networkx")
    from scipy.sparse import csr_matrix
    from scipy.sparse.csgraph import maximum_flow
    rng = np.random.default_rng(9)
    for trial in range(60):
        nv = int(rng.integers(2, 40))
        E = _random_network(rng, nv, float(rng.uniform(0.05, 0.4)), 100000)
        v, _, _ = hxo.maxflow_edges(nv, E, 0, 1)
        M = np.zeros((nv, nv), np.int32)
        G = nx.DiGraph()
        G.add_nodes_from(range(nv))
        for a, b, c in E:
            M[a, b] += c
            G.add_edge(a, b, capacity=c)
        assert v == maximum_flow(csr_matrix(M), 0, 1).flow_value
        assert v == nx.maximum_flow_value(G, 0, 1)


def _random_flownet(rng, N, maxP, maxD, cap_choices):
    dims = (maxP, maxD, maxP * maxD)
    fn = dict(n_p=np.zeros(N, np.int32), n_d=np.zeros(N, np.int32))
    for k, rows in (("src_cap", maxP), ("p_cap", maxP), ("kv_cap", maxP * maxD), ("d_cap", maxD),
                    ("sink_cap", maxD), ("p_slot", maxP), ("d_slot", maxD)):
        fn[k] = np.zeros((rows, N), np.int32)
    for n in range(N):
        P, D = int(rng.integers(0, maxP + 1)), int(rng.integers(0, maxD + 1))
        fn["n_p"][n], fn["n_d"][n] = P, D
        hi = int(rng.choice(cap_choices))
        for k, rows in (("src_cap", P), ("p_cap", P), ("kv_cap", P * D), ("d_cap", D), ("sink_cap", D)):
            fn[k][:rows, n] = rng.integers(0, hi + 1, rows)
            if rng.random() < 0.3:
                fn[k][:rows, n] = np.where(rng.random(rows) < 0.5, Hh.CAP_MAX, fn[k][:rows, n])
    fn["dims"] = dims
    return fn


def test_maxflow_batch_certified():
    """On random Sec. 3.3 networks: the value equals the brute-force minimum cut (small) and the
    bipartite closed form; the returned flow is valid and its residual cut certifies it."""
    rng = np.random.default_rng(21)
    fn = _random_flownet(rng, 200, 4, 4, [1, 3, 100, 5000, Hh.CAP_MAX])
    out = hxo.maxflow_batch(fn)
    Hh.check_flow(fn, out["flow_value"], out["kv_flow"], out["cut"])
    for n in range(200):
        P, D = int(fn["n_p"][n]), int(fn["n_d"][n])
        a = np.minimum(fn["src_cap"][:P, n], fn["p_cap"][:P, n]).astype(np.int64)
        b = np.minimum(fn["d_cap"][:D, n], fn["sink_cap"][:D, n]).astype(np.int64)
        c = fn["kv_cap"][:P * D, n].astype(np.int64).reshape(P, D)
        assert out["flow_value"][n] == Hh.bipartite_closed_form(a, b, c)
        if P + D <= 7:
            nv, E = Hh.network_edges(fn, n)
            assert out["flow_value"][n] == Hh.brute_force_min_cut(nv, E)


def test_maxflow_special_cases():
    """P = D = 1: the minimum of the five capacities in series.  KV edges unbounded: min(sum a, sum b)."""
    rng = np.random.default_rng(2)
    fn = _random_flownet(rng, 64, 1, 1, [1000])
    fn["n_p"][:] = 1
    fn["n_d"][:] = 1
    fn["src_cap"][0] = rng.integers(0, 1000, 64)
    fn["p_cap"][0] = rng.integers(0, 1000, 64)
    fn["kv_cap"][0] = rng.integers(0, 1000, 64)
    fn["d_cap"][0] = rng.integers(0, 1000, 64)
    fn["sink_cap"][0] = rng.integers(0, 1000, 64)
    out = hxo.maxflow_batch(fn)
    want = np.min(np.stack([fn[k][0] for k in ("src_cap", "p_cap", "kv_cap", "d_cap", "sink_cap")]), axis=0)
    assert np.array_equal(out["flow_value"], want)

    fn = _random_flownet(rng, 64, 5, 6, [10 ** 6])
    fn["kv_cap"][:] = Hh.CAP_MAX
    out = hxo.maxflow_batch(fn)
    for n in range(64):
        P, D = fn["n_p"][n], fn["n_d"][n]
        a = np.minimum(fn["src_cap"][:P, n], fn["p_cap"][:P, n]).astype(np.int64).sum()
        b = np.minimum(fn["d_cap"][:D, n], fn["sink_cap"][:D, n]).astype(np.int64).sum()
        assert out["flow_value"][n] == (min(a, b) if P and D else 0)


def test_maxflow_int32_extremes():
    """Largest networks of the refinement workload with every capacity at 2^24 - 1: the value
    (up to 64 * (2^24 - 1)) stays exact in int32."""
    rng = np.random.default_rng(4)
    fn = _random_flownet(rng, 2, 64, 64, [Hh.CAP_MAX])
    fn["n_p"][:] = 64
    fn["n_d"][:] = 64
    for k in ("src_cap", "p_cap", "kv_cap", "d_cap", "sink_cap"):
        fn[k][:] = Hh.CAP_MAX
    out = hxo.maxflow_batch(fn)
    assert (out["flow_value"] == 64 * Hh.CAP_MAX).all()


# ------------------------------------------------------------------ argmax

def test_best_candidate():
    rng = np.random.default_rng(1)
    for N in (1, 2, 7, 1000):
        fv = rng.integers(-4, 50, N).astype(np.int32)
        i, v = hxo.best_candidate(fv)
        assert i == int(np.argmax(fv)) and v == int(fv.max())
    with pytest.raises(ValueError):
        hxo.best_candidate(np.zeros(0, np.int32))


def test_score_batch_threads_agree():
    prob = I.make_problem(2, n_cand=300)
    r1 = hxo.score_batch(prob, n_threads=1)
    r4 = hxo.score_batch(prob, n_threads=4)
    assert np.array_equal(r1["flow_value"], r4["flow_value"]) and r1["best"] == r4["best"]
    c = hxo.cost_eval(prob)
    f = hxo.build_flownet(prob, c)
    m = hxo.maxflow_batch(f)
    assert np.array_equal(m["flow_value"], r1["flow_value"])
    Hh.check_flow(f, m["flow_value"], m["kv_flow"], m["cut"])
