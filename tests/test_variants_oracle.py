"""Pins of the oracle's cost-model variants (no GPU).

Pipelined decode capacity (variant bit 0): a decode replica's batches leave at the pace of its
slowest stage, x = 1000 b / max_j T_j with T_j = comp_j + TP_j + PP_j (the link into the next
stage counted with stage j); the latency and prefill capacities are unchanged.  Checked against
what that definition fixes: one stage changes nothing; the stage times bound the summed
latency (lat / pp <= max T_j <= lat); identical GPUs on free links give the closed form
max T_j = ceil(L/pp) * (per-layer time); and a batch's decode capacities can only rise while its
prefill capacities stay as they were.

KV stage-order search (variant bit 1): a KV edge's time is minimised over the stage orders of
both replicas.  Checked on hand-derived cases whose ascending orders pair the slow links and
whose best orders pair the fast ones (two and eight stages a side), against brute force over
every order pair (up to five stages a side), and by what a search over every order fixes: it
never exceeds the ascending time, leaves single stages alone, and cannot tell in which order the
stage blocks were handed to it.

Asymmetric layer split (variant bit 2): hand-derived splits, the invariants of the rule (sum L,
at least one layer each, faster stages never fewer but the leftover, one type = uniform), whole
batches unchanged on a one-type cluster, a free-link latency closed form, and a KV edge whose
stages share the split's 40 layers.
"""
import dataclasses
import itertools

import numpy as np
import pytest

from oracle import hxo
from paper_2502_07903_amd import inputs as I

PIPE = 1


def _random_groups(prob, rng, n):
    G = prob.n_gpus
    out = []
    while len(out) < n:
        tp = int(rng.choice([1, 2, 4, 8]))
        pp = int(rng.integers(1, min(8, G // tp) + 1))
        members = sorted(rng.choice(G, tp * pp, replace=False).tolist())
        out.append((members, tp, pp))
    return out


def test_pipelined_single_stage_and_prefill_unchanged():
    prob = I.make_problem(3, n_cand=4)
    rng = np.random.default_rng(1)
    for members, tp, pp in _random_groups(prob, rng, 300):
        for role in (0, 1):
            a = hxo.strategy_cost(prob, members, tp, pp, role, variant=0)
            b = hxo.strategy_cost(prob, members, tp, pp, role, variant=PIPE)
            assert a[:3] == b[:3]                      # feasibility, b_max, latency
            if role == 0 or pp == 1:
                assert a[3] == b[3]


def test_pipelined_bounds_by_latency():
    """lat / pp <= max_j T_j <= lat, i.e. x_sum <= x_pipe <= pp x_sum (to rounding)."""
    rng = np.random.default_rng(2)
    for cfg in (2, 3):
        prob = I.make_problem(cfg, n_cand=4)
        seen = 0
        for members, tp, pp in _random_groups(prob, rng, 400):
            ok, bmax, lat, xs = hxo.strategy_cost(prob, members, tp, pp, 1, variant=0)
            if not ok:
                continue
            _, _, _, xp = hxo.strategy_cost(prob, members, tp, pp, 1, variant=PIPE)
            assert xs * (1 - 1e-14) <= xp <= pp * xs * (1 + 1e-14)
            seen += pp > 1
        assert seen > 20


def test_pipelined_free_links_closed_form():
    """Four identical GPUs, alpha = 0 and beta -> inf: T_j = l_j (12 H^2 B s_out / (t m) +
    24 b s_out H^2 / (t c)), so the slowest stage holds ceil(L / pp) layers."""
    prob = I.make_problem(2, n_cand=4)
    cl = prob.cluster
    free = I.Cluster(cl.gpu_type, cl.type_flops, cl.type_hbm_bw, cl.type_mem,
                     np.full_like(cl.beta, 1e300), np.zeros_like(cl.alpha))
    md = dict(prob.model)
    H, B = md["hidden"], md["bytes_per_elem"]
    c, m = 312e12, 2.0e12                                  # node 0 is type A
    for L in (48, 47, 45):
        md["n_layers"] = L
        p2 = dataclasses.replace(prob, cluster=free, model=dict(md))
        for tp, pp in [(1, 4), (2, 2), (1, 3), (1, 2)]:
            members = list(range(tp * pp))
            ok, b, lat, xs = hxo.strategy_cost(p2, members, tp, pp, 1, variant=0)
            if not ok:
                continue
            _, _, _, xp = hxo.strategy_cost(p2, members, tp, pp, 1, variant=PIPE)
            per_layer = 12.0 * H * H * B * p2.s_out / (tp * m) + 24.0 * b * p2.s_out * H * H / (tp * c)
            assert xp == pytest.approx(1000.0 * b / (-(-L // pp) * per_layer), rel=1e-12)
            assert xs == pytest.approx(1000.0 * b / (L * per_layer), rel=1e-12)


def test_pipelined_batch_raises_only_decode():
    for cfg in (2, 3):
        prob = I.make_problem(cfg, n_cand=300)
        base = hxo.cost_eval(prob)
        pipe = hxo.cost_eval(dataclasses.replace(prob, variant=PIPE))
        dec = prob.role == 1
        pre = prob.role == 0
        assert np.array_equal(base["cap"][pre], pipe["cap"][pre])
        assert (pipe["cap"][dec] >= base["cap"][dec]).all()
        assert (pipe["cap"][dec] > base["cap"][dec]).any()


# ------------------------------------------------------------------ KV stage-order search

ORDER = 2


def _crossed_cluster():
    """Four GPUs of one type; links 0<->3 and 1<->2 at 300 GB/s, every other link 10 GB/s, alpha 0."""
    G = 4
    beta = np.full((G, G), 10e9)
    for a, b in ((0, 3), (1, 2)):
        beta[a, b] = beta[b, a] = 300e9
    np.fill_diagonal(beta, 0.0)
    t = np.array([I.GPU_TYPES["A"]], np.float64)
    return I.Cluster(np.zeros(G, np.int32), t[:, 0].copy(), t[:, 1].copy(), t[:, 2].copy(),
                     np.ascontiguousarray(beta.reshape(-1)), np.zeros(G * G))


def test_kv_order_hand_case():
    """Prefill {0, 1} and decode {2, 3}, one GPU per stage, two stages of 24 layers each.
    Ascending orders pair 0->2 and 1->3 (10 GB/s); putting decode stage {3} first pairs 0->3 and
    1->2 (300 GB/s).  Each link carries a stage's KV cache, 2 s_in H_kv B * 24 bytes."""
    from tests import helpers as Hh
    cl = _crossed_cluster()
    a, r = I.placement_from_groups([[0, 1], [2, 3]], [I.PREFILL, I.DECODE], 4, 2)
    prob = Hh.problem(cl, dict(I.OPT_30B), a, r, s_in=512.0, s_out=128.0, tp=(1,), pp=(2,))
    V = 2.0 * 512.0 * 7168 * 2 * 24
    assert hxo.kv_time(prob, [0, 1], 1, 2, [2, 3], 1, 2) == pytest.approx(V / 10e9, rel=1e-15)
    assert hxo.kv_time(prob, [0, 1], 1, 2, [2, 3], 1, 2, best_order=True) == pytest.approx(V / 300e9, rel=1e-15)
    # the whole network: the KV edge capacity follows the searched order only with the variant
    plain = hxo.build_flownet(prob, hxo.cost_eval(prob))
    p2 = dataclasses.replace(prob, variant=ORDER)
    searched = hxo.build_flownet(p2, hxo.cost_eval(p2))
    assert int(plain["kv_cap"][0, 0]) == int(np.floor(1000.0 / (V / 10e9)))
    assert int(searched["kv_cap"][0, 0]) == int(np.floor(1000.0 / (V / 300e9)))


def _stage_blocks(members, tp, perm):
    return [g for s in perm for g in members[s * tp:(s + 1) * tp]]


def test_kv_order_search_properties():
    """On random replica pairs of the 32-GPU cluster, up to five stages a side: the searched time
    never exceeds the ascending one, equals it for single stages, and does not change when the
    stage blocks are handed over in another order (the search covers every order)."""
    prob = I.make_problem(3, n_cand=4)
    rng = np.random.default_rng(5)
    checked = strict = 0
    for _ in range(300):
        ptp, dtp = int(rng.choice([1, 2, 4])), int(rng.choice([1, 2, 4]))
        ppp, dpp = int(rng.integers(1, 6)), int(rng.integers(1, 6))
        if ptp * ppp + dtp * dpp > prob.n_gpus:
            continue
        g = rng.permutation(prob.n_gpus)
        pm = sorted(g[:ptp * ppp].tolist())
        dm = sorted(g[ptp * ppp:ptp * ppp + dtp * dpp].tolist())
        asc = hxo.kv_time(prob, pm, ptp, ppp, dm, dtp, dpp)
        best = hxo.kv_time(prob, pm, ptp, ppp, dm, dtp, dpp, best_order=True)
        assert best <= asc
        if ppp == 1 and dpp == 1:
            assert best == asc
            continue
        checked += 1
        strict += best < asc
        pm2 = _stage_blocks(pm, ptp, rng.permutation(ppp))
        dm2 = _stage_blocks(dm, dtp, rng.permutation(dpp))
        assert hxo.kv_time(prob, pm2, ptp, ppp, dm2, dtp, dpp, best_order=True) == best
    assert checked > 50 and strict > 10


@pytest.mark.parametrize("ppp,dpp,ptp,dtp,seed", [(2, 3, 2, 1, 1), (3, 3, 1, 2, 2), (4, 3, 1, 1, 3), (3, 5, 2, 1, 4),
                                                  (4, 4, 1, 2, 5), (5, 4, 1, 1, 6), (2, 6, 2, 1, 7), (6, 2, 1, 4, 8),
                                                  (5, 5, 1, 1, 9)])
def test_kv_order_search_brute_force(ppp, dpp, ptp, dtp, seed):
    """The search's minimum equals the smallest KV time over every pair of stage orders, each
    order pair's time taken by the oracle's plain walk with explicit orders."""
    prob = I.make_problem(4, n_cand=1)
    rng = np.random.default_rng(seed)
    g = rng.permutation(prob.n_gpus)
    pm = sorted(g[:ptp * ppp].tolist())
    dm = sorted(g[ptp * ppp:ptp * ppp + dtp * dpp].tolist())
    brute = min(hxo.kv_time_orders(prob, pm, ptp, ppp, op, dm, dtp, dpp, od)
                for op in itertools.permutations(range(ppp)) for od in itertools.permutations(range(dpp)))
    assert hxo.kv_time(prob, pm, ptp, ppp, dm, dtp, dpp, best_order=True) == brute
    assert hxo.kv_time_orders(prob, pm, ptp, ppp, range(ppp), dm, dtp, dpp, range(dpp)) == \
        hxo.kv_time(prob, pm, ptp, ppp, dm, dtp, dpp)


def _hidden_pairing_cluster(fast):
    """16 GPUs of one type: prefill GPUs 0-7, decode GPUs 8-15; the link i -> 8 + t is 300 GB/s
    when fast(i, t), 10 GB/s otherwise; alpha 0."""
    G = 16
    beta = np.full((G, G), 10e9)
    for i in range(8):
        for t in range(8):
            if fast(i, t):
                beta[i, 8 + t] = beta[8 + t, i] = 300e9
    np.fill_diagonal(beta, 0.0)
    tt = np.array([I.GPU_TYPES["A"]], np.float64)
    return I.Cluster(np.zeros(G, np.int32), tt[:, 0].copy(), tt[:, 1].copy(), tt[:, 2].copy(),
                     np.ascontiguousarray(beta.reshape(-1)), np.zeros(G * G))


@pytest.mark.parametrize("dpp", [8, 4])
def test_kv_order_deep_hand_case(dpp):
    """Eight one-GPU prefill stages against eight or four one-GPU decode stages, 48 layers.  A hidden pairing makes some links 300 GB/s and the rest 10 GB/s; an order that puts
    every overlapping pair of positions on a fast link exists, so the minimum is the fast time of
    the largest overlap.
      dpp = 8: positions a and b share 6 layers iff a = b; link i -> t is fast iff t = pi(i) for
               a permutation pi, so ordering decode stages as pi of the prefill order makes all
               eight links fast: 2 s_in H_kv B * 6 / 300e9.
      dpp = 4: decode position b (12 layers) shares 6 layers with prefill positions 2b and 2b+1;
               link i -> t is fast iff pi(i) // 2 = t, so each decode stage has two fast prefill
               stages; placing them at 2b, 2b+1 makes every link fast: again 6 layers at 300 GB/s.
    The ascending orders hit a slow link (pi is not the identity pairing)."""
    pi = [3, 6, 0, 7, 2, 5, 1, 4]
    fast = (lambda i, t: pi[i] == t) if dpp == 8 else (lambda i, t: pi[i] // 2 == t)
    from tests import helpers as Hh
    cl = _hidden_pairing_cluster(fast)
    groups = [list(range(8)), list(range(8, 8 + dpp))]
    a, r = I.placement_from_groups(groups, [I.PREFILL, I.DECODE], 16, 2)
    prob = Hh.problem(cl, dict(I.OPT_30B), a, r, s_in=512.0, s_out=128.0, tp=(1,), pp=(4, 8))
    V6 = 2.0 * 512.0 * 7168 * 2 * 6
    best = hxo.kv_time(prob, groups[0], 1, 8, groups[1], 1, dpp, best_order=True)
    assert best == V6 / 300e9
    assert hxo.kv_time(prob, groups[0], 1, 8, groups[1], 1, dpp) == V6 / 10e9
    # an optimal order pair, checked with the plain walk
    if dpp == 8:
        od = pi
    else:
        od = [0, 1, 2, 3]
        op = sorted(range(8), key=lambda i: (pi[i] // 2, i))
    op = list(range(8)) if dpp == 8 else op
    assert hxo.kv_time_orders(prob, groups[0], 1, 8, op, groups[1], 1, dpp, od) == best


def test_kv_order_rejects_deep_pp_mask():
    """The search covers pipelines of up to 8 stages: with it, a PP mask past 8 is refused."""
    prob = I.make_problem(2, n_cand=4)
    p2 = dataclasses.replace(prob, variant=ORDER, pp_mask=prob.pp_mask | (1 << 8))
    with pytest.raises(ValueError):
        hxo.build_flownet(p2, hxo.cost_eval(dataclasses.replace(p2, variant=0)))


# ------------------------------------------------------------------ asymmetric layer split

ASYM = 4


def test_asym_split_hand_cases():
    """16-GPU cluster: GPUs 0-3 type A (312 TFLOP/s), 4-7 B (125), 8-11 C (65); L = 48.
    (A | C): shares of 46 are 46*312/377 = 38.07 and 46*65/377 = 7.93, floors 38 and 7, one
    layer left over for stage 0: (1+38+1, 1+7) = (40, 8).  (A A | B B): 46*312/437 = 32.84 and
    46*125/437 = 13.16: (34, 14).  One type: the uniform split."""
    prob = I.make_problem(2, n_cand=1)
    assert hxo.layer_split(prob, [0, 8], 1, 2, ASYM) == [40, 8]
    assert hxo.layer_split(prob, [0, 1, 4, 5], 2, 2, ASYM) == [34, 14]
    assert hxo.layer_split(prob, [0, 1, 2], 1, 3, ASYM) == [16, 16, 16]
    assert hxo.layer_split(prob, [0, 8], 1, 2, 0) == [24, 24]


def test_asym_split_invariants():
    prob = I.make_problem(3, n_cand=1)
    rng = np.random.default_rng(6)
    flops = np.asarray(prob.cluster.type_flops)[np.asarray(prob.cluster.gpu_type)]
    L = prob.model["n_layers"]
    for _ in range(300):
        tp = int(rng.choice([1, 2, 4]))
        pp = int(rng.integers(1, 9))
        members = sorted(rng.choice(prob.n_gpus, tp * pp, replace=False).tolist())
        lay = hxo.layer_split(prob, members, tp, pp, ASYM)
        assert sum(lay) == L and min(lay) >= 1
        c = [flops[members[j * tp:(j + 1) * tp]].min() for j in range(pp)]
        for i in range(pp):
            for j in range(pp):
                if c[i] > c[j]:
                    assert lay[i] >= lay[j] - 1          # faster stages never get fewer layers (but the leftover)
        if len(set(c)) == 1:
            assert lay == hxo.layer_split(prob, members, tp, pp, 0)


def test_asym_is_uniform_on_one_type():
    """A cluster of one GPU type: the asymmetric split is the uniform one, so every capacity, KV
    edge and flow is unchanged."""
    prob = I.make_problem(3, n_cand=200)
    cl = prob.cluster
    one = I.Cluster(np.zeros_like(cl.gpu_type), cl.type_flops, cl.type_hbm_bw, cl.type_mem, cl.beta, cl.alpha)
    p0 = dataclasses.replace(prob, cluster=one)
    a = hxo.score_batch(p0)
    b = hxo.score_batch(dataclasses.replace(p0, variant=ASYM))
    for k in ("tp", "pp", "bmax", "cap", "lat"):
        assert np.array_equal(a["cost"][k], b["cost"][k])
    assert np.array_equal(a["flownet"]["kv_cap"], b["flownet"]["kv_cap"])
    assert np.array_equal(a["flow_value"], b["flow_value"])


def test_asym_free_links_closed_form_and_kv():
    """Free links: a prefill group (A | C) has latency 24 s_in H^2 (40 / c_A + 8 / c_C).  Two (A | C)
    replicas over links of one bandwidth: the uniform split puts 24 layers (29.6 GB of weights) on
    the 16 GB C GPU, so neither replica is feasible; the asymmetric split gives it 8 and both
    are, and their stage 0s share 40 layers, so the KV time is that of 40 layers."""
    prob = I.make_problem(2, n_cand=1)
    cl = prob.cluster
    H = prob.model["hidden"]
    free = I.Cluster(cl.gpu_type, cl.type_flops, cl.type_hbm_bw, cl.type_mem,
                     np.full_like(cl.beta, 1e300), np.zeros_like(cl.alpha))
    p2 = dataclasses.replace(prob, cluster=free, variant=ASYM)
    ok, b, lat, x = hxo.strategy_cost(p2, [0, 8], 1, 2, 0)
    assert ok
    assert lat == pytest.approx(24.0 * p2.s_in * H * H * (40 / 312e12 + 8 / 65e12), rel=1e-12)
    flat = I.Cluster(cl.gpu_type, cl.type_flops, cl.type_hbm_bw, cl.type_mem,
                     np.full_like(cl.beta, 20e9), np.zeros_like(cl.alpha))
    a, r = I.placement_from_groups([[0, 8], [1, 9]], [I.PREFILL, I.DECODE], 16, 2)
    from tests import helpers as Hh
    base = Hh.problem(flat, prob.model, a, r, s_in=prob.s_in, s_out=prob.s_out, tp=(1,), pp=(2,))
    V1 = 2.0 * prob.s_in * (H * prob.model["n_kv_heads"] // prob.model["n_heads"]) * 2
    uni = hxo.cost_eval(base)
    assert (uni["cap"][:2, 0] == 0).all()
    pv = dataclasses.replace(base, variant=ASYM)
    cost = hxo.cost_eval(pv)
    assert list(cost["pp"][:2, 0]) == [2, 2] and (cost["cap"][:2, 0] > 0).all()
    fn = hxo.build_flownet(pv, cost)
    assert int(fn["kv_cap"][0, 0]) == int(np.floor(1000.0 / ((V1 * 40) / 20e9)))
