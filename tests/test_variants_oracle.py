"""Pins of the oracle's cost-model variants (no GPU).

Pipelined decode capacity (variant bit 0): a decode replica's batches leave at the pace of its
slowest stage, x = 1000 b / max_j T_j with T_j = comp_j + TP_j + PP_j (the link into the next
stage counted with stage j); the latency and prefill capacities are unchanged.  Checked against
what that definition fixes: one stage changes nothing; the stage times bound the summed
latency (lat / pp <= max T_j <= lat); identical GPUs on free links give the closed form
max T_j = ceil(L/pp) * (per-layer time); and a batch's decode capacities can only rise while its
prefill capacities and every latency stay as they were.
"""
import dataclasses

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
