"""Pins of the oracle's per-GPU flow network (one flow node per GPU), no GPU.

The paper's network has one node per replica (Sec. 3.3); the per-GPU network refines it with
the same units (requests on every edge): a GPU node carries its share of its replica's
requests, and a KV edge carries whole requests' KV caches over one link.  Pinned by
hand-derived networks (tests/golden/per_gpu_network.txt), by the identity with the replica
network when every replica is one GPU, and by maximum flows certified by brute-force minimum
cuts.
"""
import dataclasses

import numpy as np
import pytest

from oracle import hxo
from paper_2502_07903_amd import inputs as I
from tests import helpers as Hh

CASES = Hh.parse_golden("per_gpu_network.txt")


def _golden_problem(case):
    groups = [Hh.ints(g.replace("/", ",")) for g in case["groups"].split(";")]
    roles = [Hh.ROLE[r] for r in case["roles"].split(",")]
    cl = Hh.cluster_c1()
    a, r = I.placement_from_groups(groups, roles, cl.n_gpus, len(groups))
    prob = Hh.problem(cl, Hh.MODELS["opt30b"], a, r, granularity=1)
    K = len(groups)
    tp = np.zeros((K, 1), np.uint8)
    pp = np.zeros((K, 1), np.uint8)
    for k, s in enumerate(case["strategy"].split(",")):
        t, p = (int(x) for x in s.split("x"))
        tp[k, 0], pp[k, 0] = t, p
    cap = np.array(Hh.ints(case["cap"]), np.int32).reshape(K, 1)
    cost = dict(tp=tp, pp=pp, cap=cap, bmax=np.zeros((K, 1), np.int32), lat=np.zeros((K, 1)))
    return prob, cost


@pytest.mark.parametrize("case", CASES, ids=lambda c: c["name"])
def test_per_gpu_network_golden(case):
    prob, cost = _golden_problem(case)
    f = hxo.build_flownet(prob, cost)
    pg, dg = Hh.ints(case["p_gpus"]), Hh.ints(case["d_gpus"])
    P, D = len(pg), len(dg)
    assert (int(f["n_p"][0]), int(f["n_d"][0])) == (P, D)
    assert f["p_slot"][:P, 0].tolist() == pg
    assert f["d_slot"][:D, 0].tolist() == dg
    assert f["p_cap"][:P, 0].tolist() == Hh.ints(case["p_cap"])
    assert f["d_cap"][:D, 0].tolist() == Hh.ints(case["d_cap"])
    assert f["src_cap"][:P, 0].tolist() == [Hh.CAP_MAX] * P
    assert f["sink_cap"][:D, 0].tolist() == [Hh.CAP_MAX] * D
    assert f["kv_cap"][:P * D, 0].tolist() == Hh.ints(case["kv_cap"])
    # the flow value, by the oracle and by enumerating every cut of the explicit network
    assert int(hxo.maxflow_batch(f)["flow_value"][0]) == int(case["flow"])
    nv, edges = Hh.network_edges(f, 0)
    assert Hh.brute_force_min_cut(nv, edges) == int(case["flow"])


def test_kv_gpu_time_hand_values():
    """The link time alone: the whole request's KV cache over one link, at any replica size."""
    prob, _ = _golden_problem(CASES[0])
    V1L = 2.0 * 512 * 7168 * 2 * 48
    assert V1L == 704643072.0
    assert hxo.kv_gpu_time(prob, 2, 0) == 1e-5 + V1L / 300e9
    assert hxo.kv_gpu_time(prob, 5, 0) == 5e-5 + V1L / 12.5e9
    assert hxo.quantize(1000.0 / hxo.kv_gpu_time(prob, 2, 0)) == 423942
    assert hxo.quantize(1000.0 / hxo.kv_gpu_time(prob, 5, 0)) == 17723


@pytest.mark.parametrize("cfg", [1, 2])
def test_single_gpu_replicas_match_replica_network(cfg):
    """When every replica is one GPU, the per-GPU network is the replica network: the same node
    capacities, and every KV edge the replica KV edge of the same two GPUs."""
    wl = I.WORKLOADS[cfg]
    base = I.make_problem(cfg, n_cand=1)
    G = base.n_gpus
    rng = np.random.default_rng(2502)
    cands = []
    for _ in range(40):
        roles = rng.integers(0, 2, G)
        roles[0], roles[1] = 0, 1
        used = rng.random(G) < 0.8
        used[0] = used[1] = True
        groups = [[g] for g in range(G) if used[g]]
        cands.append(I.placement_from_groups(groups, [int(roles[g]) for g in range(G) if used[g]], G, G))
    a, r = I.stack_candidates(cands)
    rep = dataclasses.replace(base, assign=a, role=r, max_groups=G, granularity=0,
                              tp_mask=wl.tp_mask, pp_mask=wl.pp_mask)
    per = dataclasses.replace(rep, granularity=1)
    cost = hxo.cost_eval(rep)
    assert np.array_equal(cost["tp"], hxo.cost_eval(per)["tp"])
    fr = hxo.build_flownet(rep, cost)
    fg = hxo.build_flownet(per, cost)
    assert np.array_equal(fr["n_p"], fg["n_p"]) and np.array_equal(fr["n_d"], fg["n_d"])
    for n in range(rep.n_cand):
        P, D = int(fr["n_p"][n]), int(fr["n_d"][n])
        # group k holds GPU gk, numbered in GPU order, so node i is the same GPU in both networks
        gp = [int(np.flatnonzero(a[:, n] == k)[0]) for k in fr["p_slot"][:P, n]]
        gd = [int(np.flatnonzero(a[:, n] == k)[0]) for k in fr["d_slot"][:D, n]]
        assert gp == fg["p_slot"][:P, n].tolist() and gd == fg["d_slot"][:D, n].tolist()
        for key, rows in (("p_cap", P), ("src_cap", P), ("d_cap", D), ("sink_cap", D), ("kv_cap", P * D)):
            assert np.array_equal(fr[key][:rows, n], fg[key][:rows, n]), (key, n)
    vr = hxo.maxflow_batch(fr, want_flows=False)["flow_value"]
    vg = hxo.maxflow_batch(fg, want_flows=False)["flow_value"]
    assert np.array_equal(vr, vg)
    assert (vr > 0).sum() > 10


def test_per_gpu_kv_edges_on_refinement_workload():
    """On the 128-GPU refinement workload every KV edge between feasible replicas is the
    one-GPU-replica edge of its two GPUs (the replica rule with one stage pair and one rank
    pair), independent of both replicas' sizes."""
    prob = I.make_problem(5, n_cand=3)
    cost = hxo.cost_eval(prob)
    f = hxo.build_flownet(prob, cost)
    checked = 0
    for n in range(prob.n_cand):
        P, D = int(f["n_p"][n]), int(f["n_d"][n])
        for i in range(0, P, 5):
            for j in range(0, D, 3):
                g, h = int(f["p_slot"][i, n]), int(f["d_slot"][j, n])
                kp, kd = int(prob.assign[g, n]), int(prob.assign[h, n])
                feasible = cost["tp"][kp, n] > 0 and cost["tp"][kd, n] > 0
                want = hxo.quantize(1000.0 / hxo.kv_time(prob, [g], 1, 1, [h], 1, 1)) if feasible else 0
                assert int(f["kv_cap"][i * D + j, n]) == want
                checked += feasible
    assert checked > 20
