"""Pins of the oracle's request classes (per-bucket workloads), no GPU.

With classes, a strategy must fit every class in memory; the replica's latency is the class
mix's mean and its capacity the weighted harmonic mean of its per-class capacities (the mix's
time per request is the weighted sum of per-class times), and a KV edge's time is the mix's
mean.  Checked against what those definitions fix: one class of weight 1 is the single task;
identical classes are the single task to rounding; the mix capacity lies between the per-class
capacities; a class that fits no memory makes every strategy infeasible; and the kept strategy
of every group is the one a search over its strategies, scored class by class with the single-
task cost (pinned on its own), selects.  The class buckets partition the drawn requests, so
their weighted means are the overall means.
"""
import dataclasses

import numpy as np
import pytest

from oracle import hxo
from paper_2502_07903_amd import inputs as I


def _with_classes(prob, rows):
    return dataclasses.replace(prob, classes=np.asarray(rows, np.float64))


def _single(prob, s_in, s_out):
    return dataclasses.replace(prob, s_in=float(s_in), s_out=float(s_out), classes=None)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_length_classes_partition_requests(cfg):
    wl = I.WORKLOADS[cfg]
    cls = I.length_classes(wl)
    a, b = I.request_lengths(wl)
    assert cls.shape == (4, 3)
    assert cls[:, 2].sum() == pytest.approx(1.0, abs=1e-15)
    assert (np.diff(cls[:, 0]) >= 0).all()
    assert (cls[:, 2] * cls[:, 0]).sum() == pytest.approx(a.mean(), rel=1e-13)
    assert (cls[:, 2] * cls[:, 1]).sum() == pytest.approx(b.mean(), rel=1e-13)
    # a bucket's prompts never exceed the next bucket's
    order = np.lexsort((np.arange(len(a)), b, a))
    q = len(a) // 4
    for k in range(3):
        assert a[order[(k + 1) * q - 1]] <= a[order[(k + 1) * q]]


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_one_class_is_the_single_task(cfg):
    prob = I.make_problem(cfg, n_cand=48)
    one = _with_classes(prob, [[prob.s_in, prob.s_out, 1.0]])
    a, b = hxo.cost_eval(prob), hxo.cost_eval(one)
    for k in ("tp", "pp", "bmax", "lat"):
        assert np.array_equal(a[k], b[k]), k
    # x = 1 / (1 / x) can move the last bit, so the quantised capacity by at most one
    assert np.abs(a["cap"].astype(np.int64) - b["cap"]).max() <= 1
    fa, fb = hxo.build_flownet(prob, a), hxo.build_flownet(one, a)
    assert np.array_equal(fa["kv_cap"], fb["kv_cap"])


def test_identical_classes_are_the_single_task():
    prob = I.make_problem(3, n_cand=32)
    four = _with_classes(prob, [[prob.s_in, prob.s_out, 0.25]] * 4)
    a, b = hxo.cost_eval(prob), hxo.cost_eval(four)
    for k in ("tp", "pp", "bmax"):
        assert np.array_equal(a[k], b[k]), k
    np.testing.assert_allclose(b["lat"], a["lat"], rtol=1e-15)
    assert np.abs(a["cap"].astype(np.int64) - b["cap"]).max() <= 1
    fa, fb = hxo.build_flownet(prob, a), hxo.build_flownet(four, a)
    assert np.abs(fa["kv_cap"].astype(np.int64) - fb["kv_cap"]).max() <= 1


def _groups(prob, n):
    """(members, role) of the present groups of the first n candidates."""
    out = []
    for c in range(n):
        col = prob.assign[:, c]
        for k in range(prob.max_groups):
            r = int(prob.role[k, c])
            if r in (I.PREFILL, I.DECODE):
                m = np.flatnonzero(col == k).tolist()
                if m:
                    out.append((m, r))
    return out


def _strategies(prob, n):
    out = []
    for tp in (1, 2, 4, 8):
        if not (prob.tp_mask >> (tp - 1)) & 1 or n % tp:
            continue
        pp = n // tp
        if (prob.pp_mask >> (pp - 1)) & 1 and pp <= prob.model["n_layers"]:
            out.append((tp, pp))
    return out


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_selection_matches_per_class_search(cfg):
    """The kept strategy, found by a search over the group's strategies with every class scored
    on its own single task: lowest mix latency for prefill, highest harmonic-mean capacity for
    decode, ties to the smaller tp; infeasible in any class = not a candidate."""
    prob = I.make_problem(cfg, n_cand=24)
    cls = I.length_classes(I.WORKLOADS[cfg])
    mix = _with_classes(prob, cls)
    seen = [0, 0]
    for members, role in _groups(prob, 24):
        best = None
        for tp, pp in _strategies(prob, len(members)):
            rows = [hxo.strategy_cost(_single(prob, i, o), members, tp, pp, role, variant=0) for i, o, _ in cls]
            if not all(r[0] for r in rows):
                continue
            lat, tau = 0.0, 0.0
            for (ok, bk, lk, xk), w in zip(rows, cls[:, 2]):
                lat = lat + w * lk
                tau = tau + w / xk
            x = 1.0 / tau
            bmax = min(r[1] for r in rows)
            if best is None or (lat < best[4] if role == I.PREFILL else x > best[5]):
                best = (tp, pp, bmax, None, lat, x)
            lo, hi = min(r[3] for r in rows), max(r[3] for r in rows)
            assert lo * (1 - 1e-15) <= x <= hi * (1 + 1e-15)
        got = hxo.group_select(mix, members, role)
        if best is None:
            assert got == (0, 0, 0, 0, 0.0)
            continue
        seen[role] += 1
        exp = (best[0], best[1], best[2], hxo.quantize(best[5]), best[4])
        assert got == exp, (members, role)
    assert min(seen) > 0


def test_class_that_fits_nowhere_makes_groups_infeasible():
    """A class whose KV cache alone exceeds every GPU's memory admits no batch of one."""
    prob = I.make_problem(2, n_cand=16)
    mix = _with_classes(prob, [[prob.s_in, prob.s_out, 0.5], [4.0e7, prob.s_out, 0.5]])
    out = hxo.cost_eval(mix)
    assert (out["tp"] == 0).all() and (out["cap"] == 0).all()
    assert (hxo.cost_eval(prob)["tp"] > 0).any()


@pytest.mark.parametrize("cfg", [2, 3])
def test_kv_mix_is_weighted_mean_of_class_times(cfg):
    prob = I.make_problem(cfg, n_cand=64)
    cls = I.length_classes(I.WORKLOADS[cfg])
    mix = _with_classes(prob, cls)
    cost = hxo.cost_eval(mix)
    f = hxo.build_flownet(mix, cost)
    checked = 0
    for n in range(prob.n_cand):
        nd = int(f["n_d"][n])
        for i in range(int(f["n_p"][n])):
            for j in range(nd):
                kp, kd = int(f["p_slot"][i, n]), int(f["d_slot"][j, n])
                if cost["tp"][kp, n] == 0 or cost["tp"][kd, n] == 0:
                    continue
                pm = np.flatnonzero(prob.assign[:, n] == kp).tolist()
                dm = np.flatnonzero(prob.assign[:, n] == kd).tolist()
                t = 0.0
                for s_in, s_out, w in cls:
                    t = t + w * hxo.kv_time(_single(prob, s_in, s_out), pm, int(cost["tp"][kp, n]),
                                            int(cost["pp"][kp, n]), dm, int(cost["tp"][kd, n]),
                                            int(cost["pp"][kd, n]))
                assert f["kv_cap"][i * nd + j, n] == hxo.quantize(1000.0 / t)
                checked += 1
    assert checked > 10


def test_classes_refused_with_stage_order_or_asym_split():
    prob = I.make_problem(1, n_cand=4)
    cls = I.length_classes(I.WORKLOADS[1])
    for v in (2, 4):
        with pytest.raises(ValueError):
            hxo.cost_eval(dataclasses.replace(_with_classes(prob, cls), variant=v))
    hxo.cost_eval(dataclasses.replace(_with_classes(prob, cls), variant=1))


def test_kv_mix_per_gpu_nodes():
    """Per-GPU nodes (128 GPUs): each GPU edge's time is the mix's mean of its per-class times."""
    prob = I.make_problem(5, n_cand=2)
    cls = I.length_classes(I.WORKLOADS[5])
    mix = _with_classes(prob, cls)
    cost = hxo.cost_eval(mix)
    f = hxo.build_flownet(mix, cost)
    checked = 0
    for n in range(prob.n_cand):
        nd = int(f["n_d"][n])
        for i in range(0, int(f["n_p"][n]), 7):
            for j in range(0, nd, 5):
                g, h = int(f["p_slot"][i, n]), int(f["d_slot"][j, n])
                kp, kd = int(prob.assign[g, n]), int(prob.assign[h, n])
                if cost["tp"][kp, n] == 0 or cost["tp"][kd, n] == 0:
                    continue
                t = 0.0
                for s_in, s_out, w in cls:
                    t = t + w * hxo.kv_gpu_time(_single(prob, s_in, s_out), g, h)
                assert f["kv_cap"][i * nd + j, n] == hxo.quantize(1000.0 / t)
                checked += 1
    assert checked > 10
