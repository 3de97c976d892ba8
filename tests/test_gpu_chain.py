"""Workload 5 as a chain, through the C-ABI: 16 rounds of 131,072 single-step perturbations of the
128-GPU cluster (per-GPU flow nodes), each round perturbing the previous round's best placement.

Per round, against the oracle on the same seeded inputs:
  * 4,096 seeded sample candidates and the GPU's 16 highest-scoring ones: flow values bit-exact;
  * the argmax certified over the whole batch: every candidate's flow is at most its upper bound
    min(sum of prefill replica capacities, sum of decode replica capacities), taken from the
    oracle's cost model (a GPU node's share of its replica's capacity sums back to the capacity,
    and coordinator edges are unbounded), so the oracle scores every candidate whose bound exceeds
    the GPU's best value, and every candidate below the GPU's index whose bound reaches it: none
    may beat it, none may tie it at a lower index;
  * the next round's base is that candidate, the one the oracle's own argmax picks.
"""
import os
import sys

import numpy as np
import pytest

from oracle import hxo
from paper_2502_07903_amd import hx
from paper_2502_07903_amd import inputs as I

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


def test_refinement_chain(torch):
    wl = I.WORKLOADS[5]
    n, rounds = wl.n_cand, wl.rounds
    assert (n, rounds) == (131072, 16)
    cur = I.base_placement(wl)
    dp = ws = None
    rng = np.random.default_rng(2516)
    bests = []
    for r in range(rounds):
        prob = I.make_problem(5, n_cand=n, rnd=r, base=cur)
        say(f"chain round {r}: scoring {n} candidates on the GPU")
        if dp is None:
            # every candidate is one move from the same placement (the shared-groups hint)
            dp = hx.DeviceProblem.upload(prob).with_hint()
            ws = hx.Workspace.for_problem(dp, flows=False)
        else:
            dp.tensors["assign"].copy_(torch.from_numpy(prob.assign))
            dp.tensors["role"].copy_(torch.from_numpy(prob.role))
        hx.score(dp, ws)
        torch.cuda.synchronize()
        fv = ws.flow_value.cpu().numpy()
        bi, bv = (int(x) for x in ws.best.cpu().numpy())
        assert fv[bi] == bv and bv == fv.max() and np.flatnonzero(fv == bv)[0] == bi
        # sampled values and the GPU's top 16
        top = np.argsort(-fv.astype(np.int64), kind="stable")[:16]
        idx = np.unique(np.concatenate([rng.choice(n, 4096, replace=False), top]))
        want = hxo.score_batch(prob.subset(idx), n_threads=N_THREADS)["flow_value"]
        bad = np.flatnonzero(fv[idx] != want)
        assert bad.size == 0, f"round {r}: flow values differ at {idx[bad[:8]].tolist()}"
        # the argmax over the whole batch, certified by the oracle's upper bounds
        cap = hxo.cost_eval(prob)["cap"].astype(np.int64)
        a = np.where(prob.role == I.PREFILL, cap, 0).sum(0)
        b = np.where(prob.role == I.DECODE, cap, 0).sum(0)
        ub = np.minimum(a, b)
        assert (fv <= ub).all()
        check = np.flatnonzero((ub > bv) | ((ub == bv) & (np.arange(n) < bi)))
        say(f"chain round {r}: best {bv} at {bi}; certifying over {check.size} candidates")
        if check.size:
            vals = hxo.score_batch(prob.subset(check), n_threads=N_THREADS)["flow_value"]
            assert vals.max() <= bv
            assert not ((vals == bv) & (check < bi)).any()
        bests.append(bv)
        cur = (prob.assign[:, bi].copy(), prob.role[:, bi].copy())
    # a round's batch holds single-step variants of the previous best, not the placement itself,
    # so the best may also drop from one round to the next
    say(f"chain bests: {bests}")
