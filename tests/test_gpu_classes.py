"""GPU parity of request classes (per-bucket workloads) against the oracle, through the C-ABI:
with the requests costed as four prompt-length classes every strategy choice, batch limit,
capacity and latency, the networks built on them, every flow value and the best candidate must
equal the oracle's (integers bit-exact, latencies to 1e-5 relative and expected
bit-identical), alone and with the pipelined decode capacity, at both flow-node granularities,
on ragged batch sizes, and on a class mix that no group can hold."""
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


def _classes(prob, cfg, variant=0):
    return dataclasses.replace(prob, classes=I.length_classes(I.WORKLOADS[cfg]), variant=variant)


def _gpu(torch, prob):
    dp = hx.DeviceProblem.upload(prob)
    assert dp.workload.n_classes == len(prob.classes)
    ws = hx.Workspace.for_problem(dp)
    hx.score(dp, ws)
    torch.cuda.synchronize()
    return ({k: getattr(ws.cost, k).cpu().numpy() for k in ("tp", "pp", "bmax", "cap", "lat")}, ws.net.host(),
            ws.flow_value.cpu().numpy(), tuple(int(x) for x in ws.best.cpu().numpy()))


def _check(cost, fn, fv, best, want):
    for k in ("tp", "pp", "bmax", "cap"):
        bad = cost[k] != want["cost"][k]
        assert not bad.any(), f"{k} differs at {np.argwhere(bad)[:5].tolist()}"
    rel = np.abs(cost["lat"] - want["cost"]["lat"]) / np.maximum(np.abs(want["cost"]["lat"]), 1e-300)
    assert (rel <= 1e-5).all()
    assert np.array_equal(cost["lat"], want["cost"]["lat"])
    Hh.compare_flownet(fn, want["flownet"])
    assert np.array_equal(fv, want["flow_value"])
    assert best == want["best"]


@pytest.mark.parametrize("cfg,n,variant", [(1, None, 0), (2, None, 0), (3, None, 0), (3, 4097, 1), (4, None, 0),
                                           (4, 4096, 1), (2, 1, 0)])
def test_classes_parity(torch, cfg, n, variant):
    prob = _classes(I.make_problem(cfg, n_cand=n), cfg, variant)
    say(f"request classes: workload {cfg}, N={prob.n_cand}, variant {variant}")
    got = _gpu(torch, prob)
    want = hxo.score_batch(prob, n_threads=N_THREADS)
    _check(*got, want)
    assert (got[0]["tp"] > 0).any()


def test_classes_per_gpu_nodes(torch):
    """Per-GPU flow nodes (128 GPUs), on a seeded sample of round 0."""
    prob = _classes(I.make_problem(5, n_cand=1024), 5)
    say("request classes: per-GPU nodes, N=1024")
    got = _gpu(torch, prob)
    want = hxo.score_batch(prob, n_threads=N_THREADS)
    _check(*got, want)


def test_classes_one_class_holds_nothing(torch):
    """A class whose KV cache exceeds every GPU's memory: every group infeasible, no flow."""
    prob = I.make_problem(2, n_cand=512)
    prob = dataclasses.replace(prob, classes=np.array([[prob.s_in, prob.s_out, 0.5], [4.0e7, prob.s_out, 0.5]]))
    say("request classes: an unservable class, N=512")
    got = _gpu(torch, prob)
    want = hxo.score_batch(prob, n_threads=N_THREADS)
    _check(*got, want)
    assert (got[0]["tp"] == 0).all() and (got[2] == 0).all()


def test_classes_refused_with_order_search(torch):
    prob = _classes(I.make_problem(1, n_cand=8), 1, variant=2)
    dp = hx.DeviceProblem.upload(prob)
    ws = hx.Workspace.for_problem(dp)
    with pytest.raises(hx.HxError):
        hx.score(dp, ws)
