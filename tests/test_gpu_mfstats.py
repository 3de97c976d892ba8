"""GPU check of the max-flow diagnostic counters (hx_maxflow_stats), through the C-ABI: the flow
values equal hx_maxflow_batch's, and the candidates counted per path equal a host classification
of the same networks by the rules that pick the path (no flow possible; one side with a single
node that can carry flow; every KV arc at least min(a_i, b_j); at most six such nodes on the
smaller side when only values are wanted; push-relabel otherwise), for the packed plans of the
32-GPU workload with and without flow assignments and for the per-workgroup plans of the
128-GPU refinement workload (where a pre-pass settles the no-flow and dominant networks)."""
import sys

import numpy as np
import pytest

from paper_2502_07903_amd import hx
from paper_2502_07903_amd import inputs as I

pytestmark = pytest.mark.gpu
ENUM_MAX = 6


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


def _classify(net, value_only: bool, packed: bool):
    """Host classification of every candidate's path."""
    n_p, n_d = net["n_p"], net["n_d"]
    N = n_p.shape[0]
    counts = dict(no_flow=0, star=0, dominant=0, min_cut=0, push_relabel=0)
    for n in range(N):
        P, D = int(n_p[n]), int(n_d[n])
        a = np.minimum(net["src_cap"][:P, n], net["p_cap"][:P, n]).astype(np.int64)
        b = np.minimum(net["d_cap"][:D, n], net["sink_cap"][:D, n]).astype(np.int64)
        pe, de = int((a > 0).sum()), int((b > 0).sum())
        if P == 0 or D == 0 or pe == 0 or de == 0:
            counts["no_flow"] += 1
            continue
        c = net["kv_cap"][:P * D, n].astype(np.int64).reshape(P, D)
        dominant = bool((c >= np.minimum(a[:, None], b[None, :])).all())
        if packed and (pe == 1 or de == 1):
            counts["star"] += 1
        elif dominant:
            counts["dominant"] += 1
        elif packed and value_only and min(pe, de) <= ENUM_MAX:
            counts["min_cut"] += 1
        else:
            counts["push_relabel"] += 1
    return counts


def _run(torch, prob, flows: bool):
    dp = hx.DeviceProblem.upload(prob)
    ws = hx.Workspace.for_problem(dp, flows=flows)
    hx.score(dp, ws)
    torch.cuda.synchronize()
    ref = ws.flow_value.clone()
    fv = torch.full_like(ws.flow_value, -7)
    kv = torch.zeros_like(ws.kv_flow) if flows else None
    cut = torch.zeros_like(ws.cut) if flows else None
    st = hx.maxflow_stats(ws.net, fv, kv, cut)
    assert torch.equal(fv, ref)
    return st, ws.net.host()


@pytest.mark.parametrize("flows", [False, True])
def test_packed_plan_paths(torch, flows):
    prob = I.make_problem(3, n_cand=8192)
    say(f"max-flow counters: workload 3, N=8192, flows={flows}")
    st, net = _run(torch, prob, flows)
    want = _classify(net, value_only=not flows, packed=True)
    for k, v in want.items():
        assert st[k] == v, (k, st[k], v)
    assert st["prepass"] == 0
    assert (st["pushes"] > 0) == (st["push_relabel"] > 0)
    assert st["rounds"] >= (1 if st["push_relabel"] else 0)


def test_workgroup_plan_paths(torch):
    prob = I.make_problem(5, n_cand=512)
    say("max-flow counters: refinement workload round 0, N=512")
    st, net = _run(torch, prob, flows=False)
    want = _classify(net, value_only=True, packed=False)
    assert st["prepass"] == want["no_flow"] + want["dominant"]
    assert st["push_relabel"] == want["push_relabel"]
    assert st["star"] == st["min_cut"] == st["dominant"] == st["no_flow"] == 0
