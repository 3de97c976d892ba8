"""The cost-model entry point that allocates nothing (hx_cost_eval_static, libhx's static device
scratch) against hx_cost_eval with a caller-owned workspace, through the C-ABI: two calls in a row,
the second on a smaller batch, every output bit-exact.  (Its host-side refusal of a batch whose
scratch exceeds the static array is a CPU test in test_abi.py.)"""
import sys

import numpy as np
import pytest

from paper_2502_07903_amd import hx
from paper_2502_07903_amd import inputs as I

pytestmark = pytest.mark.gpu


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


def _garbage(torch, buf: hx.CostBuffers, byte: int) -> None:
    for t in (buf.tp, buf.pp, buf.bmax, buf.cap, buf.lat, buf.members):
        t.view(torch.uint8).fill_(byte)


def _host(buf: hx.CostBuffers):
    return {k: getattr(buf, k).cpu().numpy().view(np.uint8) for k in ("tp", "pp", "bmax", "cap", "lat", "members")}


@pytest.mark.parametrize("order", ["large_then_small"])
def test_cost_eval_static_matches_workspace_call(torch, order):
    L = hx.lib()
    cases = [(3, 65536), (2, 777)]  # the second call smaller than the first
    for cfg, n in cases:
        prob = I.make_problem(cfg, n_cand=n)
        need = int(L.hx_cost_workspace_bytes(prob.n_gpus, prob.max_groups, n))
        assert need <= int(L.hx_static_scratch_bytes())
        say(f"no-alloc cost model: workload {cfg}, N={n}, scratch {need} bytes")
        dp = hx.DeviceProblem.upload(prob)
        ref = hx.CostBuffers.empty(dp.max_groups, n, dp.n_gpus)
        got = hx.CostBuffers.empty(dp.max_groups, n, dp.n_gpus)
        _garbage(torch, ref, 0x5A)
        _garbage(torch, got, 0xA5)
        hx.cost_eval(dp, ref)
        hx.cost_eval_static(dp, got)
        torch.cuda.synchronize()
        a, b = _host(ref), _host(got)
        for k in a:
            assert np.array_equal(a[k], b[k]), f"{k} differs (workload {cfg}, N={n})"
        assert (ref.cap.cpu().numpy() > 0).any()
