"""Host-side checks of the C-ABI library (no GPU): it loads, exports every function that
include/hx.h declares, and hx_validate accepts and rejects arguments as documented without
any device access (the pointers below are never dereferenced)."""
import ctypes as C
import os
import re

import pytest

from paper_2502_07903_amd import hx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "hx.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(hx_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_function():
    names = _declared_functions()
    assert "hx_maxflow_batch" in names and "hx_cost_eval" in names
    lib = hx.lib()
    for name in names:
        assert hasattr(lib, name), f"libhx.so does not export {name}"
    assert set(hx.EXPORTS) <= set(names)


def test_abi_version_and_strings():
    assert hx.lib().hx_abi_version() == 3
    for code in (0, -1, -2, -3, -4):
        assert hx.strerror(code)
    assert hx.lib().hx_last_error() is not None


FAKE = 0x1000  # a non-null address that validation must never dereference


def _args(G=32, T=4, N=100, Kmax=16, tp=0b1011, pp=0xFF, gran=0):
    cl = hx.hx_cluster(G, T, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, 0.0)
    md = hx.hx_model(80, 8192, 64, 8, 2)
    wl = hx.hx_workload(1024.0, 256.0)
    sp = hx.hx_space(tp, pp, gran)
    cand = hx.hx_candidates(N, Kmax, FAKE, FAKE)
    cost = hx.hx_cost_out(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    b = Kmax if gran == 0 else G
    net = hx.hx_flownet(N, b, b, (b // 2) * ((b + 1) // 2), *([FAKE] * 9))
    return cl, md, wl, sp, cand, cost, net


def _validate(cl, md, wl, sp, cand, cost, net):
    return hx.lib().hx_validate(C.byref(cl), md, wl, sp, C.byref(cand), C.byref(cost) if cost else None,
                                C.byref(net) if net else None)


def test_validate_accepts_workloads():
    for kw in (dict(G=8, T=2, N=256, Kmax=4), dict(G=32, N=65536, Kmax=16), dict(G=64, T=5, N=262144, Kmax=32),
               dict(G=128, T=6, N=131072, Kmax=32, gran=1)):
        assert _validate(*_args(**kw)) == hx.HX_OK
    a = list(_args())
    for v in (1, 2, 3, 4, 5):                           # HX_VARIANT_PIPELINED, _KV_ORDER, _ASYM
        a[3].variant = v
        assert _validate(*a) == hx.HX_OK
    a = list(_args())
    for n in (1, 4):                                    # request classes, alone and pipelined
        _classes(a[2], n)
        for v in (0, 1):
            a[3].variant = v
            assert _validate(*a) == hx.HX_OK


def _classes(wl, n):
    wl.n_classes = n
    for k in range(n):
        wl.cls_in[k], wl.cls_out[k], wl.cls_w[k] = 300.0 * (k + 1), 400.0, 1.0 / n


@pytest.mark.parametrize("mutate", [
    lambda a: setattr(a[0], "n_gpus", 0),
    lambda a: setattr(a[0], "n_gpus", 256),
    lambda a: setattr(a[0], "beta", None),
    lambda a: setattr(a[0], "coord_bw", -1.0),
    lambda a: setattr(a[1], "n_layers", 0),
    lambda a: setattr(a[1], "n_kv_heads", 65),
    lambda a: setattr(a[1], "n_heads", 48),          # H_kv = 8192 * 8 / 48 is not whole
    lambda a: setattr(a[2], "s_in", 0.0),
    lambda a: setattr(a[2], "s_out", float("nan")),
    lambda a: setattr(a[2], "n_classes", 5),        # more than HX_MAX_CLASSES
    lambda a: setattr(a[2], "n_classes", -1),
    lambda a: (_classes(a[2], 2), a[2].cls_w.__setitem__(1, 0.0)),
    lambda a: (_classes(a[2], 3), a[2].cls_in.__setitem__(2, float("inf"))),
    lambda a: (_classes(a[2], 1), a[2].cls_out.__setitem__(0, -5.0)),
    lambda a: (_classes(a[2], 4), setattr(a[3], "variant", 2)),   # classes with the stage-order search
    lambda a: (_classes(a[2], 4), setattr(a[3], "variant", 4)),   # classes with the asymmetric split
    lambda a: setattr(a[3], "tp_mask", 0),
    lambda a: setattr(a[3], "tp_mask", 1 << 8),      # TP degree 9 > 8
    lambda a: setattr(a[3], "pp_mask", 0),
    lambda a: setattr(a[3], "granularity", 2),
    lambda a: setattr(a[3], "variant", 8),           # unknown cost-model variant bit
    lambda a: setattr(a[3], "variant", 6),           # stage-order search with the asymmetric split
    lambda a: setattr(a[4], "n_cand", 0),
    lambda a: setattr(a[4], "max_groups", 256),
    lambda a: setattr(a[4], "role", None),
    lambda a: setattr(a[5], "lat", None),
    lambda a: setattr(a[5], "members", None),
    lambda a: setattr(a[6], "max_pd", 63),           # 16 groups may split 8/8: 64 KV edges
    lambda a: setattr(a[6], "max_p", 15),
    lambda a: setattr(a[6], "n_cand", 99),
    lambda a: setattr(a[6], "kv_cap", None),
], ids=lambda f: "")
def test_validate_rejects(mutate):
    a = list(_args())
    mutate(a)
    assert _validate(*a) == hx.HX_EINVAL


def test_validate_too_big_for_lds():
    # 255 GPUs at per-GPU granularity: 127*128 KV edges exceed the LDS plan.
    a = _args(G=255, T=6, N=10, Kmax=32, gran=1)
    assert _validate(*a) == hx.HX_ETOOBIG


def test_cost_eval_static_refuses_before_any_device_work():
    """The entry point that allocates nothing refuses, on the host and before any HIP call, a
    batch whose scratch exceeds its static array (262,144 candidates of 64 GPUs and 32 groups
    need 137 MB), and invalid arguments as hx_cost_eval does."""
    L = hx.lib()
    assert L.hx_static_scratch_bytes() == 32 << 20
    cl, md, wl, sp, cand, cost, net = _args(G=64, T=5, N=262144, Kmax=32)
    assert L.hx_cost_workspace_bytes(64, 32, 262144) > L.hx_static_scratch_bytes()
    assert L.hx_cost_eval_static(C.byref(cl), md, wl, sp, C.byref(cand), C.byref(cost), None) == hx.HX_ETOOBIG
    cand.n_cand = 0
    assert L.hx_cost_eval_static(C.byref(cl), md, wl, sp, C.byref(cand), C.byref(cost), None) == hx.HX_EINVAL
    cand.n_cand = 1000
    cost.lat = None
    assert L.hx_cost_eval_static(C.byref(cl), md, wl, sp, C.byref(cand), C.byref(cost), None) == hx.HX_EINVAL


def test_calls_reject_before_any_device_work():
    cl, md, wl, sp, cand, cost, net = _args()
    cand.n_cand = 0
    L = hx.lib()
    assert L.hx_cost_eval(C.byref(cl), md, wl, sp, C.byref(cand), C.byref(cost), FAKE, 1 << 30, None) == hx.HX_EINVAL
    cand.n_cand = 100
    need = L.hx_cost_workspace_bytes(32, 16, 100)
    assert need > 0
    ws = 0x100000  # 256-byte aligned, never dereferenced: every call below fails validation
    assert L.hx_cost_eval(C.byref(cl), md, wl, sp, C.byref(cand), C.byref(cost), ws, need - 1, None) == hx.HX_EINVAL
    assert L.hx_cost_eval(C.byref(cl), md, wl, sp, C.byref(cand), C.byref(cost), ws + 8, need, None) == hx.HX_EINVAL
    assert L.hx_cost_eval(C.byref(cl), md, wl, sp, C.byref(cand), C.byref(cost), None, need, None) == hx.HX_EINVAL
    cand.n_cand = 0
    assert L.hx_build_flownet(C.byref(cl), md, wl, sp, C.byref(cand), C.byref(cost), C.byref(net), None) == hx.HX_EINVAL
    assert L.hx_maxflow_batch(C.byref(net), None, None, None, None) == hx.HX_EINVAL
    assert L.hx_best_candidate(None, 10, FAKE, None) == hx.HX_EINVAL
    assert L.hx_best_candidate(FAKE, 0, FAKE, None) == hx.HX_EINVAL
    big = _args(G=255, T=6, N=10, Kmax=32, gran=1)[6]
    assert L.hx_maxflow_batch(C.byref(big), FAKE, None, None, None) == hx.HX_ETOOBIG
    # the diagnostic variant: same checks, plus an 8-byte aligned counter array
    assert L.hx_maxflow_stats(C.byref(net), None, None, None, FAKE, None) == hx.HX_EINVAL
    assert L.hx_maxflow_stats(C.byref(net), FAKE, None, None, None, None) == hx.HX_EINVAL
    assert L.hx_maxflow_stats(C.byref(net), FAKE, None, None, FAKE + 4, None) == hx.HX_EINVAL
    assert L.hx_maxflow_stats(C.byref(big), FAKE, None, None, FAKE, None) == hx.HX_ETOOBIG


def test_refinement_calls_reject_before_any_device_work():
    cl, md, wl, sp, cand, cost, net = _args()
    L = hx.lib()
    u8 = lambda: C.c_void_p(FAKE)
    assert L.hx_edge_classes(C.byref(net), None, FAKE, FAKE, FAKE, None) == hx.HX_EINVAL
    assert L.hx_edge_classes(C.byref(net), FAKE, None, FAKE, FAKE, None) == hx.HX_EINVAL
    assert L.hx_edge_classes(C.byref(net), FAKE, FAKE, None, FAKE, None) == hx.HX_EINVAL
    bad_net = hx.hx_flownet(0, 1, 1, 1, *([FAKE] * 9))
    assert L.hx_edge_classes(C.byref(bad_net), FAKE, FAKE, FAKE, FAKE, None) == hx.HX_EINVAL
    # guided moves: the parents' network must be built for the parent batch
    par = hx.hx_candidates(3, 16, FAKE, FAKE)
    pnet = hx.hx_flownet(3, 16, 16, 64, *([FAKE] * 9))
    ok = (32, 0, C.byref(par), C.byref(pnet), u8(), 100, u8(), u8(), u8(), u8(), None)
    for i, bad in ((0, 0), (0, 256), (1, 2), (5, 0), (4, None), (6, None), (7, None), (8, None), (9, None)):
        a = list(ok)
        a[i] = bad
        assert L.hx_guided_moves(*a) == hx.HX_EINVAL, (i, bad)
    pnet.n_cand = 4
    assert L.hx_guided_moves(*ok) == hx.HX_EINVAL
    many = hx.hx_candidates(70000, 16, FAKE, FAKE)
    mnet = hx.hx_flownet(70000, 16, 16, 64, *([FAKE] * 9))
    assert L.hx_guided_moves(32, 0, C.byref(many), C.byref(mnet), u8(), 100, u8(), u8(), u8(), u8(), None) == \
        hx.HX_EINVAL
    # gather
    src = hx.hx_candidates(10, 16, FAKE, FAKE)
    assert L.hx_gather_candidates(32, C.byref(src), None, 1, FAKE, FAKE, None) == hx.HX_EINVAL
    assert L.hx_gather_candidates(32, C.byref(src), FAKE, 0, FAKE, FAKE, None) == hx.HX_EINVAL
    assert L.hx_gather_candidates(0, C.byref(src), FAKE, 1, FAKE, FAKE, None) == hx.HX_EINVAL
    assert L.hx_gather_candidates(32, C.byref(src), FAKE, 1, None, FAKE, None) == hx.HX_EINVAL


def test_partition_calls_reject_before_any_device_work():
    cl, md, wl, sp, cand, cost, net = _args()
    L = hx.lib()
    assert L.hx_partition_workspace_bytes(1) == 0 and L.hx_partition_workspace_bytes(256) == 0
    need = L.hx_partition_workspace_bytes(32)
    assert need >= 32 * 32 * 4
    assert L.hx_spectral_order(C.byref(cl), 100, FAKE, need - 1, FAKE, None, None) == hx.HX_EINVAL
    assert L.hx_spectral_order(C.byref(cl), 100, FAKE, need, None, None, None) == hx.HX_EINVAL
    assert L.hx_spectral_order(C.byref(cl), -1, FAKE, need, FAKE, None, None) == hx.HX_EINVAL
    args = [C.byref(cl), md, wl, 16, FAKE, need, FAKE, 100, FAKE, FAKE, FAKE, None]
    for i, bad in ((3, 0), (4, None), (5, need - 1), (6, None), (7, 0), (8, None), (9, None), (10, None)):
        a = list(args)
        a[i] = bad
        assert L.hx_partition_candidates(*a) == hx.HX_EINVAL, (i, bad)
    cl.n_gpus = 1
    assert L.hx_spectral_order(C.byref(cl), 100, FAKE, need, FAKE, None, None) == hx.HX_EINVAL


def test_workspace_and_mask_sizes():
    L = hx.lib()
    assert [L.hx_member_words(g) for g in (1, 64, 65, 128, 129, 255)] == [1, 1, 2, 2, 4, 4]
    assert L.hx_member_words(0) == 0 and L.hx_member_words(256) == 0
    assert L.hx_cost_workspace_bytes(0, 16, 10) == 0
    # one unit slot per candidate and group (at most min(Kmax, G) groups) plus the histogram
    assert L.hx_cost_workspace_bytes(32, 16, 1000) >= 8 * 16 * 1000
    assert L.hx_cost_workspace_bytes(8, 16, 1000) >= 8 * 8 * 1000


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(hx, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(hx, "_lib", None)
    with pytest.raises(RuntimeError, match="not built"):
        hx.lib()
