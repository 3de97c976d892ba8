"""ctypes binding of the CPU oracle (oracle/hxo.c).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU
baseline use it to check and time the HIP path; the product path never imports
it.  It takes the numpy arrays of `paper_2502_07903_amd.inputs` and returns
numpy arrays in the same candidate-fastest layouts as the C-ABI library.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "hxo.c")
LIB = os.path.join(HERE, "libhxo.so")
CAP_MAX = 16777215

# -O2 without -march: SSE2 binary64, no FMA contraction, no fast-math.
BUILD_CMD = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
             "-Wall", "-o", LIB, SRC, "-lm", "-lpthread"]


def build() -> str:
    subprocess.run(BUILD_CMD, check=True)
    return LIB


class _Cluster(C.Structure):
    _fields_ = [("n_gpus", C.c_int32), ("n_types", C.c_int32), ("gpu_type", C.c_void_p),
                ("type_flops", C.c_void_p), ("type_hbm_bw", C.c_void_p), ("type_mem", C.c_void_p),
                ("beta", C.c_void_p), ("alpha", C.c_void_p), ("coord_bw", C.c_double),
                ("req_bytes", C.c_double)]


class _Model(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("hidden", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("bytes_per_elem", C.c_int32)]


MAX_CLASSES = 4


class _Workload(C.Structure):
    _fields_ = [("s_in", C.c_double), ("s_out", C.c_double), ("n_classes", C.c_int32),
                ("cls_in", C.c_double * MAX_CLASSES), ("cls_out", C.c_double * MAX_CLASSES),
                ("cls_w", C.c_double * MAX_CLASSES)]


def _workload(prob) -> _Workload:
    """The task t, and the request classes (rows of (s_in, s_out, weight)) when prob has them."""
    w = _Workload(float(prob.s_in), float(prob.s_out), 0)
    cls = getattr(prob, "classes", None)
    if cls is not None:
        cls = np.asarray(cls, np.float64)
        w.n_classes = len(cls)
        for k, (i, o, wt) in enumerate(cls):
            w.cls_in[k], w.cls_out[k], w.cls_w[k] = float(i), float(o), float(wt)
    return w


class _Space(C.Structure):
    _fields_ = [("tp_mask", C.c_uint32), ("pp_mask", C.c_uint32), ("granularity", C.c_int32),
                ("variant", C.c_uint32)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        _lib = C.CDLL(LIB)
        _lib.hxo_maxflow_edges.restype = C.c_int64
        _lib.hxo_kv_time.restype = C.c_double
        _lib.hxo_kv_time_best.restype = C.c_double
        _lib.hxo_kv_time_orders.restype = C.c_double
        _lib.hxo_kv_gpu_time.restype = C.c_double
        _lib.hxo_quantize.restype = C.c_int32
    return _lib


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise ValueError(f"{what}: the oracle refused the problem ({rc})")


def _p(a: np.ndarray) -> C.c_void_p:
    assert a.flags["C_CONTIGUOUS"]
    return C.c_void_p(a.ctypes.data)


class _Args:
    """Keeps the numpy arrays alive while the C structs point at them."""

    def __init__(self, prob):
        cl = prob.cluster
        self.keep = [np.ascontiguousarray(x) for x in
                     (cl.gpu_type.astype(np.int32), cl.type_flops.astype(np.float64),
                      cl.type_hbm_bw.astype(np.float64), cl.type_mem.astype(np.float64),
                      cl.beta.astype(np.float64), cl.alpha.astype(np.float64))]
        k = self.keep
        self.cluster = _Cluster(cl.n_gpus, cl.n_types, _p(k[0]), _p(k[1]), _p(k[2]), _p(k[3]),
                                _p(k[4]), _p(k[5]), float(cl.coord_bw), float(cl.req_bytes))
        m = prob.model
        self.model = _Model(m["n_layers"], m["hidden"], m["n_heads"], m["n_kv_heads"], m["bytes_per_elem"])
        self.wl = _workload(prob)
        self.space = _Space(int(prob.tp_mask), int(prob.pp_mask), int(prob.granularity),
                            int(getattr(prob, "variant", 0)))

    def refs(self):
        return C.byref(self.cluster), C.byref(self.model), C.byref(self.wl), C.byref(self.space)


def flownet_dims(prob) -> Tuple[int, int, int]:
    """(max_p, max_d, max_pd): room for any split of the replicas (or GPUs) into two sides."""
    b = prob.max_groups if prob.granularity == 0 else prob.n_gpus
    return b, b, (b // 2) * ((b + 1) // 2)


def cost_eval(prob) -> Dict[str, np.ndarray]:
    a = _Args(prob)
    K, N = prob.max_groups, prob.n_cand
    out = dict(tp=np.zeros((K, N), np.uint8), pp=np.zeros((K, N), np.uint8), bmax=np.zeros((K, N), np.int32),
               cap=np.zeros((K, N), np.int32), lat=np.zeros((K, N), np.float64))
    rc = lib().hxo_cost_eval(*a.refs(), C.c_int32(N), C.c_int32(K), _p(prob.assign), _p(prob.role),
                        _p(out["tp"]), _p(out["pp"]), _p(out["bmax"]), _p(out["cap"]), _p(out["lat"]))
    _check(rc, "hxo_cost_eval")
    return out


def _flownet_arrays(N, dims):
    mp, md, mpd = dims
    return dict(n_p=np.zeros(N, np.int32), n_d=np.zeros(N, np.int32),
                p_slot=np.zeros((mp, N), np.int32), d_slot=np.zeros((md, N), np.int32),
                src_cap=np.zeros((mp, N), np.int32), p_cap=np.zeros((mp, N), np.int32),
                kv_cap=np.zeros((mpd, N), np.int32), d_cap=np.zeros((md, N), np.int32),
                sink_cap=np.zeros((md, N), np.int32))


def build_flownet(prob, cost: Dict[str, np.ndarray], dims: Optional[Tuple[int, int, int]] = None):
    a = _Args(prob)
    dims = dims or flownet_dims(prob)
    N = prob.n_cand
    f = _flownet_arrays(N, dims)
    rc = lib().hxo_build_flownet(*a.refs(), C.c_int32(N), C.c_int32(prob.max_groups), _p(prob.assign),
                            _p(prob.role), _p(cost["tp"]), _p(cost["pp"]), _p(cost["cap"]),
                            *(C.c_int32(x) for x in dims),
                            *(_p(f[k]) for k in ("n_p", "n_d", "p_slot", "d_slot", "src_cap", "p_cap",
                                                 "kv_cap", "d_cap", "sink_cap")))
    _check(rc, "hxo_build_flownet")
    f["dims"] = dims
    return f


def maxflow_batch(f, want_flows: bool = True) -> Dict[str, np.ndarray]:
    mp, md, mpd = f["dims"]
    N = f["n_p"].shape[0]
    out = dict(flow_value=np.zeros(N, np.int32))
    kv = np.zeros((mpd, N), np.int32) if want_flows else None
    cut = np.zeros((mp + md, N), np.uint8) if want_flows else None
    lib().hxo_maxflow_batch(C.c_int32(N), C.c_int32(mp), C.c_int32(md), C.c_int32(mpd),
                            *(_p(f[k]) for k in ("n_p", "n_d", "src_cap", "p_cap", "kv_cap", "d_cap",
                                                 "sink_cap")),
                            _p(out["flow_value"]), _p(kv) if kv is not None else None,
                            _p(cut) if cut is not None else None)
    if want_flows:
        out["kv_flow"] = kv
        out["cut"] = cut
    return out


def best_candidate(flow_value: np.ndarray) -> Tuple[int, int]:
    fv = np.ascontiguousarray(flow_value, np.int32)
    best = np.zeros(2, np.int32)
    rc = lib().hxo_best_candidate(_p(fv), C.c_int32(len(fv)), _p(best))
    if rc != 0:
        raise ValueError("empty batch")
    return int(best[0]), int(best[1])


def score_batch(prob, n_threads: int = 1, dims=None) -> Dict[str, object]:
    """Cost model + flow network + max-flow + argmax over the whole batch on n_threads threads."""
    a = _Args(prob)
    dims = dims or flownet_dims(prob)
    K, N = prob.max_groups, prob.n_cand
    cost = dict(tp=np.zeros((K, N), np.uint8), pp=np.zeros((K, N), np.uint8), bmax=np.zeros((K, N), np.int32),
                cap=np.zeros((K, N), np.int32), lat=np.zeros((K, N), np.float64))
    f = _flownet_arrays(N, dims)
    fv = np.zeros(N, np.int32)
    best = np.zeros(2, np.int32)
    rc = lib().hxo_score_batch(*a.refs(), C.c_int32(N), C.c_int32(K), _p(prob.assign), _p(prob.role),
                          *(_p(cost[k]) for k in ("tp", "pp", "bmax", "cap", "lat")),
                          *(C.c_int32(x) for x in dims),
                          *(_p(f[k]) for k in ("n_p", "n_d", "p_slot", "d_slot", "src_cap", "p_cap",
                                               "kv_cap", "d_cap", "sink_cap")),
                          _p(fv), _p(best), C.c_int32(n_threads))
    _check(rc, "hxo_score_batch")
    f["dims"] = dims
    return dict(cost=cost, flownet=f, flow_value=fv, best=(int(best[0]), int(best[1])))


# ------------------------------------------------------------------ single-group entry points

def strategy_cost(prob, members: Sequence[int], tp: int, pp: int, role: int, variant: Optional[int] = None):
    """(feasible, b_max, latency, x) of one strategy of one group of prob's cluster (variant:
    prob's by default)."""
    a = _Args(prob)
    v = int(getattr(prob, "variant", 0)) if variant is None else int(variant)
    mem = np.ascontiguousarray(np.asarray(members, np.int32))
    bmax = C.c_int32()
    lat = C.c_double()
    x = C.c_double()
    ok = lib().hxo_strategy_cost_v(C.byref(a.cluster), C.byref(a.model), C.byref(a.wl), _p(mem),
                                   C.c_int32(len(mem)), C.c_int32(tp), C.c_int32(pp), C.c_int32(role),
                                   C.c_uint32(v), C.byref(bmax), C.byref(lat), C.byref(x))
    return bool(ok), bmax.value, lat.value, x.value


def group_select(prob, members: Sequence[int], role: int):
    """(tp, pp, b_max, cap, latency) of the strategy a group keeps."""
    a = _Args(prob)
    mem = np.ascontiguousarray(np.asarray(members, np.int32))
    o = [C.c_int32() for _ in range(4)]
    lat = C.c_double()
    lib().hxo_group_select(*a.refs(), _p(mem), C.c_int32(len(mem)), C.c_int32(role),
                           *(C.byref(v) for v in o), C.byref(lat))
    return o[0].value, o[1].value, o[2].value, o[3].value, lat.value


def kv_time(prob, pm: Sequence[int], ptp: int, ppp: int, dm: Sequence[int], dtp: int, dpp: int,
            best_order: bool = False) -> float:
    """KV time of one request between two replicas (ascending stage orders, or the stage-order
    search when best_order)."""
    a = _Args(prob)
    p = np.ascontiguousarray(np.asarray(pm, np.int32))
    d = np.ascontiguousarray(np.asarray(dm, np.int32))
    fn = lib().hxo_kv_time_best if best_order else lib().hxo_kv_time
    return fn(C.byref(a.cluster), C.byref(a.model), C.byref(a.wl), _p(p), C.c_int32(ptp),
              C.c_int32(ppp), _p(d), C.c_int32(dtp), C.c_int32(dpp))


def kv_time_orders(prob, pm: Sequence[int], ptp: int, ppp: int, ord_p: Sequence[int], dm: Sequence[int], dtp: int,
                   dpp: int, ord_d: Sequence[int]) -> float:
    """KV time of one request with explicit stage orders (ord_p[a]: the prefill stage serving
    pipeline position a; ord_d likewise)."""
    a = _Args(prob)
    arr = lambda v: np.ascontiguousarray(np.asarray(v, np.int32))
    p, d, op, od = arr(pm), arr(dm), arr(ord_p), arr(ord_d)
    return lib().hxo_kv_time_orders(C.byref(a.cluster), C.byref(a.model), C.byref(a.wl), _p(p), C.c_int32(ptp),
                                    C.c_int32(ppp), _p(op), _p(d), C.c_int32(dtp), C.c_int32(dpp), _p(od))


def kv_gpu_time(prob, g: int, h: int) -> float:
    """Per-GPU flow nodes: seconds for one request's whole KV cache over the link g -> h."""
    a = _Args(prob)
    return lib().hxo_kv_gpu_time(C.byref(a.cluster), C.byref(a.model), C.byref(a.wl), C.c_int32(g),
                                 C.c_int32(h))


def quantize(x: float) -> int:
    return lib().hxo_quantize(C.c_double(x))


def maxflow_edges(nv: int, edges: List[Tuple[int, int, int]], s: int, t: int):
    """(value, per-edge flow, residual-reachable set from s) of an explicit network."""
    ne = len(edges)
    fr = np.ascontiguousarray(np.array([e[0] for e in edges] or [0], np.int32))
    to = np.ascontiguousarray(np.array([e[1] for e in edges] or [0], np.int32))
    cp = np.ascontiguousarray(np.array([e[2] for e in edges] or [0], np.int64))
    fl = np.zeros(max(ne, 1), np.int64)
    reach = np.zeros(nv, np.uint8)
    v = lib().hxo_maxflow_edges(C.c_int32(nv), C.c_int32(ne), _p(fr), _p(to), _p(cp), C.c_int32(s),
                                C.c_int32(t), _p(fl), _p(reach))
    return int(v), fl[:ne].copy(), reach.astype(bool)


# ------------------------------------------------------------------ refinement (Sec. 3.4)

def edge_classes(f) -> Dict[str, np.ndarray]:
    """Bottleneck (bit 0) / underutilized (bit 1) classes of every edge of every network.

    node_cls [max_p + max_d][N]: node edges in bits 0-1, coordinator edges in bits 2-3;
    kv_cls [max_pd][N]: KV edges.  Rows past a network's counts stay 0.
    """
    mp, md, mpd = f["dims"]
    N = f["n_p"].shape[0]
    node = np.zeros((mp + md, N), np.uint8)
    kv = np.zeros((mpd, N), np.uint8)
    lib().hxo_edge_classes(C.c_int32(N), C.c_int32(mp), C.c_int32(md), C.c_int32(mpd),
                           *(_p(f[k]) for k in ("n_p", "n_d", "src_cap", "p_cap", "kv_cap", "d_cap",
                                                "sink_cap")),
                           _p(node), _p(kv))
    return dict(node_cls=node, kv_cls=kv)


def guided_moves(n_gpus: int, max_groups: int, granularity: int, p_assign: np.ndarray, p_role: np.ndarray,
                 f, cls: Dict[str, np.ndarray], rnd: np.ndarray) -> Dict[str, np.ndarray]:
    """Children of the parent placements (columns of p_assign / p_role, scored into network f
    with edge classes cls): child c descends from parent c mod M; one guided move each."""
    M = p_assign.shape[1]
    mp = f["dims"][0]
    rnd = np.ascontiguousarray(rnd, np.uint64)
    Nc = rnd.shape[0]
    out = dict(assign=np.zeros((n_gpus, Nc), np.uint8), role=np.zeros((max_groups, Nc), np.uint8),
               move=np.zeros(Nc, np.int32))
    lib().hxo_guided_moves(C.c_int32(n_gpus), C.c_int32(max_groups), C.c_int32(granularity), C.c_int32(M),
                           _p(np.ascontiguousarray(p_assign, np.uint8)), _p(np.ascontiguousarray(p_role, np.uint8)),
                           C.c_int32(mp), _p(f["n_p"]), _p(f["n_d"]), _p(f["p_slot"]), _p(f["d_slot"]),
                           _p(cls["node_cls"]), _p(cls["kv_cls"]), C.c_int32(Nc), _p(rnd),
                           _p(out["assign"]), _p(out["role"]), _p(out["move"]))
    return out


# ------------------------------------------------------------------ graph partition (Sec. 3.2)

def spectral_order(prob, iters: int = 1000) -> Tuple[np.ndarray, np.ndarray]:
    """(order, fiedler): GPUs sorted by the power-iteration Fiedler direction, and that vector."""
    a = _Args(prob)
    G = prob.n_gpus
    order = np.zeros(G, np.int32)
    x = np.zeros(G, np.float64)
    lib().hxo_spectral_order(C.byref(a.cluster), C.c_int32(iters), _p(order), _p(x))
    return order, x


def partition_groups(prob) -> int:
    a = _Args(prob)
    lib().hxo_partition_groups.restype = C.c_int32
    return int(lib().hxo_partition_groups(C.byref(a.cluster), C.byref(a.model), C.byref(a.wl)))


def kl_refine(prob, grp: np.ndarray) -> Tuple[np.ndarray, int]:
    """Kernighan-Lin refinement of one grouping of prob's GPUs (group ids < 256): (the refined
    grouping, the number of passes that lowered the cut)."""
    a = _Args(prob)
    g = np.ascontiguousarray(np.asarray(grp, np.int32).copy())
    passes = lib().hxo_kl_refine(C.byref(a.cluster), _p(g))
    return g, int(passes)


def partition_candidates(prob, order: np.ndarray, rnd: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Candidates of the first phase (initial partition, Kernighan-Lin, coarsen and max-cut split,
    projection), one per draw: assign [G][N], role [max_groups][N]."""
    a = _Args(prob)
    rnd = np.ascontiguousarray(rnd, np.uint64)
    N = rnd.shape[0]
    assign = np.zeros((prob.n_gpus, N), np.uint8)
    role = np.zeros((prob.max_groups, N), np.uint8)
    lib().hxo_partition_candidates(C.byref(a.cluster), C.byref(a.model), C.byref(a.wl),
                                   _p(np.ascontiguousarray(order, np.int32)), C.c_int32(prob.max_groups),
                                   C.c_int32(N), _p(rnd), _p(assign), _p(role))
    return assign, role


def layer_split(prob, members: Sequence[int], tp: int, pp: int, variant: int) -> List[int]:
    """Layers of each stage of a (tp, pp) strategy of a group (uniform, or asymmetric with bit 2)."""
    a = _Args(prob)
    mem = np.ascontiguousarray(np.asarray(members, np.int32))
    out = np.zeros(max(pp, 1), np.int32)
    rc = lib().hxo_layer_split(C.byref(a.cluster), C.c_int32(prob.model["n_layers"]), _p(mem), C.c_int32(tp),
                               C.c_int32(pp), C.c_uint32(variant), _p(out))
    if rc != 0:
        raise ValueError("pp outside [1, min(32, L)]")
    return out[:pp].tolist()
