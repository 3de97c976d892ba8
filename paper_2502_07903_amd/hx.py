"""Python binding of libhx (include/hx.h): argument marshalling only.

Device memory and streams come from PyTorch; every step of the scoring path runs in the
HIP kernels of libhx.so.  The functions keep the C names:

    cost_eval, build_flownet, maxflow_batch, best_candidate, validate

the refinement calls of Sec. 3.4

    edge_classes, guided_moves, gather_candidates

and `DeviceProblem` uploads a seeded `inputs.Problem` once so that repeated calls read
device-resident inputs.  There is no fallback: without the built library or a GPU every
call raises.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import os
from typing import Dict, Optional, Tuple

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libhx.so")

HX_OK, HX_EINVAL, HX_ETOOBIG, HX_EHIP, HX_ENOCONV = 0, -1, -2, -3, -4
CAP_MAX = 16777215


class HxError(RuntimeError):
    def __init__(self, code: int, where: str, detail: str = ""):
        self.code = code
        super().__init__(f"{where}: {strerror(code)} ({code}){': ' + detail if detail else ''}")


class hx_cluster(C.Structure):
    _fields_ = [("n_gpus", C.c_int32), ("n_types", C.c_int32), ("gpu_type", C.c_void_p),
                ("type_flops", C.c_void_p), ("type_hbm_bw", C.c_void_p), ("type_mem", C.c_void_p),
                ("beta", C.c_void_p), ("alpha", C.c_void_p), ("coord_bw", C.c_double),
                ("req_bytes", C.c_double)]


class hx_model(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("hidden", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("bytes_per_elem", C.c_int32)]


HX_MAX_CLASSES = 4


class hx_workload(C.Structure):
    _fields_ = [("s_in", C.c_double), ("s_out", C.c_double), ("n_classes", C.c_int32),
                ("cls_in", C.c_double * HX_MAX_CLASSES), ("cls_out", C.c_double * HX_MAX_CLASSES),
                ("cls_w", C.c_double * HX_MAX_CLASSES)]


def make_workload(prob) -> hx_workload:
    """The task (s_in, s_out) and, when prob has them, its request classes (rows of
    (s_in, s_out, weight))."""
    w = hx_workload(float(prob.s_in), float(prob.s_out), 0)
    cls = getattr(prob, "classes", None)
    if cls is not None:
        cls = np.asarray(cls, np.float64)
        if cls.ndim != 2 or cls.shape[1] != 3 or len(cls) > HX_MAX_CLASSES:
            raise ValueError("classes: at most four rows of (s_in, s_out, weight)")
        w.n_classes = len(cls)
        for k, (i, o, wt) in enumerate(cls):
            w.cls_in[k], w.cls_out[k], w.cls_w[k] = float(i), float(o), float(wt)
    return w


# hx_space.variant bit (include/hx.h HX_HINT_SHARED_GROUPS): a hint, not a model variant.
HINT_SHARED_GROUPS = 1 << 16


class hx_space(C.Structure):
    _fields_ = [("tp_mask", C.c_uint32), ("pp_mask", C.c_uint32), ("granularity", C.c_int32),
                ("variant", C.c_uint32)]


class hx_candidates(C.Structure):
    _fields_ = [("n_cand", C.c_int32), ("max_groups", C.c_int32), ("assign", C.c_void_p), ("role", C.c_void_p)]


class hx_cost_out(C.Structure):
    _fields_ = [("tp", C.c_void_p), ("pp", C.c_void_p), ("bmax", C.c_void_p), ("cap", C.c_void_p),
                ("lat", C.c_void_p), ("members", C.c_void_p)]


class hx_flownet(C.Structure):
    _fields_ = [("n_cand", C.c_int32), ("max_p", C.c_int32), ("max_d", C.c_int32), ("max_pd", C.c_int32),
                ("n_p", C.c_void_p), ("n_d", C.c_void_p), ("p_slot", C.c_void_p), ("d_slot", C.c_void_p),
                ("src_cap", C.c_void_p), ("p_cap", C.c_void_p), ("kv_cap", C.c_void_p), ("d_cap", C.c_void_p),
                ("sink_cap", C.c_void_p)]


EXPORTS = ("hx_validate", "hx_cost_eval", "hx_cost_eval_static", "hx_static_scratch_bytes", "hx_cost_workspace_bytes", "hx_member_words", "hx_build_flownet",
           "hx_maxflow_batch", "hx_maxflow_stats", "hx_best_candidate", "hx_score_batch", "hx_score_workspace_bytes", "hx_edge_classes", "hx_guided_moves",
           "hx_gather_candidates",
           "hx_partition_workspace_bytes", "hx_spectral_order", "hx_partition_candidates",
           "hx_profile", "hx_profile_read", "hx_kernel_name", "hx_strerror", "hx_last_error",
           "hx_abi_version")
HX_KERNELS = 14

_lib = None


def lib() -> C.CDLL:
    """The loaded libhx.so.  Raises if it has not been built (python -m paper_2502_07903_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libhx.so not built at {LIB_PATH}; run `python -m paper_2502_07903_amd.build`")
        L = C.CDLL(LIB_PATH)
        P = C.POINTER
        L.hx_validate.argtypes = [P(hx_cluster), hx_model, hx_workload, hx_space, P(hx_candidates),
                                  P(hx_cost_out), P(hx_flownet)]
        L.hx_cost_eval.argtypes = [P(hx_cluster), hx_model, hx_workload, hx_space, P(hx_candidates),
                                   P(hx_cost_out), C.c_void_p, C.c_size_t, C.c_void_p]
        L.hx_cost_eval_static.argtypes = [P(hx_cluster), hx_model, hx_workload, hx_space, P(hx_candidates),
                                          P(hx_cost_out), C.c_void_p]
        L.hx_static_scratch_bytes.restype = C.c_size_t
        L.hx_cost_workspace_bytes.argtypes = [C.c_int32, C.c_int32, C.c_int32]
        L.hx_cost_workspace_bytes.restype = C.c_size_t
        L.hx_member_words.argtypes = [C.c_int32]
        L.hx_member_words.restype = C.c_int
        L.hx_build_flownet.argtypes = [P(hx_cluster), hx_model, hx_workload, hx_space, P(hx_candidates),
                                       P(hx_cost_out), P(hx_flownet), C.c_void_p]
        L.hx_maxflow_batch.argtypes = [P(hx_flownet), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.hx_maxflow_stats.argtypes = [P(hx_flownet), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.hx_best_candidate.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p]
        L.hx_score_workspace_bytes.argtypes = [C.c_int32, C.c_int32, C.c_int32]
        L.hx_score_workspace_bytes.restype = C.c_size_t
        L.hx_score_batch.argtypes = [P(hx_cluster), hx_model, hx_workload, hx_space, P(hx_candidates),
                                     P(hx_cost_out), P(hx_flownet), C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t,
                                     C.c_void_p]
        L.hx_edge_classes.argtypes = [P(hx_flownet), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.hx_guided_moves.argtypes = [C.c_int32, C.c_int32, P(hx_candidates), P(hx_flownet), C.c_void_p,
                                      C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.hx_gather_candidates.argtypes = [C.c_int32, P(hx_candidates), C.c_void_p, C.c_int32, C.c_void_p,
                                           C.c_void_p, C.c_void_p]
        L.hx_partition_workspace_bytes.argtypes = [C.c_int32]
        L.hx_partition_workspace_bytes.restype = C.c_size_t
        L.hx_spectral_order.argtypes = [P(hx_cluster), C.c_int32, C.c_void_p, C.c_size_t, C.c_void_p, C.c_void_p,
                                        C.c_void_p]
        L.hx_partition_candidates.argtypes = [P(hx_cluster), hx_model, hx_workload, C.c_int32, C.c_void_p, C.c_size_t,
                                              C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.hx_profile.argtypes = [C.c_int32]
        L.hx_profile.restype = C.c_int
        L.hx_profile_read.argtypes = [C.c_void_p, C.c_void_p, C.c_int32]
        L.hx_profile_read.restype = C.c_int
        L.hx_kernel_name.argtypes = [C.c_int32]
        L.hx_kernel_name.restype = C.c_char_p
        L.hx_strerror.restype = C.c_char_p
        L.hx_strerror.argtypes = [C.c_int]
        L.hx_last_error.restype = C.c_char_p
        L.hx_abi_version.restype = C.c_int
        _lib = L
    return _lib


def profile(enable: bool) -> None:
    """Diagnostic per-kernel timing: HIP events around every later libhx kernel launch."""
    _check(lib().hx_profile(1 if enable else 0), "hx_profile")


def profile_read() -> Dict[str, Tuple[float, int]]:
    """{kernel name: (total ms, launches)} since the last profile() call; clears the records."""
    ms = (C.c_double * HX_KERNELS)()
    n = (C.c_int32 * HX_KERNELS)()
    rc = lib().hx_profile_read(C.cast(ms, C.c_void_p), C.cast(n, C.c_void_p), HX_KERNELS)
    if rc < 0:
        _check(rc, "hx_profile_read")
    return {lib().hx_kernel_name(k).decode(): (float(ms[k]), int(n[k])) for k in range(HX_KERNELS)}


def strerror(code: int) -> str:
    try:
        return lib().hx_strerror(code).decode()
    except RuntimeError:
        return f"error {code}"


def _check(rc: int, where: str) -> None:
    if rc != HX_OK:
        detail = lib().hx_last_error().decode() if rc == HX_EHIP else ""
        raise HxError(rc, where, detail)


def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("libhx needs a ROCm GPU; torch.cuda.is_available() is False")
    return torch


def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


def _stream(stream=None) -> C.c_void_p:
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(int(s.cuda_stream))


def flownet_dims(max_groups: int, n_gpus: int, granularity: int) -> Tuple[int, int, int]:
    """(max_p, max_d, max_pd) large enough for any split of the replicas (or GPUs) into sides."""
    b = max_groups if granularity == 0 else n_gpus
    return b, b, (b // 2) * ((b + 1) // 2)


@dataclasses.dataclass
class DeviceProblem:
    """A scoring problem resident in device memory, with the C structs pointing at it."""
    tensors: Dict[str, object]
    cluster: hx_cluster
    model: hx_model
    workload: hx_workload
    space: hx_space
    cand: hx_candidates
    n_gpus: int
    max_groups: int

    @property
    def n_cand(self) -> int:
        return int(self.cand.n_cand)

    @classmethod
    def upload(cls, prob, device: str = "cuda") -> "DeviceProblem":
        torch = _torch()
        cl = prob.cluster
        gt = np.asarray(cl.gpu_type, np.int32)
        if gt.min(initial=0) < 0 or gt.max(initial=0) >= cl.n_types:
            raise ValueError("gpu_type outside [0, n_types)")
        dev = lambda a, dt: torch.as_tensor(np.ascontiguousarray(a), dtype=dt).to(device)
        t = dict(gpu_type=dev(gt, torch.int32),
                 type_flops=dev(cl.type_flops, torch.float64), type_hbm_bw=dev(cl.type_hbm_bw, torch.float64),
                 type_mem=dev(cl.type_mem, torch.float64), beta=dev(cl.beta, torch.float64),
                 alpha=dev(cl.alpha, torch.float64),
                 assign=dev(prob.assign, torch.uint8), role=dev(prob.role, torch.uint8))
        return cls.from_tensors(t, prob)

    @classmethod
    def from_tensors(cls, t, prob) -> "DeviceProblem":
        cl = prob.cluster
        m = prob.model
        c = hx_cluster(cl.n_gpus, cl.n_types, _ptr(t["gpu_type"]), _ptr(t["type_flops"]), _ptr(t["type_hbm_bw"]),
                       _ptr(t["type_mem"]), _ptr(t["beta"]), _ptr(t["alpha"]), float(cl.coord_bw),
                       float(cl.req_bytes))
        md = hx_model(m["n_layers"], m["hidden"], m["n_heads"], m["n_kv_heads"], m["bytes_per_elem"])
        n_cand = int(t["assign"].shape[1])
        k = hx_candidates(n_cand, int(prob.max_groups), _ptr(t["assign"]), _ptr(t["role"]))
        return cls(t, c, md, make_workload(prob),
                   hx_space(int(prob.tp_mask), int(prob.pp_mask), int(prob.granularity),
                            int(getattr(prob, "variant", 0))), k, cl.n_gpus,
                   int(prob.max_groups))

    def with_hint(self, shared_groups: bool = True) -> "DeviceProblem":
        """The same problem with the HX_HINT_SHARED_GROUPS hint set (or cleared): the batch's
        candidates share most of their groups with candidate 0, which is costed first.  The
        outputs are the same either way."""
        v = self.space.variant | HINT_SHARED_GROUPS if shared_groups else self.space.variant & ~HINT_SHARED_GROUPS
        sp = hx_space(self.space.tp_mask, self.space.pp_mask, self.space.granularity, v)
        return dataclasses.replace(self, space=sp)

    def with_candidates(self, assign, role) -> "DeviceProblem":
        """The same cluster/model/workload with another candidate batch (device uint8 tensors)."""
        t = dict(self.tensors, assign=assign, role=role)
        k = hx_candidates(int(assign.shape[1]), self.max_groups, _ptr(assign), _ptr(role))
        return dataclasses.replace(self, tensors=t, cand=k)


@dataclasses.dataclass
class CostBuffers:
    tp: object
    pp: object
    bmax: object
    cap: object
    lat: object
    members: object     # int64 [Kmax * W, N]: the group member bitmasks (uint64 bit patterns)
    workspace: object   # uint8 scratch of hx_score_workspace_bytes (>= hx_cost_workspace_bytes)

    @classmethod
    def empty(cls, max_groups: int, n_cand: int, n_gpus: int, device: str = "cuda") -> "CostBuffers":
        torch = _torch()
        z = lambda dt: torch.empty((max_groups, n_cand), dtype=dt, device=device)
        words = lib().hx_member_words(n_gpus)
        wsb = int(lib().hx_score_workspace_bytes(n_gpus, max_groups, n_cand))
        if words <= 0 or wsb <= 0:
            raise ValueError("invalid sizes for the cost-model buffers")
        return cls(z(torch.uint8), z(torch.uint8), z(torch.int32), z(torch.int32), z(torch.float64),
                   torch.empty((max_groups * words, n_cand), dtype=torch.int64, device=device),
                   torch.empty(wsb, dtype=torch.uint8, device=device))

    def struct(self) -> hx_cost_out:
        return hx_cost_out(_ptr(self.tp), _ptr(self.pp), _ptr(self.bmax), _ptr(self.cap), _ptr(self.lat),
                           _ptr(self.members))


@dataclasses.dataclass
class FlowNetBuffers:
    dims: Tuple[int, int, int]
    n_p: object
    n_d: object
    p_slot: object
    d_slot: object
    src_cap: object
    p_cap: object
    kv_cap: object
    d_cap: object
    sink_cap: object

    @classmethod
    def empty(cls, dims: Tuple[int, int, int], n_cand: int, device: str = "cuda", fill: Optional[int] = 0):
        torch = _torch()
        mp, md, mpd = dims

        def z(rows):
            shape = (rows, n_cand) if rows is not None else (n_cand,)
            if fill is None:
                return torch.empty(shape, dtype=torch.int32, device=device)
            return torch.full(shape, fill, dtype=torch.int32, device=device)
        return cls(dims, z(None), z(None), z(mp), z(md), z(mp), z(mp), z(mpd), z(md), z(md))

    @classmethod
    def from_host(cls, fn: Dict[str, np.ndarray], device: str = "cuda") -> "FlowNetBuffers":
        """Device copy of a host network (same layout), e.g. to run max-flow on given capacities."""
        torch = _torch()
        d = lambda k: torch.as_tensor(np.ascontiguousarray(fn[k], np.int32)).to(device)
        return cls(tuple(fn["dims"]), d("n_p"), d("n_d"), d("p_slot"), d("d_slot"), d("src_cap"), d("p_cap"),
                   d("kv_cap"), d("d_cap"), d("sink_cap"))

    def struct(self) -> hx_flownet:
        mp, md, mpd = self.dims
        return hx_flownet(int(self.n_p.shape[0]), mp, md, mpd, _ptr(self.n_p), _ptr(self.n_d), _ptr(self.p_slot),
                          _ptr(self.d_slot), _ptr(self.src_cap), _ptr(self.p_cap), _ptr(self.kv_cap),
                          _ptr(self.d_cap), _ptr(self.sink_cap))

    def host(self) -> Dict[str, np.ndarray]:
        out = {k: getattr(self, k).cpu().numpy() for k in ("n_p", "n_d", "p_slot", "d_slot", "src_cap", "p_cap",
                                                           "kv_cap", "d_cap", "sink_cap")}
        out["dims"] = self.dims
        return out


# ------------------------------------------------------------------ the four calls

def validate(dp: DeviceProblem, cost: Optional[CostBuffers] = None, net: Optional[FlowNetBuffers] = None) -> int:
    cs = cost.struct() if cost is not None else None
    ns = net.struct() if net is not None else None
    return lib().hx_validate(C.byref(dp.cluster), dp.model, dp.workload, dp.space, C.byref(dp.cand),
                             C.byref(cs) if cs is not None else None, C.byref(ns) if ns is not None else None)


def cost_eval(dp: DeviceProblem, out: CostBuffers, stream=None) -> CostBuffers:
    o = out.struct()
    _check(lib().hx_cost_eval(C.byref(dp.cluster), dp.model, dp.workload, dp.space, C.byref(dp.cand), C.byref(o),
                              _ptr(out.workspace), C.c_size_t(int(out.workspace.numel())), _stream(stream)),
           "hx_cost_eval")
    return out


def cost_eval_static(dp: DeviceProblem, out: CostBuffers, stream=None) -> CostBuffers:
    """hx_cost_eval_static: the cost model with libhx's static scratch (out.workspace unused)."""
    o = out.struct()
    _check(lib().hx_cost_eval_static(C.byref(dp.cluster), dp.model, dp.workload, dp.space, C.byref(dp.cand),
                                     C.byref(o), _stream(stream)), "hx_cost_eval_static")
    return out


def build_flownet(dp: DeviceProblem, cost: CostBuffers, net: FlowNetBuffers, stream=None) -> FlowNetBuffers:
    o = cost.struct()
    f = net.struct()
    _check(lib().hx_build_flownet(C.byref(dp.cluster), dp.model, dp.workload, dp.space, C.byref(dp.cand),
                                  C.byref(o), C.byref(f), _stream(stream)), "hx_build_flownet")
    return net


def maxflow_batch(net: FlowNetBuffers, flow_value, kv_flow=None, cut=None, stream=None):
    f = net.struct()
    _check(lib().hx_maxflow_batch(C.byref(f), _ptr(flow_value), _ptr(kv_flow), _ptr(cut), _stream(stream)),
           "hx_maxflow_batch")
    return flow_value


MF_STATS = ("no_flow", "star", "dominant", "min_cut", "push_relabel", "prepass", "pushes", "relabels",
            "global_relabels", "rounds")


def maxflow_stats(net: FlowNetBuffers, flow_value, kv_flow=None, cut=None, stream=None) -> Dict[str, int]:
    """hx_maxflow_batch plus its diagnostic counters (synchronises the stream to read them)."""
    torch = _torch()
    f = net.struct()
    st = torch.zeros(len(MF_STATS), dtype=torch.int64, device=flow_value.device)
    _check(lib().hx_maxflow_stats(C.byref(f), _ptr(flow_value), _ptr(kv_flow), _ptr(cut), _ptr(st), _stream(stream)),
           "hx_maxflow_stats")
    (torch.cuda.current_stream() if stream is None else stream).synchronize()
    return dict(zip(MF_STATS, (int(v) for v in st.cpu().tolist())))


def best_candidate(flow_value, best, n_cand: Optional[int] = None, stream=None):
    n = int(flow_value.shape[0]) if n_cand is None else n_cand
    _check(lib().hx_best_candidate(_ptr(flow_value), C.c_int32(n), _ptr(best), _stream(stream)),
           "hx_best_candidate")
    return best


# ------------------------------------------------------------------ whole path

@dataclasses.dataclass
class Workspace:
    """Preallocated outputs of one pass over a batch of n_cand candidates."""
    cost: CostBuffers
    net: FlowNetBuffers
    flow_value: object
    kv_flow: Optional[object]
    cut: Optional[object]
    best: object

    @classmethod
    def for_problem(cls, dp: DeviceProblem, flows: bool = False, device: str = "cuda") -> "Workspace":
        torch = _torch()
        N = dp.n_cand
        dims = flownet_dims(dp.max_groups, dp.n_gpus, dp.space.granularity)
        kv = torch.zeros((dims[2], N), dtype=torch.int32, device=device) if flows else None
        cut = torch.zeros((dims[0] + dims[1], N), dtype=torch.uint8, device=device) if flows else None
        return cls(CostBuffers.empty(dp.max_groups, N, dp.n_gpus, device), FlowNetBuffers.empty(dims, N, device),
                   torch.empty(N, dtype=torch.int32, device=device), kv, cut,
                   torch.empty(2, dtype=torch.int32, device=device))


def score(dp: DeviceProblem, ws: Workspace, stream=None) -> None:
    """Enqueues the whole hot path: cost model -> flow network -> max-flow -> argmax."""
    cost_eval(dp, ws.cost, stream)
    build_flownet(dp, ws.cost, ws.net, stream)
    maxflow_batch(ws.net, ws.flow_value, ws.kv_flow, ws.cut, stream)
    best_candidate(ws.flow_value, ws.best, dp.n_cand, stream)


def score_batch(dp: DeviceProblem, ws: Workspace, stream=None) -> None:
    """Enqueues the whole hot path in one call, value only (hx_score_batch): cost outputs, node
    rows, flow values and the best; kv_cap rows only where a network needs them."""
    o = ws.cost.struct()
    f = ws.net.struct()
    _check(lib().hx_score_batch(C.byref(dp.cluster), dp.model, dp.workload, dp.space, C.byref(dp.cand), C.byref(o),
                                C.byref(f), _ptr(ws.flow_value), _ptr(ws.best), _ptr(ws.cost.workspace),
                                C.c_size_t(int(ws.cost.workspace.numel())), _stream(stream)), "hx_score_batch")


# ------------------------------------------------------------------ refinement (Sec. 3.4)

def edge_classes(net: FlowNetBuffers, flow_value, kv_flow, node_cls, kv_cls, stream=None):
    """Bottleneck / underutilized classes of every network edge (hx_edge_classes)."""
    f = net.struct()
    _check(lib().hx_edge_classes(C.byref(f), _ptr(flow_value), _ptr(kv_flow), _ptr(node_cls), _ptr(kv_cls),
                                 _stream(stream)), "hx_edge_classes")
    return node_cls, kv_cls


def guided_moves(parents: DeviceProblem, parent_net: FlowNetBuffers, node_cls, rnd, child_assign, child_role, move,
                 stream=None):
    """Children of the parent batch, one guided move each (hx_guided_moves)."""
    f = parent_net.struct()
    _check(lib().hx_guided_moves(C.c_int32(parents.n_gpus), C.c_int32(int(parents.space.granularity)),
                                 C.byref(parents.cand), C.byref(f), _ptr(node_cls), C.c_int32(int(rnd.shape[0])),
                                 _ptr(rnd), _ptr(child_assign), _ptr(child_role), _ptr(move), _stream(stream)),
           "hx_guided_moves")
    return child_assign, child_role, move


def gather_candidates(src: DeviceProblem, index, dst_assign, dst_role, stream=None):
    """dst column m = src column index[m] (hx_gather_candidates)."""
    _check(lib().hx_gather_candidates(C.c_int32(src.n_gpus), C.byref(src.cand), _ptr(index),
                                      C.c_int32(int(index.shape[0])), _ptr(dst_assign), _ptr(dst_role),
                                      _stream(stream)), "hx_gather_candidates")
    return dst_assign, dst_role


@dataclasses.dataclass
class Refiner:
    """Max-flow guided refinement on the device (Sec. 3.4): one parent placement and a batch of
    n_child children per round.  A round enqueues, with no host synchronisation:
      1. the parent scored with a flow assignment (cost, network, max-flow with kv_flow) and
         its edge classes;
      2. the children (child 0 = the parent) by guided moves;
      3. the children scored (value only) and the best chosen (lowest index on ties);
      4. the best child gathered into the parent for the next round.
    best_value after a round is the parent's new score; a round whose best index is 0 found
    no improvement."""
    parent: DeviceProblem
    parent_ws: Workspace
    node_cls: object
    kv_cls: object
    children: DeviceProblem
    child_ws: Workspace
    move: object

    @classmethod
    def create(cls, dp: DeviceProblem, parent_col: int, n_child: int, device: str = "cuda",
               shared_groups_hint: bool = True) -> "Refiner":
        torch = _torch()
        pa = dp.tensors["assign"][:, parent_col:parent_col + 1].clone()
        pr = dp.tensors["role"][:, parent_col:parent_col + 1].clone()
        parent = dp.with_candidates(pa, pr)
        pws = Workspace.for_problem(parent, flows=True, device=device)
        mp, md, mpd = pws.net.dims
        ca = torch.empty((dp.n_gpus, n_child), dtype=torch.uint8, device=device)
        cr = torch.empty((dp.max_groups, n_child), dtype=torch.uint8, device=device)
        # child 0 is the parent and every other child one move away from it
        children = dp.with_candidates(ca, cr).with_hint(shared_groups_hint)
        return cls(parent, pws, torch.zeros((mp + md, 1), dtype=torch.uint8, device=device),
                   torch.zeros((mpd, 1), dtype=torch.uint8, device=device), children,
                   Workspace.for_problem(children, device=device),
                   torch.empty(n_child, dtype=torch.int32, device=device))

    def round(self, rnd, stream=None) -> None:
        p, pw, ch, cw = self.parent, self.parent_ws, self.children, self.child_ws
        score(p, pw, stream)
        edge_classes(pw.net, pw.flow_value, pw.kv_flow, self.node_cls, self.kv_cls, stream)
        guided_moves(p, pw.net, self.node_cls, rnd, ch.tensors["assign"], ch.tensors["role"], self.move, stream)
        score_batch(ch, cw, stream)
        gather_candidates(ch, cw.best[:1], p.tensors["assign"], p.tensors["role"], stream)


# ------------------------------------------------------------------ graph partition (Sec. 3.2)

def partition_workspace(dp: DeviceProblem, device: str = "cuda"):
    torch = _torch()
    nb = int(lib().hx_partition_workspace_bytes(dp.n_gpus))
    if nb <= 0:
        raise ValueError("the partition needs 2..255 GPUs")
    return torch.empty(nb, dtype=torch.uint8, device=device)


def spectral_order(dp: DeviceProblem, workspace, order, fiedler=None, iters: int = 1000, stream=None):
    """GPUs sorted along the Fiedler direction of the device graph (hx_spectral_order)."""
    _check(lib().hx_spectral_order(C.byref(dp.cluster), C.c_int32(iters), _ptr(workspace),
                                   C.c_size_t(int(workspace.numel())), _ptr(order), _ptr(fiedler), _stream(stream)),
           "hx_spectral_order")
    return order


def partition_candidates(dp: DeviceProblem, workspace, order, rnd, assign, role, stream=None):
    """One first-phase candidate per draw (hx_partition_candidates) into assign [G][N] / role [Kmax][N]."""
    _check(lib().hx_partition_candidates(C.byref(dp.cluster), dp.model, dp.workload, C.c_int32(dp.max_groups),
                                         _ptr(workspace), C.c_size_t(int(workspace.numel())), _ptr(order),
                                         C.c_int32(int(rnd.shape[0])), _ptr(rnd), _ptr(assign), _ptr(role),
                                         _stream(stream)), "hx_partition_candidates")
    return assign, role
