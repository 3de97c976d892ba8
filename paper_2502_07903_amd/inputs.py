"""Seeded synthetic inputs for batched placement scoring.

This module only *draws* problem instances: heterogeneous clusters (GPU types,
bandwidth and latency matrices), a model shape, request-length means and
candidate placements (a group id per GPU and a role per group).  It holds none
of the scoring arithmetic: no cost model, no flow network, no max-flow.  Both
the HIP path and the CPU oracle read the arrays it returns, so it is the only
code they share.

The problem statement it follows is the paper's (Sec. 3.1 and 3.2): a device
graph whose nodes are GPUs (with compute, memory bandwidth and memory limit,
Table 1 legend) and whose edges carry the pairwise bandwidth beta and latency
alpha; a placement partitions the GPUs into groups, each a prefill or a decode
replica.  The paper's own clusters, measured bandwidth matrices and Azure
request traces are not available, so the five workloads below are synthetic
stand-ins with the shapes and value ranges of the paper's experiments
(Sec. 5.1: H100/A100/L40/A6000-class GPUs, OPT-30B and Llama-2-70B, prompt and
output lengths from a few tens to a few thousand tokens).

Array layouts (all candidate-fastest, "structure of arrays"):
  assign  uint8 [n_gpus][n_cand]      group id of each GPU, 0xFF = GPU unused
  role    uint8 [max_groups][n_cand]  0 = prefill, 1 = decode, 0xFF = no group
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

UNUSED = 0xFF
PREFILL = 0
DECODE = 1
GPUS_PER_NODE = 4

# GPU types in SI units: (tensor FLOP/s, HBM bytes/s, memory bytes).
# A, B, C are the three types the workload definitions name; D, E, F are
# H100-, L40- and A6000-class datasheet values, the paper's mix (Sec. 5.1).
GPU_TYPES: Dict[str, Tuple[float, float, float]] = {
    "A": (312e12, 2.0e12, 80e9),
    "B": (125e12, 0.9e12, 24e9),
    "C": (65e12, 0.6e12, 16e9),
    "D": (989e12, 3.35e12, 80e9),
    "E": (181e12, 0.864e12, 48e9),
    "F": (155e12, 0.768e12, 48e9),
}

# Model shapes: layers L, hidden size H, attention heads, KV heads, bytes per element.
OPT_30B = dict(n_layers=48, hidden=7168, n_heads=56, n_kv_heads=56, bytes_per_elem=2)
LLAMA2_70B = dict(n_layers=80, hidden=8192, n_heads=64, n_kv_heads=8, bytes_per_elem=2)

BETA_INTRA = 300e9     # bytes/s between GPUs of one node
ALPHA_INTRA = 1e-5     # s
ALPHA_INTER = 5e-5     # s
N_REQUESTS = 4096      # requests drawn per workload; their mean lengths are the task t


def _mask(degrees) -> int:
    m = 0
    for d in degrees:
        m |= 1 << (d - 1)
    return m


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic scoring workload."""
    cfg: int
    name: str
    n_gpus: int
    types: str                 # type letter of node i is types[i % len(types)]
    inter_bw: Tuple[str, float, float]   # ("fixed", v, v) | ("pair_stream", lo, hi) | ("pair_seed", lo, hi) in GB/s
    model: Dict[str, int]
    lengths: str               # "fixed" | "uniform" | "lognormal"
    n_cand: int
    k_range: Tuple[int, int]
    tp: Tuple[int, ...]
    pp: Tuple[int, ...]
    max_groups: int
    granularity: int = 0       # 0: one flow node per replica, 1: one per GPU
    rounds: int = 1            # refinement rounds (each a fresh batch of n_cand)

    @property
    def tp_mask(self) -> int:
        return _mask(self.tp)

    @property
    def pp_mask(self) -> int:
        return _mask(self.pp)


WORKLOADS: Dict[int, Workload] = {
    1: Workload(1, "8 GPUs/2 nodes/2 types, OPT-30B, 512/128 tokens, 256 candidates",
                8, "AB", ("fixed", 12.5, 12.5), OPT_30B, "fixed", 256, (2, 4),
                (1, 2, 4), (1, 2), 4),
    2: Workload(2, "16 GPUs/4 nodes/3 types, OPT-30B, uniform lengths, 4,096 candidates",
                16, "ABC", ("pair_stream", 5.0, 25.0), OPT_30B, "uniform", 4096, (2, 8),
                (1, 2, 4, 8), (1, 2, 4), 8),
    3: Workload(3, "32 GPUs/8 nodes/4 types, Llama-2-70B, lognormal lengths, 65,536 candidates",
                32, "ABCD", ("pair_stream", 5.0, 25.0), LLAMA2_70B, "lognormal", 65536, (2, 16),
                (1, 2, 4, 8), tuple(range(1, 9)), 16),
    4: Workload(4, "64 GPUs/16 nodes/5 types, Llama-2-70B, two-tier fabric, 262,144 candidates",
                64, "ABCDE", ("pair_seed", 3.0, 25.0), LLAMA2_70B, "lognormal", 262144, (2, 32),
                (1, 2, 4, 8), tuple(range(1, 9)), 32),
    5: Workload(5, "128 GPUs/32 nodes/6 types, Llama-2-70B, 16 refinement rounds x 131,072 "
                   "perturbations, per-GPU flow nodes",
                128, "ABCDEF", ("pair_seed", 3.0, 25.0), LLAMA2_70B, "lognormal", 131072, (32, 32),
                (1, 2, 4, 8), tuple(range(1, 9)), 32, granularity=1, rounds=16),
}


@dataclasses.dataclass
class Cluster:
    gpu_type: np.ndarray      # int32 [G]
    type_flops: np.ndarray    # float64 [T]  c_d
    type_hbm_bw: np.ndarray   # float64 [T]  memory bandwidth (decode weight scan)
    type_mem: np.ndarray      # float64 [T]  memory limit in bytes
    beta: np.ndarray          # float64 [G*G] bytes/s, row = sending GPU; diagonal unused
    alpha: np.ndarray         # float64 [G*G] seconds; diagonal unused
    coord_bw: float = 0.0     # coordinator link bandwidth (0: source/sink edges unbounded)
    req_bytes: float = 0.0    # bytes per request on coordinator links

    @property
    def n_gpus(self) -> int:
        return int(self.gpu_type.shape[0])

    @property
    def n_types(self) -> int:
        return int(self.type_flops.shape[0])


@dataclasses.dataclass
class Problem:
    """Everything one scoring call reads."""
    cluster: Cluster
    model: Dict[str, int]
    s_in: float
    s_out: float
    tp_mask: int
    pp_mask: int
    granularity: int
    max_groups: int
    assign: np.ndarray        # uint8 [G][N]
    role: np.ndarray          # uint8 [max_groups][N]
    variant: int = 0          # cost-model variant bits (bit 0: pipelined decode capacity)
    classes: Optional[np.ndarray] = None   # float64 [n][3]: request classes (s_in, s_out, weight)

    @property
    def n_cand(self) -> int:
        return int(self.assign.shape[1])

    @property
    def n_gpus(self) -> int:
        return int(self.assign.shape[0])

    def subset(self, idx) -> "Problem":
        """The same problem restricted to candidates idx (a slice or index array)."""
        return dataclasses.replace(self, assign=np.ascontiguousarray(self.assign[:, idx]),
                                   role=np.ascontiguousarray(self.role[:, idx]))


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([2502, 7903, *key])))


# --------------------------------------------------------------------------- clusters

def make_cluster(wl: Workload) -> Cluster:
    """Cluster of wl.n_gpus GPUs, GPUS_PER_NODE per node, node i of type types[i % T]."""
    G = wl.n_gpus
    n_nodes = G // GPUS_PER_NODE
    letters = sorted(set(wl.types), key=wl.types.index)
    tids = {c: i for i, c in enumerate(letters)}
    node_type = np.array([tids[wl.types[i % len(wl.types)]] for i in range(n_nodes)], np.int32)
    gpu_type = np.repeat(node_type, GPUS_PER_NODE).astype(np.int32)
    tab = np.array([GPU_TYPES[c] for c in letters], np.float64)

    kind, lo, hi = wl.inter_bw
    inter = np.zeros((n_nodes, n_nodes), np.float64)
    if kind == "fixed":
        inter[:] = lo * 1e9
    elif kind == "pair_stream":
        rng = _rng(wl.cfg, 0)
        for u in range(n_nodes):
            for v in range(u + 1, n_nodes):
                inter[u, v] = inter[v, u] = rng.uniform(lo, hi) * 1e9
    elif kind == "pair_seed":
        for u in range(n_nodes):
            for v in range(u + 1, n_nodes):
                inter[u, v] = inter[v, u] = _rng(wl.cfg, 0, u, v).uniform(lo, hi) * 1e9
    else:
        raise ValueError(kind)
    return cluster_from_nodes(gpu_type, tab, inter)


def cluster_from_nodes(gpu_type: np.ndarray, type_table: np.ndarray, inter_node_bw: np.ndarray,
                       beta_intra: float = BETA_INTRA, alpha_intra: float = ALPHA_INTRA,
                       alpha_inter: float = ALPHA_INTER) -> Cluster:
    """Two-tier fabric: GPUs g, h share a node iff g // GPUS_PER_NODE == h // GPUS_PER_NODE."""
    G = len(gpu_type)
    node = np.arange(G) // GPUS_PER_NODE
    same = node[:, None] == node[None, :]
    beta = np.where(same, beta_intra, inter_node_bw[node[:, None], node[None, :]])
    alpha = np.where(same, alpha_intra, alpha_inter)
    np.fill_diagonal(beta, 0.0)
    np.fill_diagonal(alpha, 0.0)
    tt = np.asarray(type_table, np.float64)
    return Cluster(np.asarray(gpu_type, np.int32), tt[:, 0].copy(), tt[:, 1].copy(), tt[:, 2].copy(),
                   np.ascontiguousarray(beta.reshape(-1)), np.ascontiguousarray(alpha.reshape(-1)))


# --------------------------------------------------------------------------- request lengths

def request_lengths(wl: Workload) -> Tuple[np.ndarray, np.ndarray]:
    """N_REQUESTS seeded (prompt, output) token counts."""
    rng = _rng(wl.cfg, 1)
    n = N_REQUESTS
    if wl.lengths == "fixed":
        return np.full(n, 512, np.int64), np.full(n, 128, np.int64)
    if wl.lengths == "uniform":
        return rng.integers(128, 2049, n).astype(np.int64), rng.integers(32, 513, n).astype(np.int64)
    if wl.lengths == "lognormal":
        s_in = np.clip(np.rint(np.exp(rng.normal(np.log(1024.0), 1.0, n))), 1, 4096)
        s_out = np.clip(np.rint(np.exp(rng.normal(np.log(256.0), 1.0, n))), 1, 2048)
        return s_in.astype(np.int64), s_out.astype(np.int64)
    raise ValueError(wl.lengths)


def mean_lengths(wl: Workload) -> Tuple[float, float]:
    """The task t's s_in and s_out: exact integer sums over the drawn requests / count."""
    a, b = request_lengths(wl)
    return float(int(a.sum())) / len(a), float(int(b.sum())) / len(b)


MAX_CLASSES = 4


def length_classes(wl: Workload, n: int = MAX_CLASSES) -> np.ndarray:
    """Request classes: the drawn requests sorted by prompt length (ties by output length, then
    draw index) and cut into n runs of equal count (the first N_REQUESTS mod n one longer); a
    class's lengths are its run's exact means and its weight the run's share of the requests.
    Rows (s_in, s_out, weight), float64 [n][3]."""
    if not 1 <= n <= MAX_CLASSES:
        raise ValueError(n)
    a, b = request_lengths(wl)
    order = np.lexsort((np.arange(len(a)), b, a))
    out = np.zeros((n, 3), np.float64)
    start = 0
    for k in range(n):
        cnt = len(a) // n + (1 if k < len(a) % n else 0)
        idx = order[start:start + cnt]
        start += cnt
        out[k] = (float(int(a[idx].sum())) / cnt, float(int(b[idx].sum())) / cnt, cnt / len(a))
    return out


# --------------------------------------------------------------------------- candidates

def admissible_sizes(n_gpus: int, tp: Tuple[int, ...], pp: Tuple[int, ...], n_layers: int) -> np.ndarray:
    """ok[n] is True iff a group of n GPUs has some tp*pp == n with tp, pp in the sets."""
    ok = np.zeros(n_gpus + 1, bool)
    for t in tp:
        for p in pp:
            if t * p <= n_gpus and p <= n_layers:
                ok[t * p] = True
    return ok


def _renumber(assign_ng: np.ndarray, role_nk: np.ndarray, max_groups: int) -> Tuple[np.ndarray, np.ndarray]:
    """Renumber groups so that group ids ascend with each group's smallest GPU id.

    assign_ng: [N][G] (UNUSED allowed), role_nk: [N][max_groups].  Returns the same layouts.
    """
    N, G = assign_ng.shape
    big = np.int64(G + 1)
    minmem = np.full((N, max_groups + 1), big, np.int64)   # last column collects UNUSED
    rows = np.arange(N)
    a = np.where(assign_ng == UNUSED, max_groups, assign_ng).astype(np.int64)
    for g in range(G - 1, -1, -1):
        minmem[rows, a[:, g]] = np.minimum(minmem[rows, a[:, g]], g)
    minmem = minmem[:, :max_groups]
    order = np.argsort(minmem, axis=1, kind="stable")        # order[r] = old id of new id r
    newid = np.empty_like(order)
    np.put_along_axis(newid, order, np.broadcast_to(np.arange(max_groups), order.shape), axis=1)
    present = np.take_along_axis(minmem, order, axis=1) < big
    new_assign = np.where(assign_ng == UNUSED, UNUSED,
                          np.take_along_axis(newid, np.minimum(a, max_groups - 1), axis=1))
    new_role = np.take_along_axis(role_nk, order, axis=1)
    new_role = np.where(present, new_role, UNUSED)
    return new_assign.astype(np.uint8), new_role.astype(np.uint8)


def random_candidates(wl: Workload, n_cand: Optional[int] = None, stream: int = 2) -> Tuple[np.ndarray, np.ndarray]:
    """Seeded random placements: K ~ U{lo..hi} groups, a random composition of the GPUs into
    K groups whose sizes each admit a strategy (up to 1000 redraws, then kept as drawn),
    GPUs shuffled across groups, roles uniform with at least one prefill and one decode.
    Returns assign [G][N] and role [max_groups][N]."""
    rng = _rng(wl.cfg, stream)
    N = wl.n_cand if n_cand is None else n_cand
    G, Kmax = wl.n_gpus, wl.max_groups
    ok_size = admissible_sizes(G, wl.tp, wl.pp, wl.model["n_layers"])
    K = rng.integers(wl.k_range[0], wl.k_range[1] + 1, N)
    grp = np.zeros((N, G), np.int64)                       # group of composition slot i
    todo = np.arange(N)
    for _ in range(1000):
        if len(todo) == 0:
            break
        m = len(todo)
        keys = rng.random((m, G - 1))
        ranks = np.argsort(np.argsort(keys, axis=1), axis=1)
        cut = ranks < (K[todo] - 1)[:, None]
        g = np.concatenate([np.zeros((m, 1), np.int64), np.cumsum(cut, axis=1)], axis=1)
        grp[todo] = g
        sizes = np.zeros((m, Kmax), np.int64)
        np.add.at(sizes, (np.repeat(np.arange(m), G), g.reshape(-1)), 1)
        kk = np.arange(Kmax)[None, :]
        bad = ((kk < K[todo][:, None]) & ~ok_size[sizes]).any(axis=1)
        todo = todo[bad]
    perm = np.argsort(rng.random((N, G)), axis=1)          # slot i holds GPU perm[i]
    assign_ng = np.empty((N, G), np.int64)
    np.put_along_axis(assign_ng, perm, grp, axis=1)
    role = rng.integers(0, 2, (N, Kmax))
    kk = np.arange(Kmax)[None, :]
    for _ in range(1000):
        live = kk < K[:, None]
        n_p = ((role == PREFILL) & live).sum(1)
        bad = (n_p == 0) | (n_p == K)
        if not bad.any():
            break
        role[bad] = rng.integers(0, 2, (int(bad.sum()), Kmax))
    role = np.where(kk < K[:, None], role, UNUSED)
    a, r = _renumber(assign_ng.astype(np.uint8), role.astype(np.uint8), Kmax)
    return np.ascontiguousarray(a.T), np.ascontiguousarray(r.T)


def base_placement(wl: Workload) -> Tuple[np.ndarray, np.ndarray]:
    """Refinement round-0 base: each node's GPUs form one group; roles alternate by node."""
    G = wl.n_gpus
    assign = (np.arange(G) // GPUS_PER_NODE).astype(np.uint8)
    n_groups = G // GPUS_PER_NODE
    role = np.full(wl.max_groups, UNUSED, np.uint8)
    role[:n_groups] = np.arange(n_groups) % 2
    return assign, role


def perturbations(wl: Workload, base_assign: np.ndarray, base_role: np.ndarray, rnd: int,
                  n_cand: Optional[int] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Round rnd of a refinement batch: n_cand single-step perturbations of a base placement.
    45%: move one GPU to another existing group; 45%: exchange two GPUs of different groups;
    10%: merge two groups, keeping the larger group's role (ties: the lower id's).  No size
    filter.  Groups are renumbered by smallest member.  Returns assign [G][N], role [Kmax][N]."""
    rng = _rng(wl.cfg, 3 + rnd)
    N = wl.n_cand if n_cand is None else n_cand
    G, Kmax = wl.n_gpus, wl.max_groups
    base_assign = np.asarray(base_assign, np.uint8)
    base_role = np.asarray(base_role, np.uint8)
    used = base_assign != UNUSED
    groups = np.unique(base_assign[used]).astype(np.int64)
    n_groups = len(groups)
    sizes = np.bincount(base_assign[used].astype(np.int64), minlength=Kmax)
    a = np.broadcast_to(base_assign.astype(np.int64), (N, G)).copy()
    role = np.broadcast_to(base_role.astype(np.int64), (N, Kmax)).copy()
    kind = rng.choice(3, size=N, p=[0.45, 0.45, 0.10])
    rows = np.arange(N)
    used_idx = np.flatnonzero(used)
    if n_groups >= 2:
        # move
        g = used_idx[rng.integers(0, len(used_idx), N)]
        cur = base_assign[g].astype(np.int64)
        pos = np.searchsorted(groups, cur)
        j = rng.integers(0, n_groups - 1, N)
        j = np.where(j >= pos, j + 1, j)
        sel = kind == 0
        a[rows[sel], g[sel]] = groups[j[sel]]
        # exchange
        g1 = used_idx[rng.integers(0, len(used_idx), N)]
        g2 = used_idx[rng.integers(0, len(used_idx), N)]
        for _ in range(200):
            same = base_assign[g1] == base_assign[g2]
            if not same.any():
                break
            g2[same] = used_idx[rng.integers(0, len(used_idx), int(same.sum()))]
        sel = (kind == 1) & (base_assign[g1] != base_assign[g2])
        a[rows[sel], g1[sel]] = base_assign[g2[sel]]
        a[rows[sel], g2[sel]] = base_assign[g1[sel]]
        # merge
        k1 = rng.integers(0, n_groups, N)
        k2 = rng.integers(0, n_groups - 1, N)
        k2 = np.where(k2 >= k1, k2 + 1, k2)
        ga, gb = groups[k1], groups[k2]
        lo, hi = np.minimum(ga, gb), np.maximum(ga, gb)
        keep = np.where(sizes[hi] > sizes[lo], hi, lo)
        drop = np.where(keep == hi, lo, hi)
        sel = kind == 2
        a[sel] = np.where(a[sel] == drop[sel][:, None], keep[sel][:, None], a[sel])
    a, r = _renumber(a.astype(np.uint8), role.astype(np.uint8), Kmax)
    return np.ascontiguousarray(a.T), np.ascontiguousarray(r.T)


# --------------------------------------------------------------------------- problems

def make_problem(cfg: int, n_cand: Optional[int] = None, rnd: int = 0,
                 base: Optional[Tuple[np.ndarray, np.ndarray]] = None) -> Problem:
    """The seeded problem of workload cfg (1..5).  For the refinement workload (5), round rnd
    perturbs `base` (default: the round-0 base placement)."""
    wl = WORKLOADS[cfg]
    cl = make_cluster(wl)
    s_in, s_out = mean_lengths(wl)
    if wl.rounds > 1:
        b = base_placement(wl) if base is None else base
        assign, role = perturbations(wl, b[0], b[1], rnd, n_cand)
    else:
        assign, role = random_candidates(wl, n_cand)
    return Problem(cl, dict(wl.model), s_in, s_out, wl.tp_mask, wl.pp_mask, wl.granularity,
                   wl.max_groups, assign, role)


GUIDED_STREAM = 1 << 20   # seed stream of guided refinement round r: GUIDED_STREAM + r


PARTITION_STREAM = 1 << 21   # seed stream of the graph-partition candidate draws


def partition_draws(cfg: int, n: int) -> np.ndarray:
    """Uniform 64-bit draws, one per candidate of the graph-partition generator."""
    return _rng(cfg, PARTITION_STREAM).integers(0, 2**64, size=n, dtype=np.uint64, endpoint=False)


def move_draws(cfg: int, rnd: int, n: int) -> np.ndarray:
    """The uniform 64-bit draws of guided refinement round rnd of workload cfg, one per child
    (the move generator takes its random choices from them)."""
    return _rng(cfg, GUIDED_STREAM + rnd).integers(0, 2**64, size=n, dtype=np.uint64, endpoint=False)


def placement_from_groups(groups: List[List[int]], roles: List[int], n_gpus: int,
                          max_groups: int) -> Tuple[np.ndarray, np.ndarray]:
    """One candidate from explicit groups (lists of GPU ids) and roles, as [G][1] / [Kmax][1]."""
    assign = np.full((n_gpus, 1), UNUSED, np.uint8)
    role = np.full((max_groups, 1), UNUSED, np.uint8)
    for k, (members, r) in enumerate(zip(groups, roles)):
        for g in members:
            assign[g, 0] = k
        role[k, 0] = r
    return assign, role


def stack_candidates(cands: List[Tuple[np.ndarray, np.ndarray]]) -> Tuple[np.ndarray, np.ndarray]:
    return (np.ascontiguousarray(np.concatenate([c[0] for c in cands], axis=1)),
            np.ascontiguousarray(np.concatenate([c[1] for c in cands], axis=1)))
