"""Pins of the oracle's max-flow guided refinement (Sec. 3.4): edge classes and guided moves.

The edge classes are checked against their definitions by brute force: an edge is a
bottleneck when raising its capacity by one raises the maximum flow, and underutilized when
lowering it by one keeps the maximum flow; the maximum flows come from exhaustive minimum-cut
enumeration (tiny networks) or scipy's solver, never from the oracle's own max-flow.  The
guided moves are checked for what the move rules fix: every child is its parent with one
move applied whose donor and receiver have the classes the rule requires (classes recomputed
by brute force), the first children are the parents, and random choices spread evenly.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import hxo
from paper_2502_07903_amd import inputs as I
from tests import helpers as Hh


def _scipy_value(nv, E):
    from scipy.sparse import csr_matrix
    from scipy.sparse.csgraph import maximum_flow
    M = np.zeros((nv, nv), np.int64)
    for a, b, c in E:
        M[a, b] += c
    return int(maximum_flow(csr_matrix(M.astype(np.int32)), 0, 1).flow_value)


def _brute_classes(fn, n, solver):
    """{edge index: class bits} of candidate n by re-solving with every capacity +1 and -1."""
    nv, E = Hh.network_edges(fn, n)
    base = solver(nv, E)
    out = []
    for e, (a, b, c) in enumerate(E):
        up = list(E)
        up[e] = (a, b, c + 1)
        k = 1 if solver(nv, up) > base else 0
        if c >= 1:
            dn = list(E)
            dn[e] = (a, b, c - 1)
            if solver(nv, dn) == base:
                k |= 2
        out.append(k)
    return E, out


def _oracle_edge_bits(fn, cls, n):
    """Class bits of candidate n in network_edges order, read from the oracle's rows."""
    P, D = int(fn["n_p"][n]), int(fn["n_d"][n])
    mp = fn["dims"][0]
    bits = []
    for i in range(P):
        c = int(cls["node_cls"][i, n])
        bits += [(c >> 2) & 3, c & 3]
    for i in range(P):
        for j in range(D):
            bits.append(int(cls["kv_cls"][i * D + j, n]) & 3)
    for j in range(D):
        c = int(cls["node_cls"][mp + j, n])
        bits += [c & 3, (c >> 2) & 3]
    return bits


def _small_flownet(rng, N, maxP, maxD, hi_choices):
    fn = dict(n_p=np.zeros(N, np.int32), n_d=np.zeros(N, np.int32))
    for k, rows in (("src_cap", maxP), ("p_cap", maxP), ("kv_cap", maxP * maxD), ("d_cap", maxD),
                    ("sink_cap", maxD), ("p_slot", maxP), ("d_slot", maxD)):
        fn[k] = np.zeros((rows, N), np.int32)
    for n in range(N):
        P, D = int(rng.integers(0, maxP + 1)), int(rng.integers(0, maxD + 1))
        fn["n_p"][n], fn["n_d"][n] = P, D
        hi = int(rng.choice(hi_choices))
        for k, rows in (("src_cap", P), ("p_cap", P), ("kv_cap", P * D), ("d_cap", D), ("sink_cap", D)):
            fn[k][:rows, n] = rng.integers(0, hi + 1, rows)
    fn["dims"] = (maxP, maxD, maxP * maxD)
    return fn


def test_edge_classes_brute_force_min_cut():
    """Tiny networks: classes = the +-1 capacity definitions, max flows by exhaustive min cut."""
    rng = np.random.default_rng(34)
    fn = _small_flownet(rng, 160, 3, 3, [1, 2, 4, 9])
    cls = hxo.edge_classes(fn)
    for n in range(160):
        if int(fn["n_p"][n]) + int(fn["n_d"][n]) > 5:
            continue
        E, want = _brute_classes(fn, n, Hh.brute_force_min_cut)
        assert _oracle_edge_bits(fn, cls, n) == want, (n, E)


def test_edge_classes_scipy_workload_networks():
    """Networks of real candidates (8- and 16-GPU workloads): classes = the +-1 definitions
    with scipy's maximum flow."""
    pytest.importorskip("scipy")
    for cfg, n_cand in ((1, 48), (2, 24)):
        prob = I.make_problem(cfg, n_cand=n_cand)
        fn = hxo.build_flownet(prob, hxo.cost_eval(prob))
        cls = hxo.edge_classes(fn)
        for n in range(n_cand):
            E, want = _brute_classes(fn, n, _scipy_value)
            assert _oracle_edge_bits(fn, cls, n) == want, (cfg, n)


def test_edge_classes_kv_summary_bit():
    """Bit 4 of a node's class = some KV edge at that node is a bottleneck."""
    rng = np.random.default_rng(13)
    fn = _small_flownet(rng, 300, 4, 4, [3, 50])
    cls = hxo.edge_classes(fn)
    mp = fn["dims"][0]
    for n in range(300):
        P, D = int(fn["n_p"][n]), int(fn["n_d"][n])
        kv = cls["kv_cls"][:P * D, n].reshape(P, D) & 1
        for i in range(P):
            assert bool(cls["node_cls"][i, n] & 16) == bool(kv[i].any())
        for j in range(D):
            assert bool(cls["node_cls"][mp + j, n] & 16) == bool(kv[:, j].any())


def test_edge_classes_properties():
    """No edge is both a bottleneck and underutilized; in a series chain of distinct
    capacities the smallest edge is the one bottleneck and every other edge underutilized."""
    rng = np.random.default_rng(8)
    fn = _small_flownet(rng, 400, 4, 4, [3, 50, 1000])
    cls = hxo.edge_classes(fn)
    for n in range(400):
        bits = _oracle_edge_bits(fn, cls, n)
        assert all(b != 3 for b in bits)
    # series chain s -> p -> d -> t with one strictly smallest edge: exactly that edge is a
    # bottleneck, every other edge underutilized
    fn = _small_flownet(rng, 50, 1, 1, [10])
    caps = np.zeros((5, 50), np.int64)
    for n in range(50):
        fn["n_p"][n] = fn["n_d"][n] = 1
        c = rng.permutation([5, 6, 7, 8, 9])
        caps[:, n] = c
        fn["src_cap"][0, n], fn["p_cap"][0, n], fn["kv_cap"][0, n], fn["d_cap"][0, n], fn["sink_cap"][0, n] = c
    cls = hxo.edge_classes(fn)
    for n in range(50):
        bits = _oracle_edge_bits(fn, cls, n)
        smallest = int(np.argmin(caps[:, n]))
        assert bits == [1 if e == smallest else 2 for e in range(5)]


# ------------------------------------------------------------------ guided moves

def _parents_with_classes(cfg, n_par, seed_skip=0):
    prob = I.make_problem(cfg, n_cand=n_par + seed_skip).subset(np.arange(seed_skip, seed_skip + n_par))
    fn = hxo.build_flownet(prob, hxo.cost_eval(prob))
    return prob, fn, hxo.edge_classes(fn)


def _eligibility(prob, fn, n, edge_bits):
    """Donor GPUs, receiver groups and flip-eligible groups of parent n, from class bits in
    network_edges order (the move rules' definitions)."""
    G, K = prob.n_gpus, prob.max_groups
    P, D = int(fn["n_p"][n]), int(fn["n_d"][n])
    a = prob.assign[:, n].astype(int)
    r = prob.role[:, n].astype(int)
    grp = [int(a[g]) if a[g] < K and r[a[g]] in (0, 1) else -1 for g in range(G)]
    node_b, node_u, kv_b = {}, {}, {}
    for i in range(P):
        node_b[("p", i)] = edge_bits[2 * i + 1] & 1
        node_u[("p", i)] = edge_bits[2 * i + 1] >> 1 & 1
        kv_b[("p", i)] = any(edge_bits[2 * P + i * D + j] & 1 for j in range(D))
    for j in range(D):
        b = edge_bits[2 * P + P * D + 2 * j]
        node_b[("d", j)] = b & 1
        node_u[("d", j)] = b >> 1 & 1
        kv_b[("d", j)] = any(edge_bits[2 * P + i * D + j] & 1 for i in range(P))

    def node_of(g):
        if grp[g] < 0:
            return None
        key = grp[g] if prob.granularity == 0 else g
        if r[grp[g]] == 0:
            hits = [i for i in range(P) if fn["p_slot"][i, n] == key]
            return ("p", hits[0]) if hits else None
        hits = [j for j in range(D) if fn["d_slot"][j, n] == key]
        return ("d", hits[0]) if hits else None

    donors = {g for g in range(G) if grp[g] < 0 or (node_of(g) is not None and node_u[node_of(g)])}
    recv = set()
    for g in range(G):
        v = node_of(g)
        if v is not None and (node_b[v] or kv_b[v]):
            recv.add(grp[g])
    groups = {k for k in grp if k >= 0}
    flip = set()
    for k in groups - recv:
        if all(g in donors for g in range(G) if grp[g] == k) and any(r[q] != r[k] for q in recv):
            flip.add(k)
    return grp, donors, recv, flip


@pytest.mark.parametrize("cfg", [1, 2])
def test_guided_children_apply_one_eligible_move(cfg):
    prob, fn, cls = _parents_with_classes(cfg, 6)
    M = prob.n_cand
    rnd = I.move_draws(cfg, 0, 3000)
    ch = hxo.guided_moves(prob.n_gpus, prob.max_groups, prob.granularity, prob.assign, prob.role, fn, cls, rnd)
    elig = {}
    for m in range(M):
        _, want = _brute_classes(fn, m, _scipy_value)
        elig[m] = _eligibility(prob, fn, m, want)
    kinds = np.zeros(4, int)
    for c in range(3000):
        m = c % M
        pa, pr = prob.assign[:, m], prob.role[:, m]
        ca, cr = ch["assign"][:, c], ch["role"][:, c]
        mv = int(ch["move"][c])
        t, x, y = mv & 0xFF, mv >> 8 & 0xFF, mv >> 16 & 0xFF
        kinds[t] += 1
        grp, donors, recv, flip = elig[m]
        da = set(np.flatnonzero(ca != pa).tolist())
        dr = set(np.flatnonzero(cr != pr).tolist())
        if c < M:
            assert mv == 0 and not da and not dr
        elif t == 0:
            assert not da and not dr
            # no move had a choice: no receiver with an outside donor, and no flip
            assert not flip
            assert not any(d for k in recv for d in donors if grp[d] != k)
        elif t == 1:
            assert da == {x} and not dr and ca[x] == y
            assert y in recv and x in donors and grp[x] != y
        elif t == 2:
            assert da == {x, y} and not dr
            assert ca[x] == pa[y] and ca[y] == pa[x]
            assert grp[x] in recv and y in donors and grp[y] != grp[x]
        else:
            assert not da and dr == {x} and x in flip and cr[x] == 1 - pr[x]
    assert kinds[0] >= M


def test_guided_first_type_and_choice_spread():
    """The type field picks MOVE / SWAP / FLIP in thirds, and a receiver among m in near-equal
    shares, over an exhaustive sweep of the draw's bits."""
    prob, fn, cls = _parents_with_classes(2, 1, seed_skip=3)
    _, want = _brute_classes(fn, 0, _scipy_value)
    grp, donors, recv, flip = _eligibility(prob, fn, 0, want)
    if not recv or not any(d for d in donors if grp[d] not in recv):
        pytest.skip("parent has no MOVE choice")
    # u0 = 0 starts with MOVE; sweep the receiver field over 4096 evenly spaced values
    u1 = (np.arange(4096, dtype=np.uint64) << np.uint64(12)) << np.uint64(16)
    rnd = np.concatenate([np.zeros(1, np.uint64), u1])
    ch = hxo.guided_moves(prob.n_gpus, prob.max_groups, prob.granularity, prob.assign, prob.role, fn, cls, rnd)
    mv = ch["move"][1:]
    assert np.all(mv & 0xFF == 1)
    got = np.bincount((mv >> 16) & 0xFF, minlength=256)
    counts = got[sorted(recv)]
    assert counts.sum() == 4096 and counts.max() - counts.min() <= 1
    # type field over all 2^16 values: MOVE first for the lowest third
    u0 = np.arange(0, 1 << 16, 16, dtype=np.uint64)
    t0 = (u0 * np.uint64(3)) >> np.uint64(16)
    assert np.bincount(t0.astype(int)).max() - np.bincount(t0.astype(int)).min() <= 1


def test_guided_moves_relieve_decode_bottleneck():
    """The case study's situation (Appendix, light prefill / heavy decode): a prefill replica
    with spare capacity feeding a decode replica that limits the flow.  Guided MOVEs then take
    a prefill (or unused) GPU into the decode replica, and FLIPs turn prefill into decode."""
    cl = Hh.cluster_c1()
    model = dict(I.OPT_30B)
    # 8 GPUs (node 0 = A, node 1 = B): prefill {0,1,2,3} TP4 on A, decode {4,5,6,7} TP4 on B
    assign, role = I.placement_from_groups([[0, 1, 2, 3], [4, 5, 6, 7]], [I.PREFILL, I.DECODE], 8, 4)
    prob = Hh.problem(cl, model, assign, role, s_in=512.0, s_out=128.0, tp=(1, 2, 4), pp=(1, 2))
    fn = hxo.build_flownet(prob, hxo.cost_eval(prob))
    cls = hxo.edge_classes(fn)
    assert int(fn["p_cap"][0, 0]) > int(fn["d_cap"][0, 0]) > 0
    assert cls["node_cls"][0, 0] & 3 == 2                       # prefill node: underutilized
    assert cls["node_cls"][fn["dims"][0], 0] & 3 == 1           # decode node: bottleneck
    rnd = I.move_draws(1, 0, 2000)
    ch = hxo.guided_moves(8, 4, 0, assign, role, fn, cls, rnd)
    mv = ch["move"]
    t = mv & 0xFF
    assert set(np.unique(t[1:]).tolist()) <= {1, 2, 3}
    for c in np.flatnonzero(t == 1):
        g, k = int(mv[c] >> 8 & 0xFF), int(mv[c] >> 16 & 0xFF)
        assert k == 1 and g in (0, 1, 2, 3)
    for c in np.flatnonzero(t == 2):
        g, h = int(mv[c] >> 8 & 0xFF), int(mv[c] >> 16 & 0xFF)
        assert g in (4, 5, 6, 7) and h in (0, 1, 2, 3)
    for c in np.flatnonzero(t == 3):
        assert int(mv[c] >> 8 & 0xFF) == 0 and ch["role"][0, c] == I.DECODE
