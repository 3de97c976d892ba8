"""Pins of the oracle's graph-partition phase (Sec. 3.2), no GPU.

Spectral step: the power-iteration vector is orthogonal to the constant vector, has unit
length, and its Rayleigh quotient is the Laplacian's second-smallest eigenvalue from numpy's
symmetric eigensolver; on the two-node cluster it separates the nodes.  Candidates: checked
against what the partition rules fix, with every cut recomputed explicitly from the pairwise
weights (not the oracle's gain bookkeeping): the number of groups follows K = floor(total
memory / replica memory) shifted by the draw; no Kernighan-Lin swap that keeps the two groups'
memory gap from widening lowers the cut (a local optimum); no single flip of a super node
raises the coarse cut while both sides stay occupied; groups are numbered by smallest member;
both roles are present.  Kernighan-Lin: a hand-derived case (tests/golden/kl_worked.txt) where
no single swap lowers the cut but a pass that first takes a swap of negative gain does, reaching
the smallest cut of all balanced splits (brute force); on random graphs the refinement never
raises the cut and ends at a local optimum of single swaps.
"""
import dataclasses
import itertools

import numpy as np
import pytest

from oracle import hxo
from paper_2502_07903_amd import inputs as I
from tests import helpers as Hh


def _weights(prob):
    G = prob.n_gpus
    b = np.asarray(prob.cluster.beta, np.float64).reshape(G, G)
    w = np.clip(np.floor(((b + b.T) * 0.5) / 1e6), 0, 2 ** 47).astype(np.int64)
    np.fill_diagonal(w, 0)
    return w


def _laplacian(w):
    return np.diag(w.sum(1)).astype(np.float64) - w.astype(np.float64)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_spectral_vector(cfg):
    prob = I.make_problem(cfg, n_cand=1)
    order, x = hxo.spectral_order(prob, iters=4000)
    Lap = _laplacian(_weights(prob))
    ev = np.linalg.eigvalsh(Lap)
    assert abs(x.sum()) < 1e-9 and abs(np.dot(x, x) - 1.0) < 1e-12
    rq = float(x @ Lap @ x)
    assert rq == pytest.approx(ev[1], rel=2e-3, abs=1e-6 * ev[-1])
    assert sorted(order.tolist()) == list(range(prob.n_gpus))
    assert all((x[order[i]], order[i]) <= (x[order[i + 1]], order[i + 1]) for i in range(prob.n_gpus - 1))


def test_spectral_two_nodes():
    """Two nodes of four GPUs, 300 GB/s inside and 12.5 GB/s across: the Fiedler direction has one
    sign per node, so the spectral order keeps each node's GPUs together."""
    prob = I.make_problem(1, n_cand=1)
    order, x = hxo.spectral_order(prob)
    assert len(set(np.sign(x[:4]))) == 1 and len(set(np.sign(x[4:]))) == 1 and np.sign(x[0]) != np.sign(x[4])
    assert set(order[:4].tolist()) in ({0, 1, 2, 3}, {4, 5, 6, 7})


def test_partition_group_count():
    """K = floor(total memory / (12 H^2 B L + 32 * 2 (s_in + s_out) H_kv B L))."""
    for cfg in (1, 2, 3, 4, 5):
        prob = I.make_problem(cfg, n_cand=1)
        cl = prob.cluster
        m = prob.model
        H, B, L = m["hidden"], m["bytes_per_elem"], m["n_layers"]
        Hkv = H * m["n_kv_heads"] // m["n_heads"]
        total = float(np.floor(np.asarray(cl.type_mem)[np.asarray(cl.gpu_type)]).sum())
        rep = 12.0 * H * H * B * L + 32.0 * 2.0 * (prob.s_in + prob.s_out) * Hkv * B * L
        assert hxo.partition_groups(prob) == int(np.floor(total / rep))


def _cut(w, grp):
    diff = grp[:, None] != grp[None, :]
    return int((w * diff).sum() // 2)


@pytest.mark.parametrize("cfg,n", [(1, 64), (2, 48), (3, 24), (4, 3)])
def test_partition_candidates_are_local_optima(cfg, n):
    prob = I.make_problem(cfg, n_cand=1)
    order, _ = hxo.spectral_order(prob)
    rnd = I.partition_draws(cfg, n)
    assign, role = hxo.partition_candidates(prob, order, rnd)
    w = _weights(prob)
    G, Kmax = prob.n_gpus, prob.max_groups
    mem = np.floor(np.asarray(prob.cluster.type_mem)[np.asarray(prob.cluster.gpu_type)]).astype(np.int64)
    k_est = hxo.partition_groups(prob)
    for c in range(n):
        grp = assign[:, c].astype(np.int64)
        used = int(grp.max()) + 1
        # numbering by smallest member, every group used
        firsts = [int(np.flatnonzero(grp == k)[0]) for k in range(used)]
        assert firsts == sorted(firsts)
        # the draw's K (groups may only merge away when a cut chunk is empty)
        K = min(max(k_est + int(rnd[c] & np.uint64(7)) % 5 - 2, 2), min(G, Kmax, 32))
        assert used <= K
        # Kernighan-Lin local optimum under the balance rule
        base = _cut(w, grp)
        gmem = np.bincount(grp, weights=mem, minlength=used).astype(np.int64)
        for u in range(G):
            for v in range(u + 1, G):
                A, Bk = grp[u], grp[v]
                if A == Bk:
                    continue
                gap0 = abs(gmem[A] - gmem[Bk])
                gap1 = abs((gmem[A] - mem[u] + mem[v]) - (gmem[Bk] - mem[v] + mem[u]))
                if gap1 > gap0:
                    continue
                g2 = grp.copy()
                g2[u], g2[v] = Bk, A
                assert _cut(w, g2) >= base, (c, u, v)
        # roles: both present, and no single flip raises the coarse cut
        side = role[:used, c].astype(np.int64)
        assert set(side.tolist()) == {0, 1} and (role[used:, c] == I.UNUSED).all()
        S = np.zeros((used, used), np.int64)
        for d in range(G):
            for e in range(G):
                if grp[d] != grp[e]:
                    S[grp[d], grp[e]] += w[d, e]
        cut0 = int((S * (side[:, None] != side[None, :])).sum())
        for k in range(used):
            s2 = side.copy()
            s2[k] ^= 1
            if len(set(s2.tolist())) < 2:
                continue
            assert int((S * (s2[:, None] != s2[None, :])).sum()) <= cut0


def _graph_problem(w, mem=None):
    """A cluster whose device-graph weights are exactly w (whole MB/s): beta = (w + 1/2) MB/s."""
    G = w.shape[0]
    beta = (w.astype(np.float64) + 0.5) * 1e6
    np.fill_diagonal(beta, 0.0)
    mem = np.full(G, 80e9) if mem is None else np.asarray(mem, np.float64)
    types, gpu_type = np.unique(mem, return_inverse=True)
    T = len(types)
    cl = I.Cluster(gpu_type.astype(np.int32), np.full(T, 312e12), np.full(T, 2e12), types.astype(np.float64),
                   np.ascontiguousarray(beta.reshape(-1)), np.zeros(G * G))
    a = np.zeros((G, 1), np.uint8)
    r = np.zeros((1, 1), np.uint8)
    return Hh.problem(cl, Hh.MODELS["opt30b"], a, r)


def _swap_gains(w, grp, mem):
    """Cut change of every balance-keeping single swap, from explicit cuts."""
    base = _cut(w, grp)
    gmem = {k: int(mem[grp == k].sum()) for k in set(grp.tolist())}
    out = []
    for u in range(len(grp)):
        for v in range(u + 1, len(grp)):
            A, B = grp[u], grp[v]
            if A == B:
                continue
            if abs((gmem[A] - mem[u] + mem[v]) - (gmem[B] - mem[v] + mem[u])) > abs(gmem[A] - gmem[B]):
                continue
            g2 = grp.copy()
            g2[u], g2[v] = B, A
            out.append(base - _cut(w, g2))
    return out


def test_kl_worked_case():
    case = Hh.parse_golden("kl_worked.txt")[0]
    w = np.array([Hh.ints(row) for row in case["weights"].split(";")], np.int64)
    assert (w == w.T).all()
    prob = _graph_problem(w)
    assert np.array_equal(_weights(prob), w)
    start = np.array(Hh.ints(case["start"]), np.int64)
    mem = np.full(len(start), 80_000_000_000, np.int64)
    assert _cut(w, start) == int(case["start_cut"])
    assert max(_swap_gains(w, start, mem)) == int(case["best_single_swap_gain"])  # greedy stops here
    got, passes = hxo.kl_refine(prob, start)
    assert got.tolist() == Hh.ints(case["result"])
    assert _cut(w, got.astype(np.int64)) == int(case["result_cut"])
    assert passes == int(case["improving_passes"])
    best = min(_cut(w, np.array([0 if i in S else 1 for i in range(8)])) for S in itertools.combinations(range(8), 4))
    assert best == int(case["result_cut"])


def test_kl_random_graphs():
    """Random weighted graphs, groups and memories: the refined grouping keeps the group sizes'
    memory balance rule (no swap it made widened a gap, so no group is emptied), never has a
    larger cut than the start, and no single balance-keeping swap lowers its cut."""
    rng = np.random.default_rng(3502)
    improved = 0
    for trial in range(60):
        G = int(rng.integers(4, 13))
        K = int(rng.integers(2, min(G, 4) + 1))
        w = rng.integers(0, 50, (G, G))
        w = np.triu(w, 1)
        w = w + w.T
        mem = rng.choice([16e9, 24e9, 80e9], G)
        prob = _graph_problem(w, mem)
        start = np.arange(G) % K
        rng.shuffle(start)
        got, _ = hxo.kl_refine(prob, start)
        got = got.astype(np.int64)
        memi = mem.astype(np.int64)
        assert sorted(set(got.tolist())) == sorted(set(start.tolist()))
        assert _cut(w, got) <= _cut(w, start)
        assert max(_swap_gains(w, got, memi), default=0) <= 0
        improved += _cut(w, got) < _cut(w, start)
    assert improved > 20
