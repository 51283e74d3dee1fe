"""Pins for the oracle's fanout sampler, dedup and relabel.

The sampler's choice has a plain definition: for a row of length d > fanout,
the fanout positions with the smallest (Philox key, position); otherwise
every position. Checked by brute force over every subset on tiny graphs, by
exact BFS when the fanout covers every row, and by a chi^2 test of
uniformity (the paper samples a fixed-size uniform neighbour set).
"""
import itertools
import math

import numpy as np
import pytest

import oracle
from helpers import tiny_problem, workload_problem


def _keys(v, d, t, k, seed=0):
    out = []
    for j in range(d):
        w = oracle.philox4x32_10([j // 4, v, t, k], [seed & 0xFFFFFFFF, seed >> 32])
        out.append(w[j % 4])
    return out


def _check_block_structure(prob, st, seeds):
    """Invariants of one step's blocks (frontier prefix, relabel, row sizes)."""
    K = len(prob.fanout)
    F = st.nodes
    assert len(set(F.tolist())) == len(F), "frontier has repeats"
    assert list(F[:len(seeds)]) == list(seeds)
    for k in range(K):
        nprev, nk = st.n[k], st.n[k + 1]
        new = F[nprev:nk]
        assert np.all(np.diff(new) > 0), "new nodes are not ascending"
        ip, ix = st.indptr[k], st.indices[k]
        assert ip[0] == 0 and ip[-1] == st.e[k] == len(ix)
        sampled = set()
        for i in range(nprev):
            v = F[i]
            nb = prob.neighbours(v)
            row = ix[ip[i]:ip[i + 1]]
            assert np.all((row >= 0) & (row < nk))
            ids = F[row]
            assert len(row) == min(len(nb), prob.fanout[k])
            assert len(set(ids.tolist())) == len(ids), "repeated neighbour"
            pos = np.searchsorted(nb, ids)
            assert np.all(nb[pos] == ids), "sampled id is not a neighbour"
            assert np.all(np.diff(pos) > 0), "row not in ascending CSR position"
            sampled.update(ids.tolist())
        # new = exactly the sampled ids not already in F_{k-1}
        assert set(new.tolist()) == sampled - set(F[:nprev].tolist())


@pytest.mark.parametrize("gseed", [1, 2, 3, 4])
def test_bruteforce_subsets_tiny(gseed):
    prob = tiny_problem(n_local=5, n_halo=7, p=0.6, seed=gseed, fanout=(3, 2))
    orc = prob.oracle()
    checked = 0
    for t in range(6):
        seeds = np.array([t % prob.L, (t + 2) % prob.L], np.int32)
        st = orc.sample(seeds)
        orc.evict_step()
        _check_block_structure(prob, st, seeds)
        F = st.nodes
        for k in range(2):
            fo = prob.fanout[k]
            ip, ix = st.indptr[k], st.indices[k]
            for i in range(st.n[k]):
                v = int(F[i])
                nb = prob.neighbours(v)
                d = len(nb)
                chosen = np.searchsorted(nb, F[ix[ip[i]:ip[i + 1]]]).tolist()
                if d <= fo:
                    assert chosen == list(range(d))
                    continue
                keys = _keys(v, d, t, k + 1)
                winners = []
                for S in itertools.combinations(range(d), fo):
                    rest = [j for j in range(d) if j not in S]
                    if max((keys[j], j) for j in S) < min((keys[j], j) for j in rest):
                        winners.append(list(S))
                assert len(winners) == 1
                assert chosen == winners[0]
                checked += 1
    assert checked > 10


def test_full_fanout_is_exact_bfs():
    prob = tiny_problem(n_local=8, n_halo=12, p=0.3, seed=7, fanout=(50, 50, 50))
    orc = prob.oracle()
    seeds = np.array([0, 3], np.int32)
    st = orc.sample(seeds)
    # K-hop neighbourhood by plain BFS
    frontier, seen = set(seeds.tolist()), set(seeds.tolist())
    for k in range(3):
        nxt = set()
        for v in range(st.n[k]):
            nxt.update(prob.neighbours(int(st.nodes[v])).tolist())
        seen |= nxt
        assert set(st.nodes[:st.n[k + 1]].tolist()) == seen
        for i in range(st.n[k]):
            row = st.nodes[st.indices[k][st.indptr[k][i]:st.indptr[k][i + 1]]]
            assert row.tolist() == prob.neighbours(int(st.nodes[i])).tolist()


def test_uniform_subsets_chi2():
    # One local node with 6 neighbours, fanout 2: 15 subsets, equally likely.
    L, H = 1, 6
    indptr = np.array([0, 6] + [6 + i + 1 for i in range(6)], np.int64)
    indices = np.array([1, 2, 3, 4, 5, 6] + [0] * 6, np.int32)
    from helpers import Problem
    prob = Problem(L, H, indptr, indices, np.arange(H, dtype=np.int32), np.ones(H, np.int64),
                   np.zeros((1, 1), np.float32), np.zeros((H, 1), np.float32), 1, "f32",
                   (2,), 0, 0.9, 1000)
    orc = prob.oracle()
    counts = {}
    T = 3000
    for t in range(T):
        st = orc.sample(np.array([0], np.int32))
        orc.evict_step()
        key = tuple(sorted(st.nodes[st.indices[0]].tolist()))
        counts[key] = counts.get(key, 0) + 1
    assert len(counts) == 15
    exp = T / 15
    chi2 = sum((c - exp) ** 2 / exp for c in counts.values())
    assert chi2 < 36.1  # 14 dof, p = 0.001


def test_block_invariants_cl10k():
    prob, sched, w = workload_problem("cl10k")
    orc = prob.oracle()
    for t in range(3):
        seeds = sched.seeds(t)
        st = orc.sample(seeds)
        orc.evict_step()
        _check_block_structure(prob, st, seeds)


def test_rejects_bad_seeds():
    prob = tiny_problem()
    orc = prob.oracle()
    with pytest.raises(ValueError):
        orc.sample(np.array([prob.L], np.int32))        # a halo node is not a seed
    with pytest.raises(ValueError):
        orc.sample(np.array([1, 1], np.int32))          # duplicate seed
    st = orc.sample(np.array([1, 2], np.int32))         # state unharmed
    assert st.n[0] == 2
    with pytest.raises(ValueError):
        orc.sample(np.array([1, 2], np.int32))          # the round call is owed first
