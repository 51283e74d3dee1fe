"""Property-based runs of the oracle on random tiny partitions (hypothesis,
derandomised so that every run draws the same cases): random graph density,
halo size (none included), feature width, hops and fanouts, f from 0 to
100%, gamma in (0, 1], Delta, and seed batches of any size. Every step is
checked against what the definitions fix (the NeighborSampler of
Algorithm 2, the buffer policy of Algorithm 2 and Section IV-B, Eq. 1):
  * blocks: each row's sampled neighbours are distinct true neighbours,
    min(d, fanout) of them, in ascending CSR position; fanout >= d keeps the
    whole row; the new nodes are the ascending unique sampled ids not in the
    frontier; relabelled indices point at those ids;
  * classes and rows: local / hit / miss against the buffer before the step,
    gathered bytes equal the source rows;
  * the policy: the independent Python replay of the buffer (same frontiers)
    gives the same hits, misses, evictions, replacements and scores after
    every step, and the halo rank is numpy's lexsort of (gid, -degree)."""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from helpers import rank_order, tiny_problem
from test_oracle_buffer import _replay


@st.composite
def cases(draw):
    n_local = draw(st.integers(1, 12))
    n_halo = draw(st.integers(0, 20))
    K = draw(st.integers(1, 3))
    fanout = tuple(draw(st.integers(1, 6)) for _ in range(K))
    gamma = draw(st.sampled_from([1.0, 0.95, 0.8, 0.5, 0.3]))
    prob = tiny_problem(n_local=n_local, n_halo=n_halo, p=draw(st.floats(0.05, 0.9)),
                        seed=draw(st.integers(0, 10_000)), d=draw(st.integers(1, 9)), fanout=fanout,
                        buffer_pct=draw(st.integers(0, 100)), gamma=gamma, delta=draw(st.integers(1, 5)),
                        dtype=draw(st.sampled_from(["f32", "bf16"])))
    steps = draw(st.integers(1, 24))
    most = draw(st.integers(1, n_local))  # small batches leave slots unsampled, so rounds evict
    batches = [draw(st.lists(st.integers(0, n_local - 1), min_size=1, max_size=most, unique=True))
               for _ in range(steps)]
    return prob, batches


def _check_blocks(prob, st_, seeds):
    F = st_.nodes
    assert np.array_equal(F[:len(seeds)], seeds)
    assert len(np.unique(F)) == len(F)
    for k, fo in enumerate(prob.fanout):
        n0, n1 = st_.n[k], st_.n[k + 1]
        ip, ix = st_.indptr[k], st_.indices[k]
        assert len(ip) == n0 + 1 and ip[0] == 0 and len(ix) == st_.e[k] == ip[-1]
        assert np.all((ix >= 0) & (ix < n1))
        sampled = F[ix]
        for i in range(n0):
            nb = prob.neighbours(int(F[i]))
            got = sampled[ip[i]:ip[i + 1]]
            assert len(got) == min(len(nb), fo)
            pos = np.searchsorted(nb, got)  # CSR rows are sorted and duplicate-free
            assert np.all(pos < len(nb)) and np.array_equal(nb[np.minimum(pos, len(nb) - 1)], got)
            assert np.all(np.diff(pos) > 0), "not in ascending position"
            if fo >= len(nb):
                assert np.array_equal(got, nb)
        new = np.setdiff1d(np.unique(sampled), F[:n0])
        assert np.array_equal(F[n0:n1], new)


@settings(max_examples=300, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
@given(cases())
def test_oracle_on_random_tiny_partitions(case):
    prob, batches = case
    orc = prob.oracle()
    rk = orc.rank()
    if prob.H:
        assert np.array_equal(np.argsort(rk, kind="stable"), rank_order(prob))
    b = prob.row_bytes
    lf = prob.local_feat.view(np.uint8).reshape(prob.L, b)
    hs = prob.halo_store.view(np.uint8).reshape(prob.H, b)
    frontiers, got = [], []
    for seeds in batches:
        seeds = np.array(seeds, np.int32)
        sid_before = orc.state()[0].copy()
        s = orc.sample(seeds)
        _check_blocks(prob, s, seeds)
        F = s.nodes
        inbuf = np.zeros(max(prob.H, 1), bool)
        inbuf[sid_before] = True
        halo = F >= prob.L
        want = np.where(~halo, 0, np.where(inbuf[np.where(halo, F - prob.L, 0)], 1, 2))
        assert np.array_equal(s.mask, want.astype(np.uint8))
        src = np.where(halo[:, None], hs[np.maximum(F - prob.L, 0)] if prob.H else 0, lf[np.minimum(F, prob.L - 1)])
        assert np.array_equal(s.feat, src)
        rnd = orc.evict_step()
        frontiers.append(F.copy())
        got.append((s.hits, s.misses, rnd, orc.state()))
    rep = _replay(prob, frontiers, rk)
    for (hits, misses, rnd, (sid, se, sa)), (r_hits, r_misses, r_rnd, r_slot, r_se, r_sa) in zip(got, rep):
        assert (hits, misses) == (r_hits, r_misses)
        if r_rnd is None or not r_rnd[0]:
            assert rnd.k == 0
        else:
            E, ev, R = r_rnd
            assert rnd.slots.tolist() == E and rnd.evicted.tolist() == ev and rnd.replaced.tolist() == R
        assert sid.tolist() == r_slot
        assert np.array_equal(se.view(np.uint32), np.array(r_se, np.float32).view(np.uint32))
        assert np.array_equal(sa.view(np.uint32), r_sa.view(np.uint32))
