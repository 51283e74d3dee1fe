"""GPU parity at the edges of the argument ranges: one hop and the maximum of
eight, fanouts at the top of their range (where the sampler's candidate list
is nearly full), a partition without halo nodes, a CSR with more than 2^31
entries (64-bit row offsets past the 32-bit range), long rows by few blocks,
and host-link kernels at grids that do not divide their work."""
import time

import numpy as np
import pytest

from gpu_util import log, make_gpu, require_gpu, run_parity, to_dev
from helpers import Problem, tiny_problem, workload_problem

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()


def test_one_hop():
    prob, sched, w = workload_problem("cl10k", fanout=(1,), delta=2)
    rounds, _, _ = run_parity("cl10k K=1", prob, sched.seeds, 8, buffer_rows_every=2)
    assert rounds >= 3


def test_eight_hops():
    prob, sched, w = workload_problem("cl10k", fanout=(3, 2, 2, 2, 1, 1, 1, 1), delta=3)
    rounds, _, _ = run_parity("cl10k K=8", prob, sched.seeds, 7, buffer_rows_every=3)
    # eight hops reach most of the halo, so most buffered slots are hit every
    # step and a due round may evict nothing
    assert rounds >= 1


@pytest.mark.parametrize("fo", [200, 255, 256])
def test_largest_fanouts(fo):
    # rows up to ~1.5K long: every row longer than fo selects from a nearly
    # full candidate list
    prob, sched, w = workload_problem("cl170k", fanout=(fo,), delta=2)
    assert max(np.diff(prob.indptr)) > fo
    rounds, _, _ = run_parity("cl170k fo=%d" % fo, prob, sched.seeds, 5, state_every=2)
    assert rounds == 2


def test_no_halo():
    # a partition whose nodes have no remote neighbours: empty buffer, no misses
    prob = tiny_problem(n_local=40, n_halo=0, p=0.2, seed=5, fanout=(4, 3), buffer_pct=25, delta=2)
    assert prob.H == 0
    rng = np.random.default_rng(5)
    seeds = [rng.permutation(prob.L)[:8].astype(np.int32) for _ in range(6)]
    rounds, hits, misses = run_parity("no halo", prob, lambda t: seeds[t], 6)
    assert rounds == 0 and hits == 0 and misses == 0


def _offset_problem():
    """L = 1024 local nodes with 2.2M neighbour positions each (2.25e9 CSR
    entries), H = 2^20 halo nodes with empty rows. Row v holds the ids
    (v * 7919 + j * 104729) mod (L + H), j < 2.2M."""
    L, H, d = 1024, 1 << 20, 2_200_000
    R = L + H
    indptr = np.zeros(R + 1, np.int64)
    indptr[1:L + 1] = np.arange(1, L + 1, dtype=np.int64) * d
    indptr[L + 1:] = indptr[L]
    assert indptr[-1] > 2 ** 31
    base = (np.arange(d, dtype=np.int64) * 104729 % R).astype(np.int64)
    indices = np.empty(int(indptr[-1]), np.int32)
    for v in range(L):
        row = base + (v * 7919) % R
        row[row >= R] -= R
        indices[v * d:(v + 1) * d] = row
    rng = np.random.default_rng(7)
    halo_gid = rng.permutation(H).astype(np.int32)
    halo_degree = rng.integers(0, 100, H).astype(np.int64)
    feats = rng.standard_normal((R, 4)).astype(np.float32)
    return Problem(L, H, indptr, indices, halo_gid, halo_degree, np.ascontiguousarray(feats[:L]),
                   np.ascontiguousarray(feats[L:]), 4, "f32", (5,), 25, 0.9, 2)


@pytest.mark.timeout(600)
def test_row_offsets_past_2_31():
    import oracle
    t0 = time.time()
    prob = _offset_problem()
    log("offset graph: %d CSR entries (%.0fs)" % (prob.indptr[-1], time.time() - t0))
    gm = make_gpu(prob)
    bb = gm.alloc_batch(prob.L)
    L, H = prob.L, prob.H
    seeds = np.arange(L, dtype=np.int32)[::-1].copy()  # every local row, the highest offsets first
    fo = prob.fanout[0]
    hs = np.ascontiguousarray(prob.halo_store).view(np.uint8).reshape(H, prob.row_bytes)
    for t in range(3):
        sid, _, _, _ = gm.state()
        log("offsets t=%d" % t)
        res = gm.sample(to_dev(seeds), bb)
        assert res.n[0] == L and res.e[0] == L * fo
        F = bb.nodes[:res.n[1]].cpu().numpy()
        assert np.array_equal(F[:L], seeds)
        ip = bb.indptr[0][:L + 1].cpu().numpy().astype(np.int64)
        assert np.array_equal(np.diff(ip), np.full(L, fo))
        sampled = F[bb.indices[0][:res.e[0]].cpu().numpy()]
        assert np.array_equal(F[L:], np.setdiff1d(np.unique(sampled), seeds))
        # rows whose offsets lie past 2^31, and a sample of the others
        past = np.nonzero(prob.indptr[seeds] >= 2 ** 31)[0]
        assert len(past) > 0
        rows = np.union1d(past, np.random.default_rng(t).choice(L, 32, replace=False))
        for i in rows:
            want = oracle.sample_row(prob.indptr, prob.indices, int(seeds[i]), t, 1, fo, prob.seed)
            assert np.array_equal(sampled[ip[i]:ip[i + 1]], want), (t, i)
        # classes and rows against the buffer as it stood before the step
        inbuf = np.zeros(H, bool)
        inbuf[sid] = True
        mask = bb.mask[:res.n[1]].cpu().numpy()
        halo = F >= L
        want = np.where(~halo, 0, np.where(inbuf[np.where(halo, F - L, 0)], 1, 2)).astype(np.uint8)
        assert np.array_equal(mask, want)
        feat = bb.feat[:res.n[1]].cpu().numpy()
        lf = np.ascontiguousarray(prob.local_feat).view(np.uint8).reshape(L, prob.row_bytes)
        src = np.where(halo[:, None], hs[np.where(halo, F - L, 0)], lf[np.minimum(F, L - 1)])
        assert np.array_equal(feat, src)
        gm.evict_step()
    log("offsets: done (%.0fs)" % (time.time() - t0))


@pytest.mark.parametrize("big_row,big_blocks", [(256, 3), (300, 2048)])
def test_long_rows_by_blocks(monkeypatch, big_row, big_blocks):
    # rows longer than big_row are sampled by a whole block (four waves over
    # consecutive quarters of the row); few blocks make each walk many rows
    monkeypatch.setenv("MASSIVE_BIG_ROW", str(big_row))
    monkeypatch.setenv("MASSIVE_BIG_BLOCKS", str(big_blocks))
    prob, sched, w = workload_problem("cl170k", delta=2)
    deg = np.diff(prob.indptr)
    assert np.sum(deg > big_row) > 100
    rounds, _, _ = run_parity("cl170k big rows > %d, %d blocks" % (big_row, big_blocks), prob, sched.seeds, 5,
                              state_every=2)
    assert rounds == 2
    prob, sched, w = workload_problem("cl10k", fanout=(200, 30), delta=3)
    run_parity("cl10k fanout 200 big rows > %d" % big_row, prob, sched.seeds, 6)


@pytest.mark.parametrize("host_blocks,refill_blocks", [(1, 1), (5, 3)])
def test_host_link_grids(monkeypatch, host_blocks, refill_blocks):
    # the host-link kernels at grids that do not divide their work: with one
    # block the miss gather's block 0 moves every row, stamps every
    # written-through slot and then publishes the step; refills in flight on
    # every step (a round every second step)
    monkeypatch.setenv("MASSIVE_HOST_BLOCKS", str(host_blocks))
    monkeypatch.setenv("MASSIVE_REFILL_BLOCKS", str(refill_blocks))
    prob, sched, w = workload_problem("cl170k", delta=2)
    rounds, hits, misses = run_parity("cl170k host grid %d, refill grid %d" % (host_blocks, refill_blocks), prob,
                                      sched.seeds, 7, state_every=2, buffer_rows_every=2)
    assert rounds == 3 and misses > 0


def test_timing_groups():
    # only the selected kernel groups carry HIP events; a mask outside the
    # groups is refused
    from paper_2410_22697_amd import MassiveError, TIMING_GROUPS
    prob, sched, w = workload_problem("cl10k", delta=2)
    gm = make_gpu(prob)
    bb = gm.alloc_batch(w.batch)
    gm.set_timing(["gather_hbm", "classify"])
    for t in range(3):
        gm.sample(to_dev(sched.seeds(t)), bb)
        gm.evict_step()
    tim = gm.timing()
    assert set(tim) == set(TIMING_GROUPS)
    assert tim["gather_hbm"][1] == 3 and tim["classify"][1] == 3 and tim["gather_hbm"][0] > 0
    assert all(tim[g][1] == 0 for g in TIMING_GROUPS if g not in ("gather_hbm", "classify"))
    gm.set_timing(True)
    gm.sample(to_dev(sched.seeds(3)), bb)
    gm.evict_step()
    tim = gm.timing()
    assert tim["sample_dedup"][1] == 1 and tim["gather_hbm"][1] == 1 and tim["gather_miss"][1] == 1
    assert tim["sample_last_hop"][1] == 1 and 0 < tim["sample_last_hop"][0] <= tim["sample_dedup"][0]
    with pytest.raises(MassiveError) as ei:
        gm._check(gm._lib.massive_set_timing(gm._h, 1 << len(TIMING_GROUPS)))
    assert ei.value.code == -1
