"""GPU parity of the staged host link (MASSIVE_LINK_STAGED): the rows that
cross the host link (misses, hits on slots still refilling, refill rows) are
gathered by the context's host threads into pinned staging memory, copied to
the device by the DMA engines and scattered by a kernel, so no kernel reads
host memory. Outputs, states, eviction sets and buffer rows must equal the
oracle's exactly as in the loads mode: with staging entries of a few rows (the
ring wraps many times per step), one or three gathering threads, a round after
every step, refills in flight under two or three batches in flight, rows of
every vector width, no halo and no buffer."""
import numpy as np
import pytest

from gpu_util import log, make_gpu, require_gpu, run_lookahead, run_parity, to_dev
from helpers import tiny_problem, workload_problem

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()


@pytest.fixture
def small_ring(monkeypatch):
    """Staging entries of 4 KiB (8 rows of 512 B): the ring wraps often."""
    monkeypatch.setenv("MASSIVE_RING_BYTES", "4096")


def staged(prob, **kw):
    return make_gpu(prob, link="staged", **kw)


def test_staged_tiny_graphs(small_ring):
    total = 0
    for seed in (1, 2, 3):
        prob = tiny_problem(n_local=6, n_halo=9, p=0.4, seed=seed, fanout=(2, 1), buffer_pct=34, delta=2, gamma=0.5)
        rng = np.random.default_rng(seed)
        seeds = [rng.permutation(prob.L)[:1].astype(np.int32) for _ in range(16)]
        rounds, _, _ = run_parity("staged tiny%d" % seed, prob, lambda t: seeds[t], 16, gm=staged(prob))
        total += rounds
    assert total >= 3


def test_staged_cl10k_full_run(small_ring):
    prob, sched, w = workload_problem("cl10k")
    rounds, _, _ = run_parity("staged cl10k", prob, sched.seeds, w.steps, buffer_rows_every=5, gm=staged(prob))
    assert rounds >= 5


@pytest.mark.parametrize("over", [dict(gamma=0.7, delta=2, buffer_pct=80),    # fewer candidates than evictions
                                  dict(buffer_pct=100, delta=2),                # no candidates at all
                                  dict(buffer_pct=0, delta=2),                  # empty buffer: every row a miss
                                  dict(gamma=0.9, delta=1)])                    # a round after every step
def test_staged_cl10k_variants(over, small_ring):
    prob, sched, w = workload_problem("cl10k", **over)
    run_parity("staged cl10k%s" % sorted(over.items()), prob, sched.seeds, 20, buffer_rows_every=4, gm=staged(prob))


def test_staged_cl170k_full_run():
    # the library's own staging entries (8 MiB)
    prob, sched, w = workload_problem("cl170k")
    rounds, _, _ = run_parity("staged cl170k", prob, sched.seeds, w.steps, state_every=8, buffer_rows_every=50,
                              gm=staged(prob))
    assert rounds >= 10


@pytest.mark.parametrize("depth", [2, 3])
def test_staged_lookahead_round_every_step(depth, small_ring):
    prob, sched, w = workload_problem("cl10k", delta=1, gamma=0.9)
    rounds, pending = run_lookahead("staged async cl10k delta 1 depth %d" % depth, prob, sched.seeds, 12, depth,
                                    link="staged")
    assert rounds >= 8


def test_staged_lookahead_cl2m45_inflight_refills():
    prob, sched, w = workload_problem("cl2m45", delta=2)
    rounds, pending = run_lookahead("staged async cl2m45", prob, sched.seeds, 6, link="staged")
    assert rounds == 2 and pending > 0  # hits on refilling slots were written through


# rows of 4, 12, 100 and 4000 bytes (fp32) and 100 bytes (bf16): one-chunk
# rows, 4-byte vectors, and rows longer than a staging entry's share
@pytest.mark.parametrize("d,dtype", [(1, "f32"), (3, "f32"), (25, "f32"), (1000, "f32"), (50, "bf16")])
def test_staged_row_sizes(d, dtype, small_ring):
    prob, sched, w = workload_problem("cl10k", delta=2, gamma=0.8, d=d, dtype=dtype)
    rounds, pending = run_lookahead("staged async cl10k d=%d %s" % (d, dtype), prob, sched.seeds, 10, link="staged")
    assert rounds >= 3 and pending > 0


@pytest.mark.parametrize("threads", [1, 3])
def test_staged_gather_threads(threads, small_ring):
    prob, sched, w = workload_problem("cl10k", delta=3, gamma=0.8)
    rounds, _ = run_lookahead("staged threads=%d" % threads, prob, sched.seeds, 12, 3, link="staged",
                              link_threads=threads)
    assert rounds >= 2


def test_staged_no_halo():
    prob = tiny_problem(n_local=40, n_halo=0, p=0.2, seed=5, fanout=(4, 3), buffer_pct=25, delta=2)
    assert prob.H == 0
    rng = np.random.default_rng(5)
    seeds = [rng.permutation(prob.L)[:8].astype(np.int32) for _ in range(6)]
    rounds, hits, misses = run_parity("staged no halo", prob, lambda t: seeds[t], 6, gm=staged(prob))
    assert rounds == 0 and hits == 0 and misses == 0


def test_staged_timing_groups():
    # the worker's ranges: one per step with host rows, one per non-empty refill chunk
    prob, sched, w = workload_problem("cl10k", delta=2)
    gm = staged(prob)
    bb = gm.alloc_batch(w.batch)
    gm.set_timing(True)
    misses = 0
    for t in range(5):
        misses += gm.sample(to_dev(sched.seeds(t)), bb).host_rows > 0
        gm.evict_step()
    tim = gm.timing()
    log("staged timing %s" % tim)
    assert tim["gather_miss"][1] == misses and misses > 0 and tim["gather_miss"][0] > 0
    assert tim["refill"][1] >= 1 and tim["refill"][0] > 0
    assert tim["sample_dedup"][1] == 5 and tim["gather_hbm"][1] == 5


def test_staged_and_loads_give_the_same_bytes(small_ring):
    # the two modes side by side on one problem with rounds and look-ahead
    import torch
    prob, sched, w = workload_problem("cl10k", delta=2, gamma=0.8)
    ga, gb = make_gpu(prob), staged(prob)
    ba, bb = ga.alloc_batch(w.batch), gb.alloc_batch(w.batch)
    for t in range(10):
        s = to_dev(sched.seeds(t))
        ra, rb = ga.sample(s, ba), gb.sample(s, bb)
        assert (ra.n, ra.e, ra.hits, ra.misses, ra.host_rows) == (rb.n, rb.e, rb.hits, rb.misses, rb.host_rows), t
        n = ra.n[-1]
        assert torch.equal(ba.feat[:n], bb.feat[:n]), t
        assert ga.evict_step() == gb.evict_step(), t
    assert np.array_equal(ga.buffer_rows(), gb.buffer_rows())
    assert ga.counters() == gb.counters()
