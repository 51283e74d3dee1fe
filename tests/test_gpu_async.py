"""GPU parity of the look-ahead pipeline: massive_sample_async with two or three
batches in flight and eviction rounds enqueued without waiting, against the oracle
run step by step. With a short eviction interval on the products-sized graph
the refills (hundreds of thousands of rows over the host link) are still in
flight when the next steps classify, so hits on refilled slots are served
from the host store and written through into their slots (the refill then
skips them); the outputs and the buffer rows must not change."""
import numpy as np
import pytest

from gpu_util import compare_step, log, make_gpu, require_gpu, run_lookahead, to_dev
from helpers import workload_problem

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()


@pytest.mark.parametrize("depth", [2, 3])
def test_lookahead_cl10k(depth):
    prob, sched, w = workload_problem("cl10k", delta=3, gamma=0.8)
    assert run_lookahead("async cl10k depth %d" % depth, prob, sched.seeds, 24, depth)[0] >= 3


def test_lookahead_cl2m45_inflight_refills():
    prob, sched, w = workload_problem("cl2m45", delta=2)
    rounds, pending = run_lookahead("async cl2m45", prob, sched.seeds, 6)
    assert rounds == 2 and pending > 0  # hits on refilling slots were written through


@pytest.mark.parametrize("depth", [2, 3])
def test_lookahead_round_every_step(depth):
    # delta 1: a round after every step, each refill in one chunk that the
    # next round must flush first, with two or three batches in flight
    prob, sched, w = workload_problem("cl10k", delta=1, gamma=0.9)
    rounds, pending = run_lookahead("async cl10k delta 1 depth %d" % depth, prob, sched.seeds, 12, depth)
    assert rounds >= 8


def test_invalid_seeds_with_later_steps_in_flight():
    # a step whose seeds are invalid cannot be taken back once a later step
    # was issued: its wait reports the seeds, the batch issued after it is
    # refused (it ran at a step count the failed step had already advanced),
    # and the context refuses further work; every kernel completes normally
    from paper_2410_22697_amd import MassiveError
    prob, sched, w = workload_problem("cl10k")
    gm = make_gpu(prob)
    bbs = [gm.alloc_batch(w.batch) for _ in range(3)]
    seeds = [to_dev(sched.seeds(0)), to_dev(np.array([3, 3], np.int32)), to_dev(sched.seeds(2))]
    for t in range(3):
        gm.sample_async(seeds[t], bbs[t])
        gm.evict_step(wait=False)
    gm.wait(bbs[0])
    with pytest.raises(MassiveError) as ei:
        gm.wait(bbs[1])
    assert ei.value.code == -1
    with pytest.raises(MassiveError) as ei:
        gm.wait(bbs[2])
    assert ei.value.code == -5
    with pytest.raises(MassiveError) as ei:
        gm.sample_async(seeds[0], bbs[0])
    assert ei.value.code == -5


@pytest.mark.parametrize("order", ["in order", "later batch first"])
def test_failed_step_invalidates_later_batches(order, monkeypatch):
    # A step that fails on the device (here forced from the host: zero
    # threshold passes make every row longer than its fanout report a failed
    # search; every kernel still exits normally) skips its dedup scan and
    # classify, leaving bitmap marks and frontier positions set that later
    # steps sample against. The batch before it stays valid; the failed one
    # reports EHIP; every batch issued after it reports ESTATE, whichever is
    # waited for first; the context then refuses further work.
    from paper_2410_22697_amd import MassiveError
    prob, sched, w = workload_problem("cl10k")
    gm_ok = make_gpu(prob)
    monkeypatch.setenv("MASSIVE_TAU_ITERS", "0")
    gm = make_gpu(prob)
    monkeypatch.delenv("MASSIVE_TAU_ITERS")
    orc = prob.oracle()
    bbs = [gm.alloc_batch(w.batch) for _ in range(3)]
    seeds = [to_dev(sched.seeds(t)) for t in range(3)]
    # step 0 with an empty batch (nothing to sample: valid), then two full ones
    empty = to_dev(np.zeros(0, np.int32))
    log("failed step test (%s): enqueue" % order)
    gm.sample_async(empty, bbs[0])
    gm.evict_step(wait=False)
    for t in (1, 2):
        gm.sample_async(seeds[t], bbs[t])
        gm.evict_step(wait=False)
    res0 = gm.wait(bbs[0])
    st0 = orc.sample(np.zeros(0, np.int32))
    compare_step("failed-step test t=0", st0, res0, bbs[0], len(prob.fanout))
    if order == "in order":
        with pytest.raises(MassiveError) as ei:
            gm.wait(bbs[1])
        assert ei.value.code == -4
        with pytest.raises(MassiveError) as ei:
            gm.wait(bbs[2])
        assert ei.value.code == -5
    else:
        with pytest.raises(MassiveError) as ei:
            gm.wait(bbs[2])
        assert ei.value.code == -5
        with pytest.raises(MassiveError) as ei:
            gm.wait(bbs[1])
        assert ei.value.code == -4
    with pytest.raises(MassiveError) as ei:
        gm.sample_async(seeds[0], bbs[0])
    assert ei.value.code == -5
    gm.close()
    # a context made without the limit samples normally
    bb = gm_ok.alloc_batch(w.batch)
    orc2 = prob.oracle()
    compare_step("control t=0", orc2.sample(sched.seeds(0)), gm_ok.sample(seeds[0], bb), bb, len(prob.fanout))


def test_lookahead_rejects_one_batch_too_many():
    from paper_2410_22697_amd import MAX_INFLIGHT, MassiveError
    prob, sched, w = workload_problem("cl10k")
    gm = make_gpu(prob)
    n = MAX_INFLIGHT + 1
    bbs = [gm.alloc_batch(w.batch) for _ in range(n)]
    s = [to_dev(sched.seeds(t)) for t in range(n)]
    for t in range(MAX_INFLIGHT):
        gm.sample_async(s[t], bbs[t])
        gm.evict_step(wait=False)
    with pytest.raises(MassiveError) as ei:
        gm.sample_async(s[n - 1], bbs[n - 1])
    assert ei.value.code == -5
    # a batch still in flight cannot be enqueued again either
    gm.wait(bbs[0])
    with pytest.raises(MassiveError) as ei:
        gm.sample_async(s[n - 1], bbs[1])
    assert ei.value.code == -5
    for t in range(1, MAX_INFLIGHT):
        gm.wait(bbs[t])


# Rows of 4, 8, 12, 16, 100 and 4000 bytes (fp32) and 4 and 100 bytes (bf16):
# one-chunk rows, 4- and 8-byte vectors, and refill rows longer than a
# wavefront; every step after a round has hits on refilling slots.
@pytest.mark.parametrize("d,dtype", [(1, "f32"), (2, "f32"), (3, "f32"), (4, "f32"), (25, "f32"), (1000, "f32"),
                                     (2, "bf16"), (50, "bf16")])
def test_lookahead_row_sizes(d, dtype):
    prob, sched, w = workload_problem("cl10k", delta=2, gamma=0.8, d=d, dtype=dtype)
    assert w.row_bytes == d * (4 if dtype == "f32" else 2)
    rounds, pending = run_lookahead("async cl10k d=%d %s" % (d, dtype), prob, sched.seeds, 10)
    assert rounds >= 3 and pending > 0
