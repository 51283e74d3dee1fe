"""GPU parity: libmassive (through the C ABI) against the oracle, element by
element: sampled blocks, frontier, masks, gathered rows, eviction sets and
scores. Sizes span several tiles and ragged tails; the oracle finishes each in
seconds."""
import numpy as np
import pytest

from gpu_util import log, make_gpu, pinned_store, require_gpu, run_parity, to_dev
from helpers import matched_problem, subnormal_order_schedule, tiny_problem, workload_problem

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()


def test_tiny_graphs():
    total = 0
    for seed in (1, 2, 3):
        prob = tiny_problem(n_local=6, n_halo=9, p=0.4, seed=seed, fanout=(2, 1), buffer_pct=34, delta=2, gamma=0.5)
        rng = np.random.default_rng(seed)
        seeds = [rng.permutation(prob.L)[:1].astype(np.int32) for _ in range(16)]
        rounds, _, _ = run_parity("tiny%d" % seed, prob, lambda t: seeds[t], 16)
        total += rounds
    assert total >= 3


def test_cl10k_full_run():
    prob, sched, w = workload_problem("cl10k")
    rounds, _, _ = run_parity("cl10k", prob, sched.seeds, w.steps, buffer_rows_every=5)
    assert rounds >= 5


@pytest.mark.parametrize("over", [dict(gamma=0.8, delta=3, buffer_pct=50),
                                  dict(gamma=0.7, delta=2, buffer_pct=80),    # fewer candidates than evictions
                                  dict(buffer_pct=100, delta=2),                # no candidates at all
                                  dict(buffer_pct=0, delta=2),                  # empty buffer
                                  dict(gamma=1.0, delta=2),                     # nothing ever decays below alpha
                                  dict(fanout=(40, 30, 2), delta=5),            # rows up to 320 long, long-row path
                                  dict(gamma=0.9, delta=1)])                    # a round after every step
def test_cl10k_variants(over):
    prob, sched, w = workload_problem("cl10k", **over)
    run_parity("cl10k%s" % sorted(over.items()), prob, sched.seeds, 20, buffer_rows_every=4)


def test_cl170k_full_run():
    # the whole stated run: 200 minibatches (11 per epoch), rounds every 16
    prob, sched, w = workload_problem("cl170k")
    rounds, _, _ = run_parity("cl170k", prob, sched.seeds, w.steps, state_every=8, buffer_rows_every=50)
    assert rounds >= 10


def test_cl2m45_short_interval():
    # products-sized graph, 3 hops, hub rows of ~11K neighbours; delta lowered
    # so that two rounds fit in a short run.
    prob, sched, w = workload_problem("cl2m45", delta=2)
    rounds, _, _ = run_parity("cl2m45", prob, sched.seeds, 5, state_every=2)
    assert rounds == 2


def test_cl2m45_bf16_rows():
    # 200-byte bf16 rows (8-byte vectors), fanout (20,15,10), f = 50%, gamma 0.8;
    # batch lowered to keep the oracle within seconds.
    prob, sched, w = workload_problem("cl2m45_bf16", batch=512)
    from synth import Schedule
    sch = Schedule(prob.L, w.train_pct, 512, w.seed)
    rounds, _, _ = run_parity("cl2m45_bf16", prob, sch.seeds, 5, state_every=2)
    assert rounds == 1


@pytest.mark.timeout(900)
def test_cl2m45_bf16_stated_batch():
    # the stated shape: batch 4096, fanout (20,15,10), bf16 rows, f 50%,
    # gamma 0.8, Delta 4; every step element by element through the first
    # round (after t = 4) and two steps after it (the oracle takes ~10 s a step)
    prob, sched, w = workload_problem("cl2m45_bf16")
    assert w.batch == 4096
    rounds, _, _ = run_parity("cl2m45_bf16 batch 4096", prob, sched.seeds, 7, state_every=1, buffer_rows_every=4)
    assert rounds == 1


def _subnormals(x):
    return int(((x > 0) & (x < np.float32(2.0 ** -126))).sum())


def test_subnormal_scores_cl10k():
    # gamma 0.3, Delta 80: alpha = 0.3^80 is subnormal, unsampled slots' S_E
    # pass through 2^-126..2^-149 to 0, and the round at t = 160 moves
    # subnormal S_E into S_A (the swap of Section IV-B). S_E and S_A bits are
    # compared after every one of 241 steps (rounds at 80, with nothing below
    # alpha yet, 160 and 240).
    prob, sched, w = workload_problem("cl10k", gamma=0.3, delta=80)
    orc, gm = prob.oracle(), make_gpu(prob)
    assert 0 < np.float32(orc.alpha) < np.float32(2.0 ** -126)
    r1, _, _ = run_parity("cl10k subnormal", prob, sched.seeds, 161, gm=gm, orc=orc)
    _, se, sa = orc.state()
    assert r1 >= 1 and _subnormals(se) > 0 and _subnormals(sa) > 0
    r2, _, _ = run_parity("cl10k subnormal, steps 161-240", prob, lambda t: sched.seeds(161 + t), 80, gm=gm, orc=orc)
    assert r2 >= 1


def test_subnormal_S_A_outranks_zero():
    # a candidate whose S_A is subnormal (2^-141, from a swap) must be chosen
    # ahead of a better-ranked candidate whose S_A is exactly 0: the three
    # rounds of helpers.subnormal_order_schedule, state bits after every step
    prob = matched_problem([6, 5, 4, 3, 2, 1], buffer_pct=50, gamma=0.5, delta=140)
    orc, gm = prob.oracle(), make_gpu(prob)
    rounds, _, _ = run_parity("subnormal order", prob, subnormal_order_schedule(), 421, gm=gm, orc=orc,
                              batch_max=3)
    assert rounds == 3
    sid, se, _, _ = gm.state()
    assert sid.tolist() == [5, 3, 1] and int(se.view(np.uint32)[2]) == 1 << 8


def test_empty_and_ragged_batches():
    prob, sched, w = workload_problem("cl10k", delta=2)
    sizes = [0, 1, 63, 64, 65, 250, 0, 7, 129, 1]
    rng = np.random.default_rng(5)
    seeds = [rng.permutation(prob.L)[:n].astype(np.int32) for n in sizes]
    run_parity("cl10k ragged", prob, lambda t: seeds[t], len(sizes), batch_max=250)


def test_invalid_seeds_leave_state_unchanged():
    from paper_2410_22697_amd import MassiveError
    prob, sched, w = workload_problem("cl10k")
    gm = make_gpu(prob)
    orc = prob.oracle()
    bb = gm.alloc_batch(256)
    for bad in ([prob.L], [-1], [3, 3]):
        log("invalid seeds %s" % bad)
        with pytest.raises(MassiveError) as ei:
            gm.sample(to_dev(np.array(bad, np.int32)), bb)
        assert ei.value.code == -1
    log("valid step after the rejections")
    from gpu_util import compare_step
    st = orc.sample(sched.seeds(0))
    res = gm.sample(to_dev(sched.seeds(0)), bb)
    compare_step("after invalid", st, res, bb, len(prob.fanout))
    with pytest.raises(MassiveError) as ei:
        gm.sample(to_dev(sched.seeds(1)), bb)         # evict call is owed first
    assert ei.value.code == -5


def test_output_capacity_is_checked():
    from paper_2410_22697_amd import MassiveError
    prob, sched, w = workload_problem("cl10k")
    gm = make_gpu(prob)
    bb = gm.alloc_batch(100)
    with pytest.raises(MassiveError) as ei:
        gm.sample(to_dev(sched.seeds(0)), bb)         # 250 seeds > bound of 100
    assert ei.value.code == -2


def test_deterministic_bytes():
    import torch
    prob, sched, w = workload_problem("cl170k")
    outs = []
    store = pinned_store(prob)
    for rep in range(2):
        log("determinism run %d" % rep)
        gm = make_gpu(prob, store=store)
        bb = gm.alloc_batch(w.batch)
        digest = []
        for t in range(18):
            r = gm.sample(to_dev(sched.seeds(t)), bb)
            nK = r.n[-1]
            digest.append((bb.nodes[:nK].cpu().numpy().tobytes(), bb.feat[:nK].cpu().numpy().tobytes(),
                           bb.indices[2][:r.e[2]].cpu().numpy().tobytes(), bb.mask[:nK].cpu().numpy().tobytes()))
            gm.evict_step()
        sid, se, sa, _ = gm.state()
        outs.append((digest, sid.tobytes(), se.tobytes(), sa.tobytes()))
        gm.close()
        torch.cuda.synchronize()
    assert outs[0] == outs[1]
