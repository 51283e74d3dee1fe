"""GPU parity with S_A kept over every global id (MASSIVE_SCORES_BY_GID, the
O(|V|) array of Section IV-B) instead of over the halo in rank order: the
same states, eviction and replacement sets as the oracle, element by element,
on the cases that stress the round (many rounds, fewer candidates than
evictions, no candidates, an empty buffer, a round every step, subnormal
scores, random tiny partitions); and the argument checks of that layout."""
import numpy as np
import pytest

from gpu_util import log, make_gpu, run_parity
from helpers import matched_problem, subnormal_order_schedule, tiny_problem, workload_problem

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    from gpu_util import require_gpu
    require_gpu()


def test_gid_layout_cl10k_full_run():
    prob, sched, w = workload_problem("cl10k")
    gm = make_gpu(prob, score_layout="gid", n_global=w.n)
    rounds, _, _ = run_parity("cl10k gid", prob, sched.seeds, w.steps, buffer_rows_every=5, gm=gm)
    assert rounds >= 5


@pytest.mark.parametrize("over", [dict(gamma=0.7, delta=2, buffer_pct=80),    # fewer candidates than evictions
                                  dict(buffer_pct=100, delta=2),                # no candidates
                                  dict(buffer_pct=0, delta=2),                  # empty buffer
                                  dict(gamma=0.9, delta=1)])                    # a round after every step
def test_gid_layout_cl10k_variants(over):
    prob, sched, w = workload_problem("cl10k", **over)
    gm = make_gpu(prob, score_layout="gid", n_global=w.n)
    run_parity("cl10k gid %s" % sorted(over.items()), prob, sched.seeds, 20, buffer_rows_every=4, gm=gm)


def test_gid_layout_cl170k_full_run():
    prob, sched, w = workload_problem("cl170k")
    gm = make_gpu(prob, score_layout="gid", n_global=w.n)
    rounds, _, _ = run_parity("cl170k gid", prob, sched.seeds, w.steps, state_every=8, buffer_rows_every=50, gm=gm)
    assert rounds >= 10


def test_gid_layout_subnormal_order():
    # the subnormal S_A ahead of a better-ranked S_A of 0 (three rounds), with
    # a global id space larger than the halo (ids 100..105 of 1000)
    prob = matched_problem([6, 5, 4, 3, 2, 1], buffer_pct=50, gamma=0.5, delta=140)
    gm = make_gpu(prob, score_layout="gid", n_global=1000)
    rounds, _, _ = run_parity("subnormal order gid", prob, subnormal_order_schedule(), 421, gm=gm, batch_max=3)
    assert rounds == 3


def test_gid_layout_random_tiny():
    total = 0
    for seed in range(12):
        rng = np.random.default_rng(100 + seed)
        prob = tiny_problem(n_local=int(rng.integers(3, 10)), n_halo=int(rng.integers(1, 14)), p=float(rng.uniform(0.2, 0.7)),
                            seed=seed, fanout=(2, 2), buffer_pct=int(rng.integers(0, 101)),
                            gamma=float(rng.uniform(0.3, 1.0)), delta=int(rng.integers(1, 4)))
        seeds = [rng.permutation(prob.L)[:int(rng.integers(0, prob.L + 1))].astype(np.int32) for _ in range(12)]
        gm = make_gpu(prob, score_layout="gid", n_global=1000)
        rounds, _, _ = run_parity("tiny gid %d" % seed, prob, lambda t: seeds[t], 12, gm=gm,
                                  batch_max=max(1, prob.L))
        total += rounds
    assert total >= 5


def test_gid_layout_argument_checks():
    from paper_2410_22697_amd import MassiveError
    prob, _, w = workload_problem("cl10k")
    log("gid layout: n_global below a halo id")
    with pytest.raises(MassiveError) as ei:
        make_gpu(prob, score_layout="gid", n_global=int(prob.halo_gid.max()))
    assert ei.value.code == -1 and "n_global" in str(ei.value)
    log("gid layout: a repeated halo id")
    bad = prob.halo_gid.copy()
    bad[1] = bad[0]
    from helpers import Problem
    import dataclasses
    with pytest.raises(MassiveError) as ei:
        make_gpu(dataclasses.replace(prob, halo_gid=bad), score_layout="gid", n_global=w.n)
    assert ei.value.code == -1 and "repeats" in str(ei.value)
