"""massive_sample_noalloc (the entry point for callers that cannot allocate)
against massive_sample: the same step, element by element, with its per-step
scratch in the library's static device array instead of the context's
buffers. Two calls in a row, the second with a smaller batch; contexts of
different graphs sharing the one array; the no-alloc step between ordinary
ones; and the size limit."""
import numpy as np
import pytest

from gpu_util import log, make_gpu, pinned_store, require_gpu, to_dev
from helpers import Problem, workload_problem

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()


def _outputs(res, bb, K):
    nK = res.n[-1]
    return dict(sizes=(res.n, res.e, res.local, res.hits, res.misses, res.host_rows),
                nodes=bb.nodes[:nK].cpu().numpy().copy(), mask=bb.mask[:nK].cpu().numpy().copy(),
                feat=bb.feat[:nK].cpu().numpy().copy(),
                indptr=[bb.indptr[k][:res.n[k] + 1].cpu().numpy().copy() for k in range(K)],
                indices=[bb.indices[k][:res.e[k]].cpu().numpy().copy() for k in range(K)])


def _assert_same(tag, a, b):
    assert a["sizes"] == b["sizes"], (tag, a["sizes"], b["sizes"])
    for key in ("nodes", "mask", "feat"):
        assert np.array_equal(a[key], b[key]), (tag, key)
    for k, (x, y) in enumerate(zip(a["indptr"], b["indptr"])):
        assert np.array_equal(x, y), (tag, "indptr", k)
    for k, (x, y) in enumerate(zip(a["indices"], b["indices"])):
        assert np.array_equal(x, y), (tag, "indices", k)


def _assert_same_state(tag, g1, g2):
    s1, s2 = g1.state(), g2.state()
    assert s1[3] == s2[3], tag
    assert np.array_equal(s1[0], s2[0]), tag + " slot_id"
    assert np.array_equal(s1[1].view(np.uint32), s2[1].view(np.uint32)), tag + " S_E"
    assert np.array_equal(s1[2].view(np.uint32), s2[2].view(np.uint32)), tag + " S_A"


def _pair(name, **over):
    prob, sched, w = workload_problem(name, **over)
    store = pinned_store(prob)
    ref, na = make_gpu(prob, store=store), make_gpu(prob, store=store)
    return prob, sched, w, store, ref, na, ref.alloc_batch(w.batch), na.alloc_batch(w.batch)


def test_noalloc_matches_sample_second_call_smaller():
    # products-sized graph (frontiers of ~200K rows, many scan tiles; 1000
    # seeds keep the frontier bound, 1,056,000 rows, inside the array), a round
    # after every step so that refill chunks run beside the no-alloc steps
    prob, sched, w, store, ref, na, bb_ref, bb_na = _pair("cl2m45", delta=1, gamma=0.8)
    K = len(prob.fanout)
    for t, seeds in enumerate([sched.seeds(0)[:1000], sched.seeds(1)[:300]]):
        log("no-alloc cl2m45 t=%d n0=%d" % (t, len(seeds)))
        r_ref = ref.sample(to_dev(seeds), bb_ref)
        r_na = na.sample_noalloc(to_dev(seeds), bb_na)
        _assert_same("cl2m45 t=%d" % t, _outputs(r_ref, bb_ref, K), _outputs(r_na, bb_na, K))
        assert ref.evict_step() == na.evict_step()
        _assert_same_state("cl2m45 t=%d" % t, ref, na)
    assert np.array_equal(ref.buffer_rows(), na.buffer_rows())


def test_noalloc_contexts_share_the_array():
    # two graphs interleaved on one GPU: each call clears what the other left
    # in the array (sizes, scan flags), and ordinary steps of the same context
    # (their own buffers and scan epochs) sit between no-alloc ones
    a = _pair("cl10k", delta=2)
    b = _pair("cl170k", delta=3)
    plan = [(a, "na"), (b, "na"), (a, "na"), (b, "sample"), (a, "sample"), (b, "na"), (a, "na"), (b, "na")]
    steps = {id(a): 0, id(b): 0}
    for i, (p, kind) in enumerate(plan):
        prob, sched, w, store, ref, na, bb_ref, bb_na = p
        K = len(prob.fanout)
        t = steps[id(p)]
        seeds = sched.seeds(t) if i % 3 else sched.seeds(t)[: max(1, len(sched.seeds(t)) // 4)]
        log("shared array: %s t=%d %s n0=%d" % ("cl10k" if p is a else "cl170k", t, kind, len(seeds)))
        r_ref = ref.sample(to_dev(seeds), bb_ref)
        r_na = na.sample_noalloc(to_dev(seeds), bb_na) if kind == "na" else na.sample(to_dev(seeds), bb_na)
        _assert_same("plan %d" % i, _outputs(r_ref, bb_ref, K), _outputs(r_na, bb_na, K))
        assert ref.evict_step() == na.evict_step()
        steps[id(p)] = t + 1
    for p in (a, b):
        _assert_same_state("shared array end", p[4], p[5])


def test_noalloc_size_limit():
    # 1.4M isolated local nodes: a batch of 1.4M seeds has a frontier bound
    # above the array's 1,310,720 rows and is refused; massive_sample takes it
    from paper_2410_22697_amd import MassiveError
    n = 1_400_000
    rng = np.random.default_rng(0)
    feats = rng.standard_normal((n, 1)).astype(np.float32)
    prob = Problem(n, 0, np.zeros(n + 1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.int32),
                   np.zeros(0, np.int64), feats, np.zeros((0, 1), np.float32), 1, "f32", (1,), 25, 0.9, 4)
    gm = make_gpu(prob)
    bb = gm.alloc_batch(n)
    seeds = to_dev(rng.permutation(n).astype(np.int32))
    with pytest.raises(MassiveError) as ei:
        gm.sample_noalloc(seeds, bb)
    assert ei.value.code == -2 and "no-alloc" in str(ei.value)
    r = gm.sample(seeds, bb)
    assert r.n == [n, n] and r.e == [0] and r.local == n
    gm.evict_step()
    small = to_dev(np.arange(1000, dtype=np.int32))
    r2 = gm.sample_noalloc(small, bb)
    assert r2.n == [1000, 1000] and np.array_equal(bb.nodes[:1000].cpu().numpy(), np.arange(1000))
    assert np.array_equal(bb.feat[:1000].cpu().numpy(), feats[:1000].view(np.uint8))
