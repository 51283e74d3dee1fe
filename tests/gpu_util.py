"""Shared driver for the GPU parity tests: the HIP path (through the C ABI)
against the oracle, step by step, on the same seeded inputs."""
import sys
import time

import numpy as np
import pytest

from helpers import Problem


def require_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2410_22697_amd import massive
    massive.load()  # raises if the HIP library is missing: no fallback


def log(msg):
    print("[gpu] " + msg, flush=True)
    sys.stdout.flush()


def pinned_store(prob: Problem):
    import torch
    hs = np.ascontiguousarray(prob.halo_store).view(np.uint8).reshape(prob.H, prob.row_bytes)
    t = torch.empty((max(prob.H, 1), prob.row_bytes), dtype=torch.uint8, pin_memory=True)
    if prob.H:
        t[:prob.H].copy_(torch.from_numpy(hs))
    return t


def make_gpu(prob: Problem, store=None, **over):
    """A context on prob; over may set fanout, buffer_pct, gamma, delta, seed,
    score_layout ("rank" or "gid", with n_global) and link ("loads" or
    "staged", with link_threads)."""
    from paper_2410_22697_amd import Massive
    kw = dict(fanout=prob.fanout, buffer_pct=prob.buffer_pct, gamma=prob.gamma, delta=prob.delta, seed=prob.seed,
              score_layout="rank", n_global=0, link="loads", link_threads=0)
    kw.update(over)
    if store is None:
        store = pinned_store(prob)
    lf = np.ascontiguousarray(prob.local_feat).view(np.uint8).reshape(prob.L, prob.row_bytes)
    return Massive(prob.L, prob.H, prob.indptr, prob.indices, prob.halo_gid, prob.halo_degree, lf, store,
                   prob.row_bytes, kw["fanout"], kw["buffer_pct"], kw["gamma"], kw["delta"], kw["seed"],
                   score_layout=kw["score_layout"], n_global=kw["n_global"], link=kw["link"],
                   link_threads=kw["link_threads"])


def to_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()


def compare_step(tag, st, res, bb, K):
    """Element-by-element equality of one step's outputs."""
    assert res.n == st.n, (tag, res.n, st.n)
    assert res.e == st.e, (tag, res.e, st.e)
    assert (res.local, res.hits, res.misses) == (st.local, st.hits, st.misses), tag
    nK = st.n[K]
    assert np.array_equal(bb.nodes[:nK].cpu().numpy(), st.nodes), tag + " nodes"
    for k in range(K):
        assert np.array_equal(bb.indptr[k][:st.n[k] + 1].cpu().numpy(), st.indptr[k]), "%s indptr hop %d" % (tag, k + 1)
        assert np.array_equal(bb.indices[k][:st.e[k]].cpu().numpy(), st.indices[k]), "%s indices hop %d" % (tag, k + 1)
    assert np.array_equal(bb.mask[:nK].cpu().numpy(), st.mask), tag + " mask"
    assert np.array_equal(bb.feat[:nK].cpu().numpy(), st.feat), tag + " feat"


def compare_state(tag, orc, gm, exact_scores=True):
    sid_o, se_o, sa_o = orc.state()
    sid_g, se_g, sa_g, t_g = gm.state()
    assert t_g == orc.t, tag
    assert np.array_equal(sid_g, sid_o), tag + " slot_id"
    # scores: fp32 within 1e-5 relative (in practice bit-exact: same fp32 products)
    np.testing.assert_allclose(se_g, se_o, rtol=1e-5, atol=0, err_msg=tag + " S_E")
    np.testing.assert_allclose(sa_g, sa_o, rtol=1e-5, atol=0, err_msg=tag + " S_A")
    if exact_scores:
        assert np.array_equal(se_g.view(np.uint32), se_o.view(np.uint32)), tag + " S_E bits"
        assert np.array_equal(sa_g.view(np.uint32), sa_o.view(np.uint32)), tag + " S_A bits"


def run_parity(name, prob: Problem, seeds_of, steps, state_every=1, buffer_rows_every=0, gm=None, orc=None,
               batch_max=None):
    """Runs `steps` steps on both sides; returns (rounds with k > 0, hits, misses)."""
    import torch
    orc = orc or prob.oracle()
    gm = gm or make_gpu(prob)
    K = len(prob.fanout)
    if batch_max is None:
        batch_max = max(len(seeds_of(t)) for t in range(steps))
    bb = gm.alloc_batch(batch_max)
    cap = gm.cap
    assert cap == orc.cap and np.float32(gm.alpha) == np.float32(orc.alpha)
    compare_state(name + " init", orc, gm)
    ev, sl, rp = (torch.empty(max(cap, 1), dtype=torch.int32, device="cuda") for _ in range(3))
    rounds = hits = misses = 0
    t0 = time.time()
    for t in range(steps):
        seeds = seeds_of(t)
        tag = "%s t=%d n0=%d" % (name, t, len(seeds))
        st = orc.sample(seeds)
        log(tag + " sample")
        res = gm.sample(to_dev(seeds), bb)
        compare_step(tag, st, res, bb, K)
        hits += st.hits
        misses += st.misses
        ro = orc.evict_step()
        k = gm.evict_step((ev, sl, rp))
        assert k == ro.k, (tag, k, ro.k)
        if k:
            rounds += 1
            assert np.array_equal(sl[:k].cpu().numpy(), ro.slots), tag + " slots"
            assert np.array_equal(ev[:k].cpu().numpy(), ro.evicted), tag + " evicted"
            assert np.array_equal(rp[:k].cpu().numpy(), ro.replaced), tag + " replaced"
        if state_every and (t % state_every == 0 or k or t == steps - 1):
            compare_state(tag, orc, gm)
        if buffer_rows_every and (t % buffer_rows_every == 0 or k):
            assert np.array_equal(gm.buffer_rows(), orc.buffer_rows()), tag + " buffer rows"
    log("%s: %d steps, %d rounds, hit rate %.3f, %.1fs" % (name, steps, rounds, hits / max(hits + misses, 1),
                                                           time.time() - t0))
    return rounds, hits, misses


def run_lookahead(name, prob, seeds_of, steps, depth=None, **over):
    """Steps 0..steps-1 with `depth` batches in flight (step t is enqueued
    before step t - depth + 1 is waited for), against the oracle step by
    step; `over` goes to make_gpu. Returns (rounds, pending hits served over
    the host link)."""
    import torch
    from paper_2410_22697_amd import MAX_INFLIGHT
    depth = depth or MAX_INFLIGHT
    orc = prob.oracle()
    gm = make_gpu(prob, **over)
    K = len(prob.fanout)
    batch_max = max(len(seeds_of(t)) for t in range(steps))
    bbs = [gm.alloc_batch(batch_max) for _ in range(depth)]
    cap = gm.cap
    outs = [tuple(torch.full((max(cap, 1),), -7, dtype=torch.int32, device="cuda") for _ in range(3))
            for _ in range(steps)]
    seeds_dev = [to_dev(seeds_of(t)) for t in range(steps)]
    rounds_o, evicted_o = [], 0
    pending = []

    def check(t):
        res = gm.wait(bbs[t % depth])
        pending.append(res.host_rows - res.misses)
        st = orc.sample(seeds_of(t))
        compare_step("%s t=%d" % (name, t), st, res, bbs[t % depth], K)
        ro = orc.evict_step()
        rounds_o.append(ro)
        return ro.k

    for t in range(steps):
        log("%s t=%d enqueue" % (name, t))
        gm.sample_async(seeds_dev[t], bbs[t % depth])
        gm.evict_step(outs[t], wait=False)
        if t >= depth - 1:
            evicted_o += check(t - depth + 1)
    for t in range(max(0, steps - depth + 1), steps):
        evicted_o += check(t)
    torch.cuda.synchronize()
    n_rounds = 0
    for t, ro in enumerate(rounds_o):
        if ro.k:
            n_rounds += 1
            ev, sl, rp = (x[:ro.k].cpu().numpy() for x in outs[t])
            assert np.array_equal(sl, ro.slots) and np.array_equal(ev, ro.evicted) and np.array_equal(rp, ro.replaced), t
    compare_state(name + " end", orc, gm)
    assert np.array_equal(gm.buffer_rows(), orc.buffer_rows())
    assert gm.counters() == (n_rounds, evicted_o)
    # the refill copies each replacement at most once, and none a miss gather wrote through
    assert cap <= gm.refilled_rows() <= cap + evicted_o
    log("%s: %d steps, %d rounds, %d evicted, pending hits per step %s" % (name, steps, n_rounds, evicted_o, pending))
    assert min(pending) >= 0
    return n_rounds, sum(pending)
