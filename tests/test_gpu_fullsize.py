"""Full-size checks on the papers-sized share (partition 0 of 64 of a
111M-node Chung-Lu graph: the workload and launch configuration the bench
times) and on the products-sized configurations (fp32 and the bf16 stress
setting). The whole-run oracle is too slow here (tens of seconds per step), so
every checked step is verified on outputs the oracle computes one by one and
on properties that hold at any size:
  * sampled rows: each checked row equals the oracle's choice for that row
    (several thousand rows per hop, the longest ones included);
  * dedup/relabel: the new nodes of each hop are exactly the ascending unique
    sampled ids not in the previous frontier;
  * masks: every row's class against the buffer as it stood before the step;
  * features: gathered bytes equal the source rows (local slab / host store);
  * scores: S_A += 1 on misses, S_E *= gamma (fp32) on unsampled slots;
  * an eviction round: E, the replacements (a numpy lexsort of the
    candidates), the score swap and the refilled rows.
The steps between checked ones run with look-ahead, as in the bench.
"""
import time

import numpy as np
import pytest

from gpu_util import log, require_gpu, to_dev

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(1200)]

_W = {}


def _inputs(name):
    if _W.get("name") != name:
        import torch
        import synth
        _W.clear()
        w = synth.get(name)
        t0 = time.time()
        log("generating %s" % w.name)
        g = synth.partition_graph(w)
        log("graph: L=%d H=%d nnz=%d (%.0fs)" % (g.L, g.H, g.nnz, time.time() - t0))
        rb = w.row_bytes
        local = np.empty((g.L, rb), np.uint8)
        synth.fill_features(g.local_gid, w.d, w.dtype, w.seed, local.ctypes.data)
        store = torch.empty((g.H, rb), dtype=torch.uint8, pin_memory=True)
        synth.fill_features(g.halo_gid, w.d, w.dtype, w.seed, store.data_ptr())
        log("features done (%.0fs)" % (time.time() - t0))
        _W.update(name=name, w=w, g=g, local=local, store=store,
                  sched=synth.Schedule(g.L, w.train_pct, w.batch, w.seed))
    return _W


def _check_step(tag, gm, bb, res, seeds, t, w, g, local, store_np, pre, rng):
    import oracle
    K = len(w.fanout)
    F = bb.nodes[:res.n[K]].cpu().numpy()
    assert len(np.unique(F)) == len(F), tag
    assert np.array_equal(F[:len(seeds)], seeds), tag
    deg = lambda v: g.indptr[v + 1] - g.indptr[v]  # noqa: E731
    for k in range(K):
        fo = w.fanout[k]
        n0, n1 = res.n[k], res.n[k + 1]
        ip = bb.indptr[k][:n0 + 1].cpu().numpy().astype(np.int64)
        ix = bb.indices[k][:res.e[k]].cpu().numpy()
        d = deg(F[:n0])
        assert np.array_equal(np.diff(ip), np.minimum(d, fo)), "%s hop %d row sizes" % (tag, k + 1)
        assert ix.min(initial=0) >= 0 and ix.max(initial=-1) < n1
        sampled = F[ix]
        new = np.setdiff1d(np.unique(sampled), F[:n0], assume_unique=True)
        assert np.array_equal(F[n0:n1], new), "%s hop %d new nodes" % (tag, k + 1)
        # rows the oracle recomputes one by one: a random sample plus the longest
        rows = np.union1d(rng.choice(n0, size=min(n0, 1500), replace=False), np.argsort(d)[-200:])
        for i in rows:
            want = oracle.sample_row(g.indptr, g.indices, int(F[i]), t, k + 1, fo, w.philox_seed)
            got = sampled[ip[i]:ip[i + 1]]
            assert np.array_equal(got, want), "%s hop %d row %d (d=%d)" % (tag, k + 1, i, d[i])
    # classes against the buffer before the step
    sid, se, sa = pre
    inbuf = np.zeros(g.H, bool)
    inbuf[sid] = True
    mask = bb.mask[:res.n[K]].cpu().numpy()
    halo = F >= g.L
    want = np.where(~halo, 0, np.where(inbuf[np.where(halo, F - g.L, 0)], 1, 2)).astype(np.uint8)
    assert np.array_equal(mask, want), tag + " mask"
    assert (res.local, res.hits, res.misses) == (int((~halo).sum()), int((want == 1).sum()), int((want == 2).sum()))
    # gathered rows (a random subset of 40K rows)
    pick = rng.choice(len(F), size=min(len(F), 40000), replace=False)
    feat = bb.feat[:res.n[K]].cpu().numpy()[pick]
    v = F[pick]
    src = np.where((v < g.L)[:, None], local[np.minimum(v, g.L - 1)], store_np[np.maximum(v - g.L, 0)])
    assert np.array_equal(feat, src), tag + " feat"
    # scores after the step
    sid2, se2, sa2, _ = gm.state()
    assert np.array_equal(sid2, sid)
    miss_h = F[mask == 2] - g.L
    sa_want = sa.copy()
    sa_want[miss_h] += np.float32(1.0)
    assert np.array_equal(sa2, sa_want), tag + " S_A"
    hit_slots = np.zeros(g.H, bool)
    hit_slots[F[mask == 1] - g.L] = True
    used = hit_slots[sid]
    se_want = np.where(used, se, (se * np.float32(w.gamma)).astype(np.float32)).astype(np.float32)
    assert np.array_equal(se2.view(np.uint32), se_want.view(np.uint32)), tag + " S_E"


# (workload, steps checked one by one, the round step whose selection is checked)
CASES = [("cl111m_p64", (0, 1, 2, 31, 32, 33), 32),    # papers-sized share, delta 32
         ("cl2m45", (0, 1, 31, 32, 33), 32),            # products-sized, delta 32, 7 minibatches per epoch
         ("cl2m45_bf16", (0, 1, 3, 4, 5, 8, 9), 4)]     # bf16 rows, f 50%, gamma 0.8, delta 4, batch 4096


@pytest.mark.parametrize("name,checked,round_t", CASES)
def test_full_size(name, checked, round_t):
    require_gpu()
    import torch
    from paper_2410_22697_amd import Massive
    W = _inputs(name)
    w, g, local, store, sched = W["w"], W["g"], W["local"], W["store"], W["sched"]
    store_np = store.numpy()
    gm = Massive(g.L, g.H, g.indptr, g.indices, g.halo_gid, g.halo_degree, local, store, w.row_bytes,
                 w.fanout, w.buffer_pct, w.gamma, w.delta, w.philox_seed)
    rng = np.random.default_rng(0)
    order = np.lexsort((g.halo_gid, -g.halo_degree))
    rank = np.empty(g.H, np.int64)
    rank[order] = np.arange(g.H)
    sid0, _, _, _ = gm.state()
    assert np.array_equal(sid0, order[:gm.cap])
    assert np.array_equal(gm.buffer_rows()[:: max(1, gm.cap // 20000)],
                          store_np[sid0[:: max(1, gm.cap // 20000)]])
    bbs = [gm.alloc_batch(w.batch), gm.alloc_batch(w.batch)]
    checked = set(checked)
    last = max(checked) + 1
    cap = gm.cap
    ev, sl, rp = (torch.empty(cap, dtype=torch.int32, device="cuda") for _ in range(3))
    t = 0
    while t < last:
        seeds = sched.seeds(t)
        if t in checked:
            pre = gm.state()[:3]
            log("full size t=%d: checked step" % t)
            res = gm.sample(to_dev(seeds), bbs[0])
            _check_step("t=%d" % t, gm, bbs[0], res, seeds, t, w, g, local, store_np, pre, rng)
            if t == round_t:
                sid, se, sa, _ = gm.state()
                k = gm.evict_step((ev, sl, rp))
                E = np.nonzero(se < np.float32(gm.alpha))[0]
                cand = np.nonzero(sa >= 0)[0]
                cand = cand[np.lexsort((rank[cand], -sa[cand]))]
                kk = min(len(E), len(cand))
                assert k == kk and k > 0
                assert np.array_equal(sl[:k].cpu().numpy(), E[:k])
                assert np.array_equal(ev[:k].cpu().numpy(), sid[E[:k]])
                R = rp[:k].cpu().numpy()
                assert np.array_equal(R, cand[:k])
                sid2, se2, sa2, _ = gm.state()
                assert np.array_equal(sa2[sid[E]], se[E]) and np.array_equal(se2[E], sa[R])
                assert np.all(sa2[R] == -1.0) and np.array_equal(sid2[E], R)
                rows = gm.buffer_rows()
                probe = rng.choice(cap, size=20000, replace=False)
                assert np.array_equal(rows[probe], store_np[sid2[probe]])
                log("round t=%d: %d slots evicted and refilled" % (t, k))
            else:
                k = gm.evict_step()
                assert k == 0 or (t > 0 and t % w.delta == 0)
            t += 1
            continue
        # look-ahead run up to the next checked step
        stop = min(x for x in checked | {last} if x > t)
        log("full size t=%d..%d: look-ahead" % (t, stop - 1))
        for u in range(t, stop + 1):
            if u < stop:
                gm.sample_async(to_dev(sched.seeds(u)), bbs[u % 2])
                gm.evict_step(wait=False)
            if u > t:
                gm.wait(bbs[(u - 1) % 2])
        t = stop
    log("full size: done")
