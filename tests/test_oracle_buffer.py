"""Pins for the oracle's prefetch buffer: initialisation, scoring, eviction.

Closed forms used (Algorithm 1/2, Section IV-B, Eq. 1):
  * init: BUF = the cap highest-ranked halo nodes (numpy lexsort), S_E = 1,
    S_A = -1 on BUF and 0 elsewhere, alpha = gamma^Delta (fp32 products);
  * before the first round, S_A[h] of an unbuffered node equals the number of
    steps in which it was sampled, and S_E[s] equals gamma applied once per
    step in which the slot's node was not sampled;
  * the first round evicts exactly the initial slots never sampled in steps
    0..Delta, and picks replacements as a lexsort prefix of (S_A desc, rank);
  * gamma = 1 never evicts; f = 0 never hits; Delta beyond the run is a
    static cache;
plus invariants after every step of a long run and an independent Python
replay of the policy over several rounds.
"""
import numpy as np
import pytest

from helpers import fp32_decay, rank_order, tiny_problem, workload_problem


def _halo_sets(prob, nodes):
    return set((nodes[nodes >= prob.L] - prob.L).tolist())


def _check_gather(prob, st):
    b = prob.row_bytes
    lf = prob.local_feat.view(np.uint8).reshape(prob.L, b)
    hs = prob.halo_store.view(np.uint8).reshape(prob.H, b)
    v = st.nodes
    loc = v < prob.L
    assert np.array_equal(st.feat[loc], lf[v[loc]])
    assert np.array_equal(st.feat[~loc], hs[v[~loc] - prob.L])


def test_initial_state():
    prob, _, w = workload_problem("cl10k")
    orc = prob.oracle()
    cap = prob.H * prob.buffer_pct // 100
    assert orc.cap == cap
    sid, se, sa = orc.state()
    order = rank_order(prob)
    assert np.array_equal(sid, order[:cap])
    assert np.all(se == np.float32(1.0))
    want = np.zeros(prob.H, np.float32)
    want[order[:cap]] = -1.0
    assert np.array_equal(sa, want)
    assert np.float32(orc.alpha) == fp32_decay(1.0, prob.gamma, prob.delta)
    # the rank the oracle reports is the inverse of that order
    r = orc.rank()
    assert np.array_equal(r[order], np.arange(prob.H))


@pytest.mark.parametrize("name_over", [("cl10k", {}), ("cl10k", {"gamma": 0.8, "delta": 3})])
def test_first_round_closed_form(name_over):
    name, over = name_over
    prob, sched, w = workload_problem(name, **over)
    orc = prob.oracle()
    cap, L, D = orc.cap, prob.L, prob.delta
    order = rank_order(prob)
    init_buf = order[:cap]
    in_buf = np.zeros(prob.H, bool)
    in_buf[init_buf] = True
    seen_count = np.zeros(prob.H, np.int64)
    for t in range(D + 1):
        st = orc.sample(sched.seeds(t))
        halo = st.nodes[st.nodes >= L] - L
        # mask against the initial buffer (no round has run yet)
        want = np.where(st.nodes < L, 0, np.where(in_buf[np.maximum(st.nodes - L, 0)], 1, 2))
        assert np.array_equal(st.mask, want.astype(np.uint8))
        assert st.hits == int(in_buf[halo].sum()) and st.misses == int((~in_buf[halo]).sum())
        _check_gather(prob, st)
        seen_count[halo] += 1
        if t < D:
            assert orc.evict_step().k == 0
    sid, se, sa = orc.state()
    want_sa = np.where(in_buf, -1.0, seen_count).astype(np.float32)
    assert np.array_equal(sa, want_sa)
    unused = (D + 1) - seen_count[init_buf]
    want_se = np.array([fp32_decay(1.0, prob.gamma, int(u)) for u in unused], np.float32)
    assert np.array_equal(se, want_se)

    rnd = orc.evict_step()
    never = np.nonzero(seen_count[init_buf] == 0)[0]
    cand = np.nonzero(sa >= 0)[0]
    rk = orc.rank()
    cand_sorted = cand[np.lexsort((rk[cand], -sa[cand]))]
    k = min(len(never), len(cand))
    assert rnd.k == k
    assert np.array_equal(rnd.slots, never[:k])
    assert np.array_equal(rnd.evicted, init_buf[never[:k]])
    assert np.array_equal(rnd.replaced, cand_sorted[:k])
    sid2, se2, sa2 = orc.state()
    assert np.array_equal(sa2[rnd.evicted], se[rnd.slots])       # S_A := last S_E
    assert np.array_equal(se2[rnd.slots], sa[rnd.replaced])      # S_E := last S_A
    assert np.all(sa2[rnd.replaced] == -1.0)
    assert np.array_equal(sid2[rnd.slots], rnd.replaced)
    keep = np.setdiff1d(np.arange(cap), rnd.slots)
    assert np.array_equal(sid2[keep], sid[keep]) and np.array_equal(se2[keep], se[keep])
    # refilled rows are the replacements' store rows
    hs = prob.halo_store.view(np.uint8).reshape(prob.H, prob.row_bytes)
    assert np.array_equal(orc.buffer_rows(), hs[sid2])


def test_gamma_one_never_evicts():
    prob, sched, w = workload_problem("cl10k", gamma=1.0)
    orc = prob.oracle()
    sid0, _, _ = orc.state()
    for t in range(3 * prob.delta + 1):
        orc.sample(sched.seeds(t))
        assert orc.evict_step().k == 0
    sid, se, _ = orc.state()
    assert np.array_equal(sid, sid0) and np.all(se == 1.0)


def test_empty_buffer_never_hits():
    prob, sched, w = workload_problem("cl10k", buffer_pct=0)
    orc = prob.oracle()
    assert orc.cap == 0
    for t in range(2 * prob.delta + 1):
        st = orc.sample(sched.seeds(t))
        assert st.hits == 0 and st.misses == int((st.nodes >= prob.L).sum())
        assert orc.evict_step().k == 0


def test_long_interval_is_static_cache():
    prob, sched, w = workload_problem("cl10k", delta=1000)
    orc = prob.oracle()
    sid0, _, _ = orc.state()
    for t in range(20):
        orc.sample(sched.seeds(t))
        assert orc.evict_step().k == 0
    assert np.array_equal(orc.state()[0], sid0)


def test_full_buffer_has_no_candidates():
    prob, sched, w = workload_problem("cl10k", buffer_pct=100)
    orc = prob.oracle()
    for t in range(2 * prob.delta + 1):
        st = orc.sample(sched.seeds(t))
        assert st.misses == 0
        assert orc.evict_step().k == 0


def _replay(prob, steps, orc_rank):
    """Independent replay of the buffer policy from the sampled frontiers."""
    L, H = prob.L, prob.H
    cap = H * prob.buffer_pct // 100
    order = np.argsort(orc_rank, kind="stable")
    slot = [int(h) for h in order[:cap]]
    SE = [np.float32(1.0)] * cap
    SA = {h: np.float32(0.0) for h in range(H)}
    for h in slot:
        SA[h] = np.float32(-1.0)
    g = np.float32(prob.gamma)
    alpha = fp32_decay(1.0, prob.gamma, prob.delta)
    out = []
    for t, nodes in enumerate(steps):
        sampled = set((nodes[nodes >= L] - L).tolist())
        buf = set(slot)
        hits = sampled & buf
        misses = sampled - buf
        for s in range(cap):
            if slot[s] not in sampled:
                SE[s] = np.float32(SE[s] * g)
        for h in misses:
            SA[h] = np.float32(SA[h] + np.float32(1.0))
        rnd = None
        if t > 0 and t % prob.delta == 0:
            E = [s for s in range(cap) if SE[s] < alpha]
            C = sorted((h for h in range(H) if SA[h] >= 0), key=lambda h: (-SA[h], orc_rank[h]))
            k = min(len(E), len(C))
            if k < len(E):
                E = sorted(sorted(E, key=lambda s: (SE[s], orc_rank[slot[s]]))[:k])
            R = C[:k]
            olds = [(SE[s], SA[r]) for s, r in zip(E, R)]
            ev = []
            for (s, r), (se, sa) in zip(zip(E, R), olds):
                e = slot[s]
                ev.append(e)
                SA[e] = se
                SE[s] = sa
                SA[r] = np.float32(-1.0)
                slot[s] = r
            rnd = (E, ev, R)
        out.append((len(hits), len(misses), rnd, list(slot), list(SE),
                    np.array([SA[h] for h in range(H)], np.float32)))
    return out


@pytest.mark.parametrize("over", [{}, {"gamma": 0.8, "delta": 4, "buffer_pct": 50},
                                  {"buffer_pct": 80, "gamma": 0.7, "delta": 2}])
def test_python_replay_and_invariants(over):
    prob, sched, w = workload_problem("cl10k", **over)
    orc = prob.oracle()
    rk = orc.rank()
    T = 40
    steps, rounds, states = [], [], []
    hs = prob.halo_store.view(np.uint8).reshape(prob.H, prob.row_bytes)
    for t in range(T):
        st = orc.sample(sched.seeds(t))
        sid, se, sa = orc.state()
        # invariants on the pre-round state
        assert len(set(sid.tolist())) == orc.cap
        buffered = np.zeros(prob.H, bool)
        buffered[sid] = True
        assert np.all(sa[buffered] == -1.0) and np.all(sa[~buffered] >= 0.0)
        hit_h = st.nodes[st.mask == 1] - prob.L
        assert np.all(buffered[hit_h]), "a hit is not resident"
        miss_h = st.nodes[st.mask == 2] - prob.L
        assert not np.any(buffered[miss_h])
        _check_gather(prob, st)
        assert np.array_equal(orc.buffer_rows(), hs[sid])
        rnd = orc.evict_step()
        steps.append(st.nodes.copy())
        rounds.append((st.hits, st.misses, rnd))
        states.append(orc.state())
    rep = _replay(prob, steps, rk)
    n_rounds = 0
    for t in range(T):
        hits, misses, rnd = rounds[t]
        r_hits, r_misses, r_rnd, r_slot, r_se, r_sa = rep[t]
        assert (hits, misses) == (r_hits, r_misses)
        if r_rnd is None:
            assert rnd.k == 0
        else:
            E, ev, R = r_rnd
            assert rnd.slots.tolist() == E and rnd.evicted.tolist() == ev and rnd.replaced.tolist() == R
            n_rounds += rnd.k > 0
        sid, se, sa = states[t]
        assert sid.tolist() == r_slot
        assert np.array_equal(se, np.array(r_se, np.float32))
        assert np.array_equal(sa, r_sa)
    assert n_rounds >= 3
