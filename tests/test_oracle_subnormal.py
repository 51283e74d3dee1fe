"""Pins for the subnormal range of the scores (Eq. 1 and the decay and swap of
Section IV-B): alpha = gamma^Delta and the decayed S_E of an unsampled slot
fall below 2^-126 for small gamma or long intervals, and the swap carries such
an S_E into S_A, where it outranks every candidate whose S_A is 0. The
oracle keeps subnormals (gradual underflow, no flush to zero); these pins
check it against binary32 rounding written out with Python integers
(tests/helpers.py fp32_round), which no FPU mode can change, so an oracle
built or run with flush-to-zero fails them."""
from fractions import Fraction

import numpy as np
import pytest

from helpers import (fp32_bits, fp32_decay_exact, fp32_round, matched_problem, subnormal_order_schedule,
                     workload_problem)

TWO = Fraction(2)


def test_exact_rounding_reference():
    """The integer-arithmetic rounding against facts fixed by IEEE 754 binary32."""
    tiny = TWO ** -149                                 # smallest subnormal
    assert fp32_bits(tiny) == 1
    assert fp32_bits(TWO ** -126) == 0x00800000        # smallest normal
    assert fp32_bits(Fraction(1)) == 0x3F800000
    assert fp32_round(TWO ** -150) == 0                # half the spacing: tie to even (0)
    assert fp32_round(3 * TWO ** -151) == tiny         # 0.75 of the spacing rounds up
    assert fp32_round(Fraction(5, 2) * tiny) == 2 * tiny   # tie to even
    assert fp32_round(Fraction(7, 2) * tiny) == 4 * tiny   # tie to even
    assert fp32_round(1 + TWO ** -24) == 1             # tie to even in the normal range
    assert fp32_round(1 + 3 * TWO ** -24) == 1 + TWO ** -22
    assert fp32_bits(fp32_round(Fraction(0.3))) == 0x3E99999A
    # normal-range products agree with the FPU's binary32 multiply
    rng = np.random.default_rng(0)
    for x, y in rng.uniform(1e-3, 1e3, (200, 2)).astype(np.float32):
        want = np.float32(x) * np.float32(y)
        assert fp32_bits(fp32_round(Fraction(float(x)) * Fraction(float(y)))) == int(want.view(np.uint32))


def _state_bits(orc):
    sid, se, sa = orc.state()
    return sid, se.view(np.uint32).astype(np.int64), sa.view(np.uint32).astype(np.int64)


def test_unsampled_slots_decay_through_subnormals_halving():
    """gamma = 1/2: after u unsampled steps S_E = 2^-u exactly down to the
    smallest subnormal 2^-149 (bits 1 << (149 - u) from u = 127), then 0 from
    u = 150 (2^-150 is a tie that rounds to even, 0). Empty batches sample
    nothing, so every slot decays at every step."""
    prob, sched, w = workload_problem("cl10k", gamma=0.5, delta=100000)
    orc = prob.oracle()
    assert orc.cap > 0
    empty = np.zeros(0, np.int32)
    for t in range(160):
        orc.sample(empty)
        assert orc.evict_step().k == 0
        u = t + 1
        _, se, _ = _state_bits(orc)
        want = fp32_bits(TWO ** -u) if u <= 149 else 0
        if 127 <= u <= 149:
            assert want == 1 << (149 - u)
        assert np.all(se == want), (u, se[:4], want)


@pytest.mark.parametrize("gamma,delta", [(0.3, 80), (0.3, 86), (0.5, 140), (0.9, 900)])
def test_alpha_in_the_subnormal_range(gamma, delta):
    """alpha = Delta binary32 products of gamma (Eq. 1), subnormal here."""
    prob, _, _ = workload_problem("cl10k", gamma=gamma, delta=delta)
    orc = prob.oracle()
    want = fp32_decay_exact(1.0, gamma, delta)
    assert 0 < want < TWO ** -126
    assert int(np.float32(orc.alpha).view(np.uint32)) == fp32_bits(want)


def test_unsampled_slots_decay_through_subnormals_gamma_03():
    """gamma = 0.3 (not a power of two): every product rounds. S_E after each
    step equals the integer-arithmetic sequence, through the subnormal range
    (from u = 73) and down to 0 (u = 87)."""
    prob, _, _ = workload_problem("cl10k", gamma=0.3, delta=100000)
    orc = prob.oracle()
    empty = np.zeros(0, np.int32)
    v = Fraction(1)
    g = fp32_round(Fraction(0.3))
    seen_sub = 0
    for t in range(100):
        orc.sample(empty)
        orc.evict_step()
        v = fp32_round(v * g)
        _, se, _ = _state_bits(orc)
        assert np.all(se == fp32_bits(v)), (t, se[:2], fp32_bits(v))
        seen_sub += 0 < v < TWO ** -126
    assert v == 0 and seen_sub >= 10


def test_subnormal_S_A_outranks_zero():
    """The swap moves a subnormal S_E into S_A; that candidate must come ahead
    of a better-ranked candidate whose S_A is exactly 0 (the scenario of
    helpers.subnormal_order_schedule, derived by hand)."""
    prob = matched_problem([6, 5, 4, 3, 2, 1], buffer_pct=50, gamma=0.5, delta=140)
    seeds = subnormal_order_schedule()
    orc = prob.oracle()
    assert orc.cap == 3 and int(np.float32(orc.alpha).view(np.uint32)) == fp32_bits(TWO ** -140)
    sid, _, _ = _state_bits(orc)
    assert sid.tolist() == [0, 1, 2]
    rounds = {}
    for t in range(421):
        st = orc.sample(seeds(t))
        if t == 0:
            assert (st.hits, st.misses) == (2, 1)
        r = orc.evict_step()
        if r.k:
            rounds[t] = (r.slots.tolist(), r.evicted.tolist(), r.replaced.tolist(), _state_bits(orc))
    assert sorted(rounds) == [140, 280, 420]
    # round 1: h1 never sampled (S_E 2^-141 < alpha) makes way for h3 (S_A 1)
    slots, ev, rep, (sid, se, sa) = rounds[140]
    assert (slots, ev, rep) == ([1], [1], [3])
    assert sa[1] == fp32_bits(TWO ** -141) == 1 << 8       # subnormal S_A
    assert se[1] == fp32_bits(Fraction(1))
    # round 2: h0 decayed to exactly 0 is evicted (S_A 0); h5 (S_A 1) is chosen
    slots, ev, rep, (sid, se, sa) = rounds[280]
    assert (slots, ev, rep) == ([0], [0], [5])
    assert sa[0] == 0 and sa[1] == 1 << 8 and sa[4] == 0
    # round 3: h1 (S_A 2^-141, rank 1) ahead of h0 (S_A 0, rank 0)
    slots, ev, rep, (sid, se, sa) = rounds[420]
    assert (slots, ev, rep) == ([2], [2], [1])
    assert sid.tolist() == [5, 3, 1]
    assert se[2] == 1 << 8                                   # the slot's S_E := 2^-141
    assert sa[2] == 0 and sa[0] == 0
