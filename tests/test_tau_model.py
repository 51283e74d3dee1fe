"""A model of the sampler's threshold search (TauSearch in the sampler):
starting from tau = mu / d * 2^32 + 1, it multiplies tau by 4 (up to 2^32)
while fewer than fanout keys lie below it, then bisects between the last
tau with too few and the first with too many, until fanout <= count <= the
candidate list's capacity; it gives up once the two bounds are adjacent (a
run of equal keys longer than the slack). The model checks, on random key
sets with and without runs of equal keys, that the search ends within the
kernel's 64 passes, that an accepted tau has an acceptable count, and that it
gives up only when no tau has one. It restates the kernel's steps; the GPU
tests exercise the kernel itself."""
import bisect
import math
import random

import pytest

FULL = 1 << 32
CAP = 320
PASSES = 64


def mu(fo):
    return min(fo + 3 * math.sqrt(fo) + 3, 0.5 * (fo + CAP))


def search(keys_sorted, fo):
    d = len(keys_sorted)
    t = mu(fo) * FULL / d + 1.0
    tau = FULL if t >= FULL else int(t)
    lo, hi = 0, FULL + 1
    for passes in range(1, PASSES + 1):
        cnt = bisect.bisect_left(keys_sorted, tau)  # keys below tau
        if fo <= cnt <= CAP:
            return tau, cnt, passes, False
        if cnt < fo:
            lo = tau
            tau = (min(tau * 4, FULL)) if hi > FULL else (lo + hi) // 2
        else:
            hi = tau
            tau = (lo + hi) // 2
        if hi <= FULL and hi - lo <= 1:
            return tau, cnt, passes, True
    return tau, None, PASSES, None  # out of passes: never expected


def acceptable_exists(keys_sorted, fo):
    # counts below tau are the distinct values' positions, plus d at 2^32
    counts = {bisect.bisect_left(keys_sorted, k) for k in keys_sorted} | {len(keys_sorted)}
    return any(fo <= c <= CAP for c in counts)


@pytest.mark.parametrize("fo", [1, 5, 10, 25, 200, 256])
def test_search_on_random_keys(fo):
    rnd = random.Random(fo)
    for d in (fo + 1, fo + 2, 2 * fo + 3, 300, 1000, 5000):
        for _ in range(20):
            keys = sorted(rnd.getrandbits(32) for _ in range(d))
            tau, cnt, passes, gave_up = search(keys, fo)
            assert gave_up is False and passes <= PASSES, (fo, d)
            assert fo <= cnt <= CAP and cnt == bisect.bisect_left(keys, tau)


@pytest.mark.parametrize("fo", [5, 25, 256])
def test_search_with_runs_of_equal_keys(fo):
    rnd = random.Random(100 + fo)
    for run in (2, 50, CAP - fo, CAP - fo + 1, CAP - fo + 2, 400):
        for _ in range(10):
            d = max(fo + 1, run + rnd.randrange(0, 600))
            v = rnd.getrandbits(32)
            keys = sorted([v] * run + [rnd.getrandbits(32) for _ in range(d - run)])
            tau, cnt, passes, gave_up = search(keys, fo)
            assert gave_up is not None and passes <= PASSES
            if gave_up:
                assert not acceptable_exists(keys, fo), (fo, run, d)
            else:
                assert fo <= cnt <= CAP and cnt == bisect.bisect_left(keys, tau)


def test_adversarial_start_points():
    # every key at 0 or at 2^32 - 1: growth from the first tau to 2^32 takes
    # the most passes (16), then bisection over the whole range (33)
    for fo, low, high in ((5, 3, 500), (5, 10, 500), (25, 0, 400), (25, 300, 10), (256, 200, 1000)):
        keys = sorted([0] * low + [FULL - 1] * high)
        tau, cnt, passes, gave_up = search(keys, fo)
        assert passes <= PASSES
        assert gave_up == (not acceptable_exists(keys, fo))


def test_a_key_at_tau_is_not_below_it():
    # four keys below the first tau and one exactly at it: only four are
    # below, so the search must move on (counting the key at tau would stop
    # it at a count of five that the candidate list does not hold)
    fo, d = 5, 300
    t0 = int(mu(fo) * FULL / d + 1.0)
    keys = sorted([1, 2, 3, 4, t0] + [FULL - 1 - i for i in range(d - 5)])
    tau, cnt, passes, gave_up = search(keys, fo)
    assert gave_up is False and passes > 1
    assert cnt == bisect.bisect_left(keys, tau) and fo <= cnt <= CAP
