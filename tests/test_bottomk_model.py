"""A model of the sampler's bottom-k choice in one wavefront (the
NeighborSampler of Algorithm 2, with uniform sampling read as the fanout
positions of smallest (key, j)).

Filter: lane q of an iteration holds the four keys of positions 4q..4q+3;
four ballots mark the keys below tau, and a candidate's list index is the
running count plus the marked keys of lower lanes (all four words) plus the
lane's own earlier words, so the list is in ascending j; it is cut at 320
entries but counted in full. In an iteration whose positions all exist, the
marks are only taken if some lane's smallest key is below tau, and when no
lane has two marked keys, a marked lane's entry is its smallest key at the
running count plus the marked lanes below it. A block splits a row into four
consecutive quarters of groups, one per wave, and concatenates the lists.

Select: list entry i sits in slot i // 64 of lane i % 64. A bitwise search
from tau's top bit finds T, the largest value with fewer than fanout keys
below it (the fanout-th smallest key); every key below T is taken, and the
ties at T in list order until fanout are reached; emission is slot-major,
lane-minor, which is list order.

The model restates those steps (the keys are given: Philox itself is pinned
elsewhere) and checks them against sorting by (key, j), with ties, rows whose
length is not a multiple of four or 256, and tau at 2^32. It restates the
kernel's steps; the GPU tests exercise the kernel itself."""
import random

import pytest

WAVE = 64
CAP = 320


def lanes_below(mask, lane):
    return bin(mask & ((1 << lane) - 1)).count("1")


PATHS = {"skip": 0, "one_per_lane": 0, "general": 0}  # iterations by the kernel's branch


def filter_groups(keys, g0, g1, tau):
    d = len(keys)
    tm1 = tau - 1
    gf = min(g1, d // 4)  # groups below gf have all four positions
    c, cnt = [None] * CAP, 0
    for q0 in range(g0, g1, WAVE):
        m = [0, 0, 0, 0]
        for lane in range(WAVE):
            q = q0 + lane
            for s in range(4):
                j = 4 * q + s
                if q < g1 and j < d and keys[j] <= tm1:
                    m[s] |= 1 << lane
        whole = q0 + WAVE <= gf
        if whole:
            mins = [min(keys[4 * (q0 + lane):4 * (q0 + lane) + 4]) for lane in range(WAVE)]
            if not any(mn <= tm1 for mn in mins):
                PATHS["skip"] += 1
                continue
            anym = m[0] | m[1] | m[2] | m[3]
            if sum(bin(ms).count("1") for ms in m) == bin(anym).count("1"):
                PATHS["one_per_lane"] += 1
                for lane in range(WAVE):
                    if (anym >> lane) & 1:
                        s = next(x for x in range(4) if (m[x] >> lane) & 1)
                        p = cnt + lanes_below(anym, lane)
                        if p < CAP:
                            c[p] = (mins[lane] << 32) | (4 * (q0 + lane) + s)
                cnt += bin(anym).count("1")
                continue
            PATHS["general"] += 1
        for lane in range(WAVE):
            q = q0 + lane
            p = cnt + sum(lanes_below(ms, lane) for ms in m)
            for s in range(4):
                if (m[s] >> lane) & 1:
                    if p < CAP:
                        c[p] = (keys[4 * q + s] << 32) | (4 * q + s)
                    p += 1
        cnt += sum(bin(ms).count("1") for ms in m)
    return c, cnt


def select_emit(lst, cnt, fo, tau):
    S = (cnt + WAVE - 1) // WAVE
    slot = [[lst[s * WAVE + lane] if s * WAVE + lane < cnt else None for lane in range(WAVE)]
            for s in range(S)]

    def count_below(x):
        return sum(1 for row in slot for e in row if e is not None and (e >> 32) < x)

    T, tm1 = 0, tau - 1
    top = tm1.bit_length() - 1 if tm1 else 0
    for b in range(top, -1, -1):
        trial = T | (1 << b)
        if count_below(trial) < fo:
            T = trial
    n_lt = count_below(T)
    need = fo - n_lt
    out, eq_before = [], 0
    for row in slot:
        eq_mask = sum(1 << ln for ln, e in enumerate(row) if e is not None and (e >> 32) == T)
        for ln, e in enumerate(row):
            if e is None:
                continue
            k = e >> 32
            if k < T or (k == T and eq_before + lanes_below(eq_mask, ln) < need):
                out.append(e & 0xFFFFFFFF)
        eq_before += bin(eq_mask).count("1")
    return out


def reference(keys, fo):
    return sorted(sorted(range(len(keys)), key=lambda j: (keys[j], j))[:fo])


def acceptable_taus(keys, fo):
    # tau values with fo <= count(key < tau) <= CAP: each key value, and 2^32
    sk = sorted(keys)
    out = []
    for v in sorted(set(keys)) + [1 << 32]:
        c = sum(1 for k in sk if k < v)
        if fo <= c <= CAP:
            out.append(v)
    return out


def sample_row(keys, fo, tau, waves=1):
    ng = (len(keys) + 3) // 4
    lst, cnt = [], 0
    for w in range(waves):  # a block: consecutive quarters of the groups
        g0, g1 = ng * w // waves, ng * (w + 1) // waves
        c, n = filter_groups(keys, g0, g1, tau)
        lst += [e for e in c[:min(n, CAP)]]
        cnt += n
    assert cnt <= CAP
    return select_emit(lst, cnt, fo, tau)


@pytest.mark.parametrize("fo", [1, 5, 10, 25])
def test_bottom_k_equals_sort(fo):
    rnd = random.Random(fo)
    for d in (fo + 1, 2 * fo + 3, 257, 1000, 1027):
        keys = [rnd.getrandbits(32) for _ in range(d)]
        taus = acceptable_taus(keys, fo)
        for tau in {taus[0], taus[len(taus) // 2], taus[-1]}:
            assert sample_row(keys, fo, tau) == reference(keys, fo), (fo, d, tau)


@pytest.mark.parametrize("fo", [3, 15])
def test_ties_take_the_lower_positions(fo):
    rnd = random.Random(7 + fo)
    for d in (40, 301, 700):
        pool = [rnd.getrandbits(32) for _ in range(6)]  # few distinct keys
        keys = [rnd.choice(pool) for _ in range(d)]
        for tau in acceptable_taus(keys, fo)[:3]:
            assert sample_row(keys, fo, tau) == reference(keys, fo), (fo, d, tau)


def test_block_lists_concatenate_in_order():
    rnd = random.Random(99)
    for d in (2049, 4096, 9001):
        fo = 10
        keys = [rnd.getrandbits(32) for _ in range(d)]
        for tau in acceptable_taus(keys, fo)[::40]:
            assert sample_row(keys, fo, tau, waves=4) == reference(keys, fo), (d, tau)


def test_small_keys_and_full_range_tau():
    # keys near 0 (T's search must reach bit 0) and near 2^32 - 1 (tau = 2^32)
    for keys in ([0, 0, 1, 2, 3, 3, 3, 1] * 5, [(1 << 32) - 1 - k for k in range(70)]):
        for fo in (1, 4, 7):
            for tau in acceptable_taus(keys, fo):
                assert sample_row(keys, fo, tau) == reference(keys, fo), (fo, tau)


def test_both_append_paths_taken():
    # the tests above reach the one-per-lane append and the general one
    rnd = random.Random(5)
    before = dict(PATHS)
    for d in (1000, 4096):
        keys = [rnd.getrandbits(32) for _ in range(d)]
        for tau in acceptable_taus(keys, 10)[::20]:
            assert sample_row(keys, 10, tau) == reference(keys, 10)
    pool = [rnd.getrandbits(32) for _ in range(4)]
    keys = [rnd.choice(pool) for _ in range(600)]  # lanes with several keys below tau
    for tau in acceptable_taus(keys, 5):
        assert sample_row(keys, 5, tau) == reference(keys, 5)
    assert PATHS["one_per_lane"] > before["one_per_lane"]
    assert PATHS["general"] > before["general"]
    assert PATHS["skip"] > before["skip"]
