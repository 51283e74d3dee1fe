"""A model of k_classify's list compaction (the hit/miss split of
Algorithm 2 written as two gather lists). Per item of a block of 256 threads
(4 waves of 64), every wave counts its rows of each list with ballots; the
block's first thread takes one base per list from a global counter (blocks
in any order); a wave's offset is the base plus the counts of the waves
before it, and a lane's slot adds the matching lanes below it. Rows of one
thread are items 0..ITEMS-1 at positions b0 + it * 256 + thread.

The model restates those steps, with blocks taking their bases in a random
order, and checks that each list holds every row of its class exactly once
(the HBM list: local rows and hits; the host list: misses and hits on slots
still refilling), that no slot is written twice or left empty, and that the
class counts match. It restates the kernel's steps; the GPU tests exercise
the kernel itself."""
import random

import pytest

NT, WAVE, ITEMS = 256, 64, 4
TILE = NT * ITEMS


def lanes_below(mask, lane):
    return bin(mask & ((1 << lane) - 1)).count("1")


def compact(cls, rnd):
    """cls[i] in {0 local, 1 hit, 2 miss, 3 hit on a refilling slot}."""
    n = len(cls)
    nblocks = -(-n // TILE)
    hbm, host = [None] * n, [None] * n
    counters = [0, 0]
    for b in rnd.sample(range(nblocks), nblocks):  # blocks reach the atomics in any order
        b0 = b * TILE
        # per (item, wave) ballots of the two lists
        wc = [[0, 0] for _ in range(NT // WAVE)]
        for it in range(ITEMS):
            for w in range(NT // WAVE):
                for lane in range(WAVE):
                    i = b0 + it * NT + w * WAVE + lane
                    c = cls[i] if i < n else -1
                    wc[w][0] += c in (0, 1)
                    wc[w][1] += c >= 2
        base = []
        for k in range(2):
            tot = sum(wc[w][k] for w in range(NT // WAVE))
            base.append(counters[k])
            counters[k] += tot
        for w in range(NT // WAVE):
            oh = base[0] + sum(wc[x][0] for x in range(w))
            om = base[1] + sum(wc[x][1] for x in range(w))
            for it in range(ITEMS):
                rows = [b0 + it * NT + w * WAVE + lane for lane in range(WAVE)]
                c = [cls[i] if i < n else -1 for i in rows]
                mh = sum(1 << ln for ln in range(WAVE) if c[ln] in (0, 1))
                mm = sum(1 << ln for ln in range(WAVE) if c[ln] >= 2)
                for ln in range(WAVE):
                    if c[ln] in (0, 1):
                        slot = oh + lanes_below(mh, ln)
                        assert hbm[slot] is None, "HBM slot written twice"
                        hbm[slot] = rows[ln]
                    elif c[ln] >= 2:
                        slot = om + lanes_below(mm, ln)
                        assert host[slot] is None, "host slot written twice"
                        host[slot] = rows[ln]
                oh += bin(mh).count("1")
                om += bin(mm).count("1")
    return hbm[:counters[0]], host[:counters[1]], counters


@pytest.mark.parametrize("n", [0, 1, 63, 64, 65, 1023, 1024, 1025, 2047, 2048, 2049, 5000])
def test_every_row_lands_once_in_its_list(n):
    rnd = random.Random(n)
    for mix in ((0.3, 0.3, 0.3), (1.0, 0.0, 0.0), (0.0, 0.0, 1.0), (0.2, 0.5, 0.2)):
        cls = []
        for _ in range(n):
            u = rnd.random()
            cls.append(0 if u < mix[0] else 1 if u < mix[0] + mix[1] else 2 if u < sum(mix) else 3)
        hbm, host, counters = compact(cls, rnd)
        assert None not in hbm and None not in host
        assert sorted(hbm) == [i for i in range(n) if cls[i] in (0, 1)]
        assert sorted(host) == [i for i in range(n) if cls[i] >= 2]
        assert counters == [sum(c in (0, 1) for c in cls), sum(c >= 2 for c in cls)]
        # the step's completion derives the counts: local rows come from the dedup scans,
        # pending hits from their own counter; hits and misses from the lists
        local, pending = sum(c == 0 for c in cls), sum(c == 3 for c in cls)
        hits, misses = counters[0] - local + pending, counters[1] - pending
        assert hits == sum(c in (1, 3) for c in cls) and misses == sum(c == 2 for c in cls)
