"""A model of the row list that k_row_scan writes for the one-wave-per-row
sampler (the NeighborSampler's per-node draws of Algorithm 2, one wavefront
per frontier row). Each block of the scan takes one tile of rows; inside the
block every row longer than the long-row limit goes to the front of an LDS
array and every other row to its back (LDS atomics, in any order); the
block's first thread then takes one base per part from two global counters
(blocks in any order), and the block writes its long rows at
list[base_long + j] and its other rows at list[end - 1 - (base_other + j)],
where end is the frontier bound. Wave w of the sampler takes list[w] if
w < n_long, list[end - 1 - (w - n_long)] if w < n, and nothing otherwise.

The model restates those steps, with blocks and the LDS appends in random
orders, and checks: every row of the frontier is taken by exactly one wave,
the waves [0, n_long) take exactly the long rows, no two parts overlap, and
the waves from n on take nothing. It restates the kernel's steps; the GPU
tests exercise the kernels."""
import random

import pytest

TILE = 4096


def row_list(deg, n, end, big_min, rnd):
    """deg: row lengths of frontier rows 0..n-1 (n <= end)."""
    lst = [None] * end
    counters = [0, 0]
    ntiles = max(1, -(-n // TILE))
    for b in rnd.sample(range(ntiles), ntiles):
        rows = list(range(b * TILE, min((b + 1) * TILE, n)))
        rnd.shuffle(rows)  # LDS atomics: any order inside the block
        lds = [None] * TILE
        big_n = small_n = 0
        for i in rows:
            if deg[i] > big_min:
                lds[big_n] = i
                big_n += 1
            else:
                lds[TILE - 1 - small_n] = i
                small_n += 1
        assert big_n + small_n <= TILE
        big_base, small_base = counters[0], counters[1]
        counters[0] += big_n
        counters[1] += small_n
        for j in range(big_n):
            assert lst[big_base + j] is None, "long row slot written twice"
            lst[big_base + j] = lds[j]
        for j in range(small_n):
            p = end - 1 - (small_base + j)
            assert 0 <= p < end and lst[p] is None, "row slot written twice"
            lst[p] = lds[TILE - 1 - j]
    return lst, counters


def wave_rows(lst, n_long, n, end, grid_waves):
    taken = []
    for w in range(grid_waves):
        if w >= n:
            continue
        taken.append((w, lst[w if w < n_long else end - 1 - (w - n_long)]))
    return taken


@pytest.mark.parametrize("n,end", [(0, 1), (1, 1), (5, 9), (4095, 4096), (4096, 4096), (4097, 5000),
                                   (9000, 9000), (12345, 20000)])
def test_every_row_taken_once_long_rows_first(n, end):
    rnd = random.Random(n * 7 + end)
    for mix in (0.0, 0.05, 0.5, 1.0):
        big_min = 2048
        deg = [rnd.randint(2049, 60000) if rnd.random() < mix else rnd.randint(0, 2048) for _ in range(n)]
        lst, (n_long, n_small) = row_list(deg, n, end, big_min, rnd)
        assert n_long + n_small == n
        assert n_long == sum(d > big_min for d in deg)
        taken = wave_rows(lst, n_long, n, end, end)  # the grid is the frontier bound
        rows = [r for _, r in taken]
        assert sorted(rows) == list(range(n)), "every row exactly once"
        assert all(deg[r] > big_min for w, r in taken if w < n_long)
        assert all(deg[r] <= big_min for w, r in taken if w >= n_long)


def test_planted_mistake_fails():
    # reading the other rows from the front (a wrong index) loses rows
    rnd = random.Random(3)
    n, end = 5000, 6000
    deg = [rnd.randint(0, 5000) for _ in range(n)]
    lst, (n_long, _) = row_list(deg, n, end, 2048, rnd)
    wrong = [lst[w] if w < n_long else lst[w] for w in range(n)]
    assert sorted(r for r in wrong if r is not None) != list(range(n))
