"""The copy kernels flatten (row, 16/8/4-byte chunk) work and recover the row
of chunk index n as n * magic >> 64 with magic = floor((2^64 - 1) / cpr) + 1,
cpr the chunks per row. This checks, with exact integers, that the quotient
is n // cpr for every cpr a row of at most 1 MiB can have (the library
refuses larger rows; test_abi.py checks that), at the chunk indices where an
error would show first: just below and at multiples of cpr, up to the
largest index whose rows fit in 2^40 bytes of memory. A model of the
flattened loop (U chunks per lane per pass) checks that every chunk is stored
exactly once and that every load, those of lanes past the end included,
stays inside the list and the row."""
import random

import pytest

MASK64 = (1 << 64) - 1


def magic(cpr):
    return MASK64 // cpr + 1


def quotient(n, cpr):
    return (n * magic(cpr)) >> 64


@pytest.mark.parametrize("vec", [4, 8, 16])
def test_quotient_exact_for_all_row_sizes(vec):
    rnd = random.Random(vec)
    max_cpr = (1 << 20) // vec
    cprs = list(range(2, 2049)) + [max_cpr, max_cpr - 1] + [rnd.randrange(2049, max_cpr) for _ in range(300)]
    for cpr in cprs:
        rows_max = (1 << 40) // (cpr * vec)  # rows of cpr * vec bytes that fit in 2^40 bytes
        for rows in (1, 2, 3, rows_max // 2, rows_max - 1, rows_max, rnd.randrange(1, rows_max + 1)):
            for n in (rows * cpr - 1, rows * cpr, rows * cpr + cpr - 1):
                assert quotient(n, cpr) == n // cpr, (cpr, n)


def flattened_passes(n, cpr, grid, block=256, U=4):
    """Every lane's (loaded, stored) chunks in the copy kernels' flattened
    loop: U chunks per lane per pass, a lane past the end re-reading its first
    chunk of the pass and storing nothing."""
    total, stride = n * cpr, grid * block
    loads, stores = [], []
    for lane in range(stride):
        c = lane
        while c < total:
            for u in range(U):
                cc = c + u * stride
                src_cc = cc if cc < total else c
                task = src_cc if cpr == 1 else quotient(src_cc, cpr)
                loads.append((task, src_cc - task * cpr))
                if cc < total:
                    stores.append((task, src_cc - task * cpr))
            c += U * stride
    return loads, stores


@pytest.mark.parametrize("n,cpr,grid", [(0, 32, 4), (1, 32, 4), (5, 1, 2), (37, 25, 3), (1000, 32, 2),
                                        (257, 2, 1), (4097, 1, 4)])
def test_every_chunk_stored_once_and_loads_in_range(n, cpr, grid):
    loads, stores = flattened_passes(n, cpr, grid)
    assert sorted(stores) == [(r, o) for r in range(n) for o in range(cpr)]
    assert all(0 <= r < n and 0 <= o < cpr for r, o in loads)
