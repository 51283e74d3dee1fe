"""A model of k_classify's hash lookup: the table is open addressing with
linear probing (entry = slot << 32 | halo id, empty = all ones, load <= 1/2),
and the kernel settles a search from one window of four entries, the two
16-byte pairs from the probe start rounded down to even, skipping the entry
before the start when it is odd, then probes on one by one from the entry
after the window. The model restates those steps and checks them against a
plain linear-probe search on random tables, with every probe start, windows
that wrap past the table's end, keys that are absent, and dense clusters. It
restates the kernel's steps; the GPU tests exercise the kernel itself."""
import random

import pytest

EMPTY = (1 << 64) - 1
M32 = 0xFFFFFFFF


def fmix32(x):
    x ^= x >> 16
    x = (x * 0x85EBCA6B) & M32
    x ^= x >> 13
    x = (x * 0xC2B2AE35) & M32
    x ^= x >> 16
    return x


def build(keys, size, home):
    tab = [EMPTY] * size
    mask = size - 1
    for s, h in enumerate(keys):
        i = home(h) & mask
        while tab[i] != EMPTY:
            i = (i + 1) & mask
        tab[i] = (s << 32) | h
    return tab


def plain_find(tab, h, home):
    mask = len(tab) - 1
    i = home(h) & mask
    while True:
        e = tab[i]
        if e & M32 == h:
            return e >> 32
        if e == EMPTY:
            return -1
        i = (i + 1) & mask


def window_find(tab, h, home):
    mask = len(tab) - 1
    p = home(h) & mask
    q = p & ~1
    window = [tab[q], tab[q + 1], tab[(q + 2) & mask], tab[((q + 2) & mask) + 1]]
    r = -2
    for x, e in enumerate(window):
        if r == -2 and x >= (p & 1):
            if e & M32 == h:
                r = e >> 32
            elif e == EMPTY:
                r = -1
    if r == -2:  # the window held neither h nor an empty entry
        i = (q + 4) & mask
        while True:
            e = tab[i]
            if e & M32 == h:
                return e >> 32
            if e == EMPTY:
                return -1
            i = (i + 1) & mask
    return r


@pytest.mark.parametrize("size,load", [(64, 0.5), (64, 0.3), (1024, 0.5), (4096, 0.45)])
def test_window_search_equals_linear_probing(size, load):
    rnd = random.Random(size)
    for trial in range(5):
        n = int(size * load)
        keys = rnd.sample(range(1 << 20), n)
        tab = build(keys, size, fmix32)
        for h in keys + rnd.sample(range(1 << 20, 1 << 21), n):
            assert window_find(tab, h, fmix32) == plain_find(tab, h, fmix32)


def test_every_probe_start_and_wrap():
    # a hash that sends every key to a chosen start: all starts, odd and
    # even, the last pair (the window wraps to entries 0 and 1), and runs of
    # occupied entries longer than the window
    size = 64
    for start in range(size):
        for run in (0, 1, 2, 3, 4, 5, 9, 31):
            keys = list(range(100, 100 + run))
            home = lambda h, s=start: s  # noqa: E731
            tab = build(keys, size, home)
            for h in keys + [7, 8]:
                assert window_find(tab, h, home) == plain_find(tab, h, home), (start, run, h)
