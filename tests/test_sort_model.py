"""A model of the library's stable LSD radix sort pass (the round's and
init's sorts of 32-bit keys with int32 values), 8 bits per pass.

Per pass: every block of 2048 keys (256 threads x 8 items, item `it` of
thread x at index base + it * 256 + x) counts its digits into hist[digit *
nb + block], digit-major; an exclusive scan of that flat array gives every
(digit, block) its output base. The scatter then walks the items in order;
within an item, a lane finds its peers (the lanes of its wave with the same
digit) by intersecting eight bit ballots, its rank among them is the number
of peers in lower lanes, the highest peer writes the wave's count for the
digit, and a key goes to base + the block's running count for the digit +
the counts of lower waves + its rank. Only the first min(n, bound) keys are
sorted.

The model restates those steps and checks every pass against Python's
stable sort by the digit, and four passes against a stable sort by key, with
keys that share digits heavily, sizes that leave a ragged last block, and a
count below the bound. It restates the kernels' steps; the GPU tests exercise
the kernels."""
import random

import pytest

NT, ITEMS, WAVE = 256, 8, 64
TILE = NT * ITEMS


def sort_pass(keys, vals, n, bound, shift):
    n = min(n, bound)
    nb = max(1, -(-bound // TILE))
    hist = [0] * (256 * nb)
    for i in range(n):
        hist[((keys[i] >> shift) & 255) * nb + i // TILE] += 1
    offs, acc = [], 0
    for h in hist:  # exclusive scan over the digit-major array
        offs.append(acc)
        acc += h
    ko, vo = list(keys), list(vals)  # entries past n are left as they were
    for b in range(nb):
        gbase = [offs[d * nb + b] for d in range(256)]
        running = [0] * 256
        for it in range(ITEMS):
            wcnt = [[0] * 256 for _ in range(NT // WAVE)]
            items = []
            for wave in range(NT // WAVE):
                lanes = []
                for lane in range(WAVE):
                    i = b * TILE + it * NT + wave * WAVE + lane
                    lanes.append((i, i < n, (keys[i] >> shift) & 255 if i < n else 0))
                valid_mask = sum(1 << ln for ln, (_, v, _) in enumerate(lanes) if v)
                for lane, (i, valid, dgt) in enumerate(lanes):
                    peers = valid_mask
                    for bit in range(8):
                        m = sum(1 << ln for ln, (_, _, d2) in enumerate(lanes) if (d2 >> bit) & 1)
                        peers &= m if (dgt >> bit) & 1 else ~m
                    below = bin(peers & ((1 << lane) - 1)).count("1")
                    if valid and (peers >> lane) >> 1 == 0:
                        wcnt[wave][dgt] = below + 1
                    items.append((i, valid, dgt, wave, below))
            for i, valid, dgt, wave, below in items:
                if valid:
                    r = running[dgt] + below + sum(wcnt[w][dgt] for w in range(wave))
                    ko[gbase[dgt] + r] = keys[i]
                    vo[gbase[dgt] + r] = vals[i]
            for d in range(256):
                running[d] += sum(wcnt[w][d] for w in range(NT // WAVE))
    return ko, vo


def padded(xs, bound):
    return xs + [0] * (max(1, -(-bound // TILE)) * TILE - len(xs))


@pytest.mark.parametrize("n,bound,spread", [(1, 1, 32), (700, 700, 4), (2048, 2048, 32),
                                             (4100, 4100, 9), (3000, 5000, 12)])
def test_pass_is_a_stable_digit_sort(n, bound, spread):
    rnd = random.Random(n + spread)
    keys = [rnd.getrandbits(spread) << (32 - spread) | rnd.getrandbits(4) for _ in range(n)]
    vals = list(range(n))
    k, v = padded(keys, bound), padded(vals, bound)
    for shift in (0, 8, 16, 24):
        ko, vo = sort_pass(k, v, n, bound, shift)
        want = sorted(range(n), key=lambda i: (keys[i] >> shift) & 255)  # stable
        assert vo[:n] == [vals[i] for i in want] and ko[:n] == [keys[i] for i in want], (n, shift)


def test_four_passes_sort_by_key_stably():
    rnd = random.Random(5)
    n = 4500
    keys = [rnd.choice([0, 1, 255, 256, 1 << 24, (1 << 32) - 1, rnd.getrandbits(32)]) for _ in range(n)]
    k, v = padded(keys, n), padded(list(range(n)), n)
    for shift in (0, 8, 16, 24):
        k, v = sort_pass(k, v, n, n, shift)
    want = sorted(range(n), key=lambda i: keys[i])
    assert v[:n] == want and k[:n] == sorted(keys)
