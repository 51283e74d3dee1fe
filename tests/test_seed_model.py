"""A model of how hop 1's row-count launch checks and places the seed batch
(the minibatch B of Algorithm 2 becomes the first frontier F_0). Each thread
takes seed i: an id outside [0, L) sets status bit 1; a local id is placed by
a compare-and-swap of pos_of[id] from -1 to i, and a failed swap (the id is
already placed) sets status bit 2; a placed id is written to F_0[i]. When the
status is nonzero, classify later clears pos_of for every local id of the
batch, so the step leaves no trace.

The model runs the threads in random orders and checks: the status bits are
exactly "some seed is out of range" and "some local seed is repeated"; a
valid batch gets F_0 = seeds and pos_of[seed] = its position; an invalid
batch leaves pos_of all -1 after the take-back. A planted mistake (placing
without the compare-and-swap) fails it. It restates the kernel's steps; the
GPU tests exercise the kernel."""
import random

import pytest


def place(seeds, L, rnd, use_cas=True):
    pos_of = [-1] * L
    nodes = [None] * len(seeds)
    status = 0
    order = list(range(len(seeds)))
    rnd.shuffle(order)
    for i in order:
        x = seeds[i]
        if not (0 <= x < L):
            status |= 1
            continue
        if use_cas:
            if pos_of[x] == -1:
                pos_of[x] = i
            else:
                status |= 2
        else:
            pos_of[x] = i
        nodes[i] = x
    if status:  # classify's take-back
        for x in seeds:
            if 0 <= x < L:
                pos_of[x] = -1
    return pos_of, nodes, status


@pytest.mark.parametrize("n", [0, 1, 2, 17, 256, 1024])
def test_status_and_placement(n):
    rnd = random.Random(n)
    L = 3000
    for case in range(200):
        kind = case % 4
        seeds = rnd.sample(range(L), n)
        if kind == 1 and n:
            seeds[rnd.randrange(n)] = rnd.choice([-1, L, L + 5, -(1 << 31)])
        if kind == 2 and n > 1:
            a, b = rnd.sample(range(n), 2)
            seeds[b] = seeds[a]
        if kind == 3 and n > 2:
            seeds[0] = L
            seeds[2] = seeds[1]
        pos_of, nodes, status = place(seeds, L, rnd)
        out_of_range = any(not (0 <= x < L) for x in seeds)
        local = [x for x in seeds if 0 <= x < L]
        repeated = len(set(local)) < len(local)
        assert status == (1 if out_of_range else 0) | (2 if repeated else 0)
        if status == 0:
            assert nodes == seeds
            assert all(pos_of[x] == i for i, x in enumerate(seeds))
            assert sum(p >= 0 for p in pos_of) == n
        else:
            assert all(p == -1 for p in pos_of), "the step left frontier marks behind"


def test_planted_mistake_fails():
    rnd = random.Random(9)
    seeds = [5, 7, 5, 9]
    _, _, status = place(seeds, 20, rnd, use_cas=False)
    # the definition asks for status bit 2 (a repeated local seed); without the
    # compare-and-swap the repetition goes unnoticed, which the check above fails
    assert status & 2 == 0
