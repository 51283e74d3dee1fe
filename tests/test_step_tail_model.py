"""A model of how the miss gather ends a step (the merged fetch of
Algorithm 2 and the step's completion in one kernel). Every block first reads
the step's host-row count from the step's sizes, then moves its share of the
rows; block 0 then publishes the sizes (reads them all and copies them to the
host mailbox); every block finally adds one to a counter held in the sizes,
and the block that sees the count reach the grid size clears the sizes for
the slot's next step.

The model runs the blocks as sequences of atomic steps under random
interleavings (each block's own steps in program order) and checks, for every
interleaving and grid size: the sizes are cleared exactly once; no block
reads its count, and block 0 does not publish, after the clear; the mailbox
holds the step's sizes; and the sizes end cleared with the counter at zero,
ready for the slot's next step. A planted mistake (the clear by block 0 after
its own publish, without the counter) fails it. It restates the kernel's
protocol; the GPU tests exercise the kernel."""
import random

import pytest


def run(nblocks, rnd, clear_by_block0=False):
    sizes = {"n_miss": 123, "hits": 7, "done": 0}
    want = dict(sizes)
    mailbox = None
    events = []
    progs = []
    for b in range(nblocks):
        prog = [("read_count", b), ("rows", b)]
        if b == 0:
            prog.append(("publish", b))
            if clear_by_block0:
                prog.append(("clear", b))
        if not clear_by_block0:
            prog.append(("count", b))
        progs.append(prog)
    pc = [0] * nblocks
    last = [False] * nblocks
    cleared = 0
    while any(pc[b] < len(progs[b]) for b in range(nblocks)):
        b = rnd.choice([x for x in range(nblocks) if pc[x] < len(progs[x])])
        op, _ = progs[b][pc[b]]
        pc[b] += 1
        if op == "read_count":
            events.append(("read", b, sizes["n_miss"]))
        elif op == "publish":
            mailbox = {k: v for k, v in sizes.items() if k != "done"}
        elif op == "count":
            old = sizes["done"]
            sizes["done"] = old + 1
            if old == nblocks - 1:
                progs[b].append(("clear", b))
        elif op == "clear":
            for k in sizes:
                sizes[k] = 0
            cleared += 1
            events.append(("clear", b, None))
    return sizes, mailbox, events, cleared, want


@pytest.mark.parametrize("nblocks", [1, 2, 3, 12, 16])
def test_clear_after_every_reader(nblocks):
    rnd = random.Random(nblocks)
    for _ in range(300):
        sizes, mailbox, events, cleared, want = run(nblocks, rnd)
        assert cleared == 1
        reads = [e for e in events if e[0] == "read"]
        assert len(reads) == nblocks and all(r[2] == want["n_miss"] for r in reads), "a block read a cleared count"
        assert events[-1][0] == "clear"
        assert mailbox == {k: v for k, v in want.items() if k != "done"}, "the mailbox missed the step's sizes"
        assert all(v == 0 for v in sizes.values()), "the slot's sizes are not clear for its next step"


def test_planted_mistake_fails():
    # block 0 clearing after its own publish, without the counter, lets a
    # later block read a cleared count in some interleaving
    rnd = random.Random(5)
    bad = 0
    for _ in range(300):
        _, _, events, _, want = run(4, rnd, clear_by_block0=True)
        bad += any(e[0] == "read" and e[2] != want["n_miss"] for e in events)
    assert bad > 0
