"""A model of the dedup/relabel route (the NeighborSampler's frontier update
of Algorithm 2 in the DGL block convention): while writing a sampled id u,
the sampler sets bit u of a bitmap over the partition-local ids if u is not
yet in the frontier (pos_of[u] < 0); k_bits_scan then gives every tile of
4096 words (1024 threads x 4 consecutive words) its exclusive popcount prefix
(block scan plus look-back across tiles), and each thread emits the set bits
of its words in ascending order as F[n_prev + prefix + ...] = 32 * word + bit,
with pos_of[u] = that position, clearing the words; relabel maps every
sampled id through pos_of.

The model restates those steps and checks them against the definition: the
new nodes are the ascending unique sampled ids not already in the frontier,
every relabelled index points at its id, and the bitmap ends empty. It
restates the kernels' steps; the GPU tests exercise the kernels."""
import random

import pytest

NT, ITEMS = 1024, 4
TILE = NT * ITEMS


def popcount(x):
    return bin(x).count("1")


def hop(F, pos_of, sampled, R, L=None):
    W = -(-R // 32)
    bits = [0] * (W + 4)
    for u in sampled:  # emit_id: mark ids not yet in the frontier
        if pos_of[u] < 0:
            bits[u >> 5] |= 1 << (u & 31)
    n_prev = len(F)
    ntiles = max(1, -(-W // TILE))
    # per tile: the block's exclusive scan of per-thread popcounts, then the
    # tile's exclusive prefix over the tiles before it (the look-back's result)
    tile_tot = []
    for b in range(ntiles):
        tile_tot.append(sum(popcount(bits[w]) for w in range(b * TILE, min((b + 1) * TILE, W))))
    newF = list(F) + [None] * sum(tile_tot)
    before = 0
    local_new = []  # written by the thread whose words hold id L (or the last tile)
    wL = None if L is None else L >> 5
    for b in range(ntiles):
        ex = 0
        for x in range(NT):
            base = b * TILE + x * ITEMS
            words = [bits[base + i] if base + i < W else 0 for i in range(ITEMS)]
            if wL is not None and wL < W and base <= wL < base + ITEMS:
                below = sum(popcount(words[i]) for i in range(ITEMS) if base + i < wL)
                below += popcount(words[wL - base] & ((1 << (L & 31)) - 1))
                local_new.append(before + ex + below)
            off = n_prev + before + ex
            for i, wd in enumerate(words):
                while wd:
                    low = wd & -wd
                    u = ((base + i) << 5) + low.bit_length() - 1
                    wd ^= low
                    assert newF[off] is None
                    newF[off] = u
                    pos_of[u] = off
                    off += 1
                if words[i]:
                    bits[base + i] = 0
            ex += sum(popcount(wd) for wd in words)
        before += tile_tot[b]
    if wL is not None and wL >= W:
        local_new.append(before)  # the last tile: every id is below L
    assert not any(bits), "bitmap not cleared"
    relabelled = [pos_of[u] for u in sampled]
    if L is None:
        return newF, relabelled
    assert len(local_new) == 1, "one writer of the local count"
    return newF, relabelled, local_new[0]


@pytest.mark.parametrize("R,density", [(1, 1.0), (31, 0.5), (33, 0.5), (4096 * 32 + 5, 0.01),
                                       (3 * 4096 * 32 + 100, 0.002), (50_000, 0.3)])
def test_new_nodes_are_ascending_unique_and_relabel_points_back(R, density):
    rnd = random.Random(R)
    pos_of = [-1] * R
    F = rnd.sample(range(R), max(1, R // 50))
    for i, v in enumerate(F):
        pos_of[v] = i
    k = max(1, int(R * density))
    sampled = [rnd.randrange(R) for _ in range(k)] + F[:3]  # repeats and ids already in F
    newF, rel = hop(F, pos_of, sampled, R)
    want_new = sorted(set(sampled) - set(F))
    assert newF[:len(F)] == F and newF[len(F):] == want_new
    assert all(newF[p] == u for p, u in zip(rel, sampled))
    assert all(pos_of[u] == p for p, u in enumerate(newF))


@pytest.mark.parametrize("R,density", [(40, 0.5), (4096 * 32 + 5, 0.01), (3 * 4096 * 32 + 100, 0.002)])
def test_local_count_is_the_prefix_at_L(R, density):
    """The new nodes below L (local ids), counted by the one thread whose
    words hold id L, for L at word boundaries, inside words, at tile
    boundaries, at 0 and at R (every id local)."""
    rnd = random.Random(R + 1)
    for L in sorted({0, 1, 31, 32, 33, R // 2, R - 1, R, TILE * 32, TILE * 32 + 7, 2 * TILE * 32 - 1} & set(range(R + 1))):
        pos_of = [-1] * R
        F = rnd.sample(range(R), max(1, R // 50))
        for i, v in enumerate(F):
            pos_of[v] = i
        sampled = [rnd.randrange(R) for _ in range(max(1, int(R * density)))]
        newF, rel, local_new = hop(F, pos_of, sampled, R, L)
        assert local_new == sum(1 for u in newF[len(F):] if u < L), (R, L)
