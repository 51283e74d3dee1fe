"""A model of the eviction round's two selections (Algorithm 2, Section IV-B).

Replacements: the candidates are the unbuffered halo nodes (S_A >= 0), held
in rank order; each gets the key ~bits(S_A), so ascending key is descending
S_A. Four radix-select passes of 8 bits, from the top, find the key T of the
k'-th candidate: each pass histograms the digit of the candidates matching
the prefix so far, picks the digit whose exclusive count is below `need` and
whose inclusive count reaches it, and lowers `need` by the count before it.
Then the candidates with key < T, in rank order, are stably sorted by key
(LSD, 8 bits a pass) into R[0 : n_lt], and the first `need` with key == T, in
rank order, fill R[n_lt : k'].

Evictions when there are fewer candidates than flagged slots: E (ascending
slot) is stably sorted by the rank of the slot's node, then by the bits of
S_E (non-negative, so bit order is value order), the first k' kept and sorted
back to ascending slot.

The model restates those steps and checks them against plain sorts by the
definitions ((S_A desc, rank asc) and (S_E asc, rank asc)), on score mixes
like the real ones (mostly zero, small miss counts, the fractional S_E an
evicted node carries), with ties straddling the threshold and k' at its
limits. It restates the kernels' steps; the GPU tests exercise the kernels."""
import random
import struct

import pytest


def f32_bits(x):
    return struct.unpack("<I", struct.pack("<f", x))[0]


def f32(x):
    return struct.unpack("<f", struct.pack("<f", x))[0]


def lsd_sort(pairs):
    # stable LSD radix sort of (key, val) by the 32-bit key, 8 bits a pass
    for shift in (0, 8, 16, 24):
        buckets = [[] for _ in range(256)]
        for kv in pairs:
            buckets[(kv[0] >> shift) & 255].append(kv)
        pairs = [kv for b in buckets for kv in b]
    return pairs


def select_replacements(S_A_by_rank, h_of_rank, k):
    """The kernels' steps: radix select of T, then emit and sort."""
    keys = [(~f32_bits(a)) & 0xFFFFFFFF if a >= 0.0 else None for a in S_A_by_rank]
    need, prefix, pmask = k, 0, 0
    if k > 0:
        for shift in (24, 16, 8, 0):
            hist = [0] * 256
            for key in keys:
                if key is not None and (key & pmask) == prefix:
                    hist[(key >> shift) & 255] += 1
            ex, pick, before = 0, -1, 0
            for d in range(256):
                if ex < need <= ex + hist[d]:
                    pick, before = d, ex
                ex += hist[d]
            assert pick >= 0, "fewer candidates than asked for"
            need -= before
            prefix |= pick << shift
            pmask |= 255 << shift
    T = prefix
    lt = [(key, h_of_rank[r]) for r, key in enumerate(keys) if key is not None and key < T]
    eq = [h_of_rank[r] for r, key in enumerate(keys) if key is not None and key == T]
    assert len(lt) == k - need and len(eq) >= need
    return [h for _, h in lsd_sort(lt)] + eq[:need]


def select_replacements_by_gid(S_A_by_gid, rank_g, h_of_rank, gid_of, k):
    """The kernels' steps with S_A over every global id, scanned in id order:
    an exact radix select over the 64-bit key (~bits(S_A), rank), 8 bits a
    pass (four on the score word, four on the rank word), then the k' keys
    at or below it, in id order, stably sorted by rank and then by score."""
    cands = [((~f32_bits(a)) & 0xFFFFFFFF, rank_g[g]) for g, a in enumerate(S_A_by_gid) if a >= 0.0]
    need, pre, msk = k, [0, 0], [0, 0]
    if k > 0:
        for word in (0, 1):
            for shift in (24, 16, 8, 0):
                hist = [0] * 256
                for c in cands:
                    if (c[0] & msk[0]) == pre[0] and (c[1] & msk[1]) == pre[1]:
                        hist[(c[word] >> shift) & 255] += 1
                ex, pick, before = 0, -1, 0
                for d in range(256):
                    if ex < need <= ex + hist[d]:
                        pick, before = d, ex
                    ex += hist[d]
                assert pick >= 0, "fewer candidates than asked for"
                need -= before
                pre[word] |= pick << shift
                msk[word] |= 255 << shift
        assert need == 1, "ranks are unique: one key at the threshold"
    T = (pre[0], pre[1])  # the k'-th smallest key
    emitted = [(c[1], h_of_rank[c[1]]) for c in cands if k > 0 and c <= T]
    assert len(emitted) == k
    by_rank = lsd_sort(emitted)
    keyed = [((~f32_bits(S_A_by_gid[gid_of[h]])) & 0xFFFFFFFF, h) for _, h in by_rank] if by_rank else []
    return [h for _, h in lsd_sort(keyed)]


def narrow_evictions(E, S_E, rank_of_slot, k):
    """The kernels' steps: two stable sorts (rank, then S_E bits), keep k, sort by slot."""
    pairs = lsd_sort([(rank_of_slot[s], s) for s in E])
    pairs = lsd_sort([(f32_bits(S_E[s]), s) for _, s in pairs])
    return [s for _, s in lsd_sort([(s, s) for _, s in pairs[:k]])]


def score_mix(rnd, n, zero_frac=0.7):
    out = []
    for _ in range(n):
        u = rnd.random()
        if u < zero_frac:
            out.append(0.0)
        elif u < zero_frac + 0.2:
            out.append(float(rnd.randrange(1, 6)))  # miss counts
        else:
            out.append(f32(0.9 ** rnd.randrange(0, 60)))  # an evicted node's S_E
    return out


@pytest.mark.parametrize("seed", range(6))
def test_replacement_select_matches_sort(seed):
    rnd = random.Random(seed)
    H = rnd.choice([1, 7, 300, 2500])
    h_of_rank = list(range(H))
    rnd.shuffle(h_of_rank)
    S_A = score_mix(rnd, H)
    buffered = rnd.sample(range(H), rnd.randrange(0, H))
    for r in buffered:
        S_A[r] = -1.0
    ncand = sum(a >= 0.0 for a in S_A)
    for k in sorted({0, 1, ncand // 3, ncand // 2, max(ncand - 1, 0), ncand}):
        want = [h_of_rank[r] for r in sorted((r for r in range(H) if S_A[r] >= 0.0),
                                             key=lambda r: (-S_A[r], r))][:k]
        assert select_replacements(S_A, h_of_rank, k) == want, (seed, H, k)


def test_replacement_ties_straddle_threshold():
    # all candidates equal, or one value repeated across the k'-th place:
    # the first candidates in rank order among the tied ones are taken
    for S_A, k in (([0.0] * 50, 17), ([2.0] * 10 + [1.0] * 30 + [0.0] * 10, 25),
                   ([1.0, 0.0] * 40, 41), ([3.0] * 5 + [-1.0] * 5 + [3.0] * 5, 7)):
        h_of_rank = list(range(100, 100 + len(S_A)))
        order = sorted((r for r in range(len(S_A)) if S_A[r] >= 0.0), key=lambda r: (-S_A[r], r))
        assert select_replacements(S_A, h_of_rank, k) == [h_of_rank[r] for r in order[:k]]


def test_keys_order_nonnegative_floats():
    # ~bits(a) is strictly decreasing in a over the non-negative floats the
    # scores take (+0 included); the select depends on nothing else
    vals = sorted({0.0, f32(1e-30), f32(0.9 ** 59), f32(0.5), 1.0, 2.0, 3.0, f32(1e20)})
    keys = [(~f32_bits(a)) & 0xFFFFFFFF for a in vals]
    assert keys == sorted(keys, reverse=True) and len(set(keys)) == len(keys)


@pytest.mark.parametrize("seed", range(6))
def test_eviction_narrowing_matches_sort(seed):
    rnd = random.Random(50 + seed)
    cap = rnd.choice([3, 40, 900])
    rank_of_slot = rnd.sample(range(10 * cap), cap)
    S_E = [f32(0.9 ** rnd.randrange(0, 8)) if rnd.random() < 0.8 else 0.0 for _ in range(cap)]
    E = sorted(rnd.sample(range(cap), rnd.randrange(0, cap + 1)))
    for k in sorted({0, 1, len(E) // 2, len(E)}):
        want = sorted(sorted(E, key=lambda s: (S_E[s], rank_of_slot[s]))[:k])
        assert narrow_evictions(E, S_E, rank_of_slot, k) == want, (seed, cap, k)


@pytest.mark.parametrize("seed", range(6))
def test_replacement_select_by_global_id_matches_sort(seed):
    # S_A over a global id space larger than the halo (non-halo ids hold -1),
    # halo nodes at random ids: the same replacements, in the same order, as
    # the rank-ordered layout and a plain sort by (S_A desc, rank asc)
    rnd = random.Random(100 + seed)
    H = rnd.choice([1, 7, 300, 2500])
    n_global = H + rnd.choice([0, 5, 3 * H])
    gid_of = rnd.sample(range(n_global), H)          # halo h -> its global id
    h_of_rank = list(range(H))
    rnd.shuffle(h_of_rank)
    S_by_rank = score_mix(rnd, H)
    for r in rnd.sample(range(H), rnd.randrange(0, H)):
        S_by_rank[r] = -1.0
    S_by_gid, rank_g = [-1.0] * n_global, [-1] * n_global
    for r, h in enumerate(h_of_rank):
        S_by_gid[gid_of[h]] = S_by_rank[r]
        rank_g[gid_of[h]] = r
    ncand = sum(a >= 0.0 for a in S_by_rank)
    for k in sorted({0, 1, ncand // 3, ncand // 2, max(ncand - 1, 0), ncand}):
        want = [h_of_rank[r] for r in sorted((r for r in range(H) if S_by_rank[r] >= 0.0),
                                             key=lambda r: (-S_by_rank[r], r))][:k]
        assert select_replacements_by_gid(S_by_gid, rank_g, h_of_rank, gid_of, k) == want, (seed, H, k)
        assert select_replacements(S_by_rank, h_of_rank, k) == want
