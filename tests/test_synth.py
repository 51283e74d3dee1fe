"""The seeded input generator against its own definitions: Chung-Lu weights
and edge probabilities (the expected edge count and isolated-node count,
computed by brute force over all pairs), the random-range partition (an exact
split of the ids), the partition view G_p (a well-formed symmetric CSR whose
halo nodes each touch a local node), thread-count independence, the N(0,1)
features and their bf16 rounding, and the seed schedule. The recorded sizes
of the small workload are pinned too."""
import ctypes
import math

import numpy as np
import pytest
from scipy import stats

import synth
from synth.workloads import Workload


def small(n=6000, beta=2.1, mean=10.0, sym=False, parts=1, seed=3):
    return Workload("t", n, beta, mean, sym, parts, 8, "f32", 10, 64, (5,), 25, 0.95, 4, 1, seed=seed)


def raw_graph(w, part, threads=0):
    lib = synth._load()
    gp = lib.synth_partition_graph(w.n, w.beta, w.mean_deg, int(w.sym), w.parts, part, w.seed, threads)
    assert gp
    g = gp.contents
    R = g.L + g.H
    out = dict(L=g.L, H=g.H,
               indptr=np.ctypeslib.as_array(g.indptr, (R + 1,)).copy(),
               indices=np.ctypeslib.as_array(g.indices, (max(g.nnz, 1),))[:g.nnz].copy(),
               local_gid=np.ctypeslib.as_array(g.local_gid, (max(g.L, 1),))[:g.L].copy(),
               halo_gid=np.ctypeslib.as_array(g.halo_gid, (max(g.H, 1),))[:g.H].copy(),
               halo_degree=np.ctypeslib.as_array(g.halo_degree, (max(g.H, 1),))[:g.H].copy(),
               edges=(g.edges_a, g.edges_b))
    lib.synth_graph_free(gp)
    return out


def pair_probabilities(w, sym):
    """Yield, per block of rows u, the matrix p_uv over v (u != v), as defined."""
    S = w.sum()
    n = len(w)
    for u0 in range(0, n, 500):
        p = np.minimum(1.0, np.outer(w[u0:u0 + 500], w) / S)
        if sym:
            p = 1.0 - (1.0 - p) ** 2
        idx = np.arange(u0, min(u0 + 500, n))
        p[idx - u0, idx] = 0.0
        yield u0, p


def test_weights_follow_the_power_law():
    lib = synth._load()
    for n, beta, mean in ((6000, 2.1, 10.0), (2_450_000, 2.0, 50.0)):
        w = np.empty(n)
        i0 = ctypes.c_double()
        assert lib.synth_weights(n, beta, mean, w.ctypes.data, ctypes.byref(i0)) == 0
        assert w[0] == pytest.approx(math.sqrt(n * mean), rel=1e-12)
        assert np.all(np.diff(w) <= 0)
        assert w.mean() == pytest.approx(mean, rel=1e-6 if n < 65536 else 1e-4)
        a, b = n // 10, n // 2  # log-slope in (i + i0) is -1 / (beta - 1)
        slope = math.log(w[a] / w[b]) / math.log((a + i0.value) / (b + i0.value))
        assert slope == pytest.approx(-1.0 / (beta - 1.0), rel=1e-9)


@pytest.mark.parametrize("sym", [False, True])
def test_edge_count_and_isolated_nodes_match_the_pair_probabilities(sym):
    wl = small(sym=sym, mean=7.0 if sym else 10.0)
    g = raw_graph(wl, 0)
    assert g["H"] == 0 and g["L"] == wl.n  # one partition: the whole graph
    m = g["edges"][0] + g["edges"][1]
    assert g["indptr"][-1] == 2 * m
    w = synth.weights(wl.n, wl.beta, wl.mean_deg)
    e_m = var_m = e_iso = 0.0
    for u0, p in pair_probabilities(w, sym):
        e_m += p.sum() / 2
        var_m += (p * (1 - p)).sum() / 2
        e_iso += np.exp(np.log1p(-np.minimum(p, 1 - 1e-300)).sum(axis=1)).sum()
    assert abs(m - e_m) < 6 * math.sqrt(var_m), (m, e_m, math.sqrt(var_m))
    iso = int((np.diff(g["indptr"]) == 0).sum())
    assert abs(iso - e_iso) < 6 * math.sqrt(e_iso) + 1, (iso, e_iso)


def test_random_range_partition_splits_the_ids_exactly():
    wl = small(parts=4)
    seen = []
    for p in range(4):
        g = raw_graph(wl, p)
        lo, hi = p * wl.n // 4, (p + 1) * wl.n // 4
        assert g["L"] == hi - lo
        seen.append(g["local_gid"])
        assert np.all(np.diff(g["local_gid"]) > 0) and np.all(np.diff(g["halo_gid"]) > 0)
        assert not np.intersect1d(g["local_gid"], g["halo_gid"]).size
    allg = np.concatenate(seen)
    assert np.array_equal(np.sort(allg), np.arange(wl.n))


@pytest.mark.parametrize("part", [0, 2])
def test_partition_view_is_a_symmetric_csr_with_a_true_halo(part):
    wl = small(parts=4, n=8000)
    g = raw_graph(wl, part)
    L, H, ip, ix = g["L"], g["H"], g["indptr"], g["indices"]
    R = L + H
    assert ip[0] == 0 and np.all(np.diff(ip) >= 0) and len(ip) == R + 1
    rows = np.repeat(np.arange(R), np.diff(ip))
    assert np.all((ix >= 0) & (ix < R)) and not np.any(ix == rows)
    # rows ascending without repeats
    same_row = rows[1:] == rows[:-1]
    assert np.all(ix[1:][same_row] > ix[:-1][same_row])
    fwd = set(zip(rows.tolist(), ix.tolist()))
    assert all((v, u) in fwd for u, v in fwd)
    assert np.array_equal(g["halo_degree"], np.diff(ip)[L:])
    # every halo node has a local neighbour (its row starts with a local id)
    assert np.all(ix[ip[L:R]] < L) and np.all(np.diff(ip)[L:] > 0)
    assert 2 * (g["edges"][0] + g["edges"][1]) == ip[-1]


def test_independent_of_thread_count():
    wl = small(parts=4, n=8000)
    a, b = raw_graph(wl, 1, threads=1), raw_graph(wl, 1, threads=3)
    for k in ("indptr", "indices", "local_gid", "halo_gid", "halo_degree"):
        assert np.array_equal(a[k], b[k]), k
    gids = np.arange(0, 4000, 3, dtype=np.int32)
    f1 = np.empty((len(gids), 33), np.float32)
    f3 = np.empty_like(f1)
    synth.fill_features(gids, 33, "f32", 5, f1.ctypes.data, threads=1)
    synth.fill_features(gids, 33, "f32", 5, f3.ctypes.data, threads=3)
    assert np.array_equal(f1, f3)


def test_small_workload_sizes():
    g = synth.partition_graph(synth.get("cl10k"))
    assert (g.L, g.H, g.nnz, int(np.diff(g.indptr).max())) == (2500, 5310, 88216, 320)


def test_features_are_standard_normal_per_global_id():
    gids = np.arange(20000, dtype=np.int32)
    f = synth.features(gids, 64, "f32", 11)
    x = f.astype(np.float64).ravel()
    assert abs(x.mean()) < 5 / math.sqrt(x.size)
    assert x.var() == pytest.approx(1.0, abs=5 * math.sqrt(2.0 / x.size))
    assert stats.kstest(x[:200000], "norm").pvalue > 1e-4
    assert abs(np.corrcoef(f[:, 0], f[:, 1])[0, 1]) < 5 / math.sqrt(len(gids))
    # a row depends on (seed, global id) only
    g2 = np.array([17, 5, 17], np.int32)
    f2 = synth.features(g2, 64, "f32", 11)
    assert np.array_equal(f2[0], f[17]) and np.array_equal(f2[1], f[5]) and np.array_equal(f2[2], f[17])
    assert not np.array_equal(synth.features(g2, 64, "f32", 12)[0], f[17])
    # odd width: the leading columns are those of the even width
    assert np.array_equal(synth.features(g2, 5, "f32", 11), f2[:, :5])


def test_bf16_features_round_to_nearest_even():
    gids = np.arange(3000, dtype=np.int32)
    f = synth.features(gids, 40, "f32", 2)
    b = synth.features(gids, 40, "bf16", 2)
    u = f.view(np.uint32).astype(np.uint64)
    want = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    assert np.array_equal(b, want)
    # and the rounding is to nearest: |bf16 - f32| <= half a bf16 ulp
    back = (b.astype(np.uint32) << 16).view(np.float32)
    ulp = np.ldexp(1.0, np.frexp(np.abs(f))[1] - 8)
    assert np.all(np.abs(back.astype(np.float64) - f) <= ulp / 2 + 1e-30)


def test_seed_schedule():
    L, pct, batch = 1000, 37, 64
    s = synth.Schedule(L, pct, batch, seed=9)
    assert s.train_size == 370 and s.steps_per_epoch == 6
    e0, e1 = s.epoch_order(0).copy(), s.epoch_order(1).copy()
    assert len(e0) == 370 and len(set(e0.tolist())) == 370 and e0.min() >= 0 and e0.max() < L
    assert set(e0.tolist()) == set(e1.tolist()) and not np.array_equal(e0, e1)
    batches = [s.seeds(t) for t in range(6)]
    assert [len(x) for x in batches] == [64] * 5 + [50]
    assert np.array_equal(np.concatenate(batches), e0)
    assert np.array_equal(s.seeds(6), e1[:64])
