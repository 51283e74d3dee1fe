"""Seeded inputs for tests: tiny random graphs and the named synthetic workloads."""
import os
import sys
from dataclasses import dataclass
from typing import Optional, Tuple

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import synth  # noqa: E402


@dataclass
class Problem:
    """Everything an initialiser needs for one partition."""
    L: int
    H: int
    indptr: np.ndarray
    indices: np.ndarray
    halo_gid: np.ndarray
    halo_degree: np.ndarray
    local_feat: np.ndarray    # [L, d] fp32 or uint16 (bf16 bits)
    halo_store: np.ndarray    # [H, d]
    d: int
    dtype: str
    fanout: Tuple[int, ...]
    buffer_pct: int
    gamma: float
    delta: int
    seed: int = 0

    @property
    def row_bytes(self) -> int:
        return self.local_feat.dtype.itemsize * self.d

    def oracle(self, **over):
        import oracle
        kw = dict(fanout=self.fanout, buffer_pct=self.buffer_pct, gamma=self.gamma,
                  delta=self.delta, seed=self.seed)
        kw.update(over)
        return oracle.Oracle(self.L, self.H, self.indptr, self.indices, self.halo_gid,
                             self.halo_degree, self.local_feat, self.halo_store, self.row_bytes,
                             kw["fanout"], kw["buffer_pct"], kw["gamma"], kw["delta"], kw["seed"])

    def neighbours(self, v: int) -> np.ndarray:
        return self.indices[self.indptr[v]:self.indptr[v + 1]]


def tiny_problem(n_local=6, n_halo=8, p=0.5, seed=1, d=4, fanout=(3, 2), buffer_pct=25,
                 gamma=0.9, delta=2, dtype="f32") -> Problem:
    """Erdos-Renyi graph on n_local + n_halo nodes; ids [0,L) local, [L,L+H) halo."""
    rng = np.random.default_rng(seed)
    R = n_local + n_halo
    adj = np.triu(rng.random((R, R)) < p, 1)
    adj = adj | adj.T
    indptr = np.zeros(R + 1, np.int64)
    indptr[1:] = np.cumsum(adj.sum(1))
    indices = np.concatenate([np.nonzero(adj[v])[0] for v in range(R)]).astype(np.int32)
    halo_gid = (rng.permutation(1000)[:n_halo]).astype(np.int32)
    halo_degree = (indptr[n_local + 1:] - indptr[n_local:-1]).astype(np.int64)
    feats = rng.standard_normal((R, d)).astype(np.float32)
    if dtype == "bf16":
        feats = (feats.view(np.uint32) >> 16).astype(np.uint16)
    return Problem(n_local, n_halo, indptr, indices, halo_gid, halo_degree,
                   np.ascontiguousarray(feats[:n_local]), np.ascontiguousarray(feats[n_local:]),
                   d, dtype, tuple(fanout), buffer_pct, gamma, delta)


_CACHE = {}


def workload_problem(name: str, **over) -> Tuple[Problem, "synth.Schedule", "synth.Workload"]:
    """A named synthetic workload (graph cached per process)."""
    w = synth.get(name)
    if name not in _CACHE:
        g = synth.partition_graph(w)
        lf = synth.features(g.local_gid, w.d, w.dtype, w.seed)
        hs = synth.features(g.halo_gid, w.d, w.dtype, w.seed)
        _CACHE[name] = (g, lf, hs)
    g, lf, hs = _CACHE[name]
    w = w.with_(**over) if over else w
    if (w.d, w.dtype) != (lf.shape[1], synth.get(name).dtype):  # other row sizes: features drawn afresh
        lf = synth.features(g.local_gid, w.d, w.dtype, w.seed)
        hs = synth.features(g.halo_gid, w.d, w.dtype, w.seed)
    prob = Problem(g.L, g.H, g.indptr, g.indices, g.halo_gid, g.halo_degree, lf, hs, w.d, w.dtype,
                   w.fanout, w.buffer_pct, w.gamma, w.delta, w.philox_seed)
    sched = synth.Schedule(g.L, w.train_pct, w.batch, w.seed)
    return prob, sched, w


def rank_order(prob: Problem) -> np.ndarray:
    """Halo ids sorted by (degree desc, global id asc), via numpy lexsort."""
    return np.lexsort((prob.halo_gid, -prob.halo_degree)).astype(np.int32)


def fp32_decay(x: float, gamma: float, times: int) -> np.float32:
    """x multiplied by gamma `times` times, rounding to fp32 after each product."""
    v = np.float32(x)
    g = np.float32(gamma)
    for _ in range(times):
        v = np.float32(v * g)
    return v


# ------------------------------------------------------------------ exact fp32
# Binary32 rounding written from the IEEE 754 definition with Python integers
# (fractions), so that it does not depend on the FPU's flush-to-zero or
# denormals-are-zero modes: round to nearest, ties to even, with gradual
# underflow (spacing 2^-149 below 2^-126). Non-negative values only, which is
# all the decay needs.
from fractions import Fraction  # noqa: E402

_TWO = Fraction(2)


def fp32_round(q: Fraction) -> Fraction:
    """The binary32 value nearest to q >= 0 (ties to even, subnormals kept)."""
    q = Fraction(q)
    if q < 0:
        raise ValueError("non-negative values only")
    if q == 0:
        return Fraction(0)
    e = q.numerator.bit_length() - q.denominator.bit_length()
    if _TWO ** e > q:
        e -= 1                       # now 2^e <= q < 2^(e+1)
    ulp = _TWO ** (max(e, -126) - 23)
    scaled = q / ulp
    m = scaled.numerator // scaled.denominator
    rem = scaled - m
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and m % 2 == 1):
        m += 1
    return m * ulp


def fp32_bits(q: Fraction) -> int:
    """The bit pattern of a binary32 value given exactly as a fraction."""
    q = Fraction(q)
    if q == 0:
        return 0
    e = q.numerator.bit_length() - q.denominator.bit_length()
    if _TWO ** e > q:
        e -= 1
    if e < -126:                     # subnormal: q = m * 2^-149
        m = q / _TWO ** -149
        assert m.denominator == 1 and 0 < m < 2 ** 23
        return int(m)
    m = q / _TWO ** (e - 23)
    assert m.denominator == 1 and 2 ** 23 <= m < 2 ** 24
    return ((e + 127) << 23) | (int(m) - 2 ** 23)


def fp32_decay_exact(x: float, gamma: float, times: int) -> Fraction:
    """x multiplied `times` times by gamma (both taken as binary32), each
    product rounded to binary32: the decay's exact result."""
    g = fp32_round(Fraction(gamma))
    v = fp32_round(Fraction(x))
    for _ in range(times):
        v = fp32_round(v * g)
    return v


def matched_problem(degrees, buffer_pct, gamma, delta, d=4, seed=3) -> Problem:
    """len(degrees) local nodes, each adjacent to exactly one halo node (local
    i to halo i), one hop of fanout 1: seeding local i samples halo i and
    nothing else, so a seed schedule fixes the sampled halo set of every step.
    halo_degree is given, so it fixes the halo rank order."""
    n = len(degrees)
    R = 2 * n
    indptr = np.arange(R + 1, dtype=np.int64)
    indices = np.concatenate([np.arange(n, 2 * n), np.arange(n)]).astype(np.int32)
    rng = np.random.default_rng(seed)
    feats = rng.standard_normal((R, d)).astype(np.float32)
    return Problem(n, n, indptr, indices, np.arange(100, 100 + n, dtype=np.int32),
                   np.asarray(degrees, np.int64), np.ascontiguousarray(feats[:n]),
                   np.ascontiguousarray(feats[n:]), d, "f32", (1,), buffer_pct, gamma, delta)


def subnormal_order_schedule():
    """Seeds of the scenario in which a halo node whose S_A is subnormal must be
    chosen ahead of a better-ranked one whose S_A is exactly 0 (six halo nodes
    h0..h5 ranked in that order, three slots, gamma 0.5, Delta 140, so
    alpha = 2^-140):
      step 0: h0, h2 hit, h3 missed (S_A 1); steps 1-140: nothing sampled.
        Round at 140: h1 (never sampled, S_E 2^-141) is evicted, S_A(h1) =
        2^-141 (subnormal); h3 replaces it.
      steps 141-280: h2, h3 hit every step; h5 missed at 141 (S_A 1).
        Round at 280: h0's S_E has underflowed to exactly 0, so h0 is
        evicted with S_A(h0) = 0; h5 (S_A 1) replaces it, ahead of h1.
      steps 281-420: h3, h5 hit. Round at 420: h2's S_E is 0, evicted; the
        candidates are h0 (S_A 0, rank 0), h1 (S_A 2^-141, rank 1), h4 (S_A 0,
        rank 4), so h1 replaces it. Flushing subnormals to zero would pick h0.
    Returns a function t -> seeds (local ids) for t in 0..420."""
    def seeds(t):
        if t == 0:
            return np.array([0, 2, 3], np.int32)
        if t <= 140:
            return np.zeros(0, np.int32)
        if t == 141:
            return np.array([2, 3, 5], np.int32)
        if t <= 280:
            return np.array([2, 3], np.int32)
        return np.array([3, 5], np.int32)
    return seeds
