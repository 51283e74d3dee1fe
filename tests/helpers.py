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
