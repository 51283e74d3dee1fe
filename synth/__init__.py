"""Seeded synthetic inputs shared by the oracle and the HIP path.

This module holds none of the method's arithmetic. It builds the partition
view G_p of a Chung-Lu power-law graph, fills N(0,1) feature rows and yields
the per-step seed batches. See synth.c for the recipes.
"""
import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import Optional

import numpy as np

from .workloads import WORKLOADS, Workload, get  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB = os.path.join(_HERE, "libsynth.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile libsynth.so with gcc (OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O3", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               "-Wall", "-Wno-unused-function", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Graph(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int64), ("H", ctypes.c_int64), ("nnz", ctypes.c_int64),
                ("indptr", ctypes.POINTER(ctypes.c_int64)),
                ("indices", ctypes.POINTER(ctypes.c_int32)),
                ("local_gid", ctypes.POINTER(ctypes.c_int32)),
                ("halo_gid", ctypes.POINTER(ctypes.c_int32)),
                ("halo_degree", ctypes.POINTER(ctypes.c_int64)),
                ("edges_a", ctypes.c_int64), ("edges_b", ctypes.c_int64),
                ("i0", ctypes.c_double)]


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        lib.synth_partition_graph.restype = ctypes.POINTER(_Graph)
        lib.synth_partition_graph.argtypes = [ctypes.c_uint64, ctypes.c_double, ctypes.c_double,
                                              ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                              ctypes.c_uint64, ctypes.c_int]
        lib.synth_graph_free.argtypes = [ctypes.POINTER(_Graph)]
        lib.synth_features.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                       ctypes.c_int32, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_int]
        lib.synth_epoch_order.restype = ctypes.c_int64
        lib.synth_epoch_order.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64,
                                          ctypes.c_int64, ctypes.c_void_p]
        lib.synth_weights.argtypes = [ctypes.c_uint64, ctypes.c_double, ctypes.c_double,
                                      ctypes.c_void_p, ctypes.c_void_p]
        _lib = lib
    return _lib


def _threads() -> int:
    return int(os.environ.get("OMP_NUM_THREADS", "0") or 0)


@dataclass
class PartitionGraph:
    """G_p: local ids [0,L), halo ids [L,L+H); symmetric CSR."""
    L: int
    H: int
    indptr: np.ndarray       # int64 [L+H+1]
    indices: np.ndarray      # int32 [nnz]
    local_gid: np.ndarray    # int32 [L]
    halo_gid: np.ndarray     # int32 [H]
    halo_degree: np.ndarray  # int64 [H] row length in G_p
    edges_local: int         # undirected edges with a local end
    edges_halo: int          # undirected halo-halo edges

    @property
    def nnz(self) -> int:
        return int(self.indptr[-1])


def weights(n: int, beta: float, mean: float) -> np.ndarray:
    lib = _load()
    w = np.empty(n, np.float64)
    if lib.synth_weights(n, beta, mean, w.ctypes.data, None):
        raise ValueError("bad Chung-Lu parameters")
    return w


class _Owner:
    """Keeps the C-allocated graph alive while numpy views of it exist."""

    def __init__(self, lib, ptr):
        self._lib, self._ptr = lib, ptr

    def __del__(self):
        if self._ptr:
            self._lib.synth_graph_free(self._ptr)
            self._ptr = None


def _view(ptr, n, owner):
    a = np.ctypeslib.as_array(ptr, (max(n, 1),))[:n]
    # numpy views do not keep `owner` alive by themselves: wrap in a subclass
    v = a.view(_Held)
    v._owner = owner
    return v


class _Held(np.ndarray):
    def __array_finalize__(self, obj):
        self._owner = getattr(obj, "_owner", None)


def partition_graph(w: Workload, threads: Optional[int] = None) -> PartitionGraph:
    lib = _load()
    gp = lib.synth_partition_graph(w.n, w.beta, w.mean_deg, int(w.sym), w.parts, 0, w.seed,
                                   threads if threads is not None else _threads())
    if not gp:
        raise MemoryError("synth_partition_graph failed")
    g = gp.contents
    own = _Owner(lib, gp)
    R = g.L + g.H
    return PartitionGraph(
        L=int(g.L), H=int(g.H),
        indptr=_view(g.indptr, R + 1, own), indices=_view(g.indices, g.nnz, own),
        local_gid=_view(g.local_gid, g.L, own), halo_gid=_view(g.halo_gid, g.H, own),
        halo_degree=_view(g.halo_degree, g.H, own),
        edges_local=int(g.edges_a), edges_halo=int(g.edges_b))


def feature_dtype(dtype: str):
    return np.float32 if dtype == "f32" else np.uint16  # bf16 kept as raw bits


def fill_features(gids: np.ndarray, d: int, dtype: str, seed: int, out_ptr: int,
                  threads: Optional[int] = None) -> None:
    """Write N(0,1) rows for `gids` into the buffer at out_ptr ([len(gids), d])."""
    lib = _load()
    g = np.ascontiguousarray(gids, dtype=np.int32)
    lib.synth_features(g.ctypes.data, len(g), d, 0 if dtype == "f32" else 1, seed, out_ptr,
                       threads if threads is not None else _threads())


def features(gids: np.ndarray, d: int, dtype: str, seed: int) -> np.ndarray:
    out = np.empty((len(gids), d), feature_dtype(dtype))
    fill_features(gids, d, dtype, seed, out.ctypes.data)
    return out


class Schedule:
    """Seed batches for global step t (the step counter runs across epochs)."""

    def __init__(self, L: int, train_pct: int, batch: int, seed: int):
        self.L, self.train_pct, self.batch, self.seed = L, train_pct, batch, seed
        self._epoch, self._order = None, None
        self.train_size = (train_pct * L + 99) // 100
        self.steps_per_epoch = -(-self.train_size // batch)

    def epoch_order(self, e: int) -> np.ndarray:
        if self._epoch != e:
            buf = np.empty(self.L, np.int32)
            T = _load().synth_epoch_order(self.L, self.train_pct, self.seed, e, buf.ctypes.data)
            if T < 0:
                raise ValueError("bad schedule parameters")
            self._epoch, self._order = e, buf[:T].copy()
        return self._order

    def seeds(self, t: int) -> np.ndarray:
        e, b = divmod(t, self.steps_per_epoch)
        order = self.epoch_order(e)
        return order[b * self.batch:(b + 1) * self.batch]
