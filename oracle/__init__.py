"""CPU oracle of MassiveGNN's per-minibatch path (arXiv 2410.22697).

TEST INFRASTRUCTURE ONLY: only tests/, __graft_entry__.smoke() and the
CPU-baseline leg of bench.py may import this package. The product path
(paper_2410_22697_amd) never imports, links or runs anything here.

The arithmetic lives in oracle.c (plain single-threaded C, compiled with
gcc). This module only builds it and marshals arguments.
"""
import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

OK, EINVAL, ENOMEM, ESTATE = 0, -1, -3, -5


def build(force: bool = True) -> str:
    """Compile liboracle.so (gcc, no fast-math: fp32 products stay IEEE)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared",
                               "-ffp-contract=off", _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


class _Args(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("H", ctypes.c_int32),
                ("indptr", ctypes.c_void_p), ("indices", ctypes.c_void_p),
                ("halo_gid", ctypes.c_void_p), ("halo_degree", ctypes.c_void_p),
                ("local_feat", ctypes.c_void_p), ("halo_store", ctypes.c_void_p),
                ("row_bytes", ctypes.c_int64), ("K", ctypes.c_int32),
                ("fanout", ctypes.c_int32 * 8), ("buffer_pct", ctypes.c_int32),
                ("gamma", ctypes.c_float), ("delta", ctypes.c_int32), ("seed", ctypes.c_uint64)]


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        lib.oracle_philox4x32_10.argtypes = [vp, vp, vp]
        lib.oracle_init.argtypes = [ctypes.POINTER(_Args), ctypes.POINTER(vp)]
        lib.oracle_init.restype = ctypes.c_int
        lib.oracle_destroy.argtypes = [vp]
        lib.oracle_sample.argtypes = [vp, vp, i32]
        lib.oracle_sample.restype = ctypes.c_int
        lib.oracle_evict_step.argtypes = [vp, vp, vp, vp, ctypes.POINTER(i64)]
        lib.oracle_evict_step.restype = ctypes.c_int
        lib.oracle_cap.argtypes = [vp]
        lib.oracle_cap.restype = i64
        lib.oracle_alpha.argtypes = [vp]
        lib.oracle_alpha.restype = ctypes.c_float
        lib.oracle_t.argtypes = [vp]
        lib.oracle_t.restype = i64
        lib.oracle_sizes.argtypes = [vp, vp, vp, vp]
        for name in ("oracle_nodes", "oracle_mask", "oracle_feat", "oracle_rank", "oracle_buffer_rows"):
            getattr(lib, name).argtypes = [vp]
            getattr(lib, name).restype = vp
        lib.oracle_block_indptr.argtypes = [vp, ctypes.c_int]
        lib.oracle_block_indptr.restype = vp
        lib.oracle_block_indices.argtypes = [vp, ctypes.c_int]
        lib.oracle_block_indices.restype = vp
        lib.oracle_get_state.argtypes = [vp, vp, vp, vp]
        lib.oracle_phase_times.argtypes = [vp, vp]
        lib.oracle_sample_row.argtypes = [vp, vp, i32, i64, i32, i32, ctypes.c_uint64, vp]
        lib.oracle_sample_row.restype = i64
        _lib = lib
    return _lib


def philox4x32_10(ctr: Sequence[int], key: Sequence[int]) -> List[int]:
    c = (ctypes.c_uint32 * 4)(*[x & 0xFFFFFFFF for x in ctr])
    k = (ctypes.c_uint32 * 2)(*[x & 0xFFFFFFFF for x in key])
    o = (ctypes.c_uint32 * 4)()
    _load().oracle_philox4x32_10(c, k, o)
    return list(o)


def sample_row(indptr: np.ndarray, indices: np.ndarray, v: int, t: int, k: int, fanout: int,
               seed: int = 0) -> np.ndarray:
    """Neighbour ids the sampler chooses for node v at step t, hop k (1-based)."""
    ip = np.ascontiguousarray(indptr, np.int64)
    ix = np.ascontiguousarray(indices, np.int32)
    d = int(ip[v + 1] - ip[v])
    out = np.zeros(max(min(d, fanout), 1), np.int32)
    m = _load().oracle_sample_row(ip.ctypes.data, ix.ctypes.data, int(v), int(t), int(k), int(fanout),
                                  int(seed), out.ctypes.data)
    if m < 0:
        raise MemoryError("oracle_sample_row")
    return out[:m]


def _arr(ptr, dtype, n):
    if n == 0:
        return np.empty(0, dtype)
    buf = (ctypes.c_char * (n * np.dtype(dtype).itemsize)).from_address(ptr)
    return np.frombuffer(buf, dtype=dtype, count=n).copy()


@dataclass
class Step:
    nodes: np.ndarray            # int32 [n_K]
    n: List[int]                 # frontier sizes n_0..n_K
    e: List[int]                 # edges per hop
    indptr: List[np.ndarray]     # per hop int32 [n_{k-1}+1]
    indices: List[np.ndarray]    # per hop int32 [e_k], relabelled
    mask: np.ndarray             # uint8 [n_K]
    feat: np.ndarray             # uint8 [n_K, row_bytes]
    local: int
    hits: int
    misses: int


@dataclass
class Round:
    k: int
    evicted: np.ndarray          # halo ids evicted, in slot order
    slots: np.ndarray            # slots they held (ascending)
    replaced: np.ndarray         # halo ids that replace them


class Oracle:
    """Stateful CPU oracle of one partition's prefetcher + sampler."""

    def __init__(self, L, H, indptr, indices, halo_gid, halo_degree, local_feat, halo_store,
                 row_bytes, fanout, buffer_pct, gamma, delta, seed=0):
        self._lib = _load()
        # keep every borrowed array alive for the oracle's lifetime
        self._keep = [np.ascontiguousarray(indptr, np.int64), np.ascontiguousarray(indices, np.int32),
                      np.ascontiguousarray(halo_gid, np.int32), np.ascontiguousarray(halo_degree, np.int64)]
        self._local = local_feat
        self._store = halo_store
        a = _Args()
        a.L, a.H = int(L), int(H)
        a.indptr, a.indices, a.halo_gid, a.halo_degree = [x.ctypes.data for x in self._keep]
        a.local_feat = _ptr(local_feat)
        a.halo_store = _ptr(halo_store)
        a.row_bytes = int(row_bytes)
        a.K = len(fanout)
        for i, f in enumerate(fanout):
            a.fanout[i] = int(f)
        a.buffer_pct, a.gamma, a.delta, a.seed = int(buffer_pct), float(gamma), int(delta), int(seed)
        self.K, self.L, self.H, self.row_bytes = len(fanout), int(L), int(H), int(row_bytes)
        h = ctypes.c_void_p()
        rc = self._lib.oracle_init(ctypes.byref(a), ctypes.byref(h))
        if rc != OK:
            raise ValueError("oracle_init failed: %d" % rc)
        self._h = h
        self.cap = int(self._lib.oracle_cap(h))
        self.alpha = float(self._lib.oracle_alpha(h))

    def close(self):
        if getattr(self, "_h", None):
            self._lib.oracle_destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    @property
    def t(self) -> int:
        return int(self._lib.oracle_t(self._h))

    def rank(self) -> np.ndarray:
        return _arr(self._lib.oracle_rank(self._h), np.int32, self.H)

    def sample(self, seeds) -> Step:
        s = np.ascontiguousarray(seeds, np.int32)
        rc = self._lib.oracle_sample(self._h, s.ctypes.data, len(s))
        if rc != OK:
            raise ValueError("oracle_sample failed: %d" % rc)
        n = np.zeros(9, np.int64)
        e = np.zeros(8, np.int64)
        cnt = np.zeros(3, np.int64)
        self._lib.oracle_sizes(self._h, n.ctypes.data, e.ctypes.data, cnt.ctypes.data)
        K = self.K
        nK = int(n[K])
        ip = [_arr(self._lib.oracle_block_indptr(self._h, k), np.int32, int(n[k]) + 1) for k in range(K)]
        ix = [_arr(self._lib.oracle_block_indices(self._h, k), np.int32, int(e[k])) for k in range(K)]
        return Step(nodes=_arr(self._lib.oracle_nodes(self._h), np.int32, nK),
                    n=[int(x) for x in n[:K + 1]], e=[int(x) for x in e[:K]],
                    indptr=ip, indices=ix,
                    mask=_arr(self._lib.oracle_mask(self._h), np.uint8, nK),
                    feat=_arr(self._lib.oracle_feat(self._h), np.uint8, nK * self.row_bytes
                              ).reshape(nK, self.row_bytes),
                    local=int(cnt[0]), hits=int(cnt[1]), misses=int(cnt[2]))

    def evict_step(self) -> Round:
        ev = np.zeros(max(self.cap, 1), np.int32)
        sl = np.zeros(max(self.cap, 1), np.int32)
        rp = np.zeros(max(self.cap, 1), np.int32)
        k = ctypes.c_int64()
        rc = self._lib.oracle_evict_step(self._h, ev.ctypes.data, sl.ctypes.data, rp.ctypes.data,
                                         ctypes.byref(k))
        if rc != OK:
            raise ValueError("oracle_evict_step failed: %d" % rc)
        kk = int(k.value)
        return Round(kk, ev[:kk].copy(), sl[:kk].copy(), rp[:kk].copy())

    def state(self):
        sid = np.zeros(max(self.cap, 1), np.int32)
        se = np.zeros(max(self.cap, 1), np.float32)
        sa = np.zeros(max(self.H, 1), np.float32)
        self._lib.oracle_get_state(self._h, sid.ctypes.data, se.ctypes.data, sa.ctypes.data)
        return sid[:self.cap].copy(), se[:self.cap].copy(), sa[:self.H].copy()

    def buffer_rows(self) -> np.ndarray:
        return _arr(self._lib.oracle_buffer_rows(self._h), np.uint8,
                    self.cap * self.row_bytes).reshape(self.cap, self.row_bytes)

    def phase_times(self) -> np.ndarray:
        out = np.zeros(6, np.float64)
        self._lib.oracle_phase_times(self._h, out.ctypes.data)
        return out


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return int(x.data_ptr())
    return int(x.ctypes.data)
