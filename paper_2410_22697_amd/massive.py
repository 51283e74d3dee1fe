"""ctypes binding of libmassive (include/massive.h); argument marshalling only.

PyTorch supplies device memory (output tensors) and the stream. All work of
the path runs in the library's HIP kernels. There is no fallback: if the
library is missing, importing this module raises.
"""
import ctypes
import os
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmassive.so")
MAX_HOPS = 8

OK, EINVAL, ECAPACITY, ENOMEM, EHIP, ESTATE = 0, -1, -2, -3, -4, -5
SCORES_BY_RANK, SCORES_BY_GID = 0, 1  # S_A layouts (Section IV-B)
LINK_LOADS, LINK_STAGED = 0, 1  # how rows cross the host link: kernel loads, or host gather + DMA copies
MAX_INFLIGHT = 3  # batches enqueued with sample_async and not yet waited for
_NAMES = {EINVAL: "EINVAL", ECAPACITY: "ECAPACITY", ENOMEM: "ENOMEM", EHIP: "EHIP", ESTATE: "ESTATE"}

EXPORTS = ("massive_init", "massive_output_bounds", "massive_sample", "massive_sample_noalloc", "massive_sample_async",
           "massive_batch_wait", "massive_evict_step", "massive_get_counters", "massive_get_state",
           "massive_get_buffer_rows", "massive_info", "massive_set_timing", "massive_get_timing",
           "massive_destroy", "massive_last_error")


class MassiveError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("%s (%d): %s" % (_NAMES.get(code, "?"), code, msg))
        self.code = code


class InitArgs(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("H", ctypes.c_int32),
                ("indptr", ctypes.c_void_p), ("indices", ctypes.c_void_p),
                ("halo_gid", ctypes.c_void_p), ("halo_degree", ctypes.c_void_p),
                ("local_feat", ctypes.c_void_p), ("halo_store", ctypes.c_void_p),
                ("row_bytes", ctypes.c_int64), ("K", ctypes.c_int32),
                ("fanout", ctypes.c_int32 * MAX_HOPS), ("buffer_pct", ctypes.c_int32),
                ("gamma", ctypes.c_float), ("delta", ctypes.c_int32), ("seed", ctypes.c_uint64),
                ("stream", ctypes.c_void_p), ("score_layout", ctypes.c_int32), ("n_global", ctypes.c_int64),
                ("link_mode", ctypes.c_int32), ("link_threads", ctypes.c_int32)]


class Batch(ctypes.Structure):
    _fields_ = [("nodes", ctypes.c_void_p), ("mask", ctypes.c_void_p), ("feat", ctypes.c_void_p),
                ("nodes_cap", ctypes.c_int64),
                ("indptr", ctypes.c_void_p * MAX_HOPS), ("indices", ctypes.c_void_p * MAX_HOPS),
                ("indptr_cap", ctypes.c_int64 * MAX_HOPS), ("indices_cap", ctypes.c_int64 * MAX_HOPS),
                ("n", ctypes.c_int64 * (MAX_HOPS + 1)), ("e", ctypes.c_int64 * MAX_HOPS),
                ("local", ctypes.c_int64), ("hits", ctypes.c_int64), ("misses", ctypes.c_int64),
                ("host_rows", ctypes.c_int64)]


_lib = None


def load():
    """Loads libmassive.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libmassive.so is not built (run __graft_entry__.build() or "
                          "python paper_2410_22697_amd/build.py)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    P = ctypes.POINTER
    lib.massive_init.argtypes = [P(InitArgs), P(vp)]
    lib.massive_output_bounds.argtypes = [vp, i32, vp, vp]
    lib.massive_sample.argtypes = [vp, vp, i32, P(Batch)]
    lib.massive_sample_noalloc.argtypes = [vp, vp, i32, P(Batch)]
    lib.massive_sample_async.argtypes = [vp, vp, i32, P(Batch)]
    lib.massive_batch_wait.argtypes = [vp, P(Batch)]
    lib.massive_evict_step.argtypes = [vp, vp, vp, vp, vp]
    lib.massive_get_counters.argtypes = [vp, P(i64), P(i64), P(i64)]
    lib.massive_get_state.argtypes = [vp, vp, vp, vp, P(i64)]
    lib.massive_get_buffer_rows.argtypes = [vp, vp]
    lib.massive_info.argtypes = [vp, P(i64), P(ctypes.c_float)]
    lib.massive_set_timing.argtypes = [vp, ctypes.c_int]
    lib.massive_get_timing.argtypes = [vp, vp, vp]
    lib.massive_destroy.argtypes = [vp]
    lib.massive_last_error.argtypes = [vp]
    lib.massive_last_error.restype = ctypes.c_char_p
    for name in EXPORTS:
        if name != "massive_last_error":
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return int(x.data_ptr())
    return int(x.ctypes.data)


def _seed_count(seeds) -> int:
    """Checks a seed batch before its device pointer goes to the library, which
    reads it as packed int32 in device memory: a torch int32 tensor on the GPU,
    contiguous. Returns the number of seeds; raises ValueError otherwise."""
    import torch
    if not isinstance(seeds, torch.Tensor):
        raise ValueError("seeds must be a torch tensor, not %s" % type(seeds).__name__)
    if seeds.dtype != torch.int32:
        raise ValueError("seeds must be int32, not %s" % seeds.dtype)
    if not seeds.is_cuda:
        raise ValueError("seeds must be a device (cuda) tensor")
    if seeds.dim() != 1 or not seeds.is_contiguous():
        raise ValueError("seeds must be a contiguous 1-d tensor")
    return int(seeds.numel())


TIMING_GROUPS = ("sample_dedup", "classify", "gather_hbm", "gather_miss", "evict_round", "refill",
                 "sample_last_hop")
TIMING_ALL = 0x7F


@dataclass
class BatchBuffers:
    """Device tensors of one batch, sized by the bounds of n_seeds_max seeds."""
    nodes: "object"
    mask: "object"
    feat: "object"
    indptr: List["object"]
    indices: List["object"]
    n_bound: List[int]
    e_bound: List[int]
    c: Batch = field(default_factory=Batch)


@dataclass
class StepResult:
    n: List[int]
    e: List[int]
    local: int
    hits: int
    misses: int
    host_rows: int = 0


class Massive:
    """One partition's sampler + prefetch buffer + gather on the GPU."""

    def __init__(self, L, H, indptr, indices, halo_gid, halo_degree, local_feat, halo_store,
                 row_bytes, fanout: Sequence[int], buffer_pct: int, gamma: float, delta: int,
                 seed: int = 0, stream=None, score_layout: str = "rank", n_global: int = 0,
                 link: str = "loads", link_threads: int = 0):
        """score_layout: "rank" (S_A over the halo, in rank order) or "gid"
        (S_A over all n_global global ids). link: "loads" (kernels read the
        pinned store) or "staged" (link_threads host threads gather the rows,
        0 for the library's default, and the DMA engines copy them)."""
        import torch
        self._torch = torch
        self._lib = load()
        if halo_store is None or not (hasattr(halo_store, "is_pinned") and halo_store.is_pinned()):
            if H > 0:
                raise ValueError("halo_store must be a pinned torch tensor (pin_memory=True)")
        self._store = halo_store  # borrowed by the library: keep it alive
        ip = np.ascontiguousarray(indptr, np.int64)
        ix = np.ascontiguousarray(indices, np.int32)
        hg = np.ascontiguousarray(halo_gid, np.int32)
        hd = np.ascontiguousarray(halo_degree, np.int64)
        lf = local_feat
        if hasattr(lf, "numpy"):
            lf = lf.contiguous()
        else:
            lf = np.ascontiguousarray(lf)
        # the library copies L rows from local_feat and reads up to H rows of halo_store
        nbytes = lambda x: x.numel() * x.element_size() if hasattr(x, "numel") else x.nbytes  # noqa: E731
        if L > 0 and nbytes(lf) < int(L) * int(row_bytes):
            raise ValueError("local_feat holds %d bytes, fewer than L * row_bytes" % nbytes(lf))
        if H > 0 and nbytes(halo_store) < int(H) * int(row_bytes):
            raise ValueError("halo_store holds %d bytes, fewer than H * row_bytes" % nbytes(halo_store))
        if len(ip) != int(L) + int(H) + 1 or len(ix) < int(ip[-1]) or len(hg) < int(H) or len(hd) < int(H):
            raise ValueError("indptr needs L + H + 1 entries, indices indptr[-1], halo_gid and halo_degree H each")
        if stream is None:
            stream = torch.cuda.current_stream()
        self.stream = stream
        a = InitArgs()
        a.L, a.H = int(L), int(H)
        a.indptr, a.indices, a.halo_gid, a.halo_degree = ip.ctypes.data, ix.ctypes.data, hg.ctypes.data, hd.ctypes.data
        a.local_feat = _ptr(lf)
        a.halo_store = _ptr(halo_store)
        a.row_bytes = int(row_bytes)
        a.K = len(fanout)
        for i, f in enumerate(fanout):
            a.fanout[i] = int(f)
        a.buffer_pct, a.gamma, a.delta, a.seed = int(buffer_pct), float(gamma), int(delta), int(seed)
        a.stream = int(stream.cuda_stream)
        if score_layout not in ("rank", "gid"):
            raise ValueError("score_layout must be 'rank' or 'gid'")
        a.score_layout = SCORES_BY_GID if score_layout == "gid" else SCORES_BY_RANK
        a.n_global = int(n_global)
        if link not in ("loads", "staged"):
            raise ValueError("link must be 'loads' or 'staged'")
        a.link_mode = LINK_STAGED if link == "staged" else LINK_LOADS
        a.link_threads = int(link_threads)
        self.score_layout = score_layout
        self.link = link
        h = ctypes.c_void_p()
        rc = self._lib.massive_init(ctypes.byref(a), ctypes.byref(h))
        if rc != OK:
            raise MassiveError(rc, self._lib.massive_last_error(None).decode())
        self._h = h
        self.L, self.H, self.K, self.row_bytes = int(L), int(H), len(fanout), int(row_bytes)
        cap, alpha = ctypes.c_int64(), ctypes.c_float()
        self._lib.massive_info(h, ctypes.byref(cap), ctypes.byref(alpha))
        self.cap, self.alpha = int(cap.value), float(alpha.value)

    # ------------------------------------------------------------------ api
    def close(self):
        if getattr(self, "_h", None):
            self._lib.massive_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check(self, rc):
        if rc != OK:
            raise MassiveError(rc, self._lib.massive_last_error(self._h).decode())

    def bounds(self, n_seeds: int):
        nb = np.zeros(MAX_HOPS + 1, np.int64)
        eb = np.zeros(MAX_HOPS, np.int64)
        self._check(self._lib.massive_output_bounds(self._h, int(n_seeds), nb.ctypes.data, eb.ctypes.data))
        return [int(x) for x in nb[:self.K + 1]], [int(x) for x in eb[:self.K]]

    def alloc_batch(self, n_seeds_max: int, device="cuda") -> BatchBuffers:
        torch = self._torch
        nb, eb = self.bounds(n_seeds_max)
        nK = max(nb[self.K], 1)
        bb = BatchBuffers(
            nodes=torch.empty(nK, dtype=torch.int32, device=device),
            mask=torch.empty(nK, dtype=torch.uint8, device=device),
            feat=torch.empty((nK, self.row_bytes), dtype=torch.uint8, device=device),
            indptr=[torch.empty(nb[k] + 1, dtype=torch.int32, device=device) for k in range(self.K)],
            indices=[torch.empty(max(eb[k], 1), dtype=torch.int32, device=device) for k in range(self.K)],
            n_bound=nb, e_bound=eb)
        c = bb.c
        c.nodes, c.mask, c.feat, c.nodes_cap = bb.nodes.data_ptr(), bb.mask.data_ptr(), bb.feat.data_ptr(), nK
        for k in range(self.K):
            c.indptr[k] = bb.indptr[k].data_ptr()
            c.indices[k] = bb.indices[k].data_ptr()
            c.indptr_cap[k] = bb.indptr[k].numel()
            c.indices_cap[k] = bb.indices[k].numel()
        return bb

    def sample(self, seeds, bb: BatchBuffers) -> StepResult:
        """seeds: int32 device tensor of distinct local ids."""
        n0 = _seed_count(seeds)
        self._check(self._lib.massive_sample(self._h, seeds.data_ptr() if n0 else None, n0,
                                             ctypes.byref(bb.c)))
        c = bb.c
        return StepResult(n=[int(c.n[k]) for k in range(self.K + 1)], e=[int(c.e[k]) for k in range(self.K)],
                          local=int(c.local), hits=int(c.hits), misses=int(c.misses), host_rows=int(c.host_rows))

    def sample_noalloc(self, seeds, bb: BatchBuffers) -> StepResult:
        """massive_sample with its per-step scratch in the library's static
        device array (the call allocates nothing); synchronous."""
        n0 = _seed_count(seeds)
        self._check(self._lib.massive_sample_noalloc(self._h, seeds.data_ptr() if n0 else None, n0,
                                                     ctypes.byref(bb.c)))
        c = bb.c
        return StepResult(n=[int(c.n[k]) for k in range(self.K + 1)], e=[int(c.e[k]) for k in range(self.K)],
                          local=int(c.local), hits=int(c.hits), misses=int(c.misses), host_rows=int(c.host_rows))

    def sample_async(self, seeds, bb: BatchBuffers) -> None:
        """Enqueues one step; bb must not be touched until wait(bb)."""
        n0 = _seed_count(seeds)
        bb._seeds = seeds  # keep the seed tensor alive while the step is in flight
        self._check(self._lib.massive_sample_async(self._h, seeds.data_ptr() if n0 else None, n0,
                                                   ctypes.byref(bb.c)))

    def wait(self, bb: BatchBuffers) -> StepResult:
        self._check(self._lib.massive_batch_wait(self._h, ctypes.byref(bb.c)))
        bb._seeds = None
        c = bb.c
        return StepResult(n=[int(c.n[k]) for k in range(self.K + 1)], e=[int(c.e[k]) for k in range(self.K)],
                          local=int(c.local), hits=int(c.hits), misses=int(c.misses), host_rows=int(c.host_rows))

    def evict_step(self, out=None, wait: bool = True) -> int:
        """Runs the round owed by the last step; out = (evicted, slots, replaced)
        int32 device tensors with room for cap entries, or None. wait=False
        only enqueues it (returns -1)."""
        ev, sl, rp = (None, None, None) if out is None else tuple(_ptr(x) for x in out)
        if not wait:
            self._check(self._lib.massive_evict_step(self._h, ev, sl, rp, None))
            return -1
        k = ctypes.c_int64()
        self._check(self._lib.massive_evict_step(self._h, ev, sl, rp, ctypes.byref(k)))
        return int(k.value)

    def counters(self):
        """(rounds that evicted, slots evicted) since init."""
        r, e = ctypes.c_int64(), ctypes.c_int64()
        self._check(self._lib.massive_get_counters(self._h, ctypes.byref(r), ctypes.byref(e), None))
        return int(r.value), int(e.value)

    def refilled_rows(self):
        """Rows the refill has copied over the host link since init (the
        initial fill included)."""
        f = ctypes.c_int64()
        self._check(self._lib.massive_get_counters(self._h, None, None, ctypes.byref(f)))
        return int(f.value)

    def state(self):
        sid = np.zeros(max(self.cap, 1), np.int32)
        se = np.zeros(max(self.cap, 1), np.float32)
        sa = np.zeros(max(self.H, 1), np.float32)
        t = ctypes.c_int64()
        self._check(self._lib.massive_get_state(self._h, sid.ctypes.data, se.ctypes.data, sa.ctypes.data,
                                                ctypes.byref(t)))
        return sid[:self.cap].copy(), se[:self.cap].copy(), sa[:self.H].copy(), int(t.value)

    def buffer_rows(self) -> np.ndarray:
        out = np.zeros((max(self.cap, 1), self.row_bytes), np.uint8)
        self._check(self._lib.massive_get_buffer_rows(self._h, out.ctypes.data))
        return out[:self.cap]

    def set_timing(self, on=True):
        """on: True (every group), False (off), or an iterable of group names
        from TIMING_GROUPS."""
        if on is True or on is False:
            mask = TIMING_ALL if on else 0
        else:
            mask = 0
            for g in on:
                mask |= 1 << TIMING_GROUPS.index(g)
        self._check(self._lib.massive_set_timing(self._h, mask))

    def timing(self):
        ms = np.zeros(len(TIMING_GROUPS), np.float64)
        calls = np.zeros(len(TIMING_GROUPS), np.int64)
        self._check(self._lib.massive_get_timing(self._h, ms.ctypes.data, calls.ctypes.data))
        return {g: (float(ms[i]), int(calls[i])) for i, g in enumerate(TIMING_GROUPS)}
