#!/usr/bin/env python3
"""Benchmark: per-minibatch sampling + halo prefetch buffer + feature gather
(MassiveGNN, arXiv 2410.22697) for one partition on one MI355X.

A step is one minibatch through the whole path: massive_sample (3-hop fanout
sampling, dedup/relabel, buffer lookup, scoring, HBM gather, miss fetch from
pinned host memory) followed by massive_evict_step (the periodic eviction
and replacement round, with its refill overlapping the next steps). Inputs
(graph, features, seed batches) are resident before any timed region.

Prints one JSON line for the papers-sized share (cl111m_p64):
  - value: minibatches/s over `--steps` steps that lie after the first
    eviction round and contain a round (the eviction regime; the window rule
    is in window_plan), with the gather kernel against the HBM roofline, the
    miss fetch against the host link, and the bound of the whole minibatch
    computed from measured fractions;
  - early_window: the `--steps` steps right after warm-up (before any round
    for a short window: the initial buffer only);
  - eviction_run: a fresh context from init through five rounds, every
    kernel group timed over its own steps, with the per-step hit rate;
  - sampler: the last hop's sampler kernel against the VALU issue rate;
  - configs: the four smaller workloads, their stated runs and the extended
    runs of those whose stated run reaches no round (child processes);
  - cpu_baseline: the CPU oracle on a bounded sample of the same workload.
"""
import argparse
import contextlib
import gc
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0       # MI355X HBM3E
PCIE_PEAK_GBPS = 64.0        # PCIe 5.0 x16, one direction
LINK_CEILING_GBPS = 55.0     # measured: zero-copy row reads of a pinned store by 16 blocks
# Batches in flight (the library allows up to three): with two, the next
# step's sampling overlaps the current step's host-link reads and never the
# HBM gather; a third lets sampling run beside the HBM gather too, which
# slows it, with no gain while the host link bounds the step.
DEFAULT_DEPTH = 2
# VALU issue peak of the sampler, in Philox keys per second: 256 CUs issue one
# wave64 VALU instruction per clock each (four SIMDs, four clocks per wave64
# instruction) at 2.4 GHz; one pass of the sampler's inner loop is 42 VALU
# instructions for 64 Philox4x32-10 blocks = 256 keys (the block function's
# 20 multiplies and 20 three-way XORs less the two hoisted products, plus the
# below-threshold test).
SAMPLER_VALU_PER_256_KEYS = 42
SAMPLER_PEAK_KEYS_PER_S = 256 * 2.4e9 * 256 / SAMPLER_VALU_PER_256_KEYS
EVICTION_RUN_ROUNDS = 5      # the eviction run covers steps 0 .. 5 delta
SAMPLER_STEPS = 16           # steps of the sampler measurement
# the smaller workloads: stated runs, and extended runs (four rounds) for
# those whose stated run ends before the first round
CONFIG_GROUPS = (("cl10k", "cl170k"), ("cl2m45",), ("cl2m45_bf16",))
EXTENDED_ROUNDS = 4
# how rows cross the host link in every context of this process (--link)
LINK = {"link": "loads", "link_threads": 0}


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def build_inputs(w, threads=None):
    import torch
    import synth
    t0 = time.time()
    g = synth.partition_graph(w, threads)
    log("graph %s: L=%d H=%d nnz=%d (%.1fs)" % (w.name, g.L, g.H, g.nnz, time.time() - t0))
    t0 = time.time()
    rb = w.row_bytes
    local = np.empty((g.L, rb), np.uint8)
    synth.fill_features(g.local_gid, w.d, w.dtype, w.seed, local.ctypes.data, threads)
    store = torch.empty((max(g.H, 1), rb), dtype=torch.uint8, pin_memory=True)
    synth.fill_features(g.halo_gid, w.d, w.dtype, w.seed, store.data_ptr(), threads)
    log("features: %d local + %d pinned halo rows of %d B (%.1fs)" % (g.L, g.H, rb, time.time() - t0))
    sched = synth.Schedule(g.L, w.train_pct, w.batch, w.seed)
    return g, local, store, sched


def save_inputs(w, g, local, store, d):
    """The inputs of a workload written once under d (/dev/shm), for child
    processes that map them instead of generating the graph again."""
    os.makedirs(d, exist_ok=True)
    for name, arr in (("indptr", g.indptr), ("indices", g.indices), ("halo_gid", g.halo_gid),
                      ("halo_degree", g.halo_degree), ("local", local), ("store", store.numpy()[:max(g.H, 1)])):
        np.save(os.path.join(d, name + ".npy"), arr)
    json.dump({"workload": w.name, "L": int(g.L), "H": int(g.H)}, open(os.path.join(d, "meta.json"), "w"))


def load_inputs(w, d):
    """A child's view of the inputs saved by save_inputs: the graph arrays
    memory-mapped, the halo store copied into pinned memory."""
    import types
    import torch
    import synth
    meta = json.load(open(os.path.join(d, "meta.json")))
    assert meta["workload"] == w.name, (meta, w.name)
    m = {k: np.load(os.path.join(d, k + ".npy"), mmap_mode="r")
         for k in ("indptr", "indices", "halo_gid", "halo_degree", "local", "store")}
    g = types.SimpleNamespace(L=meta["L"], H=meta["H"], indptr=m["indptr"], indices=m["indices"],
                              halo_gid=m["halo_gid"], halo_degree=m["halo_degree"], nnz=int(m["indices"].shape[0]))
    store = torch.empty(m["store"].shape, dtype=torch.uint8, pin_memory=True)
    store.numpy()[:] = m["store"]
    sched = synth.Schedule(g.L, w.train_pct, w.batch, w.seed)
    return g, np.asarray(m["local"]), store, sched


class SharedInputs:
    """A /dev/shm directory holding one workload's inputs for the children of
    a parent process; removed when the parent leaves the with-block."""

    def __init__(self, w, threads=None):
        self.w, self.threads = w, threads
        self.dir = "/dev/shm/massive_bench_%d" % os.getpid()

    def __enter__(self):
        g, local, store, _ = build_inputs(self.w, self.threads)
        t0 = time.time()
        save_inputs(self.w, g, local, store, self.dir)
        log("inputs shared in %s (%.1fs)" % (self.dir, time.time() - t0))
        del g, local, store
        return self.dir

    def __exit__(self, *exc):
        import shutil
        shutil.rmtree(self.dir, ignore_errors=True)
        return False


@contextlib.contextmanager
def no_gc():
    """A timed region without Python's garbage collector: a full collection
    first, none inside (one landing in a timed window cost ~37 ms after a long
    earlier context in the same process)."""
    gc.collect()
    was = gc.isenabled()
    gc.disable()
    try:
        yield
    finally:
        if was:
            gc.enable()


def window_plan(warmup, steps, delta, limit=20000):
    """The two timed windows of the default run, each [start, stop):
    early = the `steps` steps right after warm-up (before the first round when
    warmup + steps <= delta + 1); headline = `steps` steps after the first
    round (t = delta), so that refill traffic is in its steady state, that
    contain a round: a window shorter than delta is centred on a round at
    2 delta or later; a longer one starts right after the first round (any
    delta consecutive steps hold a round). The headline never overlaps the
    early window. An interval too long for this (a static buffer) gives the
    early window only (headline = early)."""
    warmup = max(1, warmup)  # step 0 runs alone
    early = (warmup, warmup + steps)
    if 2 * delta + 2 * steps + warmup > limit:
        return early, early
    if steps >= delta:
        s = max(warmup + steps, delta + 1)
    else:
        r = delta * max(2, -(-(warmup + steps + steps // 2) // delta))
        s = r - steps // 2
    return early, (s, s + steps)


def frontier_keys(indptr, nodes, fanout):
    """Philox keys one hop draws by definition: d keys for every frontier row
    longer than the fanout (shorter rows are copied whole)."""
    d = indptr[nodes + 1] - indptr[nodes]
    return int(d[d > fanout].sum())


def run_context(w, g, local, store, sched, windows, depth=None, log_steps=False, copy_probe=False,
                first_alone=True, sampler_steps=0, score_layout="rank"):
    """One context from init over steps 0..end-1 with look-ahead (`depth`
    batches in flight: step t is enqueued, after step t-1's round, before step
    t - depth + 1 is waited for, so the sampling of the next steps overlaps the
    host-link reads of earlier ones).
    first_alone: step 0 runs alone first, and its outputs and the state after
    it are kept for the oracle check.
    windows: (label, start, stop, groups), in step order: steps [start, stop)
    are timed on the host clock between two synchronisations, with HIP events
    on the kernel groups `groups` (True: every group); steps between windows
    run untimed.
    sampler_steps: that many more steps time the last hop's sampler dispatch
    and count its keys on the host (each step's frontier is copied back,
    which holds the pipeline a little)."""
    import torch
    from paper_2410_22697_amd import Massive
    depth = depth or DEFAULT_DEPTH
    torch.cuda.set_device(0)
    end = max([1] + [b for _, _, b, _ in windows])
    total = end + sampler_steps
    t0 = time.time()
    free0 = torch.cuda.mem_get_info()[0]
    gm = Massive(g.L, g.H, g.indptr, g.indices, g.halo_gid, g.halo_degree, local, store, w.row_bytes,
                 w.fanout, w.buffer_pct, w.gamma, w.delta, w.philox_seed, score_layout=score_layout,
                 n_global=w.n, link=LINK["link"], link_threads=LINK["link_threads"])
    torch.cuda.synchronize()
    init_s = time.time() - t0
    ctx_bytes = free0 - torch.cuda.mem_get_info()[0]  # device memory the context holds
    log("%s: massive_init %.2fs: cap=%d alpha=%.6g" % (w.name, init_s, gm.cap, gm.alpha))
    bbs = [gm.alloc_batch(w.batch) for _ in range(depth)]
    seeds_dev = [torch.from_numpy(np.ascontiguousarray(sched.seeds(t), np.int32)).cuda() for t in range(total)]
    torch.cuda.synchronize()

    if copy_probe:
        a = torch.empty(256 << 20, dtype=torch.uint8, device="cuda").fill_(1)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        log("copy probe: 256 MiB device-to-device copy done")
        del a, b

    first_steps = []  # the first steps' outputs, checked against the oracle
    stats = []        # per step: local, hits, misses, rows, host-link rows
    sizes = []        # per step: frontier sizes n_0..n_K and sampled edges e_1..e_K
    keys = []         # per sampler step: keys of the last hop
    count_keys = [False]
    K = len(w.fanout)

    def finish(u):
        bb = bbs[u % depth]
        r = gm.wait(bb)
        stats.append((r.local, r.hits, r.misses, r.n[-1], r.host_rows))
        sizes.append((list(r.n), list(r.e)))
        if first_alone and u < 2 and len(first_steps) == u:
            nK = r.n[-1]
            blocks = [(bb.indptr[k][:r.n[k] + 1].cpu().numpy().copy(), bb.indices[k][:r.e[k]].cpu().numpy().copy())
                      for k in range(K)]
            first_steps.append((r, bb.nodes[:nK].cpu().numpy().copy(), bb.mask[:nK].cpu().numpy().copy(),
                                bb.feat[:nK].cpu().numpy().copy(), blocks))
        if count_keys[0]:
            keys.append(frontier_keys(g.indptr, bb.nodes[:r.n[K - 1]].cpu().numpy().astype(np.int64),
                                      w.fanout[-1]))
        if log_steps:
            log("step %d local %d hits %d misses %d rows %d host %d" % (u, r.local, r.hits, r.misses, r.n[-1],
                                                                        r.host_rows))

    def run(a, b):
        inflight = []
        for t in range(a, b):
            gm.sample_async(seeds_dev[t], bbs[t % depth])
            gm.evict_step(wait=False)
            inflight.append(t)
            if len(inflight) == depth:
                finish(inflight.pop(0))
        for u in inflight:
            finish(u)

    state0 = None
    pos = 0
    if first_alone:
        run(0, 1)
        state0 = gm.state()
        pos = 1
    out_w = {}
    for label, a, b, groups in windows:
        assert a >= pos and b > a, (label, a, b, pos)
        run(pos, a)
        r0, e0 = gm.counters()
        f0 = gm.refilled_rows()
        gm.set_timing(groups)
        torch.cuda.synchronize()
        with no_gc():
            t0 = time.perf_counter()
            run(a, b)
            torch.cuda.synchronize()
            el = time.perf_counter() - t0
        tim = gm.timing()
        r1, e1 = gm.counters()
        f1 = gm.refilled_rows()
        gm.set_timing(False)
        out_w[label] = dict(start=a, stop=b, elapsed=el, tim=tim, rounds=r1 - r0, evicted=e1 - e0,
                            refilled=f1 - f0, groups=groups)
        log("%s %s: steps %d..%d in %.4fs: %.1f minibatches/s, %d rounds" % (w.name, label, a, b - 1, el,
                                                                          (b - a) / el, r1 - r0))
        pos = b
    sampler = None
    if sampler_steps:
        gm.set_timing(["sample_last_hop"])
        count_keys[0] = True
        run(pos, pos + sampler_steps)
        count_keys[0] = False
        ms, calls = gm.timing()["sample_last_hop"]
        sampler = dict(ms=ms, calls=calls, keys=list(keys), steps=(pos, pos + sampler_steps))
        gm.set_timing(False)
    out = dict(gm_cap=gm.cap, H=g.H, alpha=gm.alpha, init_s=init_s, depth=depth, ctx_bytes=ctx_bytes,
               stats=np.array(stats, np.float64), sizes=sizes, windows=out_w,
               first_steps=first_steps, state0=state0, sampler=sampler)
    del bbs, seeds_dev
    gm.close()
    torch.cuda.synchronize()
    return out


def copy_reference(nbytes, reps=20, regions=8):
    """GB/s of a plain contiguous device-to-device copy (torch copy_) that
    reads nbytes/2 and writes nbytes/2, as the gather does per launch: the
    practical ceiling for a copy of this size on this GPU. Consecutive copies
    read and write different regions (8 of each, together well over the
    256 MB Infinity Cache), so that, like the gather's rows, the data comes
    from HBM and not from the cache. Each copy is timed between events recorded
    around it alone (the markers add a little time; the kernel trace of
    --copy-probe runs times the same copies exactly)."""
    import torch
    half = int(nbytes // 2)
    stride = (half + 4095) // 4096 * 4096  # every region starts 4 KiB-aligned, as an allocation would
    a = torch.empty(regions * stride, dtype=torch.uint8, device="cuda").fill_(1)
    b = torch.empty_like(a)
    ra = [a[r * stride:r * stride + half] for r in range(regions)]
    rb = [b[r * stride:r * stride + half] for r in range(regions)]
    for i in range(3):
        rb[i % regions].copy_(ra[(i + 3) % regions])
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    torch.cuda.synchronize()
    for i, (e0, e1) in enumerate(ev):
        e0.record()
        rb[i % regions].copy_(ra[(i + 5) % regions])
        e1.record()
    torch.cuda.synchronize()
    s = float(np.median([e0.elapsed_time(e1) for e0, e1 in ev])) / 1e3
    del a, b, ra, rb
    return 2 * half / s / 1e9


def alg_hbm_bytes(n, e, loc, hit, mis, rb):
    """HBM bytes one minibatch must move by the method's definition, whatever
    the implementation: per hop, the frontier row's id and CSR offsets (16 B),
    the selected ids, the block offsets and block entries, and ~12 B per
    sampled edge for dedup/relabel; then ~13 B per input row to classify and
    mark it, the local and buffer rows read and written, the miss rows
    written, and 8 B of score traffic per halo row."""
    b = 0
    for k in range(len(e)):
        b += 16 * n[k] + 4 * e[k] + 4 * (n[k] + 1) + 4 * e[k] + 12 * e[k]
    return b + 13 * n[-1] + 2 * (loc + hit) * rb + mis * rb + 8 * (mis + hit)


MAIN_STREAM_GROUPS = ("sample_dedup", "classify")


def summarize(w, res, label):
    """One timed window: throughput, the gather against the HBM roofline, the
    miss fetch against the host link, the hit rate, and the bound of the whole
    minibatch, taken as the largest of three measured fractions: HBM
    (algorithmic bytes per second over 8 TB/s), host link (bytes that crossed
    it per second over 64 GB/s) and the main stream (the share of the step its
    sampling, dedup and classify kernels occupy, when those groups are timed)."""
    win = res["windows"][label]
    a, b = win["start"], win["stop"]
    K, rb = b - a, w.row_bytes
    st = res["stats"][a:b]
    loc, hit, mis, host_rows = st[:, 0], st[:, 1], st[:, 2], st[:, 4]
    hbm_rows = loc + hit
    tim = win["tim"]
    el = win["elapsed"]
    mbps = K / el
    g_ms, g_calls = tim["gather_hbm"]
    g_bytes = float(np.mean(2 * hbm_rows * rb + 8 * hbm_rows))
    g_avg_s = g_ms / 1e3 / g_calls if g_calls else None
    m_ms, m_calls = tim["gather_miss"]
    m_bytes = float(np.mean(host_rows * rb))
    sz = res["sizes"][a:b]
    b_alg = float(np.mean([alg_hbm_bytes(n, e, l, h, m, rb) for (n, e), (l, h, m) in zip(sz, st[:, :3])]))
    # eviction rounds, amortised: S_E/slot scans and S_A/rank scans, and the replacement rows written
    b_alg += (win["rounds"] * (12 * res["gm_cap"] + 8 * res["H"]) + win["evicted"] * rb) / K
    link_bytes = float(host_rows.sum()) * rb + win["refilled"] * rb
    link_gbps = link_bytes / el / 1e9
    hbm_gbps = mbps * b_alg / 1e9
    phases = {k: round(v[0] / K, 4) for k, v in tim.items() if v[1]}
    fr = {"hbm": hbm_gbps / HBM_PEAK_GBPS, "host_link": link_gbps / PCIE_PEAK_GBPS}
    main_ms = None
    if all(tim[gname][1] for gname in MAIN_STREAM_GROUPS):
        main_ms = sum(tim[gname][0] for gname in MAIN_STREAM_GROUPS) / K
        fr["main_stream"] = main_ms / (1e3 * el / K)
    bound = max(fr, key=fr.get)
    out = {
        "steps_timed": [a, b - 1], "eviction_rounds": win["rounds"], "evicted_rows": win["evicted"],
        "refilled_rows": win["refilled"],
        "value": round(mbps, 3), "unit": "minibatches/s", "ms_per_step": round(1e3 * el / K, 4),
        "hit_rate": round(float(hit.sum() / max(hit.sum() + mis.sum(), 1)), 4),
        "gather_hbm": None if g_avg_s is None else {
            "bytes_per_launch": round(g_bytes), "avg_us": round(g_avg_s * 1e6, 2),
            "GBps": round(g_bytes / g_avg_s / 1e9, 1), "frac_hbm": round(g_bytes / g_avg_s / 1e9 / HBM_PEAK_GBPS, 4)},
        "gather_miss": None if not m_calls else {
            "bytes_per_launch": round(m_bytes), "avg_us": round(1e3 * m_ms / m_calls, 2),
            "GBps": round(m_bytes / (m_ms / 1e3 / m_calls) / 1e9, 2) if m_ms > 0 else None},
        "minibatch_roofline": {
            "bound": {"hbm": "hbm", "host_link": "host link", "main_stream": "main stream (sampling, dedup, classify)"}[bound],
            "fractions": {k: round(v, 4) for k, v in fr.items()},
            "hbm_alg_bytes_per_step": round(b_alg), "hbm_GBps": round(hbm_gbps, 1),
            "link_bytes_per_step": round(link_bytes / K), "link_GBps": round(link_gbps, 2),
            "link_peak_GBps": PCIE_PEAK_GBPS, "link_ceiling_measured_GBps": LINK_CEILING_GBPS,
            "main_stream_ms_per_step": None if main_ms is None else round(main_ms, 4)},
        "host_rows_per_step": round(float(np.mean(host_rows)), 1),
        "refill_rows_per_step": round(win["refilled"] / K, 1),
        "remote_rows_per_step": round(float(np.mean(host_rows)) + win["refilled"] / K, 1),
        "halo_rows_per_step": round(float(np.mean(hit + mis)), 1),
        "phase_ms_per_step": phases,
        "phases_timed": "every kernel group" if win["groups"] is True else list(win["groups"] or []),
    }
    return out


def gather_traffic(window, workload):
    """HBM bytes per gather_hbm launch over the headline window, measured by
    rocprofv3 counters (FETCH_SIZE, then WRITE_SIZE, scaled by a plain copy)
    on the same command, from the committed summary; None unless the summary
    covers this workload and window and the gather kernel's source is the one
    the counters were taken on."""
    import hashlib
    prof = os.path.join(ROOT, "profiles", "gather_hbm_%s_hbm_counters.txt" % workload)
    src = open(os.path.join(ROOT, "paper_2410_22697_amd", "csrc", "buffer_kernels.hpp")).read()
    a, b = src.find("// ---------------------------------------------------------------- gather"), src.find("// misses: pinned host store")
    if not os.path.exists(prof) or a < 0 or b < 0:
        return None
    kv = dict(l.split(": ", 1) for l in open(prof).read().splitlines() if ": " in l and not l.startswith(" "))
    if kv.get("gather_source_sha256") != hashlib.sha256(src[a:b].encode()).hexdigest():
        return None
    if kv.get("window_steps") != "%d..%d" % (window[0], window[1] - 1):
        return None
    return int(kv["traffic_bytes_per_launch"])


def sampler_summary(res, w):
    s = res["sampler"]
    if not s or not s["calls"]:
        return None
    keys = float(np.mean(s["keys"]))
    avg_s = s["ms"] / 1e3 / s["calls"]
    kps = keys / avg_s
    return {"kernel": "k_sample_waves (hop %d)" % len(w.fanout), "bound": "alu", "steps": list(s["steps"]),
            "keys_per_launch": round(keys), "avg_us": round(avg_s * 1e6, 2), "achieved": round(kps / 1e12, 4),
            "peak": round(SAMPLER_PEAK_KEYS_PER_S / 1e12, 4), "unit": "T keys/s",
            "frac": round(kps / SAMPLER_PEAK_KEYS_PER_S, 4),
            "peak_from": "256 CUs x 2.4 GHz x 1 wave64 VALU instruction per clock x 256 keys per %d instructions"
                         % SAMPLER_VALU_PER_256_KEYS,
            "keys_from": "sum of row lengths over the hop's frontier rows longer than the fanout (one Philox "
                         "key per position), counted on the host from the same steps"}


def config_entry(w, res, label, kind):
    """A compact record of one run of a smaller workload."""
    sm = summarize(w, res, label)
    g = sm["gather_hbm"]
    mr = sm["minibatch_roofline"]
    return {"kind": kind, "steps": res["windows"][label]["stop"], "from_init": True,
            "value": sm["value"], "unit": "minibatches/s", "ms_per_step": sm["ms_per_step"],
            "eviction_rounds": sm["eviction_rounds"], "evicted_rows": sm["evicted_rows"],
            "hit_rate": sm["hit_rate"], "gather_frac_hbm": g["frac_hbm"] if g else None,
            "gather_GBps": g["GBps"] if g else None, "link_GBps": mr["link_GBps"],
            "bound": mr["bound"], "fractions": mr["fractions"], "init_s": round(res["init_s"], 3)}


def config_run(names, args):
    """Child mode: the smaller workloads' runs, one JSON line per workload.
    A workload whose stated run reaches no round (its run is shorter than
    delta + 1) also gets an extended run of four rounds. Every run is one
    context from init, timed from step 0 to its end with every kernel group
    timed. The 10K-node workload's stated run is short enough for the oracle:
    it is timed in full and its per-step sizes and counts compared."""
    import synth
    for name in names:
        w = synth.get(name)
        g, local, store, sched = build_inputs(w, args.threads)
        entry = {"workload": name, "stands_in_for": w.note or None, "nodes": w.n, "partitions": w.parts,
                 "L": g.L, "H": g.H, "csr_entries": g.nnz, "batch": w.batch, "fanout": list(w.fanout),
                 "row_bytes": w.row_bytes, "dtype": w.dtype, "buffer_pct": w.buffer_pct, "gamma": w.gamma,
                 "delta": w.delta, "runs": []}
        lengths = [("stated", w.steps)]
        if w.steps < w.delta + 1:
            lengths.append(("extended", EXTENDED_ROUNDS * w.delta + 1))
        for kind, n in lengths:
            res = run_context(w, g, local, store, sched, [("run", 0, n, True)], first_alone=False)
            e = config_entry(w, res, "run", kind)
            if kind == "stated" and name == "cl10k" and not args.no_cpu:
                e["cpu_baseline"] = oracle_full_run(w, g, local, store, sched, n, res)
            entry["runs"].append(e)
            log("%s %s run: %d steps, %.1f minibatches/s, %d rounds, hit rate %.3f" %
                (name, kind, n, e["value"], e["eviction_rounds"], e["hit_rate"]))
        print(json.dumps(entry), flush=True)


def oracle_full_run(w, g, local, store, sched, n, res):
    """The oracle over a whole stated run, timed; each step's sizes and class
    counts are compared with the GPU run's."""
    import oracle
    orc = oracle.Oracle(g.L, g.H, g.indptr, g.indices, g.halo_gid, g.halo_degree, local, store.numpy(),
                        w.row_bytes, w.fanout, w.buffer_pct, w.gamma, w.delta, w.philox_seed)
    with no_gc():
        t0 = time.perf_counter()
        for t in range(n):
            st = orc.sample(sched.seeds(t))
            orc.evict_step()
            (gn, ge), row = res["sizes"][t], res["stats"][t]
            if gn != st.n or ge != st.e or (int(row[0]), int(row[1]), int(row[2])) != (st.local, st.hits, st.misses):
                raise SystemExit("bench: %s step %d differs from the oracle" % (w.name, t))
        el = time.perf_counter() - t0
    return {"value": round(n / el, 3), "unit": "minibatches/s", "cores": 1, "kind": "oracle",
            "sample": "the whole %d-step run from init; every step's sizes and class counts equal the GPU's" % n}


def configs_in_children(args):
    """Runs the smaller workloads in child processes (at most two contexts
    each) and collects their lines."""
    import subprocess
    out = []
    for group in CONFIG_GROUPS:
        cmd = [sys.executable, os.path.abspath(__file__), "--config-run", ",".join(group)]
        if args.no_cpu:
            cmd.append("--no-cpu")
        if args.threads:
            cmd += ["--threads", str(args.threads)]
        cmd += ["--link", args.link, "--link-threads", str(args.link_threads)]
        log("configs %s: %s" % (",".join(group), " ".join(cmd[1:])))
        r = subprocess.run(cmd, stdout=subprocess.PIPE, text=True)
        if r.returncode != 0:
            raise SystemExit("bench: the config run %s failed with status %d" % (",".join(group), r.returncode))
        out += [json.loads(l) for l in r.stdout.splitlines() if l.startswith("{")]
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1, help="GPUs (one partition runs on one GPU: only 1)")
    ap.add_argument("--steps", type=int, default=192, help="timed minibatches per window")
    ap.add_argument("--warmup", type=int, default=8, help="untimed minibatches before the early window")
    ap.add_argument("--workload", default="cl111m_p64", help="a named synthetic workload (synth/workloads.py)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0, help="budget of the oracle baseline")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle baselines")
    ap.add_argument("--no-configs", action="store_true", help="skip the smaller workloads")
    ap.add_argument("--no-eviction-run", action="store_true", help="skip the eviction run and the sampler pass")
    ap.add_argument("--threads", type=int, default=None, help="host threads of the input generator")
    ap.add_argument("--log-steps", action="store_true", help="per-step row counts on stderr")
    ap.add_argument("--link", choices=("loads", "staged"), default="loads",
                    help="how rows cross the host link: kernel loads of the pinned store, or host threads "
                         "gathering into pinned staging and DMA copies")
    ap.add_argument("--link-threads", type=int, default=0, help="host gather threads of --link staged (0: default)")
    ap.add_argument("--depth", type=int, default=DEFAULT_DEPTH, help="batches in flight (1 to 3)")
    ap.add_argument("--delta", type=int, default=None, help="override the eviction interval")
    ap.add_argument("--gamma", type=float, default=None, help="override the decay factor")
    ap.add_argument("--buffer-pct", type=int, default=None, help="override f (percent of the halo)")
    ap.add_argument("--headline-groups", default="all",
                    help="kernel groups timed with HIP events in the headline window: 'all', or a comma list "
                         "of sample_dedup,classify,gather_hbm,gather_miss,evict_round,refill")
    ap.add_argument("--early-groups", default="all", help="kernel groups timed in the early window (as above)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="one plain 256 MiB device copy before warmup (reference for HBM byte counters)")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"), default=None,
                    help="summarise two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of this bench with "
                         "--copy-probe: the gather's HBM bytes over the headline window")
    ap.add_argument("--config-run", default=None, help=argparse.SUPPRESS)
    ap.add_argument("--inputs-dir", default=None, help=argparse.SUPPRESS)
    ap.add_argument("--sweep-point", nargs=4, default=None, metavar=("KIND", "F", "GAMMA", "DELTA"),
                    help=argparse.SUPPRESS)
    ap.add_argument("--layouts", action="store_true",
                    help="the two S_A layouts of Section IV-B (over the halo in rank order, over every global "
                         "id) on the same eviction run, each in its own process: device memory, round time, "
                         "throughput, and that both give the same results; one JSON line each")
    ap.add_argument("--layout-run", choices=("rank", "gid"), default=None, help=argparse.SUPPRESS)
    ap.add_argument("--sweep", action="store_true",
                    help="the paper's parameter grid (f in 15/25/35/50 %%, gamma in 0.95/0.995/0.9995, delta in "
                         "16..1024) on the same inputs, plus no buffer and one static run per f; one JSON line each")
    ap.add_argument("--sweep-steps", type=int, default=1032, help="timed steps per sweep point (after 8 warm-up)")
    ap.add_argument("--sweep-f", default="15,25,35,50", help="buffer sizes f (percent) of the sweep")
    ap.add_argument("--overlap", action="store_true",
                    help="Alg. 1's look-ahead against a stand-in trainer on its own stream (Section IV-C): "
                         "path alone, trainer alone, serial and overlapped steps per trainer size")
    ap.add_argument("--compare", action="store_true",
                    help="the paper's comparison on the same inputs: no buffer (f = 0), prefetch without "
                         "eviction (no round within the run) and prefetch with eviction; one JSON line each")
    ap.add_argument("--compare-mode", choices=COMPARE_MODES, default=None,
                    help="run one mode of --compare in this process (used by --compare itself)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (each partition's "
              "buffer is private to its trainer); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    LINK.update(link=args.link, link_threads=args.link_threads)
    if args.pmc_summary:
        pmc_summary(args)
        return
    if args.config_run:
        config_run(args.config_run.split(","), args)
        return
    import synth

    w = synth.get(args.workload)
    over = {k: v for k, v in (("delta", args.delta), ("gamma", args.gamma), ("buffer_pct", args.buffer_pct))
            if v is not None}
    if over:
        w = w.with_(**over)
    parent_argv = [a for a in sys.argv[1:] if a not in ("--compare", "--layouts", "--sweep")]
    if "--sweep-f" in parent_argv:  # the grid is the parent's business
        i = parent_argv.index("--sweep-f")
        del parent_argv[i:i + 2]
    if args.compare and args.compare_mode is None:
        with SharedInputs(w, args.threads) as d:
            compare(parent_argv + ["--inputs-dir", d])
        return
    if args.layouts:
        with SharedInputs(w, args.threads) as d:
            layouts(parent_argv + ["--inputs-dir", d])
        return
    if args.sweep and args.sweep_point is None:
        with SharedInputs(w, args.threads) as d:
            sweep(w, args, parent_argv + ["--inputs-dir", d])
        return
    if args.inputs_dir:
        g, local, store, sched = load_inputs(w, args.inputs_dir)
    else:
        g, local, store, sched = build_inputs(w, args.threads)
    if args.sweep_point:
        print(json.dumps(sweep_point(w, args, g, local, store, sched)), flush=True)
        return
    if args.compare:
        print(json.dumps(compare_one(w, args.compare_mode, g, local, store, sched, args)), flush=True)
        return
    if args.layout_run:
        print(json.dumps(layout_one(w, args.layout_run, g, local, store, sched, args)), flush=True)
        return
    if args.overlap:
        overlap(w, g, local, store, sched, args)
        return

    K = args.steps
    early, head = window_plan(args.warmup, K, w.delta)
    def groups(spec):
        return True if spec == "all" else [x for x in spec.split(",") if x]
    hg = groups(args.headline_groups)
    windows = [("early", early[0], early[1], groups(args.early_groups))]
    if head != early:
        windows.append(("headline", head[0], head[1], hg))
    res = run_context(w, g, local, store, sched, windows, args.depth, args.log_steps, args.copy_probe)
    hl = "headline" if head != early else "early"
    sm = summarize(w, res, hl)
    sm_early = summarize(w, res, "early")
    evr = None
    if not args.no_eviction_run:
        n_ev = EVICTION_RUN_ROUNDS * w.delta + 1 if 2 * w.delta + K < 20000 else 2 * K
        rev = run_context(w, g, local, store, sched, [("run", 0, n_ev, True)], args.depth, first_alone=False,
                          sampler_steps=SAMPLER_STEPS)
        evr = summarize(w, rev, "run")
        st = rev["stats"][:n_ev]
        evr["hit_rate_per_step"] = (st[:, 1] / np.maximum(st[:, 1] + st[:, 2], 1)).round(4).tolist()
        evr["from_init"] = True
        evr["sampler"] = sampler_summary(rev, w)

    g_ = sm["gather_hbm"]
    log("headline window steps %d..%d: %.1f minibatches/s, %d rounds, hit rate %.3f, bound %s %s" %
        (head[0], head[1] - 1, sm["value"], sm["eviction_rounds"], sm["hit_rate"], sm["minibatch_roofline"]["bound"],
         sm["minibatch_roofline"]["fractions"]))
    log("gather_hbm %d B/launch, %.1f us, %.1f GB/s (%.1f%% of HBM)" % (g_["bytes_per_launch"], g_["avg_us"],
                                                                       g_["GBps"], 100 * g_["frac_hbm"]))
    copy_gbps = copy_reference(g_["bytes_per_launch"])
    log("plain device copy moving the same bytes: %.1f GB/s; the gather reaches %.1f%% of it" %
        (copy_gbps, 100 * g_["GBps"] / copy_gbps))

    configs = None if args.no_configs else configs_in_children(args)
    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(w, g, local, store, sched, args.cpu_seconds, res["first_steps"], res["state0"])

    traffic = gather_traffic(head, w.name)
    out = {
        "metric": "sampled+gathered minibatches/s; gather GB/s (% HBM peak); halo buffer hit rate",
        "value": sm["value"],
        "unit": "minibatches/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": head[0],
        "ms_per_step": sm["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if w.dtype == "f32" else "bf16",
        "data": "synthetic (seeded Chung-Lu power-law graph, N(0,1) features)",
        "config": {"workload": w.name, "stands_in_for": w.note or None, "nodes": w.n, "partitions": w.parts,
                   "partition": 0,
                   "L": g.L, "H": g.H, "csr_entries": g.nnz, "batch": w.batch, "fanout": list(w.fanout),
                   "row_bytes": w.row_bytes, "buffer_pct": w.buffer_pct, "gamma": w.gamma, "delta": w.delta,
                   "cap": res["gm_cap"], "steps_timed": sm["steps_timed"],
                   "eviction_rounds": sm["eviction_rounds"], "evicted_rows": sm["evicted_rows"],
                   "refilled_rows": sm["refilled_rows"], "lookahead": res["depth"] - 1,
                   "warmup_requested": args.warmup,
                   "window_rule": "the timed steps lie after the first eviction round and contain a round "
                                  "(centred on one when shorter than delta); the steps before them run untimed",
                   "parallelism": "one partition on one GPU", "link": LINK["link"]},
        "gather_GBps": g_["GBps"],
        "gather_frac_hbm": g_["frac_hbm"],
        "hit_rate": sm["hit_rate"],
        "roofline": {"bound": "hbm", "kernel": "gather_hbm", "achieved": g_["GBps"], "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": g_["frac_hbm"], "traffic": traffic,
                     "traffic_from": None if traffic is None else
                     "rocprofv3 --pmc FETCH_SIZE and WRITE_SIZE runs of the same command, averaged over the "
                     "same window's launches, scaled by a plain copy's counters",
                     "bytes_per_launch": g_["bytes_per_launch"], "avg_us": g_["avg_us"],
                     "plain_copy_same_bytes_GBps_events": round(copy_gbps, 1),
                     "frac_of_plain_copy": round(g_["GBps"] / copy_gbps, 4)},
        "host_link": dict(sm["gather_miss"] or {}, kernel="gather_miss", peak=PCIE_PEAK_GBPS, unit="GB/s",
                          link_GBps_window=sm["minibatch_roofline"]["link_GBps"],
                          refill_rows_per_step=sm["refill_rows_per_step"]),
        "minibatch_roofline": sm["minibatch_roofline"],
        "phase_ms_per_step": sm["phase_ms_per_step"],
        "phases_from": "the timed window's own steps (HIP events on %s)" % sm["phases_timed"],
        "early_window": {k: sm_early[k] for k in ("steps_timed", "eviction_rounds", "value", "ms_per_step",
                                                  "hit_rate", "minibatch_roofline", "phase_ms_per_step",
                                                  "host_rows_per_step", "refill_rows_per_step")},
        "eviction_run": evr,
        "configs": configs,
        "init_s": round(res["init_s"], 3),
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def pmc_summary(args):
    """Summary of two rocprofv3 counter runs of the default bench with
    --copy-probe (FETCH_SIZE, then WRITE_SIZE): per k_gather_hbm dispatch of
    the first context, the counters over the headline window's launches
    (dispatch i of the gather is step i), each scaled by what the counter
    reads for the plain 256 MiB copy of the probe (the last copy kernel before
    step 0's first kernel). Prints the summary for profiles/."""
    import csv
    import hashlib
    fetch_dir, write_dir = args.pmc_summary

    def rows(d, counter):
        path = [os.path.join(r, f) for r, _, fs in os.walk(d) for f in fs if f.endswith("counter_collection.csv")]
        assert len(path) == 1, path
        out = []
        for r in csv.DictReader(open(path[0])):
            if r["Counter_Name"] == counter:
                out.append((int(r["Process_Id"]), int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
        out.sort(key=lambda x: (x[0], x[1]))
        pid = out[0][0]
        return [x for x in out if x[0] == pid]

    import synth
    K = args.steps
    w = synth.get(args.workload)
    _, head = window_plan(args.warmup, K, args.delta or w.delta)
    res = {}
    for name, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rs = rows(d, name)
        first_step = next(i for i, x in enumerate(rs) if "k_seed_init" in x[2] or "k_row_scan" in x[2])
        probe = [x for x in rs[:first_step] if "copyBuffer" in x[2]][-1]
        gathers = [x[3] for x in rs if "k_gather_hbm" in x[2]]
        res[name] = (probe[3], gathers)
    probe_kib = 256 * 1024
    f_scale = probe_kib / res["FETCH_SIZE"][0]
    w_scale = probe_kib / res["WRITE_SIZE"][0]
    fe = np.array(res["FETCH_SIZE"][1][head[0]:head[1]]) * f_scale * 1024
    wr = np.array(res["WRITE_SIZE"][1][head[0]:head[1]]) * w_scale * 1024
    src = open(os.path.join(ROOT, "paper_2410_22697_amd", "csrc", "buffer_kernels.hpp")).read()
    a, b = src.find("// ---------------------------------------------------------------- gather"), src.find("// misses: pinned host store")
    print("probe FETCH_SIZE %.1f KiB -> factor %.4f; WRITE_SIZE %.1f KiB -> factor %.4f" %
          (res["FETCH_SIZE"][0], f_scale, res["WRITE_SIZE"][0], w_scale))
    print("k_gather_hbm dispatches in the first context: %d; window %d..%d" % (len(res["FETCH_SIZE"][1]), head[0],
                                                                              head[1] - 1))
    print("HBM read per launch (scaled)  %.0f" % fe.mean())
    print("HBM write per launch (scaled) %.0f" % wr.mean())
    print("window_steps: %d..%d" % (head[0], head[1] - 1))
    print("traffic_bytes_per_launch: %d" % round(fe.mean() + wr.mean()))
    print("gather_source_sha256: %s" % hashlib.sha256(src[a:b].encode()).hexdigest())


def layout_one(w, layout, g, local, store, sched, args):
    """One S_A layout on the eviction run from init (five rounds), every
    kernel group timed: device memory of the context, the score arrays' bytes,
    the round's time, throughput, and a digest of every step's counts and the
    final state for the cross-check."""
    import hashlib
    n = EVICTION_RUN_ROUNDS * w.delta + 1
    res = run_context(w, g, local, store, sched, [("run", 0, n, True)], args.depth, first_alone=False,
                      score_layout=layout)
    sm = summarize(w, res, "run")
    tim = res["windows"]["run"]["tim"]
    # local, hits, misses, rows per step (the host-link rows depend on when a refill lands)
    digest = hashlib.sha256(np.ascontiguousarray(res["stats"][:n, :4]).tobytes()).hexdigest()[:16]
    score_bytes = 4 * g.H if layout == "rank" else 8 * w.n
    return {"metric": "eviction run with the S_A layout %r" % layout, "layout": layout, "workload": w.name,
            "steps": n, "value": sm["value"], "unit": "minibatches/s", "eviction_rounds": sm["eviction_rounds"],
            "evicted_rows": sm["evicted_rows"], "hit_rate": sm["hit_rate"],
            "round_ms": round(tim["evict_round"][0] / max(tim["evict_round"][1], 1), 3),
            "score_array_bytes": score_bytes, "context_device_bytes": int(res["ctx_bytes"]),
            "init_s": round(res["init_s"], 3), "counts_digest": digest}


def layouts(argv):
    """Both S_A layouts on the same run, each in a process of its own."""
    import subprocess
    outs = []
    for layout in ("rank", "gid"):
        cmd = [sys.executable, os.path.abspath(__file__)] + argv + ["--layout-run", layout]
        r = subprocess.run(cmd, stdout=subprocess.PIPE, text=True)
        if r.returncode != 0:
            raise SystemExit("bench: the layout run %s failed with status %d" % (layout, r.returncode))
        outs.append(json.loads([l for l in r.stdout.splitlines() if l.startswith("{")][-1]))
    same = outs[0]["counts_digest"] == outs[1]["counts_digest"] and outs[0]["evicted_rows"] == outs[1]["evicted_rows"]
    for o in outs:
        o["same_results_as_other_layout"] = same
        log("layout %-4s: %.1f minibatches/s, round %.3f ms, scores %.1f MB, context %.2f GB" %
            (o["layout"], o["value"], o["round_ms"], o["score_array_bytes"] / 1e6, o["context_device_bytes"] / 1e9))
        print(json.dumps(o), flush=True)
    if not same:
        raise SystemExit("bench: the two layouts gave different results")


COMPARE_MODES = ("no_buffer", "static", "eviction")


def compare_workload(w, name, total):
    """The workload of one --compare mode."""
    if name == "no_buffer":
        return w.with_(buffer_pct=0)
    if name == "static":
        return w.with_(delta=total + 1)  # no round within the run
    return w


def compare_one(w, name, g, local, store, sched, args):
    """One mode of the paper's comparison (Section V) in this process: the
    measurements of the JSON line, without the ratios to the no-buffer mode."""
    wm = compare_workload(w, name, args.warmup + args.steps)
    log("mode %s: f=%d%% delta=%d gamma=%g" % (name, wm.buffer_pct, wm.delta, wm.gamma))
    warm = max(1, args.warmup)
    res = run_context(wm, g, local, store, sched, [("run", warm, warm + args.steps, ["gather_hbm"])])
    sm = summarize(wm, res, "run")
    st = res["stats"]
    series = (st[:, 1] / np.maximum(st[:, 1] + st[:, 2], 1)).round(4).tolist()  # per step, from step 0
    return {"metric": "sampled+gathered minibatches/s; remote rows per step", "mode": name,
            "value": sm["value"], "unit": "minibatches/s", "n_gpus": 1, "steps": args.steps,
            "warmup": warm, "dtype": "f32" if wm.dtype == "f32" else "bf16",
            "config": {"workload": wm.name, "buffer_pct": wm.buffer_pct, "gamma": wm.gamma, "delta": wm.delta,
                       "cap": res["gm_cap"], "eviction_rounds": sm["eviction_rounds"],
                       "evicted_rows": sm["evicted_rows"]},
            "init_s": round(res["init_s"], 3), "init_rows_over_link": res["gm_cap"],
            "hit_rate": sm["hit_rate"],
            "halo_rows_per_step": sm["halo_rows_per_step"],
            "remote_rows_per_step": sm["remote_rows_per_step"],
            "miss_gather_rows_per_step": sm["host_rows_per_step"],
            "refill_rows_per_step": sm["refill_rows_per_step"],
            "link_GBps_window": sm["minibatch_roofline"]["link_GBps"],
            "gather_frac_hbm": sm["gather_hbm"]["frac_hbm"] if sm["gather_hbm"] else None,
            "hit_rate_per_step": series}


def compare(argv):
    """The paper's comparison (Section V) on one partition's share: no buffer
    (every halo row over the link, the baseline without prefetching), prefetch
    without eviction (the initial degree-ranked buffer kept for the whole run)
    and prefetch with eviction. Same graph, features and seed schedule; each
    mode in a process of its own, started from this one (which does not use
    the GPU)."""
    import subprocess
    outs = {}
    for name in COMPARE_MODES:
        cmd = [sys.executable, os.path.abspath(__file__)] + argv + ["--compare", "--compare-mode", name]
        r = subprocess.run(cmd, stdout=subprocess.PIPE, text=True)
        if r.returncode != 0:
            log("mode %s failed with status %d" % (name, r.returncode))
            sys.exit(r.returncode)
        outs[name] = json.loads([l for l in r.stdout.splitlines() if l.startswith("{")][-1])
    base = outs["no_buffer"]
    for name in COMPARE_MODES:
        out = outs[name]
        out["remote_rows_vs_no_buffer"] = round(out["remote_rows_per_step"] / max(base["remote_rows_per_step"], 1e-9), 4)
        out["speedup_vs_no_buffer"] = round(out["value"] / base["value"], 4)
        log("mode %s: %.1f minibatches/s, hit rate %.3f, %.0f remote rows per step (%.3f of no buffer)" %
            (name, out["value"], out["hit_rate"], out["remote_rows_per_step"], out["remote_rows_vs_no_buffer"]))
        print(json.dumps(out), flush=True)


def sweep_point(w, args, g, local, store, sched):
    """One point of the sweep in this process: a fresh context over 8 + N
    steps with every kernel group timed."""
    kind, f, gamma, delta = args.sweep_point
    warm, steps = 8, args.sweep_steps
    wm = w.with_(buffer_pct=int(f), gamma=float(gamma), delta=int(delta))
    res = run_context(wm, g, local, store, sched, [("run", warm, warm + steps, True)])
    sm = summarize(wm, res, "run")
    st = res["stats"]
    hr = st[:, 1] / np.maximum(st[:, 1] + st[:, 2], 1)
    win = [round(float(x.mean()), 4) for x in np.array_split(hr, max(1, (warm + steps) // 64))]
    tim = res["windows"]["run"]["tim"]
    return {"metric": "sampled+gathered minibatches/s; remote rows per step", "mode": kind,
            "workload": wm.name, "buffer_pct": wm.buffer_pct, "gamma": wm.gamma, "delta": wm.delta,
            "steps": steps, "warmup": warm, "value": sm["value"], "unit": "minibatches/s",
            "hit_rate": sm["hit_rate"], "eviction_rounds": sm["eviction_rounds"],
            "evicted_rows": sm["evicted_rows"], "remote_rows_per_step": sm["remote_rows_per_step"],
            "evict_ms_per_round": round(tim["evict_round"][0] / max(tim["evict_round"][1], 1), 3),
            "hit_rate_per_64_steps": win}


def sweep(w, args, argv):
    """Section V-B's analysis of f, gamma and delta (Fig. 12-13) on one
    partition's share: every point in a process of its own (the inputs are
    mapped from shared memory), from a fresh context over the same steps and
    seed schedule, against no buffer and against the static buffer of the
    same f."""
    import subprocess
    total = 8 + args.sweep_steps
    base = None

    def point(kind, f, gamma, delta):
        nonlocal base
        cmd = [sys.executable, os.path.abspath(__file__)] + argv + ["--sweep-point", kind, str(f), str(gamma),
                                                                     str(delta)]
        r = subprocess.run(cmd, stdout=subprocess.PIPE, text=True)
        if r.returncode != 0:
            raise SystemExit("bench: sweep point %s %s %s %s failed with status %d" % (kind, f, gamma, delta,
                                                                                        r.returncode))
        out = json.loads([l for l in r.stdout.splitlines() if l.startswith("{")][-1])
        if base is None:
            base = out
        out["remote_rows_vs_no_buffer"] = round(out["remote_rows_per_step"] / max(base["remote_rows_per_step"], 1e-9), 4)
        out["speedup_vs_no_buffer"] = round(out["value"] / base["value"], 4)
        log("%-9s f=%2d%% gamma=%-6g delta=%-5d %8.1f mb/s  hit %.3f  remote rows %.0f (%.3f)  rounds %d" %
            (kind, out["buffer_pct"], out["gamma"], out["delta"], out["value"], out["hit_rate"],
             out["remote_rows_per_step"], out["remote_rows_vs_no_buffer"], out["eviction_rounds"]))
        print(json.dumps(out), flush=True)

    point("no_buffer", 0, w.gamma, w.delta)
    for f in [int(x) for x in args.sweep_f.split(",") if x]:
        point("static", f, w.gamma, total + 1)
        for gamma in (0.95, 0.995, 0.9995):
            for delta in (16, 32, 64, 128, 256, 512, 1024):
                point("eviction", f, gamma, delta)


def overlap(w, g, local, store, sched, args):
    """Alg. 1's look-ahead (Section IV-C, Eqs. 2-6): minibatch t+1 is prepared
    while minibatch t trains. The trainer is a stand-in, a 2-layer MLP forward
    and backward in fp32 over every gathered row, on a stream of its own (the
    paper's DDP training is outside this path); its hidden size sets t_DDP.
    Measured per step, in order on one context: the path alone with
    look-ahead (t_Prepare), the trainer alone (t_DDP), the serial loop
    (prepare, then train: Eq. 2) and the overlapped loop (Eq. 5)."""
    import torch
    from paper_2410_22697_amd import Massive
    assert w.dtype == "f32", "the stand-in trainer reads fp32 rows"
    torch.cuda.set_device(0)
    gm = Massive(g.L, g.H, g.indptr, g.indices, g.halo_gid, g.halo_degree, local, store, w.row_bytes,
                 w.fanout, w.buffer_pct, w.gamma, w.delta, w.philox_seed, link=LINK["link"],
                 link_threads=LINK["link_threads"])
    main = torch.cuda.current_stream()
    consumer = torch.cuda.Stream()
    bbs = [gm.alloc_batch(w.batch), gm.alloc_batch(w.batch)]
    W = args.steps
    hids = (256, 1024, 4096)
    total = 8 + W + len(hids) * (2 * (8 + W))
    seeds_dev = [torch.from_numpy(np.ascontiguousarray(sched.seeds(t), np.int32)).cuda() for t in range(total)]
    torch.cuda.synchronize()
    state = {"t": 0, "ev": [None, None], "n": 0}

    class Trainer:
        def __init__(self, hid):
            gen = torch.Generator(device="cuda").manual_seed(hid)
            self.W1 = (torch.randn(w.d, hid, device="cuda", generator=gen) / w.d ** 0.5).requires_grad_()
            self.W2 = (torch.randn(hid, 1, device="cuda", generator=gen) / hid ** 0.5).requires_grad_()

        def step(self, feat, n):
            x = feat[:n].view(torch.float32)
            loss = (torch.relu(x @ self.W1) @ self.W2).square().mean()
            loss.backward()
            with torch.no_grad():
                for p in (self.W1, self.W2):
                    p -= 1e-6 * p.grad
                    p.grad = None

    stalls = []  # (end of the previous training step, start of this one) on the trainer's stream

    def train(tr, slot, n, track=False):
        with torch.cuda.stream(consumer):
            if track:
                s0 = torch.cuda.Event(enable_timing=True)
                s0.record(consumer)
                if state.get("last_end") is not None:
                    stalls.append((state["last_end"], s0))
            tr.step(bbs[slot].feat, n)
            e = torch.cuda.Event(enable_timing=track)
            e.record(consumer)
        state["ev"][slot] = e
        state["last_end"] = e if track else None

    def lookahead(steps, tr, track=False):
        t0, prev = state["t"], None
        for t in range(t0, t0 + steps + 1):
            if t < t0 + steps:
                slot = t % 2
                if state["ev"][slot] is not None:
                    main.wait_event(state["ev"][slot])  # the trainer has read this batch
                gm.sample_async(seeds_dev[t], bbs[slot])
                gm.evict_step(wait=False)
            if prev is not None:
                r = gm.wait(bbs[prev % 2])
                state["n"] = r.n[-1]
                if tr is not None:
                    train(tr, prev % 2, r.n[-1], track)
            prev = t
        state["t"] = t0 + steps

    def serial(steps, tr):
        for t in range(state["t"], state["t"] + steps):
            slot = t % 2
            gm.sample_async(seeds_dev[t], bbs[slot])
            gm.evict_step(wait=False)
            r = gm.wait(bbs[slot])
            train(tr, slot, r.n[-1])
            consumer.synchronize()
        state["t"] += steps

    def timed(fn, *a):
        torch.cuda.synchronize()
        with no_gc():
            t0 = time.perf_counter()
            fn(*a)
            torch.cuda.synchronize()
            return (time.perf_counter() - t0) / W

    lookahead(8, None)
    gm.set_timing(True)
    t_prep = timed(lookahead, W, None)
    tim = gm.timing()
    ph = {k: v[0] / W for k, v in tim.items()}  # ms per step
    eq3 = ph["sample_dedup"] + ph["classify"] + max(ph["gather_hbm"], ph["gather_miss"])
    log("path alone: %.3f ms per step; Eq. 3 terms (ms/step) %s" % (1e3 * t_prep, {k: round(v, 3) for k, v in ph.items()}))
    for hid in hids:
        tr = Trainer(hid)
        n, slot = state["n"], (state["t"] - 1) % 2
        for _ in range(3):
            train(tr, slot, n)
        consumer.synchronize()
        with no_gc():
            t0 = time.perf_counter()
            for _ in range(20):
                train(tr, slot, n)
            consumer.synchronize()
            t_ddp = (time.perf_counter() - t0) / 20
        serial(8, tr)
        T_ser = timed(serial, W, tr)
        lookahead(8, tr)
        stalls.clear()
        state["last_end"] = None
        T_ovl = timed(lookahead, W, tr, True)
        stall = sum(a.elapsed_time(b) for a, b in stalls) / 1e3 / max(len(stalls), 1)  # s per step
        state["last_end"] = None
        # the paper's reading (Section V-B): how much of the preparation the
        # trainer does not wait for
        eff_paper = 1.0 - stall / t_prep
        eff = (t_prep + t_ddp - T_ovl) / min(t_prep, t_ddp)
        out = {"metric": "ms per minibatch, prepare overlapped with a stand-in trainer", "mode": "overlap",
               "workload": w.name, "steps": W, "link": LINK["link"], "trainer": "2-layer MLP fwd+bwd fp32, hidden %d, %d rows" % (hid, n),
               "t_prepare_ms": round(1e3 * t_prep, 4), "t_ddp_ms": round(1e3 * t_ddp, 4),
               "T_serial_ms": round(1e3 * T_ser, 4), "T_overlap_ms": round(1e3 * T_ovl, 4),
               "eq5_max_ms": round(1e3 * max(t_prep, t_ddp), 4),
               "trainer_stall_ms": round(1e3 * stall, 4),
               "overlap_efficiency": round(min(1.0, max(0.0, eff_paper)), 4),
               "overlap_efficiency_from": "1 - (the trainer's idle time between consecutive training steps, "
                                          "waiting for the next minibatch) / t_prepare",
               "hidden_vs_isolated": round(min(1.0, max(0.0, eff)), 4),
               "hidden_vs_isolated_from": "(t_prepare + t_ddp - T_overlap) / min(t_prepare, t_ddp): also charges "
                                          "the slowdown of both sharing one GPU",
               "improvement_serial_over_overlap": round(T_ser / T_ovl, 4),
               "eq3_terms_ms_per_step": {k: round(v, 4) for k, v in ph.items()},
               "eq3_sum_ms": round(eq3, 4)}
        log("hidden %d: t_DDP %.3f ms, serial %.3f ms, overlapped %.3f ms per step (max(t_Prepare, t_DDP) = %.3f), "
            "trainer stall %.3f ms, overlap efficiency %.2f (hidden vs isolated %.2f)" %
            (hid, 1e3 * t_ddp, 1e3 * T_ser, 1e3 * T_ovl, 1e3 * max(t_prep, t_ddp), 1e3 * stall, eff_paper, eff))
        print(json.dumps(out), flush=True)
    torch.cuda.synchronize()
    del bbs
    gm.close()




def cpu_baseline(w, g, local, store, sched, budget_s, first_steps, state0=None):
    """The oracle, as it stands, on the same workload from step 0 until the
    budget is spent (at least one step); its first steps are also compared
    with the GPU's, element by element: sizes, frontier, every hop's block,
    masks and rows, and the prefetcher state after step 0 (bit for bit)."""
    import oracle
    t0 = time.time()
    store_np = store.numpy()
    orc = oracle.Oracle(g.L, g.H, g.indptr, g.indices, g.halo_gid, g.halo_degree, local, store_np,
                        w.row_bytes, w.fanout, w.buffer_pct, w.gamma, w.delta, w.philox_seed)
    log("oracle init %.1fs" % (time.time() - t0))
    steps = 0
    t0 = time.perf_counter()
    checked = 0
    while True:
        st = orc.sample(sched.seeds(steps))
        orc.evict_step()
        if steps < len(first_steps):
            r, nodes, mask, feat, blocks = first_steps[steps]
            same = (r.n == st.n and r.e == st.e and np.array_equal(nodes, st.nodes) and
                    np.array_equal(mask, st.mask) and np.array_equal(feat, st.feat) and
                    all(np.array_equal(ip, st.indptr[k]) and np.array_equal(ix, st.indices[k])
                        for k, (ip, ix) in enumerate(blocks)))
            if steps == 0 and state0 is not None:
                sid_o, se_o, sa_o = orc.state()
                sid_g, se_g, sa_g, _ = state0
                same = same and (np.array_equal(sid_g, sid_o) and np.array_equal(se_g.view(np.uint32), se_o.view(np.uint32))
                                 and np.array_equal(sa_g.view(np.uint32), sa_o.view(np.uint32)))
            if not same:
                raise SystemExit("bench: GPU step %d differs from the oracle" % steps)
            checked += 1
        steps += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0 - 0.0
    ph = orc.phase_times()
    log("oracle: %d steps in %.1fs (%d checked equal to the GPU); phases %s" % (steps, el, checked, np.round(ph, 2)))
    return {"value": round(steps / el, 4), "unit": "minibatches/s", "cores": 1, "kind": "oracle",
            "sample": "steps 0..%d of %s from init (single-threaded C oracle; %d steps compared bit-exact "
                      "with the GPU run: sizes, frontier, every hop's block, masks, rows, and the state after "
                      "step 0)" % (steps - 1, w.name, checked),
            "phase_s_per_step": {k: round(float(v) / steps, 4) for k, v in
                                 zip(("sample", "dedup", "classify", "score", "gather", "evict"), ph)},
            "host_cpus": os.cpu_count(), "cpu_model": cpu_model()}


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


if __name__ == "__main__":
    main()
