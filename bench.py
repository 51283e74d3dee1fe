#!/usr/bin/env python3
"""Benchmark: per-minibatch sampling + halo prefetch buffer + feature gather
(MassiveGNN, arXiv 2410.22697) for one partition on one MI355X.

A step is one minibatch through the whole path: massive_sample (3-hop fanout
sampling, dedup/relabel, buffer lookup, scoring, HBM gather, miss fetch from
pinned host memory) followed by massive_evict_step (the periodic eviction
and replacement round, with its refill overlapping the next step). Inputs
(graph, features, seed batches) are resident before the timed region.

Prints one JSON line: minibatches/s, the gather kernel against the HBM
roofline, the hit rate, the host-link rate of the miss fetch, and the CPU
oracle timed on a bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0       # MI355X HBM3E
# Batches in flight in the timed loop (the library allows up to three): with
# two, the next step's sampling overlaps the current step's host-link reads
# and never the HBM gather; a third lets sampling run beside the HBM gather
# too, which slows it, with no gain while the host link bounds the step.
DEFAULT_DEPTH = 2
PCIE_PEAK_GBPS = 64.0        # PCIe 5.0 x16, one direction


def gather_traffic(rb_per_launch):
    """HBM bytes per gather_hbm launch from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy), as a ratio to
    the algorithmic bytes applied to this run's launches; None if the gather
    kernel's source has changed since the counters were taken."""
    import hashlib
    prof = os.path.join(ROOT, "profiles", "gather_hbm_cl111m_p64_hbm_counters.txt")
    src = open(os.path.join(ROOT, "paper_2410_22697_amd", "csrc", "buffer_kernels.hpp")).read()
    a, b = src.find("// ---------------------------------------------------------------- gather"), src.find("// misses: pinned host store")
    if not os.path.exists(prof) or a < 0 or b < 0:
        return None
    kv = dict(l.split(": ", 1) for l in open(prof).read().splitlines() if l.startswith(("traffic_", "gather_source")))
    if kv.get("gather_source_sha256") != hashlib.sha256(src[a:b].encode()).hexdigest():
        return None
    return round(float(kv["traffic_over_algorithmic"]) * rb_per_launch)


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


def run_context(w, g, local, store, sched, warmup, steps, log_steps=False, copy_probe=False, depth=None,
                timed_groups=("gather_hbm",), prof_steps=64):
    """One context over steps 0..warmup+steps-1 with look-ahead (`depth`
    batches in flight); the last `steps` are timed, with HIP events only on
    `timed_groups` (every timed group adds event packets to the streams).
    Then `prof_steps` further steps with every group timed give the phase
    breakdown. Returns the raw measurements."""
    import torch
    from paper_2410_22697_amd import Massive
    depth = depth or DEFAULT_DEPTH
    warmup = max(1, warmup)  # step 0 runs alone (below)
    torch.cuda.set_device(0)
    t0 = time.time()
    gm = Massive(g.L, g.H, g.indptr, g.indices, g.halo_gid, g.halo_degree, local, store, w.row_bytes,
                 w.fanout, w.buffer_pct, w.gamma, w.delta, w.philox_seed)
    torch.cuda.synchronize()
    init_s = time.time() - t0
    log("massive_init %.2fs: cap=%d alpha=%.6g" % (init_s, gm.cap, gm.alpha))
    bbs = [gm.alloc_batch(w.batch) for _ in range(depth)]
    total = warmup + steps
    seeds_dev = [torch.from_numpy(np.ascontiguousarray(sched.seeds(t), np.int32)).cuda()
                 for t in range(total + prof_steps)]
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

    def finish(u):
        r = gm.wait(bbs[u % depth])
        stats.append((r.local, r.hits, r.misses, r.n[-1], r.host_rows))
        sizes.append((list(r.n), list(r.e)))
        if u < 2 and len(first_steps) == u:
            bb = bbs[u % depth]
            nK = r.n[-1]
            blocks = [(bb.indptr[k][:r.n[k] + 1].cpu().numpy().copy(), bb.indices[k][:r.e[k]].cpu().numpy().copy())
                      for k in range(len(r.e))]
            first_steps.append((r, bb.nodes[:nK].cpu().numpy().copy(), bb.mask[:nK].cpu().numpy().copy(),
                                bb.feat[:nK].cpu().numpy().copy(), blocks))
        if log_steps:
            log("step %d local %d hits %d misses %d rows %d host %d" % (u, r.local, r.hits, r.misses, r.n[-1],
                                                                        r.host_rows))

    def run(t0, t1):
        """Steps t0..t1-1 with look-ahead: step t is enqueued (after step t-1's
        round) before step t - depth + 1 is waited for, so the sampling of the
        next steps overlaps the host-link reads of earlier ones."""
        inflight = []
        for t in range(t0, t1):
            gm.sample_async(seeds_dev[t], bbs[t % depth])
            gm.evict_step(wait=False)
            inflight.append(t)
            if len(inflight) == depth:
                finish(inflight.pop(0))
        for u in inflight:
            finish(u)

    # step 0 alone, so that the prefetcher state after it can be read (and
    # checked against the oracle's); then the rest of the warmup with look-ahead
    run(0, 1)
    state0 = gm.state()
    run(1, warmup)
    log("warmup %d steps done" % warmup)
    r0, e0 = gm.counters()
    f0 = gm.refilled_rows()
    gm.set_timing(timed_groups)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(warmup, total)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    tim = gm.timing()
    r1, e1 = gm.counters()
    f1 = gm.refilled_rows()
    tim_prof, stats_prof = None, None
    if prof_steps:
        n_timed = len(stats)
        gm.set_timing(True)
        run(total, total + prof_steps)
        tim_prof = gm.timing()
        stats_prof = np.array(stats[n_timed:], np.float64)
        del stats[n_timed:], sizes[n_timed:]
    out = dict(gm_cap=gm.cap, H=g.H, alpha=gm.alpha, init_s=init_s, elapsed=elapsed, steps=steps, warmup=warmup,
               depth=depth,
               stats=np.array(stats, np.float64), sizes=sizes, tim=tim, rounds=r1 - r0, evicted=e1 - e0,
               refilled=f1 - f0, first_steps=first_steps, state0=state0, tim_prof=tim_prof, stats_prof=stats_prof,
               prof_steps=prof_steps)
    del bbs, seeds_dev
    gm.close()
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


def summarize(w, res):
    """Throughput, the gather against the HBM roofline, the host link, the hit rate."""
    K, rb = res["steps"], w.row_bytes
    st = res["stats"][res["warmup"]:]
    loc, hit, mis, host_rows = st[:, 0], st[:, 1], st[:, 2], st[:, 4]
    hbm_rows = loc + hit
    tim = res["tim"]
    mbps = K / res["elapsed"]
    # gather_hbm algorithmic bytes: read + write each HBM-sourced row, plus its 8-byte list entry
    g_ms, g_calls = tim["gather_hbm"]
    g_bytes = float(np.mean(2 * hbm_rows * rb + 8 * hbm_rows))
    g_avg_s = g_ms / 1e3 / max(g_calls, 1)
    # the miss gather's own rate: from the steps with every group timed, if any
    if res.get("tim_prof"):
        m_ms, m_calls = res["tim_prof"]["gather_miss"]
        m_bytes = float(np.mean(res["stats_prof"][:, 4] * rb))
    else:
        m_ms, m_calls = tim["gather_miss"]
        m_bytes = float(np.mean(host_rows * rb))
    refill_bytes = res["refilled"] * rb / max(K, 1)  # copied by refill chunks inside the timed region, per step
    sz = res["sizes"][res["warmup"]:]
    b_alg = float(np.mean([alg_hbm_bytes(n, e, l, h, m, rb) for (n, e), (l, h, m) in zip(sz, st[:, :3])]))
    # eviction rounds, amortised: S_E/slot scans and S_A/rank scans, and the replacement rows written
    b_alg += (res["rounds"] * (12 * res["gm_cap"] + 8 * res["H"]) + res["evicted"] * rb) / max(K, 1)
    link_bytes = float(np.mean(host_rows * rb)) + refill_bytes
    return dict(mbps=mbps, b_alg=b_alg, link_bytes=link_bytes, g_bytes=g_bytes, g_avg_s=g_avg_s, g_gbps=g_bytes / g_avg_s / 1e9,
                m_bytes=m_bytes, m_avg_us=1e3 * m_ms / max(m_calls, 1),
                m_gbps=m_bytes / (m_ms / 1e3 / max(m_calls, 1)) / 1e9 if m_ms > 0 else 0.0,
                hit_rate=float(hit.sum() / max(hit.sum() + mis.sum(), 1)),
                pend_bytes=float(np.mean((host_rows - mis) * rb)), refill_bytes=refill_bytes,
                host_bytes=float(np.mean(host_rows * rb)),
                evicted_bytes=res["evicted"] * rb / max(K, 1),
                link_gbps=(float(host_rows.sum()) * rb + res["refilled"] * rb) / res["elapsed"] / 1e9,
                remote_rows=float(np.mean(host_rows)) + res["refilled"] / max(K, 1),
                halo_rows=float(np.mean(hit + mis)))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1, help="GPUs (one partition runs on one GPU: only 1)")
    ap.add_argument("--steps", type=int, default=192, help="timed minibatches")
    ap.add_argument("--warmup", type=int, default=8, help="untimed minibatches before them")
    ap.add_argument("--workload", default="cl111m_p64", help="a named synthetic workload (synth/workloads.py)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0, help="budget of the oracle baseline")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle baseline")
    ap.add_argument("--threads", type=int, default=None, help="host threads of the input generator")
    ap.add_argument("--log-steps", action="store_true", help="per-step row counts on stderr")
    ap.add_argument("--depth", type=int, default=DEFAULT_DEPTH, help="batches in flight (1 to 3)")
    ap.add_argument("--delta", type=int, default=None, help="override the eviction interval")
    ap.add_argument("--gamma", type=float, default=None, help="override the decay factor")
    ap.add_argument("--buffer-pct", type=int, default=None, help="override f (percent of the halo)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="one plain 256 MiB device copy before warmup (reference for HBM byte counters)")
    ap.add_argument("--sweep", action="store_true",
                    help="the paper's parameter grid (f in 15/25/35/50 %%, gamma in 0.95/0.995/0.9995, delta in "
                         "16..1024) on the same inputs, plus no buffer and one static run per f; one JSON line each")
    ap.add_argument("--sweep-steps", type=int, default=1032, help="timed steps per sweep point (after 8 warm-up)")
    ap.add_argument("--overlap", action="store_true",
                    help="Alg. 1's look-ahead against a stand-in trainer on its own stream (Section IV-C): "
                         "path alone, trainer alone, serial and overlapped steps per trainer size")
    ap.add_argument("--compare", action="store_true",
                    help="the paper's comparison on the same inputs: no buffer (f = 0), prefetch without "
                         "eviction (no round within the run) and prefetch with eviction; one JSON line each")
    ap.add_argument("--compare-mode", choices=COMPARE_MODES, default=None,
                    help="run one mode of --compare in this process (used by --compare itself)")
    args = ap.parse_args()
    if args.compare and args.compare_mode is None:
        compare([a for a in sys.argv[1:]])
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (each partition's "
              "buffer is private to its trainer); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import synth

    w = synth.get(args.workload)
    over = {k: v for k, v in (("delta", args.delta), ("gamma", args.gamma), ("buffer_pct", args.buffer_pct))
            if v is not None}
    if over:
        w = w.with_(**over)
    g, local, store, sched = build_inputs(w, args.threads)
    if args.compare:
        print(json.dumps(compare_one(w, args.compare_mode, g, local, store, sched, args)), flush=True)
        return
    if args.sweep:
        sweep(w, g, local, store, sched, args)
        return
    if args.overlap:
        overlap(w, g, local, store, sched, args)
        return

    res = run_context(w, g, local, store, sched, args.warmup, args.steps, args.log_steps, args.copy_probe,
                      args.depth)
    sm = summarize(w, res)
    K, rb = args.steps, w.row_bytes
    log("timed %d steps in %.3fs: %.1f minibatches/s, %d rounds, %d evicted" %
        (K, res["elapsed"], sm["mbps"], res["rounds"], res["evicted"]))
    log("host link per step: %.1f MB miss gather (%.1f MB of them hits on refilling slots, written through), "
        "%.1f MB refill copied (%.1f MB evicted); %.1f GB/s over the link" %
        (sm["host_bytes"] / 1e6, sm["pend_bytes"] / 1e6, sm["refill_bytes"] / 1e6, sm["evicted_bytes"] / 1e6,
         sm["link_gbps"]))
    phases, P = (res["tim_prof"], res["prof_steps"]) if res.get("tim_prof") else (res["tim"], K)
    log("HIP-event timing: gather_hbm over the timed steps; every group over %d further steps:" % P)
    for name, (ms, calls) in phases.items():
        log("  %-13s %9.3f ms total, %5d launches, %.1f us avg" % (name, ms, calls, 1e3 * ms / max(calls, 1)))
    log("gather_hbm %.0f B/launch, %.1f us, %.1f GB/s (%.1f%% of HBM); miss fetch %.1f GB/s; hit rate %.3f" %
        (sm["g_bytes"], sm["g_avg_s"] * 1e6, sm["g_gbps"], 100 * sm["g_gbps"] / HBM_PEAK_GBPS, sm["m_gbps"],
         sm["hit_rate"]))

    copy_gbps = copy_reference(sm["g_bytes"])
    log("plain device copy moving the same bytes (%d B): %.1f GB/s; the gather reaches %.1f%% of it" %
        (round(sm["g_bytes"]), copy_gbps, 100 * sm["g_gbps"] / copy_gbps))

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(w, g, local, store, sched, args.cpu_seconds, res["first_steps"], res["state0"])

    g_gbps = sm["g_gbps"]
    out = {
        "metric": "sampled+gathered minibatches/s; gather GB/s (% HBM peak); halo buffer hit rate",
        "value": round(sm["mbps"], 3),
        "unit": "minibatches/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * res["elapsed"] / K, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if w.dtype == "f32" else "bf16",
        "data": "synthetic (seeded Chung-Lu power-law graph, N(0,1) features)",
        "config": {"workload": w.name, "nodes": w.n, "partitions": w.parts, "partition": 0,
                   "L": g.L, "H": g.H, "csr_entries": g.nnz, "batch": w.batch, "fanout": list(w.fanout),
                   "row_bytes": rb, "buffer_pct": w.buffer_pct, "gamma": w.gamma, "delta": w.delta,
                   "cap": res["gm_cap"], "steps_timed": [args.warmup, args.warmup + K - 1],
                   "eviction_rounds": res["rounds"], "evicted_rows": res["evicted"], "lookahead": res["depth"] - 1,
                   "parallelism": "one partition on one GPU"},
        "gather_GBps": round(g_gbps, 1),
        "gather_frac_hbm": round(g_gbps / HBM_PEAK_GBPS, 4),
        "hit_rate": round(sm["hit_rate"], 4),
        "roofline": {"bound": "hbm", "kernel": "gather_hbm", "achieved": round(g_gbps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(g_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": gather_traffic(sm["g_bytes"]) if w.name == "cl111m_p64" else None,
                     "bytes_per_launch": round(sm["g_bytes"]), "avg_us": round(sm["g_avg_s"] * 1e6, 2),
                     "plain_copy_same_bytes_GBps_events": round(copy_gbps, 1),
                     "frac_of_plain_copy": round(sm["g_gbps"] / copy_gbps, 4)},
        "host_link": {"kernel": "gather_miss", "achieved": round(sm["m_gbps"], 2), "peak": PCIE_PEAK_GBPS,
                      "unit": "GB/s", "bytes_per_launch": round(sm["m_bytes"]),
                      "avg_us": round(sm["m_avg_us"], 2),
                      "refill_bytes_per_step": round(sm["refill_bytes"]),
                      "link_GBps_whole_run": round(sm["link_gbps"], 2)},
        "minibatch_roofline": {"bound": "host link",
                               "hbm_alg_bytes_per_step": round(sm["b_alg"]),
                               "hbm_GBps": round(sm["mbps"] * sm["b_alg"] / 1e9, 1),
                               "hbm_frac": round(sm["mbps"] * sm["b_alg"] / 1e9 / HBM_PEAK_GBPS, 4),
                               "link_bytes_per_step": round(sm["link_bytes"]),
                               "link_GBps": round(sm["mbps"] * sm["link_bytes"] / 1e9, 2),
                               "link_peak_GBps": PCIE_PEAK_GBPS,
                               "link_frac": round(sm["mbps"] * sm["link_bytes"] / 1e9 / PCIE_PEAK_GBPS, 4)},
        "phase_ms_per_step": {k: round(v[0] / P, 4) for k, v in phases.items()},
        "phases_from": "%d steps after the timed region, every kernel group timed with HIP events" % P,
        "init_s": round(res["init_s"], 3),
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


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
    res = run_context(wm, g, local, store, sched, args.warmup, args.steps)
    sm = summarize(wm, res)
    st = res["stats"]
    series = (st[:, 1] / np.maximum(st[:, 1] + st[:, 2], 1)).round(4).tolist()  # per step, from step 0
    return {"metric": "sampled+gathered minibatches/s; remote rows per step", "mode": name,
            "value": round(sm["mbps"], 3), "unit": "minibatches/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "dtype": "f32" if wm.dtype == "f32" else "bf16",
            "config": {"workload": wm.name, "buffer_pct": wm.buffer_pct, "gamma": wm.gamma, "delta": wm.delta,
                       "cap": res["gm_cap"], "eviction_rounds": res["rounds"], "evicted_rows": res["evicted"]},
            "init_s": round(res["init_s"], 3), "init_rows_over_link": res["gm_cap"],
            "hit_rate": round(sm["hit_rate"], 4),
            "halo_rows_per_step": round(sm["halo_rows"], 1),
            "remote_rows_per_step": round(sm["remote_rows"], 1),
            "miss_gather_rows_per_step": round(sm["host_bytes"] / wm.row_bytes, 1),
            "refill_rows_per_step": round(sm["refill_bytes"] / wm.row_bytes, 1),
            "link_GBps_whole_run": round(sm["link_gbps"], 2),
            "gather_frac_hbm": round(sm["g_gbps"] / HBM_PEAK_GBPS, 4),
            "hit_rate_per_step": series}


def compare(argv):
    """The paper's comparison (Section V) on one partition's share: no buffer
    (every halo row over the link, the baseline without prefetching), prefetch
    without eviction (the initial degree-ranked buffer kept for the whole run)
    and prefetch with eviction. Same graph, features and seed schedule; each
    mode in a process of its own, started from this one (which does not use
    the GPU): with the three modes in one process, the third context was
    measured 8-29% slower, whichever mode it was."""
    import subprocess
    outs = {}
    for name in COMPARE_MODES:
        cmd = [sys.executable, os.path.abspath(__file__)] + argv + ["--compare-mode", name]
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


def sweep(w, g, local, store, sched, args):
    """Section V-B's analysis of f, gamma and delta (Fig. 12-13) on one partition's share:
    every point from a fresh context over the same steps and seed schedule,
    against no buffer and against the static buffer of the same f."""
    warm, steps = 8, args.sweep_steps
    total = warm + steps

    def point(kind, wm, base):
        res = run_context(wm, g, local, store, sched, warm, steps, timed_groups=True, prof_steps=0)
        sm = summarize(wm, res)
        st = res["stats"]
        hr = st[:, 1] / np.maximum(st[:, 1] + st[:, 2], 1)
        win = [round(float(x.mean()), 4) for x in np.array_split(hr, max(1, total // 64))]
        out = {"metric": "sampled+gathered minibatches/s; remote rows per step", "mode": kind,
               "workload": wm.name, "buffer_pct": wm.buffer_pct, "gamma": wm.gamma, "delta": wm.delta,
               "steps": steps, "warmup": warm, "value": round(sm["mbps"], 3), "unit": "minibatches/s",
               "hit_rate": round(sm["hit_rate"], 4), "eviction_rounds": res["rounds"], "evicted_rows": res["evicted"],
               "remote_rows_per_step": round(sm["remote_rows"], 1),
               "remote_rows_vs_no_buffer": round(sm["remote_rows"] / base["remote_rows"], 4) if base else 1.0,
               "speedup_vs_no_buffer": round(sm["mbps"] / base["mbps"], 4) if base else 1.0,
               "evict_ms_per_round": round(res["tim"]["evict_round"][0] / max(res["tim"]["evict_round"][1], 1), 3),
               "hit_rate_per_64_steps": win}
        log("%-9s f=%2d%% gamma=%-6g delta=%-5d %8.1f mb/s  hit %.3f  remote rows %.0f (%.3f)  rounds %d" %
            (kind, wm.buffer_pct, wm.gamma, wm.delta, sm["mbps"], sm["hit_rate"], sm["remote_rows"],
             out["remote_rows_vs_no_buffer"], res["rounds"]))
        print(json.dumps(out), flush=True)
        return sm

    base = point("no_buffer", w.with_(buffer_pct=0), None)
    for f in (15, 25, 35, 50):
        point("static", w.with_(buffer_pct=f, delta=total + 1), base)
        for gamma in (0.95, 0.995, 0.9995):
            for delta in (16, 32, 64, 128, 256, 512, 1024):
                point("eviction", w.with_(buffer_pct=f, gamma=gamma, delta=delta), base)


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
                 w.fanout, w.buffer_pct, w.gamma, w.delta, w.philox_seed)
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

    def train(tr, slot, n):
        with torch.cuda.stream(consumer):
            tr.step(bbs[slot].feat, n)
            e = torch.cuda.Event()
            e.record(consumer)
        state["ev"][slot] = e

    def lookahead(steps, tr):
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
                    train(tr, prev % 2, r.n[-1])
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
        t0 = time.perf_counter()
        for _ in range(20):
            train(tr, slot, n)
        consumer.synchronize()
        t_ddp = (time.perf_counter() - t0) / 20
        serial(8, tr)
        T_ser = timed(serial, W, tr)
        lookahead(8, tr)
        T_ovl = timed(lookahead, W, tr)
        eff = (t_prep + t_ddp - T_ovl) / min(t_prep, t_ddp)
        out = {"metric": "ms per minibatch, prepare overlapped with a stand-in trainer", "mode": "overlap",
               "workload": w.name, "steps": W, "trainer": "2-layer MLP fwd+bwd fp32, hidden %d, %d rows" % (hid, n),
               "t_prepare_ms": round(1e3 * t_prep, 4), "t_ddp_ms": round(1e3 * t_ddp, 4),
               "T_serial_ms": round(1e3 * T_ser, 4), "T_overlap_ms": round(1e3 * T_ovl, 4),
               "eq5_max_ms": round(1e3 * max(t_prep, t_ddp), 4),
               "overlap_efficiency": round(min(1.0, max(0.0, eff)), 4),
               "improvement_serial_over_overlap": round(T_ser / T_ovl, 4),
               "eq3_terms_ms_per_step": {k: round(v, 4) for k, v in ph.items()},
               "eq3_sum_ms": round(eq3, 4)}
        log("hidden %d: t_DDP %.3f ms, serial %.3f ms, overlapped %.3f ms per step (max(t_Prepare, t_DDP) = %.3f), "
            "overlap efficiency %.2f" % (hid, 1e3 * t_ddp, 1e3 * T_ser, 1e3 * T_ovl, 1e3 * max(t_prep, t_ddp), eff))
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
