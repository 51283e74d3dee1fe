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
PCIE_PEAK_GBPS = 64.0        # PCIe 5.0 x16, one direction


def gather_traffic(rb_per_launch):
    """HBM bytes per gather_hbm launch from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy), as a ratio to
    the algorithmic bytes applied to this run's launches; None if the gather
    kernel's source has changed since the counters were taken."""
    import hashlib
    prof = os.path.join(ROOT, "profiles", "gather_hbm_cl111m_p64_hbm_counters.txt")
    src = open(os.path.join(ROOT, "paper_2410_22697_amd", "csrc", "buffer_kernels.hpp")).read()
    a, b = src.find("__device__ __forceinline__ void gather_body"), src.find("// misses: pinned host store")
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=192)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default="cl111m_p64")
    ap.add_argument("--cpu-seconds", type=float, default=20.0, help="budget of the oracle baseline")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--threads", type=int, default=None)
    ap.add_argument("--log-steps", action="store_true", help="per-step row counts on stderr")
    ap.add_argument("--delta", type=int, default=None, help="override the eviction interval")
    ap.add_argument("--gamma", type=float, default=None, help="override the decay factor")
    ap.add_argument("--buffer-pct", type=int, default=None, help="override f (percent of the halo)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="one plain 256 MiB device copy before warmup (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (each partition's "
              "buffer is private to its trainer); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_2410_22697_amd import Massive

    w = synth.get(args.workload)
    over = {k: v for k, v in (("delta", args.delta), ("gamma", args.gamma), ("buffer_pct", args.buffer_pct))
            if v is not None}
    if over:
        w = w.with_(**over)
    g, local, store, sched = build_inputs(w, args.threads)
    torch.cuda.set_device(0)
    t0 = time.time()
    gm = Massive(g.L, g.H, g.indptr, g.indices, g.halo_gid, g.halo_degree, local, store, w.row_bytes,
                 w.fanout, w.buffer_pct, w.gamma, w.delta, w.philox_seed)
    torch.cuda.synchronize()
    init_s = time.time() - t0
    log("massive_init %.2fs: cap=%d alpha=%.6g" % (init_s, gm.cap, gm.alpha))
    bbs = [gm.alloc_batch(w.batch), gm.alloc_batch(w.batch)]
    total = args.warmup + args.steps
    seeds_dev = [torch.from_numpy(np.ascontiguousarray(sched.seeds(t), np.int32)).cuda() for t in range(total)]
    torch.cuda.synchronize()

    if args.copy_probe:
        a = torch.empty(256 << 20, dtype=torch.uint8, device="cuda").fill_(1)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        log("copy probe: 256 MiB device-to-device copy done")
        del a, b

    first_steps = []  # the first steps' outputs, checked against the oracle below

    def run(t0, t1, stats):
        """Steps t0..t1-1 with look-ahead: step t+1 is enqueued (after step t's
        round) before step t is waited for, so its sampling overlaps step t's
        host-link reads."""
        prev = None
        for t in range(t0, t1 + 1):
            if t < t1:
                gm.sample_async(seeds_dev[t], bbs[t % 2])
                gm.evict_step(wait=False)
            if prev is not None:
                r = gm.wait(bbs[prev % 2])
                stats.append((r.local, r.hits, r.misses, r.n[-1], r.host_rows))
                if prev < 2 and len(first_steps) == prev:
                    bb = bbs[prev % 2]
                    nK = r.n[-1]
                    first_steps.append((r, bb.nodes[:nK].cpu().numpy().copy(), bb.mask[:nK].cpu().numpy().copy(),
                                        bb.feat[:nK].cpu().numpy().copy()))
                if args.log_steps:
                    log("step %d local %d hits %d misses %d rows %d" % (prev, r.local, r.hits, r.misses, r.n[-1]))
            prev = t

    run(0, args.warmup, [])
    log("warmup %d steps done" % args.warmup)
    r0, e0 = gm.counters()

    gm.set_timing(True)
    stats = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(args.warmup, total, stats)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    tim = gm.timing()
    r1, e1 = gm.counters()
    rounds, evicted = r1 - r0, e1 - e0
    K = args.steps
    mbps = K / elapsed
    log("timed %d steps in %.3fs: %.1f minibatches/s, %d rounds, %d evicted" % (K, elapsed, mbps, rounds, evicted))

    rb = w.row_bytes
    loc = np.array([s[0] for s in stats], np.float64)
    hit = np.array([s[1] for s in stats], np.float64)
    mis = np.array([s[2] for s in stats], np.float64)
    hbm_rows = loc + hit
    # gather_hbm algorithmic bytes: read + write each HBM-sourced row, plus its 8-byte list entry
    g_ms, g_calls = tim["gather_hbm"]
    g_bytes_per_launch = float(np.mean(2 * hbm_rows * rb + 8 * hbm_rows))
    g_avg_s = g_ms / 1e3 / max(g_calls, 1)
    g_gbps = g_bytes_per_launch / g_avg_s / 1e9
    m_ms, m_calls = tim["gather_miss"]
    host_rows = np.array([s[4] for s in stats], np.float64)
    m_bytes = float(np.mean(host_rows * rb))
    m_gbps = m_bytes / (m_ms / 1e3 / max(m_calls, 1)) / 1e9
    hit_rate = float(hit.sum() / max(hit.sum() + mis.sum(), 1))
    rf_ms, rf_calls = tim["refill"]
    log("host link per step: %.1f MB miss gather (%.1f MB of them hits on refilling slots), "
        "%.1f MB refill (amortised)" % (m_bytes / 1e6, float(np.mean((host_rows - mis) * rb)) / 1e6,
                                        evicted * rb / max(K, 1) / 1e6))
    for name, (ms, calls) in tim.items():
        log("  %-13s %9.3f ms total, %5d launches, %.1f us avg" % (name, ms, calls, 1e3 * ms / max(calls, 1)))
    log("gather_hbm %.0f B/launch, %.1f us, %.1f GB/s (%.1f%% of HBM); miss fetch %.1f GB/s; hit rate %.3f" %
        (g_bytes_per_launch, g_avg_s * 1e6, g_gbps, 100 * g_gbps / HBM_PEAK_GBPS, m_gbps, hit_rate))

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(w, g, local, store, sched, args.cpu_seconds, first_steps)

    out = {
        "metric": "sampled+gathered minibatches/s; gather GB/s (% HBM peak); halo buffer hit rate",
        "value": round(mbps, 3),
        "unit": "minibatches/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * elapsed / K, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if w.dtype == "f32" else "bf16",
        "data": "synthetic (seeded Chung-Lu power-law graph, N(0,1) features)",
        "config": {"workload": w.name, "nodes": w.n, "partitions": w.parts, "partition": 0,
                   "L": g.L, "H": g.H, "csr_entries": g.nnz, "batch": w.batch, "fanout": list(w.fanout),
                   "row_bytes": rb, "buffer_pct": w.buffer_pct, "gamma": w.gamma, "delta": w.delta,
                   "cap": gm.cap, "steps_timed": [args.warmup, total - 1], "eviction_rounds": rounds,
                   "evicted_rows": evicted, "lookahead": 1, "parallelism": "one partition on one GPU"},
        "gather_GBps": round(g_gbps, 1),
        "gather_frac_hbm": round(g_gbps / HBM_PEAK_GBPS, 4),
        "hit_rate": round(hit_rate, 4),
        "roofline": {"bound": "hbm", "kernel": "gather_hbm", "achieved": round(g_gbps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(g_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": gather_traffic(g_bytes_per_launch) if w.name == "cl111m_p64" else None,
                     "bytes_per_launch": round(g_bytes_per_launch), "avg_us": round(g_avg_s * 1e6, 2)},
        "host_link": {"kernel": "gather_miss", "achieved": round(m_gbps, 2), "peak": PCIE_PEAK_GBPS,
                      "unit": "GB/s", "bytes_per_launch": round(m_bytes),
                      "avg_us": round(1e3 * m_ms / max(m_calls, 1), 2)},
        "phase_ms_per_step": {k: round(v[0] / K, 4) for k, v in tim.items()},
        "init_s": round(init_s, 3),
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def cpu_baseline(w, g, local, store, sched, budget_s, first_steps):
    """The oracle, as it stands, on the same workload from step 0 until the
    budget is spent (at least one step); its first steps are also compared
    with the GPU's."""
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
            r, nodes, mask, feat = first_steps[steps]
            same = (r.n == st.n and r.e == st.e and np.array_equal(nodes, st.nodes) and
                    np.array_equal(mask, st.mask) and np.array_equal(feat, st.feat))
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
                      "with the GPU run)" % (steps - 1, w.name, checked),
            "host_cpus": os.cpu_count()}


if __name__ == "__main__":
    main()
