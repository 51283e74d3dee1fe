"""GPU parity on random partitions. 40 tiny seeded cases drawn over graph
density, halo size (none included), row width (fp32 and bf16), hops and
fanouts, f from 0 to 100%, gamma, Delta and batch sizes. Each runs through
the C ABI against the oracle, element by element after every step: blocks,
frontier, masks, gathered rows, eviction sets, scores and buffer rows. Ten
medium cases (seeded Chung-Lu partitions of 3K-40K nodes with random shapes)
do the same where frontiers, scans and lists span many tiles."""
import numpy as np
import pytest

from gpu_util import log, require_gpu, run_parity
from helpers import tiny_problem

pytestmark = pytest.mark.gpu

N_CASES = 40


def random_cases(n=N_CASES, seed=2024):
    rng = np.random.default_rng(seed)
    out = []
    for c in range(n):
        L = int(rng.integers(1, 13))
        H = int(rng.integers(0, 21))
        K = int(rng.integers(1, 4))
        dtype = "f32" if rng.random() < 0.6 else "bf16"
        d = int(rng.integers(1, 10)) if dtype == "f32" else 2 * int(rng.integers(1, 6))  # rows of 4k bytes
        prob = tiny_problem(n_local=L, n_halo=H, p=float(rng.uniform(0.05, 0.9)), seed=int(rng.integers(0, 10_000)),
                            d=d, fanout=tuple(int(x) for x in rng.integers(1, 7, size=K)),
                            buffer_pct=int(rng.integers(0, 101)), gamma=float(rng.choice([1.0, 0.95, 0.8, 0.5, 0.3])),
                            delta=int(rng.integers(1, 6)), dtype=dtype)
        steps = int(rng.integers(1, 25))
        most = int(rng.integers(1, L + 1))
        batches = [rng.permutation(L)[:int(rng.integers(1, most + 1))].astype(np.int32) for _ in range(steps)]
        out.append(("rand%d L=%d H=%d K=%d fo=%s f=%d%% g=%.2f D=%d %s d=%d steps=%d"
                    % (c, L, H, K, prob.fanout, prob.buffer_pct, prob.gamma, prob.delta, dtype, d, steps),
                    prob, batches))
    return out


def test_random_tiny_partitions():
    require_gpu()
    rounds = 0
    for name, prob, batches in random_cases():
        log(name)
        r, _, _ = run_parity(name, prob, lambda t, b=batches: b[t], len(batches), buffer_rows_every=1)
        rounds += r
    log("random tiny partitions: %d cases, %d rounds that evicted" % (N_CASES, rounds))
    assert rounds >= 10


def random_medium_cases(n=10, seed=77):
    """Seeded Chung-Lu partitions of a few thousand to 40K nodes: frontiers,
    scans and buffers that span several tiles, with random shapes."""
    import synth
    from helpers import Problem
    from synth.workloads import Workload
    rng = np.random.default_rng(seed)
    out = []
    for c in range(n):
        dtype = "f32" if rng.random() < 0.7 else "bf16"
        d = int(rng.integers(1, 65)) if dtype == "f32" else 2 * int(rng.integers(1, 33))
        K = int(rng.integers(1, 4))
        fan = tuple(int(x) for x in rng.integers(1, 31, size=K))
        w = Workload("rm%d" % c, int(rng.integers(3000, 40001)), float(rng.uniform(1.9, 2.6)),
                     float(rng.uniform(4, 30)), bool(rng.random() < 0.3), int(rng.choice([2, 4, 8])), d, dtype,
                     10, 64, fan, int(rng.integers(0, 101)), float(rng.choice([1.0, 0.95, 0.8, 0.5])),
                     int(rng.integers(1, 7)), 1, seed=int(rng.integers(0, 1000)), philox_seed=int(rng.integers(0, 2**40)))
        g = synth.partition_graph(w)
        lf = synth.features(g.local_gid, d, dtype, w.seed)
        hs = synth.features(g.halo_gid, d, dtype, w.seed)
        prob = Problem(g.L, g.H, g.indptr, g.indices, g.halo_gid, g.halo_degree, lf, hs, d, dtype, fan,
                       w.buffer_pct, w.gamma, w.delta, w.philox_seed)
        steps = int(rng.integers(4, 11))
        most = int(rng.integers(1, min(g.L, 1500) + 1))
        batches = [rng.permutation(g.L)[:int(rng.integers(0, most + 1))].astype(np.int32) for _ in range(steps)]
        out.append(("%s n=%d P=%d L=%d H=%d nnz=%d K=%d fo=%s f=%d%% g=%.2f D=%d %s d=%d steps=%d"
                    % (w.name, w.n, w.parts, g.L, g.H, g.nnz, K, fan, w.buffer_pct, w.gamma, w.delta, dtype, d,
                       steps), prob, batches))
    return out


def test_random_medium_partitions():
    require_gpu()
    rounds = 0
    for name, prob, batches in random_medium_cases():
        log(name)
        r, _, _ = run_parity(name, prob, lambda t, b=batches: b[t], len(batches), buffer_rows_every=3,
                             batch_max=max(1, max(len(b) for b in batches)))
        rounds += r
    log("random medium partitions: %d rounds that evicted" % rounds)
    assert rounds >= 3
