"""GPU parity on random tiny partitions: 40 seeded cases drawn over graph
density, halo size (none included), row width (fp32 and bf16), hops and
fanouts, f from 0 to 100%, gamma, Delta and batch sizes. Each runs through
the C ABI against the oracle, element by element after every step: blocks,
frontier, masks, gathered rows, eviction sets, scores and buffer rows."""
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
