"""A model of the sampler's single-pass scan (decoupled look-back, as in
k_row_scan and k_bits_scan): tiles start in order but run in any
interleaving, each publishes its aggregate and then its inclusive prefix in
one epoch-tagged word, and waits by reading 64 predecessors at a time. The
model checks that every tile gets the exact exclusive prefix, with stale
flags of an older epoch present, and that the run ends. It restates the
kernel's steps; the GPU tests exercise the kernel itself. A tile publishes
its aggregate some time after it starts, so a successor can find its flag
still holding the older epoch's value and must wait."""
import random

import pytest

WAVE = 64


def run_model(ntiles, seed, start_prob=0.3):
    rnd = random.Random(seed)
    epoch = 5
    t_agg, t_inc = 2 * epoch, 2 * epoch + 1
    flags = [((2 * 3 + 1) << 32) | rnd.randrange(1000) for _ in range(ntiles)]  # an older epoch's flags
    agg = [rnd.randrange(0, 5000) for _ in range(ntiles)]
    state, started, result = {}, [], {}
    pending = list(range(ntiles))
    for _ in range(10_000_000):
        if len(result) == ntiles:
            break
        if pending and (not started or rnd.random() < start_prob):
            b = pending.pop(0)  # blocks start in order
            state[b] = None     # computing its aggregate: its flag is still an older epoch's
            started.append(b)
            continue
        live = [b for b in started if b not in result]
        if not live:
            continue
        b = rnd.choice(live)
        if state[b] is None:  # the aggregate is ready: publish it, then look back
            flags[b] = ((t_inc if b == 0 else t_agg) << 32) | agg[b]
            state[b] = [b - 1, 0]
            continue
        p, excl = state[b]
        done = p < 0
        if not done:
            vals = [flags[p - lane] if p - lane >= 0 else (t_inc << 32) for lane in range(WAVE)]
            tags = [f >> 32 for f in vals]
            ready = [t in (t_agg, t_inc) for t in tags]
            inc = [t == t_inc for t in tags]
            k = inc.index(True) if any(inc) else WAVE - 1
            if all(ready[:k + 1]):
                excl += sum(v & 0xFFFFFFFF for v in vals[:k + 1])
                if any(inc):
                    done = True
                else:
                    p -= WAVE
                    done = p < 0
            state[b] = [p, excl]
        if done:
            if b > 0:
                flags[b] = (t_inc << 32) | (excl + agg[b])
            result[b] = excl
    assert len(result) == ntiles, "the model did not finish"
    want = 0
    for b in range(ntiles):
        assert result[b] == want, (ntiles, seed, b)
        want += agg[b]


@pytest.mark.parametrize("ntiles", [1, 2, 3, 63, 64, 65, 129, 300])
def test_lookback_exclusive_prefixes(ntiles):
    for seed in range(10):
        run_model(ntiles, seed)
