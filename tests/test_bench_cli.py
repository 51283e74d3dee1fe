"""bench.py's command-line contract on the CPU: it measures one GPU and
refuses any other count before touching a device."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=120)


def test_refuses_more_than_one_gpu():
    for n in ("2", "8"):
        r = run("--gpus", n)
        assert r.returncode == 2 and r.stdout == ""
        assert "one GPU" in r.stderr and "--gpus 1" in r.stderr


def test_help_lists_the_driver_flags():
    r = run("--help")
    assert r.returncode == 0
    for flag in ("--gpus", "--steps", "--warmup"):
        assert flag in r.stdout


def test_headline_window_holds_a_round_after_the_first():
    """The headline window lies after the first eviction round (t = delta), so
    refill traffic is in its steady state, contains a round (a step t > 0
    with t mod delta = 0), and does not overlap the early window."""
    sys.path.insert(0, ROOT)
    from bench import window_plan
    for delta in (1, 2, 3, 4, 8, 16, 32, 64, 100):
        for steps in (1, 2, 5, 19, 20, 31, 32, 33, 64, 192):
            for warmup in (0, 1, 5, 8, 50, 200):
                early, head = window_plan(warmup, steps, delta)
                assert early == (max(1, warmup), max(1, warmup) + steps)
                a, b = head
                assert b - a == steps
                assert a > delta, (delta, steps, warmup, head)
                assert any(t % delta == 0 for t in range(a, b)), (delta, steps, warmup, head)
                assert a >= early[1]
    # an interval too long for a round: the early window only
    assert window_plan(5, 20, 100000) == ((5, 25), (5, 25))
    # the driver's usual call: centred on the round at 2 delta
    assert window_plan(5, 20, 32)[1] == (54, 74)
