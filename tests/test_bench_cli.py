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
