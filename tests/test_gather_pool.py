"""The host threads of the staged link mode (csrc/gather_pool.hpp), built
with g++ and run on the CPU: exact row gathers for several thread counts and
sizes, zero rows for ids outside the store, nothing written past the rows."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def test_gather_pool(tmp_path):
    if not shutil.which("g++"):
        pytest.skip("no g++")
    exe = str(tmp_path / "gather_pool_check")
    subprocess.check_call(["g++", "-std=c++17", "-O1", "-pthread", "-Wall", "-Werror", "-fsanitize=thread",
                           os.path.join(HERE, "native", "gather_pool_check.cpp"), "-o", exe])
    out = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stdout + out.stderr
    assert "mismatches 0" in out.stdout
