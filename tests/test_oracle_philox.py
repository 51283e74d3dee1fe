"""Pins for the oracle's Philox4x32-10 (SC'11), which draws the sampler's keys."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat():
    rows = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        v = [int(x, 16) for x in line.split()]
        rows.append((v[0:4], v[4:6], v[6:10]))
    return rows


def test_known_answer_vectors():
    rows = _kat()
    assert len(rows) == 3
    for ctr, key, want in rows:
        assert oracle.philox4x32_10(ctr, key) == want


_PROBE = r"""
#include <cstdio>
#include <cstdlib>
#include <rocrand/rocrand_philox4x32_10.h>
// rocRAND's open-source Philox4x32-10 engine, used on the host as an
// independent implementation of the same published block function.
struct probe : rocrand_device::philox4x32_10_engine {
  static uint4 run(uint4 c, uint2 k) { probe p; return p.ten_rounds(c, k); }
};
int main(int argc, char** argv) {
  unsigned s = (unsigned)atoi(argv[1]);
  for (int i = 0; i < 200; i++) {
    unsigned v[6];
    for (int j = 0; j < 6; j++) { s = s * 1664525u + 1013904223u; v[j] = s ^ (s >> 13); }
    uint4 c = {v[0], v[1], v[2], v[3]}; uint2 k = {v[4], v[5]};
    uint4 o = probe::run(c, k);
    printf("%u %u %u %u %u %u %u %u %u %u\n", v[0], v[1], v[2], v[3], v[4], v[5], o.x, o.y, o.z, o.w);
  }
}
"""


@pytest.mark.skipif(shutil.which("hipcc") is None or not os.path.exists("/opt/rocm/include/rocrand"),
                    reason="hipcc / rocRAND headers not available")
def test_matches_rocrand_engine(tmp_path):
    src = tmp_path / "probe.cpp"
    src.write_text(_PROBE)
    exe = tmp_path / "probe"
    subprocess.check_call(["hipcc", "-O1", str(src), "-o", str(exe)])
    out = subprocess.check_output([str(exe), "12345"], text=True)
    n = 0
    for line in out.splitlines():
        v = [int(x) for x in line.split()]
        assert oracle.philox4x32_10(v[0:4], v[4:6]) == v[6:10]
        n += 1
    assert n == 200


def test_words_are_uniform():
    # 4096 blocks -> 16384 words; top-4-bit histogram is flat (chi^2, 15 dof).
    counts = np.zeros(16)
    for j in range(4096):
        for w in oracle.philox4x32_10([j, 7, 3, 1], [0, 0]):
            counts[w >> 28] += 1
    exp = counts.sum() / 16
    chi2 = ((counts - exp) ** 2 / exp).sum()
    assert chi2 < 40.0  # p ~ 5e-4 for 15 dof
