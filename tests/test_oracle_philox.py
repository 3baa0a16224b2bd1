"""Pins for the oracle's Philox4x32-10 (not GPU)."""
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest
from scipy import stats

from oracle import philox

GOLD = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat():
    rows = []
    for line in open(GOLD):
        if line.startswith("#") or not line.strip():
            continue
        rows.append([int(x, 16) for x in line.split()])
    return rows


@pytest.mark.parametrize("row", _kat())
def test_known_answer_scalar(row):
    ctr, key, want = row[:4], row[4:6], tuple(row[6:])
    assert philox.philox4x32_10_int(ctr, key) == want


def test_known_answer_vectorised():
    rows = np.array(_kat(), dtype=np.uint64)
    out = philox.philox4x32_10(*[rows[:, i] for i in range(6)])
    assert np.array_equal(np.stack(out, 1), rows[:, 6:])


def test_vectorised_matches_scalar_random():
    g = np.random.default_rng(5)
    w = g.integers(0, 2**32, size=(64, 6), dtype=np.uint64)
    vec = np.stack(philox.philox4x32_10(*[w[:, i] for i in range(6)]), 1)
    for i in range(64):
        assert tuple(int(x) for x in vec[i]) == philox.philox4x32_10_int(w[i, :4], w[i, 4:])


def test_uniform_is_24bit_and_in_range():
    u = philox.uniform(np.uint64(123456789012345), np.arange(4096, dtype=np.uint64))
    assert u.min() >= 0 and u.max() < 1
    assert np.all(u * 2**24 == np.floor(u * 2**24))


def test_uniform_chi_square():
    u = philox.uniform(np.uint64(7), np.arange(200000, dtype=np.uint64))
    counts = np.histogram(u, bins=64, range=(0, 1))[0]
    assert stats.chisquare(counts).pvalue > 1e-4


_ROCRAND_SRC = r"""
#include <cstdio>
#include <cstdlib>
#include <rocrand/rocrand_philox4x32_10.h>
int main(int argc, char** argv) {
  // seed, ctr, stream -> word 0 of Philox(key=(seed lo, seed hi), counter=(ctr, stream, 0, 0))
  for (int i = 1; i + 2 < argc; i += 3) {
    unsigned long long seed = strtoull(argv[i], 0, 10);
    unsigned long long ctr = strtoull(argv[i + 1], 0, 10);
    unsigned long long stream = strtoull(argv[i + 2], 0, 10);
    rocrand_device::philox4x32_10_engine e(seed, 0, 4ull * (ctr + (stream << 32)));
    printf("%u\n", e.next());
  }
  return 0;
}
"""


def test_matches_rocrand_engine_on_host():
    """Independent implementation: rocRAND's philox4x32_10 engine, built for
    and run on the host CPU only."""
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "p.hip")
        exe = os.path.join(d, "p")
        open(src, "w").write(_ROCRAND_SRC)
        r = subprocess.run([hipcc, "-O1", "--offload-arch=gfx950", src, "-o", exe],
                           capture_output=True, text=True)
        if r.returncode != 0:
            pytest.skip("could not build rocRAND check: " + r.stderr[-400:])
        g = np.random.default_rng(11)
        cases = [(int(g.integers(0, 2**63)), int(g.integers(0, 2**31)), int(g.integers(0, 2000)))
                 for _ in range(40)] + [(0, 0, 0), (2**64 - 1, 4095, 999)]
        args = [str(x) for c in cases for x in c]
        out = subprocess.run([exe] + args, capture_output=True, text=True, check=True).stdout.split()
    for (seed, ctr, stream), got in zip(cases, out):
        k0, k1 = seed & 0xFFFFFFFF, seed >> 32
        assert philox.philox4x32_10_int((ctr, stream, 0, 0), (k0, k1))[0] == int(got)
        # the sampler's uniform is the top 24 bits of that word
        assert float(philox.uniform(np.uint64(seed), ctr, stream)) == (int(got) >> 8) * 2.0 ** -24
