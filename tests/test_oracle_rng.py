"""Pins of the oracle's Philox4x32-10 and of the draws made from it."""
import os
import shutil
import subprocess

import numpy as np
import pytest
from scipy import stats

from oracle import rng


def _kat(golden_dir):
    rows = []
    with open(os.path.join(golden_dir, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            v = [int(t, 16) for t in line.split()]
            rows.append((v[0:4], v[4:6], v[6:10]))
    return rows


def test_philox_known_answers(golden_dir):
    for ctr, key, out in _kat(golden_dir):
        got = rng.philox4x32_10(np.array(ctr), key)
        assert [int(g) for g in got] == out


_RR_SRC = r"""
#include <cstdio>
#include <rocrand/rocrand_philox4x32_10.h>
int main() {
  unsigned int c[4], k[2];
  while (scanf("%x %x %x %x %x %x", &c[0], &c[1], &c[2], &c[3], &k[0], &k[1]) == 6) {
    unsigned long long seed = (unsigned long long)k[0] | ((unsigned long long)k[1] << 32);
    unsigned long long sub = (unsigned long long)c[2] | ((unsigned long long)c[3] << 32);
    unsigned long long q = (unsigned long long)c[0] | ((unsigned long long)c[1] << 32);
    rocrand_device::philox4x32_10_engine e(seed, sub, 0);
    while (q) { unsigned long long s = q < (1ull << 60) ? q : (1ull << 60); e.discard(4ull * s); q -= s; }
    uint4 r = e.next4();
    printf("%08x %08x %08x %08x\n", r.x, r.y, r.z, r.w);
  }
  return 0;
}
"""


def test_philox_matches_rocrand_host_engine(tmp_path):
    """rocRAND's Philox engine (host-callable header) is an independent library
    implementation: counter (c0,c1,c2,c3) = (offset/4 as 64 bits, subsequence as 64 bits)."""
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc) or not os.path.exists("/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"):
        pytest.skip("rocRAND headers / hipcc not available")
    src = tmp_path / "rr.cpp"
    src.write_text(_RR_SRC)
    exe = tmp_path / "rr"
    r = subprocess.run([hipcc, "-O1", str(src), "-o", str(exe)], capture_output=True, text=True)
    if r.returncode != 0:
        pytest.skip("could not build the rocRAND host harness: " + r.stderr[-300:])
    g = np.random.default_rng(123)
    cases = g.integers(0, 2 ** 32, size=(64, 6), dtype=np.uint64)
    cases[:8, 0:2] = 0
    cases[8:16, 1:3] = 0
    inp = "\n".join(" ".join("%x" % int(v) for v in row) for row in cases) + "\n"
    out = subprocess.run([str(exe)], input=inp, capture_output=True, text=True, check=True).stdout.split("\n")
    for row, line in zip(cases, out):
        got = rng.philox4x32_10(row[:4], (int(row[4]), int(row[5])))
        assert " ".join("%08x" % int(v) for v in got) == line


def test_stream_counter_layout():
    w = rng.raw_words(7, 10, cell=3, gen=5, step_field=2, tag="Z")
    blk = rng.philox4x32_10(np.array([[1, 3, (5 << 16) | 2, rng.TAG["Z"]]]), (7, 0))[0]
    assert [int(x) for x in w[4:8]] == [int(x) for x in blk]


def test_uniform_map_is_exact_and_open():
    u = rng.to_uniform(np.array([0, 511, 512, 2 ** 31, 2 ** 32 - 1], dtype=np.uint64))
    assert u[0] == 2.0 ** -24 and u[1] == 2.0 ** -24
    assert u[2] == 1.5 * 2.0 ** -23
    assert u[3] == 0.5 + 2.0 ** -24
    assert u[4] == 1.0 - 2.0 ** -24
    assert np.all(u.astype(np.float32).astype(np.float64) == u)
    w = np.random.default_rng(0).integers(0, 2 ** 32, size=100000, dtype=np.uint64)
    uu = rng.to_uniform(w)
    assert np.all((uu > 0) & (uu < 1))
    assert np.all(uu.astype(np.float32).astype(np.float64) == uu)


def test_normals_distribution():
    n = rng.normals(0, 400_000, cell=1, gen=2, step_field=3, tag="Z")
    assert abs(n.mean()) < 0.01
    assert abs(n.var() - 1.0) < 0.01
    assert stats.kstest(n, "norm").pvalue > 1e-3
    # Box-Muller pairs: the two outputs of one pair are uncorrelated
    assert abs(np.corrcoef(n[0::4], n[1::4])[0, 1]) < 0.01


def test_indices_uniform_and_in_range():
    N = 37
    idx = rng.indices(0, 370_000, N, cell=0, gen=0, step_field=1)
    assert idx.min() == 0 and idx.max() == N - 1
    counts = np.bincount(idx, minlength=N)
    assert stats.chisquare(counts).pvalue > 1e-3
    # floor(w * N / 2^32) on the exact words
    w = rng.raw_words(0, 5, 0, 0, 1, "IDX")
    assert list(idx[:5]) == [int(x) * N // 2 ** 32 for x in w]
