"""Pins for the oracle's Philox4x32-10 and its uniform draw."""

import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle.philox import philox4x32_10, uniform53
from conftest import GOLDEN


def _kat_rows():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append([int(w, 16) for w in line.split()])
    return rows


def test_published_known_answers():
    rows = _kat_rows()
    assert len(rows) == 3
    for r in rows:
        out = philox4x32_10(r[0:4], r[4:6])
        assert [int(w) for w in out] == r[6:10]


def test_vectorised_matches_scalar():
    rng = np.random.default_rng(5)
    ctr = rng.integers(0, 2**32, size=(4, 50), dtype=np.uint64)
    key = rng.integers(0, 2**32, size=(2,), dtype=np.uint64)
    vec = philox4x32_10(tuple(ctr), (key[0], key[1]))
    for t in range(50):
        one = philox4x32_10(tuple(int(c) for c in ctr[:, t]), (int(key[0]), int(key[1])))
        assert [int(v[t]) for v in vec] == [int(w) for w in one]


@pytest.mark.skipif(shutil.which("hipcc") is None, reason="hipcc not available to build rocRAND's engine")
def test_against_rocrand_engine(tmp_path):
    """rocRAND's host-side Philox engine is an implementation independent of the oracle's."""
    exe = tmp_path / "kat"
    src = os.path.join(GOLDEN, "rocrand_philox_kat.cpp")
    subprocess.run(["hipcc", "--offload-arch=gfx950", "-O1", src, "-o", str(exe)], check=True,
                   capture_output=True)
    rng = np.random.default_rng(11)
    words = rng.integers(0, 2**32, size=(64, 6), dtype=np.uint64)
    words[0] = 0
    words[1, :4] = [7, 11, 13, 0]            # a (row, column, sample, 0) style counter
    stdin = "\n".join(" ".join("%08x" % int(w) for w in row) for row in words) + "\n"
    out = subprocess.run([str(exe)], input=stdin, capture_output=True, text=True, check=True).stdout
    got = [[int(w, 16) for w in line.split()] for line in out.strip().splitlines()]
    mine = philox4x32_10(tuple(words[:, t] for t in range(4)), (words[:, 4], words[:, 5]))
    assert got == [[int(mine[w][r]) for w in range(4)] for r in range(64)]


def test_uniform53_construction():
    i = np.arange(1000)
    u = uniform53(12345, i, 3, 2)
    assert np.all((u >= 0.0) & (u < 1.0))
    # exactly a multiple of 2^-53 built from (x0 >> 5, x1 >> 6)
    x0, x1, _, _ = philox4x32_10((i, 3, 2, 0), (12345, 0))
    ints = (x0 >> np.uint64(5)) * np.uint64(1 << 26) + (x1 >> np.uint64(6))
    assert np.array_equal((u * 2.0**53).astype(np.uint64), ints)
    # different keys / counters give different streams; the mean is ~1/2
    assert not np.array_equal(u, uniform53(12346, i, 3, 2))
    assert not np.array_equal(u, uniform53(12345, i, 4, 2))
    big = uniform53(7, np.arange(200000), 0, 1)
    assert abs(big.mean() - 0.5) < 0.005
    assert abs(big.var() - 1.0 / 12.0) < 0.002


def test_seed_high_word_used():
    a = uniform53(1, np.arange(10), 0, 1)
    b = uniform53(1 + (1 << 32), np.arange(10), 0, 1)
    assert not np.array_equal(a, b)
