"""Pins of the oracle's Philox4x32-10 and uniform conversion (CPU only)."""

import os
import shutil
import subprocess

import numpy as np
import pytest
from scipy import stats

from oracle import brute
from oracle import philox as ph

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat_rows():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            vals = [int(x, 16) for x in line.split()]
            rows.append((vals[:4], vals[4:6], vals[6:10]))
    return rows


def test_kat_vectors_vectorised():
    rows = _kat_rows()
    assert len(rows) == 3
    ctr = np.array([r[0] for r in rows], np.uint32)
    key = np.array([r[1] for r in rows], np.uint32)
    out = ph.philox4x32_10(ctr, key)
    assert out.tolist() == [r[2] for r in rows]


def test_kat_vectors_scalar():
    for ctr, key, expect in _kat_rows():
        assert list(brute.philox(*ctr, *key)) == expect


def test_vectorised_matches_scalar_random():
    rng = np.random.default_rng(123)
    ctr = rng.integers(0, 2 ** 32, size=(200, 4), dtype=np.uint64)
    key = rng.integers(0, 2 ** 32, size=(200, 2), dtype=np.uint64)
    out = ph.philox4x32_10(ctr, key)
    for i in range(200):
        assert tuple(int(v) for v in out[i]) == brute.philox(*map(int, ctr[i]), *map(int, key[i]))


def _hipcc():
    for p in ("/opt/rocm/bin/hipcc", shutil.which("hipcc") or ""):
        if p and os.path.exists(p):
            return p
    return None


@pytest.mark.skipif(_hipcc() is None, reason="hipcc not available to build the rocRAND probe")
def test_matches_rocrand_engine(tmp_path):
    """Independent implementation: rocRAND's open-source Philox4x32-10."""
    src = os.path.join(os.path.dirname(__file__), "philox_rocrand_probe.cpp")
    exe = tmp_path / "probe"
    subprocess.run([_hipcc(), "-x", "hip", "--offload-host-only", "-O1", src, "-o", str(exe)],
                   check=True, capture_output=True)
    rng = np.random.default_rng(7)
    ctr = rng.integers(0, 2 ** 32, size=(500, 4), dtype=np.uint64)
    key = rng.integers(0, 2 ** 32, size=(500, 2), dtype=np.uint64)
    ctr[:50, 1:] = rng.integers(0, 8, size=(50, 3))  # small counters as in the rollout
    inp = "\n".join(" ".join(f"{int(v):x}" for v in list(ctr[i]) + list(key[i]))
                    for i in range(500))
    res = subprocess.run([str(exe)], input=inp, capture_output=True, text=True, check=True)
    got = np.array([[int(x, 16) for x in line.split()] for line in res.stdout.splitlines()],
                   np.uint64)
    np.testing.assert_array_equal(got, ph.philox4x32_10(ctr, key).astype(np.uint64))


def test_uniform_conversion_exact_and_open_interval():
    x = np.array([0, 1, 511, 512, 2 ** 31, 2 ** 32 - 1], np.uint64)
    u = ph.word_to_uniform(x)
    assert u[0] == 2.0 ** -24 and u[-1] == 1.0 - 2.0 ** -24
    assert u[1] == u[0] and u[2] == u[0] and u[3] == 3 * 2.0 ** -24
    # every value is an odd multiple of 2^-24 and exactly representable in float32
    assert np.all(u.astype(np.float32).astype(np.float64) == u)
    assert np.all((u * 2 ** 24) % 2 == 1)
    assert np.all((u > 0) & (u < 1))


def test_stream_layout_blocks_and_words():
    """Uniform i of a stream is word i % 4 of block i // 4 with counter
    (block, step, traj, stream) and key (seed lo, seed hi)."""
    seed = 0x1234_5678_9ABC_DEF0
    u = ph.stream_uniforms(seed, traj=np.array([5]), step=9, stream=2, n=10)[0]
    for i in range(10):
        w = brute.philox(i // 4, 9, 5, 2, seed & 0xFFFFFFFF, seed >> 32)[i % 4]
        assert u[i] == ((w >> 9) + 0.5) * 2.0 ** -23
        assert u[i] == brute.uniform(seed, 5, 9, 2, i)


def test_uniform_statistics():
    u = ph.stream_uniforms(42, traj=np.arange(4096), step=3, stream=1, n=256).ravel()
    assert abs(u.mean() - 0.5) < 5 * np.sqrt(1 / 12 / u.size)
    assert abs(u.var() - 1 / 12) < 0.002
    counts = np.histogram(u, bins=256, range=(0, 1))[0]
    chi2 = stats.chisquare(counts)
    assert chi2.pvalue > 1e-4
    # distinct streams / steps / trajectories are not copies of each other
    a = ph.stream_uniforms(42, traj=np.arange(64), step=3, stream=0, n=64)
    b = ph.stream_uniforms(42, traj=np.arange(64), step=3, stream=1, n=64)
    c = ph.stream_uniforms(42, traj=np.arange(64), step=4, stream=0, n=64)
    d = ph.stream_uniforms(43, traj=np.arange(64), step=3, stream=0, n=64)
    for other in (b, c, d):
        assert abs(np.corrcoef(a.ravel(), other.ravel())[0, 1]) < 5 / np.sqrt(a.size)
