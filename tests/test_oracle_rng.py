"""Pins for the oracle's random vectors (Approx-Top-r draws v_j ~ N(0, I),
Section V-C, eq:random-v): the published Philox4x32-10 known answers, the
exactness of the uniform map, and distribution tests of Box-Muller."""
import os

import numpy as np
import pytest

from oracle.philox import box_muller, gaussian_vectors, philox4x32_10, uniform01

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat_rows():
    rows = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        f = [int(x, 16) for x in line.split()]
        rows.append((f[0:4], f[4:6], f[6:10]))
    return rows


@pytest.mark.parametrize("ctr,key,expect", _kat_rows())
def test_philox_known_answers(ctr, key, expect):
    out = philox4x32_10(np.array(ctr, dtype=np.uint32), tuple(key))
    assert [int(v) for v in out] == expect


def test_philox_is_a_bijection_on_a_slice():
    # for a fixed key, distinct counters give distinct outputs
    ctr = np.zeros((4096, 4), dtype=np.uint32)
    ctr[:, 0] = np.arange(4096)
    out = philox4x32_10(ctr, (12345, 678))
    assert len({tuple(r) for r in out.tolist()}) == 4096


def test_uniform_map_is_open_and_exact_in_fp32():
    x = np.array([0, 1, 511, 512, 0x80000000, 0xFFFFFFFF], dtype=np.uint32)
    u = uniform01(x)
    assert u[0] == 2.0 ** -24
    assert u[-1] == 1.0 - 2.0 ** -24
    assert np.all((u > 0) & (u < 1))
    assert np.array_equal(u.astype(np.float32).astype(np.float64), u)


def test_box_muller_moments():
    rng = np.random.default_rng(3)
    xa = rng.integers(0, 2 ** 32, size=400_000, dtype=np.uint64).astype(np.uint32)
    xb = rng.integers(0, 2 ** 32, size=400_000, dtype=np.uint64).astype(np.uint32)
    z0, z1 = box_muller(xa, xb)
    z = np.concatenate([z0, z1])
    n = z.size
    assert abs(z.mean()) < 5 / np.sqrt(n)
    assert abs(z.var() - 1) < 5 * np.sqrt(2 / n)
    assert abs((z ** 4).mean() - 3) < 5 * np.sqrt(96 / n)
    assert abs(np.mean(np.abs(z) > 3) - 0.0026998) < 5 * np.sqrt(0.0027 / n)
    assert abs(np.corrcoef(z0, z1)[0, 1]) < 5 / np.sqrt(z0.size)


def test_gaussian_vectors_layout_and_stats():
    v = gaussian_vectors(seed=7, t=3, mat=1, rows=np.arange(64), length=1001)
    assert v.shape == (64, 1001) and v.dtype == np.float32
    # a subset of rows / a prefix of the length reproduces the same values
    sub = gaussian_vectors(seed=7, t=3, mat=1, rows=[5, 40], length=13)
    assert np.array_equal(sub, v[[5, 40], :13])
    # different step, matrix or seed give different vectors
    for kw in (dict(seed=7, t=4, mat=1), dict(seed=7, t=3, mat=2), dict(seed=8, t=3, mat=1)):
        other = gaussian_vectors(rows=np.arange(64), length=1001, **kw)
        assert not np.array_equal(other, v)
    z = v.astype(np.float64).ravel()
    assert abs(z.mean()) < 5 / np.sqrt(z.size)
    assert abs(z.var() - 1) < 5 * np.sqrt(2 / z.size)
    # distinct rows are uncorrelated
    c = np.corrcoef(v.astype(np.float64))
    off = c[~np.eye(64, dtype=bool)]
    assert np.abs(off).max() < 6 / np.sqrt(1001)
