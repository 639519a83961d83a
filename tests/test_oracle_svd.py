"""Pins for the oracle's complete left singular basis (Semi-Lazy SVD refresh,
Section V-B eq-SVD-P1; U must be complete for Proposition 3's proof)."""
import itertools

import numpy as np
import pytest

from oracle.svd import left_svd, round_robin


def _rot(a):
    return np.array([[np.cos(a), -np.sin(a)], [np.sin(a), np.cos(a)]])


@pytest.mark.parametrize("n", range(1, 10))
def test_round_robin_covers_every_pair_once(n):
    seen = []
    for p, q in round_robin(n):
        rows = list(p) + list(q)
        assert len(set(rows)) == len(rows)          # disjoint inside a round
        seen += list(zip(p.tolist(), q.tolist()))
    assert sorted(seen) == sorted(itertools.combinations(range(n), 2))


def test_analytic_2x2():
    # A = R(theta) diag(3, 0.5) R(phi)^T has left singular vectors R(theta) e_k
    th, ph = 0.7, -1.1
    a = _rot(th) @ np.diag([3.0, 0.5]) @ _rot(ph).T
    u, s, _ = left_svd(a)
    assert np.allclose(s, [3.0, 0.5], atol=1e-14)
    for k in range(2):
        e = _rot(th)[:, k]
        assert abs(abs(u[:, k] @ e) - 1.0) < 1e-14


def test_analytic_2x3_orthogonal_rows():
    # rows already orthogonal: U is a permutation putting the longer row first
    a = np.array([[0.0, 1.0, 0.0], [2.0, 0.0, 0.0]])
    u, s, _ = left_svd(a)
    assert np.allclose(s, [2.0, 1.0])
    assert np.allclose(np.abs(u), [[0, 1], [1, 0]])


@pytest.mark.parametrize("d,D", [(30, 50), (17, 17), (5, 200), (64, 96)])
def test_matches_library_singular_values_and_gapped_projectors(d, D):
    rng = np.random.default_rng(d * 1000 + D)
    # planted spectrum with clear gaps so that leading projectors are defined
    k = min(d, 6)
    us = np.linalg.qr(rng.standard_normal((d, d)))[0]
    vs = np.linalg.qr(rng.standard_normal((D, d)))[0]
    s = np.concatenate([10.0 * 0.5 ** np.arange(k), 0.01 * rng.random(d - k)])
    a = (us * s) @ vs.T
    u, sig, _ = left_svd(a)
    ref = np.linalg.svd(a, compute_uv=False)
    assert np.allclose(sig, ref, rtol=1e-12, atol=1e-13 * ref[0])
    for r in range(1, k + 1):
        p = u[:, :r] @ u[:, :r].T
        pr = us[:, :r] @ us[:, :r].T
        assert np.abs(p - pr).max() < 1e-11


def test_orthonormal_complete_and_reconstructs_on_rank_deficient():
    rng = np.random.default_rng(1)
    a = rng.standard_normal((20, 5)) @ rng.standard_normal((5, 40))
    u, s, _ = left_svd(a)
    assert np.abs(u.T @ u - np.eye(20)).max() < 1e-13
    assert np.all(s[5:] < 1e-12 * s[0])
    assert np.abs(u @ (u.T @ a) - a).max() < 1e-12 * np.abs(a).max()
    # eigen-residual of A A^T for every column, including the null space
    aat = a @ a.T
    res = aat @ u - u * s ** 2
    assert np.abs(res).max() < 1e-11 * s[0] ** 2


def test_zero_matrix_and_vector_case():
    u, s, _ = left_svd(np.zeros((4, 7)))
    assert np.array_equal(u, np.eye(4)) and np.all(s == 0)
    u, s, _ = left_svd(np.array([[3.0, -4.0]]))       # d = 1 (n = 1 in the paper)
    assert np.array_equal(u, [[1.0]]) and np.isclose(s[0], 5.0)


def test_eckart_young_residual_equals_tail_energy():
    rng = np.random.default_rng(5)
    a = rng.standard_normal((24, 40)) * (0.8 ** np.arange(24))[:, None]
    u, s, _ = left_svd(a)
    for r in range(0, 25):
        p = u[:, :r]
        res = np.sum((a - p @ (p.T @ a)) ** 2)
        assert np.isclose(res, np.sum(s[r:] ** 2), rtol=1e-10, atol=1e-12)


def test_sorted_descending_with_stable_ties():
    a = np.diag([1.0, 3.0, 3.0, 2.0])
    u, s, _ = left_svd(a)
    assert np.array_equal(s, [3.0, 3.0, 2.0, 1.0])
    # equal singular values keep their row order: e_1 before e_2
    assert np.array_equal(np.abs(u), np.eye(4)[:, [1, 2, 3, 0]])
