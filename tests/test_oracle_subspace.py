"""Pins for the oracle's top-r route used when every step is a refresh
(tau = 1; Section V-B, eq-SVD-P1: only span(U[:, :r]) is consumed), and for
the step driver's use of it: against the complete one-sided Jacobi basis, the
library SVD, exact compression of low-rank matrices, Eckart-Young, and
diagonal matrices whose singular subspaces are coordinate spans."""
import numpy as np
import pytest

from oracle.method import Oracle
from oracle.subspace import orth_columns, orth_columns_r, subspace_change, top_subspace
from oracle.svd import left_svd
from synth import get_workload, gradient_batch, planted_matrix


def _gapped(rng, d, D, r, top=5.0, decay=0.93, div=3.0):
    u = np.linalg.qr(rng.standard_normal((d, d)))[0]
    v = np.linalg.qr(rng.standard_normal((D, d)))[0]
    s = top * decay ** np.arange(d)
    s[r:] /= div
    return (u * s) @ v.T


def _proj(p):
    return p @ p.T


@pytest.mark.parametrize("d,D,r", [(24, 40, 3), (64, 300, 8), (120, 500, 20)])
def test_top_subspace_matches_the_jacobi_basis(d, D, r):
    rng = np.random.default_rng(d * 7 + r)
    a = _gapped(rng, d, D, r)
    p, sig, iters, conv = top_subspace(a, r)
    u, s, _ = left_svd(a)
    assert conv
    assert np.linalg.norm(_proj(p) - _proj(u[:, :r])) < 1e-11
    assert np.abs(sig - s[:r]).max() < 1e-11 * s[0]
    assert np.abs(p.T @ p - np.eye(r)).max() < 1e-13


@pytest.mark.slow
def test_top_subspace_matches_the_jacobi_basis_512x2304():
    rng = np.random.default_rng(512)
    a = _gapped(rng, 512, 2304, 64, decay=0.99)
    p, sig, _, conv = top_subspace(a, 64)
    u, s, _ = left_svd(a)
    assert conv
    assert np.linalg.norm(_proj(p) - _proj(u[:, :64])) < 1e-10


def test_ritz_values_are_the_library_singular_values():
    rng = np.random.default_rng(3)
    a = _gapped(rng, 80, 200, 10)
    _, sig, _, _ = top_subspace(a, 10)
    ref = np.linalg.svd(a, compute_uv=False)[:10]
    assert np.allclose(sig, ref, rtol=1e-12, atol=0)
    assert np.all(np.diff(sig) <= 0)


def test_eckart_young_tail_identity():
    rng = np.random.default_rng(4)
    a = _gapped(rng, 60, 150, 7)
    p, _, _, _ = top_subspace(a, 7)
    s = np.linalg.svd(a, compute_uv=False)
    tail = np.sum((a - p @ (p.T @ a)) ** 2)
    assert abs(tail - np.sum(s[7:] ** 2)) < 1e-12 * np.sum(s ** 2)


@pytest.mark.parametrize("rank,r", [(4, 6), (6, 6), (1, 3)])
def test_exact_compression_when_rank_at_most_r(rank, r):
    rng = np.random.default_rng(rank + r)
    a = rng.standard_normal((30, rank)) @ rng.standard_normal((rank, 70))
    p, sig, _, _ = top_subspace(a, r)
    assert np.abs(p.T @ p - np.eye(r)).max() < 1e-12
    assert np.linalg.norm(a - p @ (p.T @ a)) < 1e-12 * np.linalg.norm(a)
    assert np.all(sig[rank:] < 1e-12 * sig[0])


def test_zero_matrix_gives_an_orthonormal_block():
    p, sig, _, _ = top_subspace(np.zeros((12, 30)), 4)
    assert np.all(np.isfinite(p))
    assert np.abs(p.T @ p - np.eye(4)).max() < 1e-14
    assert np.array_equal(sig, np.zeros(4))


def test_diagonal_matrix_gives_the_coordinate_span():
    d, D, r = 10, 16, 3
    a = np.zeros((d, D))
    a[np.arange(d), np.arange(d)] = np.linspace(9.0, 1.0, d)
    p, sig, _, _ = top_subspace(a, r)
    e = np.zeros((d, r))
    e[np.arange(r), np.arange(r)] = 1.0
    # the iteration stops once the sines of the angles are below 1e-12
    assert np.linalg.norm(_proj(p) - _proj(e)) < 1e-11
    assert np.allclose(sig, np.linspace(9.0, 1.0, d)[:r], rtol=0, atol=1e-12)


def test_orth_columns_is_orthonormal_and_spans_the_input():
    rng = np.random.default_rng(5)
    y = rng.standard_normal((40, 9))
    q = orth_columns(y)
    assert np.abs(q.T @ q - np.eye(9)).max() < 1e-14
    # same span: y = q (q^T y)
    assert np.linalg.norm(y - q @ (q.T @ y)) < 1e-12 * np.linalg.norm(y)
    # R of the QR reproduces y with the same Q
    rr = orth_columns_r(y)
    assert np.allclose(q @ rr, y, atol=1e-12)
    assert np.allclose(np.tril(rr, -1), 0.0)


def test_orth_columns_completes_dependent_columns():
    rng = np.random.default_rng(6)
    b = rng.standard_normal((20, 3))
    y = np.concatenate([b, b[:, :1] * 2.0 - b[:, 1:2], np.zeros((20, 2))], axis=1)   # rank 3 of 6
    q = orth_columns(y)
    assert np.abs(q.T @ q - np.eye(6)).max() < 1e-13
    assert np.linalg.norm(b - q[:, :3] @ (q[:, :3].T @ b)) < 1e-12


def test_subspace_change_is_the_sine_of_the_angle():
    th = 0.3
    a = np.array([[1.0], [0.0]])
    b = np.array([[np.cos(th)], [np.sin(th)]])
    assert abs(subspace_change(a, b) - np.sin(th)) < 1e-15


def test_closed_gap_is_reported_as_not_converged():
    a = np.zeros((8, 12))
    a[np.arange(8), np.arange(8)] = [5, 4, 3, 3, 3, 1, 1, 1]   # sigma_3 = sigma_4 at r = 3
    rng = np.random.default_rng(7)
    q = np.linalg.qr(rng.standard_normal((8, 8)))[0]
    _, _, iters, conv = top_subspace(q @ a, 3, max_iters=25)
    assert not conv and iters == 25


@pytest.mark.parametrize("name", ["tau1_left", "tau1_right"])
def test_tau1_oracle_step_route_matches_the_full_jacobi(name):
    # the two refresh routes give the same top-r span, so the whole
    # trajectory (E, X, optimizer state) agrees
    wl = get_workload(name, steps=3)
    a = Oracle.from_workload(wl)
    b = Oracle.from_workload(wl, tau1_route="full")
    planted = planted_matrix(wl, 0)
    for t in range(3):
        g = gradient_batch(wl, 0, t, planted)
        oa, ob = a.step([g], t)[0], b.step([g], t)[0]
        assert oa["converged"]
        assert np.linalg.norm(_proj(oa["P"]) - _proj(ob["P"])) < 1e-10
        for k in ("E", "X", "s1"):
            assert np.linalg.norm(oa[k] - ob[k]) <= 1e-9 * max(np.linalg.norm(ob[k]), 1e-300)


def test_approx_selection_ranks_by_the_square_of_lambda_bar():
    """Oracle.step's Approx-Top-r ranks lambdabar_j^2 (Algorithm 2: Sigma-bar =
    Lambda-bar^2), not lambdabar_j: a hand-built step where the signed ranking
    picks a different set.  t = 0 refreshes on a rank-r diagonal gradient, so
    U = I exactly and E = 0; at t = 1 row j of Mbar is a_j v_j / |v_j|^2, so
    lambdabar_j = u_j^T Mbar v_j = a_j."""
    from oracle.philox import gaussian_vectors
    d, D, r, N = 6, 16, 2, 2
    orc = Oracle(shapes=((d, D),), workers=N, rank=r, tau=10, opt="msgd", lr=0.01, seed=11)
    g0 = np.zeros((N, d, D))
    g0[:, 0, 0], g0[:, 1, 1] = 3.0, 2.0
    o0 = orc.step([g0], 0)[0]
    assert np.array_equal(np.abs(o0["U"]), np.eye(d)) and not np.any(o0["E"])
    v = gaussian_vectors(11, 1, 0, np.arange(d), D).astype(np.float64)
    a = np.array([5.0, 4.0, -10.0, 3.0, 1.0, 0.5])
    row = a[:, None] * v / np.sum(v * v, axis=1)[:, None]
    sgn = np.diag(o0["U"])            # U = diag(+-1): u_j^T Mbar v_j = sgn_j a_j
    g1 = np.stack([row * sgn[:, None]] * N)
    o1 = orc.step([g1], 1)[0]
    assert np.allclose(o1["lam"], a, rtol=1e-12)
    assert np.array_equal(o1["J"], [0, 2])              # top-2 of a^2: 100, 25
    assert not np.array_equal(np.sort(np.argsort(-a)[:r]), o1["J"])   # signed: {0, 1}


def test_next_singular_value_estimate():
    rng = np.random.default_rng(8)
    a = _gapped(rng, 40, 90, 5)
    p, _, _, _ = top_subspace(a, 5)
    from oracle.subspace import next_singular_value
    s = np.linalg.svd(a, compute_uv=False)
    est = next_singular_value(a, p, iters=60)
    assert est <= s[5] * (1 + 1e-12) and est > 0.999 * s[5]
