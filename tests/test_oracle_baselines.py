"""Pins for the oracle's baseline modes (the paper's comparison algorithms):
the Lazy-SVD operator and Algorithm 1 (Section IV), Propositions 1 and 2
through the step driver, Appendix C's non-contractive trajectory, and the
distributed Adam-type GaLore of Algorithm 5 (Appendix E)."""
import numpy as np
import pytest

from oracle.method import Oracle, adam_update
from synth import get_workload, gradient_batch, planted_matrix


def _grads(wl, T):
    planted = planted_matrix(wl, 0)
    return [gradient_batch(wl, 0, t, planted).astype(np.float64) for t in range(T)]


def test_prop1_lazy_svd_nullifies_error_feedback_through_the_driver():
    # with P kept between refreshes, C(G + E) = C(G): the runs with and without
    # error feedback update X identically until the next refresh
    wl = get_workload("mid_left", tau=5)
    a = Oracle.from_workload(wl, select="lazy", ef=True)
    b = Oracle.from_workload(wl, select="lazy", ef=False)
    for t, g in enumerate(_grads(wl, 5)):
        oa, ob = a.step([g], t)[0], b.step([g], t)[0]
        assert np.array_equal(oa["J"], ob["J"]) and np.array_equal(oa["J"], np.arange(wl.rank))
        assert np.linalg.norm(oa["ghat"] - ob["ghat"]) <= 1e-12 * np.linalg.norm(ob["ghat"])
        assert np.linalg.norm(oa["X"] - ob["X"]) <= 1e-12 * np.linalg.norm(ob["X"])
        if t > 0:
            assert np.any(oa["E"]) and not np.any(ob["E"])


def test_algorithm1_against_a_library_svd():
    # Algorithm 1: at refresh steps Ghat is the mean gradient and P the top r
    # left singular vectors of it (here from numpy's LAPACK SVD), kept until
    # the next refresh; in between Ghat = P P^T Gbar; no error feedback
    wl = get_workload("tiny_left", tau=3)
    orc = Oracle.from_workload(wl, select="lazy", ef=False, refresh="full")
    P = None
    for t, g in enumerate(_grads(wl, 8)):
        o = orc.step([g], t)[0]
        gbar = g.mean(axis=0)
        if t % wl.tau == 0:
            P = np.linalg.svd(gbar)[0][:, :wl.rank]
            expect = gbar
        else:
            expect = P @ (P.T @ gbar)
        assert np.linalg.norm(o["ghat"] - expect) <= 1e-10 * np.linalg.norm(expect), t
        assert not np.any(o["E"])


@pytest.mark.parametrize("ef", [True, False])
def test_prop2_worked_example_through_the_driver(ef):
    # G_0 = diag(2, 1): the refresh picks e1 (r = 1); G_t = diag(0, 1) after
    # it: the lazy compressor returns 0 at every later step, with or without
    # error feedback (Proposition 2: not contractive)
    orc = Oracle(shapes=((2, 2),), workers=1, rank=1, tau=100, opt="msgd", lr=0.1, beta1=0.0,
                 select="lazy", ef=ef)
    o = orc.step([np.diag([2.0, 1.0])[None]], 0)[0]
    assert np.allclose(np.abs(o["P"][:, 0]), [1.0, 0.0])
    for t in range(1, 6):
        o = orc.step([np.diag([0.0, 1.0])[None]], t)[0]
        assert np.array_equal(o["ghat"], np.zeros((2, 2)))


def test_appendix_c_trajectory_through_the_driver():
    # f(diag(x, y)) = L x^2 / 2 + L y^2 / 4 from diag(1, 1), P = e1 from the
    # first refresh, plain gradient descent gamma = 1 / (2L) (MSGD, beta 0):
    # x_k = 2^-k and y_k = 1 exactly
    L = 4.0
    orc = Oracle(shapes=((2, 2),), workers=1, rank=1, tau=10 ** 6, opt="msgd", lr=1.0 / (2 * L), beta1=0.0,
                 select="lazy", ef=False)
    st = orc.states[0]
    st.x = np.eye(2)
    for k in range(1, 80):
        x = orc.states[0].x
        g = np.diag([L * x[0, 0], L / 2 * x[1, 1]])[None]
        o = orc.step([g], k - 1)[0]
        assert o["X"][0, 0] == 2.0 ** -k and o["X"][1, 1] == 1.0
        assert o["X"][0, 1] == 0.0 and o["X"][1, 0] == 0.0


def test_galore_with_full_rank_and_the_identity_basis_is_adam():
    # r = d and a diagonal mean gradient at the refresh (so U = I exactly):
    # the subspace moments are the full-dimensional ones and Algorithm 5's
    # update is Adam's (eq-adam) on the gradient, until the next refresh
    rng = np.random.default_rng(3)
    d, D, N = 4, 7, 2
    orc = Oracle(shapes=((d, D),), workers=N, rank=d, tau=100, opt="galore_adam", lr=1e-2,
                 beta1=0.9, beta2=0.999, eps=1e-8)
    g0 = np.zeros((N, d, D))
    g0[:, np.arange(d), np.arange(d)] = np.array([4.0, 3.0, 2.0, 1.0])
    x = np.zeros((d, D))
    m1 = np.zeros((d, D))
    m2 = np.zeros((d, D))
    for t in range(6):
        g = g0 if t == 0 else rng.standard_normal((N, d, D))
        o = orc.step([g], t)[0]
        if t == 0:
            assert np.array_equal(o["U"], np.eye(d))
        x, m1, m2 = adam_update(x, m1, m2, g.mean(axis=0), 1e-2, 0.9, 0.999, 1e-8)
        assert np.linalg.norm(o["X"] - x) <= 1e-12 * np.linalg.norm(x)


def test_galore_moments_are_reset_at_every_refresh():
    # a constant gradient: every refresh restarts the subspace moments, so the
    # X increment of each refresh step equals the first one, and the
    # increments in between (moments warming up) differ from it
    wl = get_workload("tiny_left", tau=3, opt="galore_adam")
    g = _grads(wl, 1)[0]
    orc = Oracle.from_workload(wl)
    xs = [np.zeros(wl.shapes[0])]
    for t in range(9):
        o = orc.step([g], t)[0]
        assert np.array_equal(o["J"], np.arange(wl.rank))
        xs.append(o["X"])
    inc = [xs[k + 1] - xs[k] for k in range(9)]
    for k in (3, 6):
        assert np.linalg.norm(inc[k] - inc[0]) <= 1e-9 * np.linalg.norm(inc[0])
    assert np.linalg.norm(inc[1] - inc[0]) > 1e-3 * np.linalg.norm(inc[0])


def test_galore_requires_the_compressed_refresh():
    with pytest.raises(ValueError):
        Oracle(shapes=((4, 6),), workers=1, rank=2, tau=2, opt="galore_adam", refresh="full")
