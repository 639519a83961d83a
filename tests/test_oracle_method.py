"""Pins for the oracle's compressor, selection, optimizers and step driver,
against what the paper fixes: Proposition 1 (lazy SVD nullifies EF),
Proposition 2's worked example, Appendix C's trajectory, Proposition 3
(contractivity, eq:sub_problem_derivation), the optimality of top-r selection
(eq:new_sub_problem), Proposition 4 (unbiased lambda-bar^2), Lemma 2
(contractive in expectation), the bound in Lemma 4's proof, the optimizer
equations (eq-msgd, eq-adam) and exact compression of low-rank gradients."""
import itertools

import numpy as np
import pytest

from oracle.method import (Oracle, adam_update, approx_lambdas, approx_lambdas_bf16, argtop_r,
                           bf16_round, compress, exact_scores, msgd_update, oriented_to_mn)
from oracle.philox import gaussian_vectors
from oracle.svd import left_svd
from synth import get_workload, gradient_batch, planted_matrix


# ---------------------------------------------------------------- worked examples

def test_prop2_worked_example():
    # G0 = diag(2, 1): its top singular vector is e1; G_t = diag(0, 1) is
    # annihilated by P P^T, so ||C(G_t) - G_t||^2 = ||G_t||^2 = 1.
    u, s, _ = left_svd(np.diag([2.0, 1.0]))
    p = u[:, :1]
    assert np.allclose(np.abs(p[:, 0]), [1.0, 0.0])
    gt = np.diag([0.0, 1.0])
    c = compress(p, gt)
    assert np.array_equal(c, np.zeros((2, 2)))
    assert np.sum((c - gt) ** 2) == np.sum(gt ** 2) == 1.0


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_appendix_c_trajectory(dtype):
    # f(diag(x, y)) = L x^2 / 2 + L y^2 / 4, P = e1 fixed, gamma = 1/(2L),
    # plain GD (MSGD with beta = 0): (x_k, y_k) = (2^-k, 1), and the captured
    # energy ratio alpha = 2^-2tau / (2^-2tau + 1/4).
    L = 4.0
    lr = 1.0 / (2.0 * L)
    p = np.array([[1.0], [0.0]], dtype=dtype)
    x = np.eye(2, dtype=dtype)
    buf = np.zeros((2, 2), dtype=dtype)
    for k in range(1, 130):
        grad = np.diag([L * x[0, 0], L / 2 * x[1, 1]]).astype(dtype)
        x, buf = msgd_update(x, buf, compress(p, grad), dtype(lr), dtype(0.0))
        x = x.astype(dtype)
        assert x[0, 0] == dtype(2.0) ** -k and x[1, 1] == 1.0
        g = np.diag([L * x[0, 0], L / 2 * x[1, 1]]).astype(dtype)
        num = np.sum(compress(p, g) ** 2)
        den = np.sum(g ** 2)
        alpha = num / den
        assert np.isfinite(alpha)
        expect = 2.0 ** (-2 * k) / (2.0 ** (-2 * k) + 0.25)
        if dtype == np.float64 or k <= 62:
            assert np.isclose(alpha, expect, rtol=1e-6)
        if dtype == np.float32 and k > 75:
            assert alpha == 0.0   # 2^-2k underflows fp32: zero energy, no NaN


def test_prop1_lazy_svd_nullifies_error_feedback():
    rng = np.random.default_rng(0)
    p = np.linalg.qr(rng.standard_normal((12, 3)))[0]
    e = np.zeros((12, 20))
    for _ in range(6):
        g = rng.standard_normal((12, 20))
        with_ef = compress(p, g + e)
        assert np.allclose(with_ef, compress(p, g), atol=1e-12)
        e = g + e - with_ef


# ------------------------------------------------------------- selection / Prop. 3

def _random_basis(rng, d):
    return np.linalg.qr(rng.standard_normal((d, d)))[0]


@pytest.mark.parametrize("d,r", [(6, 2), (7, 3), (8, 4), (5, 1)])
def test_top_r_selection_is_the_subset_argmin(d, r):
    rng = np.random.default_rng(d + 10 * r)
    u = _random_basis(rng, d)
    g = rng.standard_normal((d, 11)) * (0.7 ** np.arange(d))[:, None]
    best = min(np.sum((g - compress(u[:, list(j)], g)) ** 2)
               for j in itertools.combinations(range(d), r))
    jsel = argtop_r(exact_scores(u, g), r)
    got = np.sum((g - compress(u[:, jsel], g)) ** 2)
    assert np.isclose(got, best, rtol=1e-12)
    # eq:sub_problem_derivation: residual = ||G||^2 - sum_{j in J} ||u_j^T G||^2
    assert np.isclose(got, np.sum(g ** 2) - exact_scores(u, g)[jsel].sum(), rtol=1e-12)
    # Proposition 3: contractive with delta = r / d
    assert got <= (1 - r / d) * np.sum(g ** 2) * (1 + 1e-12)


def test_argtop_r_ties_go_to_smaller_index():
    s = np.array([1.0, 5.0, 3.0, 5.0, 3.0, 0.0])
    assert list(argtop_r(s, 3)) == [1, 2, 3]
    assert list(argtop_r(s, 1)) == [1]
    assert list(argtop_r(s, 10)) == [0, 1, 2, 3, 4, 5]


def test_prop4_lambda_bar_squared_is_unbiased():
    # E[lambdabar_j^2] = ||u_j^T Gbar||^2; lambdabar_j ~ N(0, l_j^2), so the
    # sample mean over S draws has relative std sqrt(2 / S).
    rng = np.random.default_rng(2)
    d, D, n_w, S = 6, 40, 3, 3000
    u = _random_basis(rng, d)
    ms = rng.standard_normal((n_w, d, D))
    mbar = ms.mean(axis=0)
    target = exact_scores(u, mbar)
    acc = np.zeros(d)
    for t in range(S):
        v = gaussian_vectors(99, t, 0, np.arange(d), D).astype(np.float64)
        lam_i, lam = approx_lambdas(u, ms, v)
        # the per-worker mean equals the bilinear form on the averaged matrix
        direct = np.einsum("aj,ab,jb->j", u, mbar, v)
        assert np.allclose(lam, direct, rtol=1e-12, atol=1e-12)
        acc += lam ** 2
    assert np.all(np.abs(acc / S / target - 1) < 5 * np.sqrt(2 / S))


def test_lemma2_contractive_in_expectation():
    rng = np.random.default_rng(4)
    d, D, r, S = 8, 30, 2, 1500
    u = _random_basis(rng, d)
    g = rng.standard_normal((d, D)) * (0.6 ** np.arange(d))[:, None]
    tot = np.sum(g ** 2)
    errs = []
    for t in range(S):
        v = gaussian_vectors(5, t, 0, np.arange(d), D).astype(np.float64)
        _, lam = approx_lambdas(u, g[None], v)
        j = argtop_r(lam ** 2, r)
        errs.append(np.sum((g - compress(u[:, j], g)) ** 2))
    errs = np.array(errs)
    mean, se = errs.mean(), errs.std() / np.sqrt(S)
    assert mean <= (1 - r / d) * tot + 4 * se
    # and never better than the exact (greedy) choice
    best = np.sum((g - compress(u[:, argtop_r(exact_scores(u, g), r)], g)) ** 2)
    assert errs.min() >= best * (1 - 1e-12)


# ------------------------------------------------------------------ optimizers

def test_msgd_closed_form():
    x, b = msgd_update(np.array([1.0]), np.array([0.5]), np.array([2.0]), 0.1, 0.9)
    # b = 0.9*0.5 + 0.1*2 = 0.65 ; x = 1 - 0.1*0.65 = 0.935
    assert np.allclose(b, 0.65) and np.allclose(x, 0.935)


def test_adam_closed_form_no_bias_correction():
    x, m1, m2 = adam_update(np.array([0.0]), np.array([0.0]), np.array([0.0]),
                            np.array([2.0]), 0.1, 0.9, 0.999, 1e-8)
    # m1 = 0.2, m2 = 0.004, x = -0.1 * 0.2 / (sqrt(0.004) + 1e-8)
    assert np.allclose(m1, 0.2) and np.allclose(m2, 0.004)
    assert np.allclose(x, -0.1 * 0.2 / (np.sqrt(0.004) + 1e-8), rtol=1e-15)
    assert not np.allclose(x, -0.1)          # a bias-corrected Adam would give -0.1


# ------------------------------------------------------------------ step driver

def _run(wl, steps=None, **kw):
    orc = Oracle.from_workload(wl, **kw)
    planted = [planted_matrix(wl, l) for l in range(len(wl.shapes))]
    outs = []
    for t in range(wl.steps if steps is None else steps):
        grads = [gradient_batch(wl, l, t, planted[l]) for l in range(len(wl.shapes))]
        outs.append((grads, orc.step(grads, t)))
    return orc, outs


# ---------------------------------------------------------------- bf16 rounding
# (the mixed-precision selection mode; bfloat16 = the upper half of a binary32)

@pytest.mark.parametrize("x,want", [
    (1.0, 1.0),
    (1.0 + 2.0 ** -8, 1.0),                         # tie, kept half even: down
    (1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -6),         # tie, kept half odd: up
    (1.0 + 2.0 ** -8 + 2.0 ** -20, 1.0 + 2.0 ** -7),  # above the tie
    (1.0 + 2.0 ** -8 - 2.0 ** -20, 1.0),            # below the tie
    (-(1.0 + 3 * 2.0 ** -8), -(1.0 + 2.0 ** -6)),   # sign-symmetric
    (2.0 - 2.0 ** -8, 2.0),                         # tie with odd fraction 127: carries into the exponent
    (3.0, 3.0), (0.0, 0.0), (2.0 ** -130, 2.0 ** -130),
    (np.float32(np.pi), 3.140625),                  # 0x40490FDB -> 0x4049
])
def test_bf16_round_values(x, want):
    assert bf16_round(np.float64(x)) == want


def test_bf16_round_is_the_nearest_bf16_with_ties_to_even():
    # brute force over every low half of a few binary32 patterns: the result is
    # the nearer of the two bf16 neighbours, found by comparing distances in
    # fp64, the even one on a tie
    for upper in (0x3F80, 0x3F81, 0x4049, 0xC2F7, 0x0001, 0x7F7E):
        lows = np.arange(0x10000, dtype=np.uint64)
        bits = ((np.uint64(upper) << np.uint64(16)) | lows).astype(np.uint32)
        x = bits.view(np.float32).astype(np.float64)
        lo = np.uint32(upper << 16)
        hi = np.uint32((upper + 1) << 16)
        a = np.array([lo], dtype=np.uint32).view(np.float32).astype(np.float64)[0]
        b = np.array([hi], dtype=np.uint32).view(np.float32).astype(np.float64)[0]
        da, db = np.abs(x - a), np.abs(x - b)
        want = np.where(da < db, a, np.where(db < da, b, a if upper % 2 == 0 else b))
        assert np.array_equal(bf16_round(x), want), hex(upper)


def test_bf16_round_bound_and_idempotence():
    rng = np.random.default_rng(5)
    x = rng.standard_normal(20000) * np.exp(rng.uniform(-30, 30, 20000))
    y = bf16_round(x)
    x32 = x.astype(np.float32).astype(np.float64)
    # 8 significant bits: unit roundoff 2^-8 (half an ulp at the bottom of a binade)
    assert np.all(np.abs(y - x32) <= 2.0 ** -8 * np.abs(x32))
    assert np.array_equal(bf16_round(y), y)
    o = np.sort(x)
    assert np.all(np.diff(bf16_round(o)) >= 0)        # monotone


def test_bf16_lambdas_equal_the_exact_ones_on_bf16_inputs():
    # on inputs that bf16 holds exactly, the mode's lambdas are Algorithm 2's
    rng = np.random.default_rng(6)
    d, D, N = 12, 20, 3
    u = rng.integers(-8, 9, (d, d)) * 2.0 ** -4
    ms = rng.integers(-64, 65, (N, d, D)) * 2.0 ** -6
    ms[1:] = ms[0]                       # identical workers: their mean is exact too
    v = rng.standard_normal((d, D))
    _, lam = approx_lambdas(u, ms, v)
    assert np.allclose(approx_lambdas_bf16(u, ms[0], v), lam, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("name", ["tiny_left", "ragged_right", "mixed_small"])
@pytest.mark.parametrize("select", ["approx", "exact", "approx_bf16"])
def test_step_invariants(name, select):
    wl = get_workload(name)
    _, outs = _run(wl, select=select)
    e_prev = {}
    for grads, res in outs:
        for l, o in enumerate(res):
            m, n = wl.shapes[l]
            d = min(m, n)
            p, q, e = o["P"], o["Q"], o["E"]
            g = np.asarray(grads[l], dtype=np.float64)
            gc = np.swapaxes(g, 1, 2) if m > n else g
            scale = max(np.abs(g).max(), 1e-300)
            # E^(i) + P Q^(i) = M^(i) = G^(i) + E^(i)_{t-1}  (eq-ef)
            mi = gc + e_prev.get(l, 0.0)
            assert np.allclose(e + np.einsum("ak,ikb->iab", p, q), mi, atol=1e-12 * scale * d)
            e_prev[l] = e
            # P has orthonormal columns
            assert np.abs(p.T @ p - np.eye(p.shape[1])).max() < 1e-12
            # the residual is orthogonal to P, and E + P Q reproduces M
            assert np.abs(np.einsum("ak,iab->ikb", p, e)).max() < 1e-12 * scale * d
            # R-bar is P^T M-bar (linearity of the mean)
            assert np.allclose(o["Rbar"], p.T @ o["mbar"], atol=1e-12 * scale * d)
            # Ghat = P Rbar, in the m x n layout
            assert o["ghat"].shape == (m, n)
            assert np.allclose(oriented_to_mn(p @ o["Rbar"], m, n), o["ghat"], atol=1e-13 * scale * d)
            # Proposition 3 on the averaged matrix, for exact selection
            if select == "exact" or o["refresh"]:
                tot = np.sum(o["mbar"] ** 2)
                res_e = np.sum((o["mbar"] - compress(p, o["mbar"])) ** 2)
                assert res_e <= (1 - p.shape[1] / d) * tot * (1 + 1e-12) + 1e-300
            if o["refresh"]:
                # Eckart-Young at a refresh step: mean error = tail energy
                res_e = np.sum((o["mbar"] - compress(p, o["mbar"])) ** 2)
                sig = o["sigma"]
                assert np.isclose(res_e, np.sum(sig[p.shape[1]:] ** 2), rtol=1e-9,
                                  atol=1e-24 + 1e-14 * np.sum(sig ** 2))


def test_orientation_transpose_symmetry():
    # an m > n matrix is the transposed m <= n problem; X comes back transposed
    wl = get_workload("ragged_right")
    wlt = get_workload("ragged_right", shapes=((72, 200),))
    o1 = Oracle.from_workload(wl)
    o2 = Oracle.from_workload(wlt)
    planted = planted_matrix(wl, 0)
    for t in range(5):
        g = gradient_batch(wl, 0, t, planted)
        r1 = o1.step([g], t)[0]
        r2 = o2.step([np.swapaxes(g, 1, 2).copy()], t)[0]
        assert r1["X"].shape == (200, 72) and r2["X"].shape == (72, 200)
        assert np.allclose(r1["X"], r2["X"].T, rtol=0, atol=1e-13)
        assert np.array_equal(r1["J"], r2["J"])


def test_exact_compression_of_low_rank_gradients():
    # rank(M) <= r: the compressor is exact, E stays 0, Ghat = Mbar
    # (fed in fp64: rounding to fp32 would make the input full rank at 1e-8)
    wl = get_workload("lowrank_exact")
    orc = Oracle.from_workload(wl)
    planted = [planted_matrix(wl, l) for l in range(len(wl.shapes))]
    for t in range(wl.steps):
        res = orc.step([np.stack([pl * (1.0 + 0.1 * i) for i in range(wl.workers)])
                        for pl in planted], t)
        for o in res:
            scale = np.abs(o["mbar"]).max()
            assert np.abs(o["E"]).max() < 1e-12 * scale
            m, n = o["X"].shape
            assert np.allclose(o["ghat"], oriented_to_mn(o["mbar"], m, n), atol=1e-12 * scale)


def test_rank_at_least_d_and_vector_case():
    # r >= d: P = U, nothing is dropped; d = 1 is the vector problem (n = 1)
    wl = get_workload("mixed_small")
    _, outs = _run(wl, steps=4)
    for _, res in outs:
        for l, o in enumerate(res):
            m, n = wl.shapes[l]
            if min(m, n) <= wl.rank:
                assert np.abs(o["E"]).max() < 1e-12 * max(1.0, np.abs(o["mbar"]).max())
            if min(m, n) == 1:
                assert np.array_equal(np.abs(o["U"]), [[1.0]])


def test_zero_gradients_stay_finite():
    wl = get_workload("zero_grad")
    orc, outs = _run(wl)
    for _, res in outs:
        for o in res:
            assert np.all(o["X"] == 0) and np.all(o["E"] == 0)


def test_refresh_full_resets_error_and_bounds_it():
    # Algorithm 3: E = 0 and Ghat = Mbar at refresh steps; in between,
    # ||Ebar_t|| <= ||Ebar_{t-1}|| + ||mean raw gradient_t|| (Lemma 4's proof)
    wl = get_workload("tiny_left")
    _, outs = _run(wl, refresh="full")
    prev = 0.0
    for grads, res in outs:
        o = res[0]
        ebar = o["E"].mean(axis=0)
        nrm = np.linalg.norm(ebar)
        if o["refresh"]:
            assert np.all(o["E"] == 0)
            assert np.allclose(o["ghat"], o["mbar"])
            prev = 0.0
        else:
            graw = np.linalg.norm(np.asarray(grads[0], dtype=np.float64).mean(axis=0))
            assert nrm <= prev + graw + 1e-12
            prev = nrm


def test_steps_must_run_in_order():
    wl = get_workload("tiny_left")
    orc = Oracle.from_workload(wl)
    with pytest.raises(ValueError):
        orc.step([gradient_batch(wl, 0, 1)], 1)


def test_deterministic():
    wl = get_workload("tiny_left")
    a, _ = _run(wl, steps=6)
    b, _ = _run(wl, steps=6)
    assert np.array_equal(a.states[0].x, b.states[0].x)


@pytest.mark.parametrize("name,refresh", [("mid_left", "compressed"), ("ragged_right", "compressed"),
                                          ("ragged_right", "full")])
def test_column_oracle_follows_the_full_oracle(name, refresh):
    # the column-restricted step, fed the full oracle's P, reproduces the full
    # oracle's columns of E, E-bar, X and the optimizer state at every step
    from oracle.method import ColumnOracle
    wl = get_workload(name, steps=7)
    full = Oracle.from_workload(wl, refresh=refresh)
    m, n = wl.shapes[0]
    D = max(m, n)
    cols = np.array([0, 3, D // 2, D - 1])
    col = ColumnOracle(wl.shapes[0], cols, wl.workers, opt=wl.opt, lr=wl.lr, beta1=wl.beta1,
                       beta2=wl.beta2, eps=wl.eps, refresh=refresh)
    planted = planted_matrix(wl, 0)
    for t in range(wl.steps):
        g = gradient_batch(wl, 0, t, planted)
        o = full.step([g], t)[0]
        go = np.swapaxes(g, 1, 2) if m > n else g
        c = col.step(go[:, :, cols], o["P"], o["refresh"])

        def close(a, b):
            # the same products summed in another order (a BLAS call over the
            # sample instead of the whole matrix): agreement to rounding
            return np.linalg.norm(a - b) <= 1e-12 * max(np.linalg.norm(b), 1e-300)

        assert close(c["E"], o["E"][:, :, cols])
        assert close(c["Ebar"], o["E"][:, :, cols].mean(axis=0))
        tr = (lambda a: a.T) if m > n else (lambda a: a)
        assert close(c["X"], tr(o["X"])[:, cols])
        assert close(c["S1"], tr(o["s1"])[:, cols])
        if wl.opt == "adam":
            assert close(c["S2"], tr(o["s2"])[:, cols])
