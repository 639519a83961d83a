"""Complete left singular basis by one-sided (Hestenes) Jacobi, fp64.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

The Semi-Lazy SVD operator needs, at every refresh step, the SVD of the
averaged matrix and the *whole* orthonormal U, not only its first r columns
(Section V-B, eq-SVD-P1; Algorithm 3 returns U; the proof of Proposition 3
uses sum_j ||u_j^T G||^2 = ||G||^2, which needs U complete; the memory
discussion prices U at min(m, n)^2).  The paper does not say how the SVD is
computed.  The oracle uses the textbook one-sided Jacobi method (Hestenes 1958):
plane rotations orthogonalise the d rows of A (d x D, d <= D) pairwise until
every pair is numerically orthogonal; the accumulated rotations form U^T, the
row norms are the singular values.  U is complete and orthogonal even when A
is rank-deficient (zero rows stay where they are).

Ordering of the pairs: cyclic, by rounds of the round-robin ("circle")
tournament, so that each round holds d/2 disjoint pairs.  Rotations inside a
round touch disjoint rows and are applied together; that does not change the
arithmetic of any rotation.

Pins: analytic 2x2 SVDs, library SVD singular values and gapped projectors,
orthonormality, completeness on rank-deficient inputs, Eckart-Young
(tests/test_oracle_svd.py).
"""
from __future__ import annotations

import numpy as np


def round_robin(n: int):
    """Rounds of disjoint pairs covering every pair of 0..n-1 exactly once.

    Circle method on an even number of seats; a seat numbered n (when n is
    odd) is a bye.  Returns a list of (p, q) index arrays with p < q.
    """
    seats = n + (n % 2)
    rounds = []
    if seats < 2:
        return rounds
    last = seats - 1
    for k in range(seats - 1):
        ps, qs = [], []
        pairs = [(k, last)]
        for i in range(1, seats // 2):
            pairs.append(((k + i) % last, (k - i) % last))
        for a, b in pairs:
            if a >= n or b >= n:
                continue
            ps.append(min(a, b))
            qs.append(max(a, b))
        if ps:
            rounds.append((np.array(ps), np.array(qs)))
    return rounds


def left_svd(a, tol: float | None = None, max_sweeps: int = 80):
    """(U, sigma, sweeps) with A = U diag(sigma) V^T, U complete (d x d).

    A is d x D with d <= D.  sigma is sorted descending; equal values keep
    their row order (stable sort).  Stops when every pair has
    |w_p . w_q| <= tol * ||w_p|| ||w_q|| during a whole sweep.
    """
    w = np.array(a, dtype=np.float64, copy=True)
    d = w.shape[0]
    if tol is None:
        tol = max(d, 16) * 2.0 ** -52
    ut = np.eye(d)
    rounds = round_robin(d)
    sweeps = 0
    for sweeps in range(1, max_sweeps + 1):
        off = 0.0
        for p, q in rounds:
            wp, wq = w[p], w[q]
            alpha = np.einsum("ij,ij->i", wp, wp)
            beta = np.einsum("ij,ij->i", wq, wq)
            gamma = np.einsum("ij,ij->i", wp, wq)
            scale = np.sqrt(alpha * beta)
            rel = np.zeros_like(gamma)
            nz = scale > 0.0
            rel[nz] = np.abs(gamma[nz]) / scale[nz]
            if rel.size:
                off = max(off, float(rel.max()))
            rot = rel > tol
            if not rot.any():
                continue
            p, q = p[rot], q[rot]
            al, be, ga = alpha[rot], beta[rot], gamma[rot]
            # zero the (p, q) inner product: tan(theta) is the smaller root of
            # t^2 + 2 zeta t - 1 = 0 with zeta = (beta - alpha) / (2 gamma)
            zeta = (be - al) / (2.0 * ga)
            sgn = np.where(zeta >= 0.0, 1.0, -1.0)
            t = sgn / (np.abs(zeta) + np.hypot(1.0, zeta))
            c = 1.0 / np.sqrt(1.0 + t * t)
            s = c * t
            c = c[:, None]
            s = s[:, None]
            wp, wq = w[p], w[q]
            w[p] = c * wp - s * wq
            w[q] = s * wp + c * wq
            up, uq = ut[p], ut[q]
            ut[p] = c * up - s * uq
            ut[q] = s * up + c * uq
        if off <= tol:
            break
    sigma = np.sqrt(np.einsum("ij,ij->i", w, w))
    order = np.argsort(-sigma, kind="stable")
    return ut[order].T.copy(), sigma[order], sweeps
