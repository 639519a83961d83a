"""Top-r left singular block by subspace iteration and Rayleigh-Ritz, fp64.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

When every step is a refresh (tau = 1 in Algorithm 3 / Algorithm 4) the
semi-lazy operator takes J = {1..r} at every step, so only the span of the
first r left singular vectors of the averaged matrix is ever consumed
(Section V-B, eq-SVD-P1 with t mod tau = 0 always); the rest of U is never
read.  For such runs the oracle computes that block directly, with two
textbook methods:

  1. block subspace (orthogonal) iteration on Mbar Mbar^T, written as two
     half steps so that the conditioning is not squared:
         Z   = orth(Mbar^T Q)     (D x r)
         Q'  = orth(Mbar Z)       (d x r)
     orth() is Gram-Schmidt with one full re-orthogonalisation pass
     ("twice is enough", Kahan-Parlett), column by column; a column that
     vanishes (rank-deficient input) is replaced by the first coordinate
     vector that is not in the span of the columns before it, so that Q
     stays orthonormal and complete to r columns.  The iteration stops when
     the subspace change ||(I - Q Q^T) Q'||_F, the Frobenius norm of the sines
     of the principal angles between the two spans, falls below `tol`.
  2. Rayleigh-Ritz: the left singular vectors Y of B = Q^T Mbar (r x D) by
     one-sided Jacobi (oracle.svd.left_svd) applied to R^T, where B^T = Q_2 R
     is a Gram-Schmidt QR of B^T (B = R^T Q_2^T has the left singular
     vectors and values of R^T); P = Q Y, the Ritz vectors in descending
     order of Ritz value.

The top-r subspace is unique exactly when sigma_r > sigma_{r+1}; the rate of
convergence per iteration is (sigma_{r+1} / sigma_r)^2.  When the gap is
closed (error feedback can close it) the iteration stops at `max_iters` and
reports converged = False: any r-dimensional subspace is then only as good
as the energy it captures.

Pins (tests/test_oracle_subspace.py): the top-r projector of the complete
one-sided Jacobi basis on gapped matrices up to 512 x 2304, Ritz values
against the library SVD, exact compression of rank <= r matrices (including
the zero matrix), the Eckart-Young tail identity, diagonal matrices.
"""
from __future__ import annotations

import numpy as np

from .svd import left_svd


def orth_columns(y):
    """Orthonormal basis of the columns of y (n x k, k <= n), column by column
    by Gram-Schmidt with one re-orthogonalisation pass; a column left with
    (numerically) nothing after both passes is replaced by the first
    coordinate vector e_i outside the span of the columns before it."""
    y = np.array(y, dtype=np.float64, copy=True)
    n, k = y.shape
    q = np.zeros((n, k))
    scale = max(float(np.abs(y).max()) if y.size else 0.0, 1e-300)
    nxt = 0   # next coordinate vector to try as a replacement
    for j in range(k):
        v = y[:, j]
        norm0 = float(np.linalg.norm(v))
        for _ in range(2):
            v = v - q[:, :j] @ (q[:, :j].T @ v)
        nv = float(np.linalg.norm(v))
        if nv <= 1e-13 * max(norm0, scale * np.sqrt(n)):
            # replacement: the first e_i that keeps a component of length >= 1/2
            # outside span(q[:, :j]) (one exists among any j + 1 coordinates)
            while True:
                e = np.zeros(n)
                e[nxt % n] = 1.0
                nxt += 1
                for _ in range(2):
                    e = e - q[:, :j] @ (q[:, :j].T @ e)
                ne = float(np.linalg.norm(e))
                if ne >= 0.5:
                    v, nv = e, ne
                    break
        q[:, j] = v / nv
    return q


def subspace_change(q_old, q_new):
    """||(I - Q_old Q_old^T) Q_new||_F: the Frobenius norm of the sines of the
    principal angles between two spans with orthonormal bases."""
    return float(np.linalg.norm(q_new - q_old @ (q_old.T @ q_new)))


def top_subspace(mbar, r, seed=0, tol=1e-12, max_iters=200, start=None):
    """(P, sigma, iters, converged): P (d x r) the Ritz vectors of the top-r
    left singular subspace of Mbar (d x D), in descending order of the Ritz
    values sigma (r).  start: optional d x r initial block (a warm start);
    otherwise a seeded Gaussian block."""
    a = np.asarray(mbar, dtype=np.float64)
    d, D = a.shape
    r = min(r, d)
    if start is None:
        start = np.random.default_rng([int(seed), d, D, r]).standard_normal((d, r))
    q = orth_columns(start)
    converged = False
    iters = 0
    for iters in range(1, max_iters + 1):
        z = orth_columns(a.T @ q)          # D x r
        qn = orth_columns(a @ z)           # d x r
        change = subspace_change(q, qn)
        q = qn
        if change <= tol:
            converged = True
            break
    b = q.T @ a                            # r x D
    rt = orth_columns_r(b.T)               # R of the QR of B^T
    y, sigma, _ = left_svd(rt.T)
    return q @ y, sigma, iters, converged


def next_singular_value(mbar, p, iters=30, seed=0):
    """An estimate from below of sigma_{r+1}(Mbar) for the top-r block P: the
    norm reached by `iters` power iterations on the deflated matrix
    (I - P P^T) Mbar, whose largest singular value is sigma_{r+1} when P
    spans the top r (used to size the eigengap at r, not by the method)."""
    a = np.asarray(mbar, dtype=np.float64)
    d, D = a.shape
    if p.shape[1] >= d:
        return 0.0
    x = np.random.default_rng([int(seed), d, D]).standard_normal(D)
    est = 0.0
    for _ in range(iters):
        nx = float(np.linalg.norm(x))
        if nx == 0.0:
            return 0.0
        x = x / nx
        y = a @ x
        y = y - p @ (p.T @ y)
        est = float(np.linalg.norm(y))
        x = a.T @ y
    return est


def orth_columns_r(y):
    """R (k x k, upper triangular) of y = Q R by the same Gram-Schmidt with
    one re-orthogonalisation pass (columns of y in order; a vanishing column
    gives a zero row of R)."""
    y = np.asarray(y, dtype=np.float64)
    n, k = y.shape
    q = np.zeros((n, k))
    rr = np.zeros((k, k))
    for j in range(k):
        v = y[:, j].copy()
        for _ in range(2):
            c = q[:, :j].T @ v
            rr[:j, j] += c
            v = v - q[:, :j] @ c
        nv = float(np.linalg.norm(v))
        rr[j, j] = nv
        if nv > 0.0:
            q[:, j] = v / nv
    return rr
