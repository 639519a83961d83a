"""GreedyLore per-step method, fp64, step by step in the paper's order.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Notation (per layer matrix, Algorithm 4 / Appendix D): the caller's matrix is
m x n; the method works on the oriented form with d = min(m, n) rows and
D = max(m, n) columns, transposing the gradient when m > n and transposing the
reconstructed gradient back before the optimizer.  Worker i holds the error
buffer E^(i) (d x D, zero at start); all workers share U (d x d, identity at
start) and the weights X (m x n, zero at start in the synthetic workloads).

One step t, following Algorithm 4 with Approx-Top-r (Algorithm 2):
  1. M^(i) = G^(i) (or G^(i)^T) + E^(i)                      [Alg. 3/4, EF]
  2. refresh iff t mod tau == 0                               [eq-SVD-P1]
  3. refresh:  Mbar = mean_i M^(i); U, Sigma = SVD(Mbar); J = {0..r-1}
               (tau = 1, r < d: only U[:, :r] is ever read, so the top-r block
               comes from oracle.subspace instead of the complete basis)
     else:     v_j ~ N(0, I_D); lambda_j^(i) = u_j^T M^(i) v_j;
               lambdabar = mean_i lambda^(i); J = argtop_r(lambdabar^2)
               ('exact' scores ||u_j^T Mbar||^2 instead, eq-semi-lazy-svd-2)
  4. P = U[:, J]                                              [eq-semi-lazy-svd-3]
  5. Q^(i) = P^T M^(i)                                        [eq 8zhb2we09]
  6. E^(i) = M^(i) - P Q^(i)                                  [eq-ef, Alg. 4]
  7. Rbar = mean_i Q^(i)                                      [All-Reduce]
  8. Ghat = P Rbar, transposed back iff m > n                 [Alg. 4]
  9. optimizer on X with Ghat                                 [eq-msgd / eq-adam]
With refresh="full" (Algorithm 3) a refresh step instead sets E^(i) = 0 and
Ghat = Mbar (the uncompressed average).

Baseline modes of the paper's comparisons (Section IV, Algorithm 1; Appendix
E, Algorithm 5):
  * select="lazy": the Lazy-SVD operator, P_t = P_{t-1} between refreshes
    (J kept, no selection);
  * ef=False: no error feedback, M^(i) = G^(i) and E^(i) stays zero;
    Algorithm 1 is select="lazy", ef=False, refresh="full" (Ghat = the mean
    gradient at refresh steps);
  * opt="galore_adam": Algorithm 5, distributed Adam-type GaLore: Lazy-SVD P
    (select "lazy", no error feedback), Adam moments M, V kept in the r x D
    subspace and reset to zero at every refresh,
        M = b1 M + (1 - b1) Rbar,  V = b2 V + (1 - b2) Rbar^2,
        X <- X - gamma P (M / (sqrt(V) + eps))   (transposed back iff m > n).
    Algorithm 5 prints the moment updates with b1 and (1 - b1) exchanged and
    gamma applied twice; they are read as the main text's Adam (eq-adam)
    with one gamma.

Storage mode store="bf16" (mixed precision; the paper does not fix a
precision): the gradients G^(i) and the error buffers E^(i) are held in
bfloat16.  The gradient used is the bf16 rounding of what the caller passes
(bf16_round; idempotent on bf16 values), and after step 6 each E^(i) is
replaced by the bf16 rounding of its fp32 value, so the next step's M^(i) and
Mbar are formed from the stored (rounded) buffers.  Everything else, U, P, Q,
Rbar, Ghat, X and the optimizer state, keeps its precision.

Readings where the paper is loose (each listed in the design notes):
  * the residual of Algorithm 3 is written P R^T, dimensionally impossible;
    Algorithm 4's P R^(i) is used;
  * Algorithm 4 prints the transpose-back on the m <= n branch; the transpose
    is undone iff the gradient was transposed (m > n), as its text says;
  * argtop_r breaks exact ties toward the smaller index; J is kept ascending;
  * "T iterations" means t = 0..T-1; t = 0 is a refresh;
  * MSGD is the EMA form with the (1 - beta) factor; Adam has no bias
    correction and adds eps after the square root.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from .philox import gaussian_vectors
from .subspace import next_singular_value, top_subspace
from .svd import left_svd

# ----------------------------------------------------------------------------
# building blocks (each pinned in tests/test_oracle_method.py)
# ----------------------------------------------------------------------------


def compress(p, g):
    """C(G) = P P^T G (eq 2nasdn)."""
    return p @ (p.T @ g)


def argtop_r(score, r):
    """Indices of the r largest scores (descending; exact ties toward the
    smaller index), returned in ascending index order (eq-semi-lazy-svd-2)."""
    score = np.asarray(score, dtype=np.float64)
    idx = np.arange(score.size)
    order = np.lexsort((idx, -score))
    return np.sort(order[: min(r, score.size)])


def exact_scores(u, mbar):
    """||u_j^T Mbar||^2 for every column u_j of U (eq-semi-lazy-svd-2)."""
    z = u.T @ mbar
    return np.einsum("ij,ij->i", z, z)


def approx_lambdas(u, ms, v):
    """lambda_j^(i) = u_j^T M^(i) v_j per worker (Algorithm 2), and their mean
    over workers (eq:lambda-bar).  ms: N x d x D; v: d x D (row j is v_j)."""
    lam = np.empty((ms.shape[0], u.shape[1]))
    for i in range(ms.shape[0]):
        z = u.T @ ms[i]
        lam[i] = np.einsum("jb,jb->j", z, v)
    return lam, lam.mean(axis=0)


def bf16_round(x):
    """Round to bfloat16 (1 sign, 8 exponent, 7 fraction bits: the upper half
    of an IEEE binary32), to nearest with ties to even, through binary32 as
    the fp32 device values are; returned as fp64.  Finite inputs only.

    The binary32 pattern is split at bit 16: the upper half is kept and
    incremented when the lower half exceeds 0x8000, or equals it with the
    kept half odd (a carry into the exponent is the correct result)."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    upper, lower = bits >> 16, bits & 0xFFFF
    up = (lower > 0x8000) | ((lower == 0x8000) & ((upper & 1) == 1))
    upper = upper + up.astype(np.uint64)
    out = (upper << 16).astype(np.uint32).view(np.float32)
    return out.astype(np.float64)


def approx_lambdas_bf16(u, mbar, v):
    """lambdabar_j = u_j^T Mbar v_j with u_j and Mbar rounded to bf16 (the
    mixed-precision selection mode; v_j and the sums exact), on the mean
    Mbar: the mode is defined on the mean, which equals the per-worker mean
    of Algorithm 2 by linearity."""
    z = bf16_round(u).T @ bf16_round(mbar)
    return np.einsum("jb,jb->j", z, v)


def msgd_update(x, b, ghat, lr, beta):
    """M_t = beta M_{t-1} + (1 - beta) G_t;  X_{t+1} = X_t - gamma M_t (eq-msgd)."""
    b = beta * b + (1.0 - beta) * ghat
    return x - lr * b, b


def adam_update(x, m1, m2, ghat, lr, beta1, beta2, eps):
    """eq-adam: no bias correction; eps added after the square root."""
    m1 = beta1 * m1 + (1.0 - beta1) * ghat
    m2 = beta2 * m2 + (1.0 - beta2) * ghat * ghat
    return x - lr * m1 / (np.sqrt(m2) + eps), m1, m2


# ----------------------------------------------------------------------------
# the per-step driver
# ----------------------------------------------------------------------------


@dataclass
class MatrixState:
    m: int
    n: int
    e: np.ndarray            # N x d x D (oriented)
    u: np.ndarray            # d x d
    x: np.ndarray            # m x n
    s1: np.ndarray           # MSGD buffer / Adam first moment, m x n
    s2: np.ndarray | None    # Adam second moment, m x n
    sigma: np.ndarray | None = None
    j: np.ndarray | None = None      # the current index set J (Lazy-SVD keeps it)
    g1: np.ndarray | None = None     # GaLore subspace first moment, r x D (oriented)
    g2: np.ndarray | None = None     # GaLore subspace second moment, r x D

    @property
    def right(self) -> bool:
        return self.m > self.n


@dataclass
class Oracle:
    shapes: tuple
    workers: int
    rank: int
    tau: int
    opt: str = "msgd"
    lr: float = 0.01
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    seed: int = 0
    refresh: str = "compressed"   # "compressed" (Alg. 4) | "full" (Alg. 3)
    select: str = "approx"        # "approx" (Alg. 2) | "exact" (eq-semi-lazy-svd-2) | "approx_bf16"
    svd_tol: float | None = None
    # refresh route when tau == 1 and r < d: "subspace" (top-r block by
    # subspace iteration + Rayleigh-Ritz, oracle.subspace) or "full" (the
    # complete one-sided Jacobi basis); both give the top-r span
    tau1_route: str = "subspace"
    sub_tol: float = 1e-12
    sub_max_iters: int = 200
    ef: bool = True               # error feedback (False: E stays zero)
    store: str = "fp32"           # "fp32" | "bf16": storage of G^(i) and E^(i)
    states: list = field(default_factory=list)
    t_next: int = 0

    def __post_init__(self):
        if self.store not in ("fp32", "bf16"):
            raise ValueError(f"unknown store {self.store!r}")
        if self.opt == "galore_adam":
            if self.select not in ("approx", "lazy") or self.refresh != "compressed":
                raise ValueError("galore_adam is Algorithm 5: Lazy-SVD selection, compressed refresh steps")
            self.select, self.ef = "lazy", False
        self.states = []
        for (m, n) in self.shapes:
            d, D = min(m, n), max(m, n)
            r = min(self.rank, d)
            galore = self.opt == "galore_adam"
            self.states.append(MatrixState(
                m=m, n=n,
                e=np.zeros((self.workers, d, D)),
                u=np.eye(d),
                x=np.zeros((m, n)),
                s1=np.zeros((m, n)),
                s2=np.zeros((m, n)) if self.opt == "adam" else None,
                j=np.arange(r),
                g1=np.zeros((r, D)) if galore else None,
                g2=np.zeros((r, D)) if galore else None,
            ))

    @classmethod
    def from_workload(cls, wl, **kw):
        return cls(shapes=wl.shapes, workers=wl.workers, rank=wl.rank, tau=wl.tau,
                   opt=wl.opt, lr=wl.lr, beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps,
                   seed=wl.seed, **kw)

    def uses_subspace(self, d, r):
        return self.tau == 1 and r < d and self.tau1_route == "subspace"

    def step(self, grads, t: int, handoff=None):
        """One step on every matrix.  grads[l] is N x m x n (any float dtype).
        Returns one dict of intermediate values per matrix.

        handoff (optional) lets a parity harness continue from another
        implementation's basis (the state hand-off for columns of U that the
        data leave ill-defined): handoff.basis(l, t, out) is called after the
        refresh with out holding this oracle's "U" (columns u_j), "sigma" and
        "mbar", and returns the d x k basis to use from this step on (its
        first r columns become P); handoff.selection(l, t, out, J) is called
        after the selection with out holding "score", and returns the index
        set to use."""
        if t != self.t_next:
            raise ValueError(f"steps run in order: expected t={self.t_next}, got {t}")
        self.t_next += 1
        return [self._step_one(l, st, np.asarray(g, dtype=np.float64), t, handoff)
                for l, (st, g) in enumerate(zip(self.states, grads))]

    def _step_one(self, l, st: MatrixState, g, t, handoff=None):
        n_w = self.workers
        d, D = min(st.m, st.n), max(st.m, st.n)
        r = min(self.rank, d)
        if self.store == "bf16":
            g = bf16_round(g)                                     # G^(i) held in bf16
        gc = np.transpose(g, (0, 2, 1)) if st.right else g        # N x d x D
        ms = gc + st.e if self.ef else gc                         # step 1
        is_refresh = (t % self.tau) == 0                          # step 2
        out = {"refresh": is_refresh, "t": t}
        mbar = ms.sum(axis=0) / n_w
        out["mbar"] = mbar
        if is_refresh:                                            # step 3
            if self.uses_subspace(d, r):
                u, sigma, sweeps, conv = top_subspace(mbar, r, seed=self.seed + 7919 * l + t,
                                                      tol=self.sub_tol, max_iters=self.sub_max_iters)
                out["converged"] = conv
                out["sigma_next"] = next_singular_value(mbar, u)
            else:
                u, sigma, sweeps = left_svd(mbar, tol=self.svd_tol)
            out.update(sigma=sigma, sweeps=sweeps, U_oracle=u)
            if handoff is not None:
                out["U"] = u
                out["mbar"] = mbar
                u = np.asarray(handoff.basis(l, t, out), dtype=np.float64)
            st.u = u
            st.sigma = sigma
            jsel = np.arange(r)
            if st.g1 is not None:                                 # Alg. 5: subspace state reset
                st.g1 = np.zeros_like(st.g1)
                st.g2 = np.zeros_like(st.g2)
        elif self.select == "lazy":                               # Lazy-SVD: P_t = P_{t-1}
            jsel = st.j
        else:
            if self.select == "approx":
                v = gaussian_vectors(self.seed, t, l, np.arange(d), D).astype(np.float64)
                lam_i, lam = approx_lambdas(st.u, ms, v)
                score = lam * lam
                out.update(lam=lam, lam_workers=lam_i)
            elif self.select == "approx_bf16":
                v = gaussian_vectors(self.seed, t, l, np.arange(d), D).astype(np.float64)
                lam = approx_lambdas_bf16(st.u, mbar, v)
                score = lam * lam
                out.update(lam=lam)
            else:
                score = exact_scores(st.u, mbar)
            jsel = argtop_r(score, r)
            out["score"] = score
            out["J_oracle"] = jsel
            if handoff is not None:
                jsel = np.asarray(handoff.selection(l, t, out, jsel))
        st.j = jsel
        p = st.u[:, jsel]                                         # step 4
        q = np.matmul(p.T, ms)                                    # step 5: P^T M^(i) per worker
        rbar = q.sum(axis=0) / n_w                                # step 7
        if is_refresh and self.refresh == "full":
            st.e = np.zeros_like(ms)                              # Alg. 3 reset
            ghat = mbar
        else:
            if self.ef:
                st.e = ms - np.matmul(p, q)                       # step 6: M^(i) - P Q^(i)
                if self.store == "bf16":
                    st.e = bf16_round(st.e)                       # E^(i) held in bf16
            ghat = p @ rbar                                       # step 8
        if self.opt == "galore_adam":                             # Alg. 5, in the subspace
            st.g1 = self.beta1 * st.g1 + (1.0 - self.beta1) * rbar
            st.g2 = self.beta2 * st.g2 + (1.0 - self.beta2) * rbar * rbar
            step = p @ (st.g1 / (np.sqrt(st.g2) + self.eps))
            st.x = st.x - self.lr * (step.T if st.right else step)
            ghat_mn = ghat.T if st.right else ghat
        else:
            ghat_mn = ghat.T if st.right else ghat
            if self.opt == "msgd":                                # step 9
                st.x, st.s1 = msgd_update(st.x, st.s1, ghat_mn, self.lr, self.beta1)
            else:
                st.x, st.s1, st.s2 = adam_update(st.x, st.s1, st.s2, ghat_mn, self.lr,
                                                 self.beta1, self.beta2, self.eps)
        out.update(J=jsel, P=p, Q=q, Rbar=rbar, ghat=ghat_mn,
                   E=st.e.copy(), U=st.u, X=st.x.copy(), s1=st.s1.copy(),
                   s2=None if st.s2 is None else st.s2.copy(),
                   g1=None if st.g1 is None else st.g1.copy(),
                   g2=None if st.g2 is None else st.g2.copy())
        return out


def oriented_to_mn(a, m, n):
    """Map an oriented d x D (or N x d x D) array back to the m x n layout."""
    if m > n:
        return np.swapaxes(a, -1, -2)
    return a


class ColumnOracle:
    """The oracle's step restricted to a sample of columns of the oriented
    problem of one matrix, given the projector P of every step.

    Once P is fixed for a step, everything after the selection acts on the
    columns of the oriented d x D problem one at a time (Algorithm 4): for a
    column b, M^(i)[:, b] = G^(i)[:, b] + E^(i)[:, b], Q^(i)[:, b] =
    P^T M^(i)[:, b], E^(i)[:, b] = M^(i)[:, b] - P Q^(i)[:, b], Rbar[:, b] =
    mean_i Q^(i)[:, b], Ghat[:, b] = P Rbar[:, b] (or Mbar[:, b] at an
    Algorithm 3 refresh, with E = 0), and the optimizer is elementwise.  So the
    sampled columns of E^(i), X and the optimizer state follow exactly the
    full oracle's trajectory given the same P at every step, at a cost
    proportional to the sample.  X, S1 and S2 are kept oriented (the
    transpose of the caller's layout when m > n).  store="bf16" rounds the
    gradient columns and the new residual columns to bf16 as Oracle does."""

    def __init__(self, shape, cols, workers, opt="msgd", lr=0.01, beta1=0.9, beta2=0.999, eps=1e-8,
                 refresh="compressed", store="fp32"):
        m, n = shape
        d = min(m, n)
        self.cols = np.asarray(cols)
        c = len(self.cols)
        self.opt, self.lr, self.beta1, self.beta2, self.eps = opt, lr, beta1, beta2, eps
        self.refresh = refresh
        if store not in ("fp32", "bf16"):
            raise ValueError(f"unknown store {store!r}")
        self.store = store
        self.e = np.zeros((workers, d, c))
        self.x = np.zeros((d, c))
        self.s1 = np.zeros((d, c))
        self.s2 = np.zeros((d, c)) if opt == "adam" else None

    def step(self, g_cols, p, is_refresh):
        """g_cols: N x d x c, the sampled oriented columns of this step's
        gradients; p: d x r, this step's P.  Returns the new state (oriented
        columns): E (N x d x c), Ebar, X, S1, S2."""
        g_cols = np.asarray(g_cols, dtype=np.float64)
        if self.store == "bf16":
            g_cols = bf16_round(g_cols)
        ms = g_cols + self.e
        p = np.asarray(p, dtype=np.float64)
        q = np.matmul(p.T, ms)
        if is_refresh and self.refresh == "full":
            self.e = np.zeros_like(ms)
            ghat = ms.mean(axis=0)
        else:
            self.e = ms - np.matmul(p, q)
            if self.store == "bf16":
                self.e = bf16_round(self.e)
            ghat = p @ q.mean(axis=0)
        if self.opt == "msgd":
            self.x, self.s1 = msgd_update(self.x, self.s1, ghat, self.lr, self.beta1)
        else:
            self.x, self.s1, self.s2 = adam_update(self.x, self.s1, self.s2, ghat, self.lr, self.beta1,
                                                   self.beta2, self.eps)
        return {"E": self.e, "Ebar": self.e.mean(axis=0), "X": self.x, "S1": self.s1, "S2": self.s2}
