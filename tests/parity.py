"""Shared driver for the GPU parity tests: runs the HIP path (through the C
ABI) and the CPU oracle side by side on identical seeded inputs and compares
what is unique: projectors P P^T (never P itself: signs and rotations inside
equal singular values are free), E^(i), X, the optimizer state, the
selection J, and the singular values at refresh steps."""
from __future__ import annotations

import numpy as np

from oracle.method import Oracle, oriented_to_mn
from synth import gradient_batch, planted_matrix

# per-step and end-of-trajectory bars (relative Frobenius)
STEP_TOL = 1e-4
FINAL_TOL = 1e-3
MARGIN = 1e-4   # selection margin below which either choice of J is correct
# An individually selected singular vector u_j is fixed by fp32 data only up
# to about eps32 * sigma_1 / min_k |sigma_j - sigma_k|; a step whose selected
# columns sit that close to an unselected one gets the bar 64 eps32 / gap.
EPS32 = 2.0 ** -24
GAP_FACTOR = 64.0


def selection_gap(sigma, jsel):
    """min over j in J, k not in J of |sigma_j - sigma_k| / sigma_1."""
    sigma = np.asarray(sigma, dtype=np.float64)
    if sigma[0] <= 0:
        return np.inf
    mask = np.ones(len(sigma), dtype=bool)
    mask[jsel] = False
    if not mask.any():
        return np.inf
    rest = sigma[mask]
    return float(min(np.abs(sigma[j] - rest).min() for j in jsel) / sigma[0])


def rel(a, b, floor=0.0):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = max(np.linalg.norm(b), floor)
    if den == 0.0:
        return float(np.linalg.norm(a))
    return float(np.linalg.norm(a - b) / den)


def selection_margin(score, r):
    s = np.sort(np.asarray(score, dtype=np.float64))[::-1]
    if r >= len(s) or s[r - 1] <= 0:
        return np.inf
    return (s[r - 1] - s[r]) / s[r - 1]


def run_parity(glr, wl, steps=None, refresh="compressed", select="approx", cold_start=False,
               max_sweeps=30, tol=1e-6, check=None):
    """Runs both paths; returns a list of per-step dicts of relative errors.
    Raises AssertionError at the first step over the bars."""
    import torch

    T = wl.steps if steps is None else steps
    comp = glr.GreedyLore(wl.shapes, wl.workers, wl.rank, wl.tau, opt=wl.opt, lr=wl.lr,
                          beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps, refresh=refresh,
                          select=select, seed=wl.seed, max_sweeps=max_sweeps, tol=tol,
                          cold_start=cold_start)
    orc = Oracle.from_workload(wl, refresh=refresh, select=select)
    planted = [planted_matrix(wl, l) for l in range(len(wl.shapes))]
    X = [torch.zeros(m, n, dtype=torch.float32, device="cuda") for (m, n) in wl.shapes]
    log = []
    sig_last = [None] * len(wl.shapes)
    carried = [STEP_TOL] * len(wl.shapes)
    for t in range(T):
        grads = [gradient_batch(wl, l, t, planted[l]) for l in range(len(wl.shapes))]
        G = [torch.from_numpy(g).cuda() for g in grads]
        comp.step(X, G, t)
        torch.cuda.synchronize()
        res = orc.step(grads, t)
        st = comp.sync_status()
        assert st in (0, 7), f"t={t}: device status {st}"
        for l, o in enumerate(res):
            m, n = wl.shapes[l]
            d = min(m, n)
            r = min(wl.rank, d)
            rec = {"t": t, "mat": l, "refresh": o["refresh"]}
            if o["refresh"]:
                sig_last[l] = o["sigma"]
                step_tol = STEP_TOL
            else:
                gap = selection_gap(sig_last[l], o["J"]) if r < d else np.inf
                rec["gap"] = gap
                step_tol = max(STEP_TOL, GAP_FACTOR * EPS32 / gap)
            carried[l] = max(carried[l], step_tol)
            rec["tol"] = carried[l]
            ut = comp.Ut(l).double().cpu().numpy()
            jg = comp.J(l).cpu().numpy()
            pg = ut[jg].T
            po = o["P"]
            # the tau = 1 refresh defines only rows 0..r-1 of U^T (its top-r block)
            uo = ut[:r] if (wl.tau == 1 and r < d) else ut
            rec["orth"] = float(np.abs(uo @ uo.T - np.eye(uo.shape[0])).max())
            assert rec["orth"] < 1e-5, (t, l, rec)
            if not o["refresh"] and r < d:
                margin = selection_margin(o["score"], r)
                rec["margin"] = margin
                assert margin >= MARGIN, f"t={t} mat={l}: selection margin {margin:.2e} is ambiguous"
                assert np.array_equal(jg, o["J"]), f"t={t} mat={l}: J {jg} != {o['J']}"
            rec["proj"] = rel(pg @ pg.T, po @ po.T)
            mi = np.abs(np.asarray(grads[l], dtype=np.float64)).max() + np.abs(o["E"]).max()
            e_o = oriented_to_mn(o["E"], m, n)
            e_g = comp.E(l).double().cpu().numpy()
            rec["E"] = rel(e_g, e_o, floor=1e-3 * mi * np.sqrt(e_o.size))
            rec["X"] = rel(X[l].double().cpu().numpy(), o["X"])
            rec["S1"] = rel(comp.S1(l).double().cpu().numpy(), o["s1"])
            if o["s2"] is not None:
                rec["S2"] = rel(comp.S2(l).double().cpu().numpy(), o["s2"])
            rec["Ebar"] = rel(comp.Ebar(l).double().cpu().numpy(), e_o.mean(axis=0),
                              floor=1e-3 * mi * np.sqrt(m * n))
            if o["refresh"]:
                sg = comp.sigma(l).double().cpu().numpy()
                # the tau = 1 refresh returns Ritz values of its top-r block
                k = r if (wl.tau == 1 and r < d) else min(d, r + 4)
                rec["sigma"] = float(np.abs(sg[:k] - o["sigma"][:k]).max() / max(o["sigma"][0], 1e-300))
                assert rec["sigma"] < 1e-5, (t, l, rec)
            assert rec["proj"] < step_tol, f"t={t} mat={l}: proj rel {rec['proj']:.3e} ({rec})"
            for key in ("E", "X", "S1", "S2", "Ebar"):
                if key in rec:
                    assert rec[key] < carried[l], f"t={t} mat={l}: {key} rel {rec[key]:.3e} ({rec})"
            if check is not None:
                check(comp, o, t, l, rec)
            log.append(rec)
    for l in range(len(wl.shapes)):
        final = rel(X[l].double().cpu().numpy(), orc.states[l].x)
        bar = max(FINAL_TOL, 10 * carried[l])
        assert final < bar, f"mat {l}: X after {T} steps rel {final:.3e} (bar {bar:.1e})"
    return log
