"""Shared driver for the GPU parity tests: runs the HIP path (through the C
ABI) and the CPU oracle side by side on identical seeded inputs and compares
what is unique: projectors P P^T (never P itself: signs and rotations inside
equal singular values are free), E^(i), E-bar, X, the optimizer state, the
selection J, and the singular values at refresh steps.

Hand-off mode (the default).  The columns of U inside a cluster of nearly
equal singular values are fixed by the data only up to rotations inside the
cluster, yet Approx-Top-r may select such columns.  So, after every refresh
the oracle first checks the GPU's basis against its own fp64 one:
  * orthonormality ||U U^T - I||_max <= 1e-5 (rows the refresh defines);
  * the top singular values, |sigma_gpu - sigma| <= 1e-5 sigma_1;
  * Eckart-Young: | ||Mbar - P P^T Mbar||^2 - sum_{k>r} sigma_k^2 | <=
    1e-5 ||Mbar||^2 with the oracle's Mbar and sigma (holds at any gap);
  * the top-r projector, rel(P P^T) <= 1e-4 when the relative eigengap
    g = (sigma_r^2 - sigma_{r+1}^2) / sigma_1^2 of the oracle's Mbar Mbar^T
    is at least 1e-2; below that the projector moves by up to ~1/g times any
    perturbation of Mbar Mbar^T (Davis-Kahan), so the bar is 1e-4 * (1e-2/g)
    at that step only, and below g = 1e-3 (a closed gap: the top-r subspace
    is not determined by the data, and neither the GPU's iteration nor the
    oracle's converges to a unique one) the projector is not compared and the
    captured energy must be within 5e-4 ||Mbar||^2 of the oracle's;
and then continues from the GPU's basis.  At a selection step the oracle
ranks its own fp64 scores on that basis; J must equal the GPU's unless the
r-th and (r+1)-th scores are within 1e-4 relative (the margin rule), where
the oracle takes the GPU's J.  Every step, whatever happened at the refresh,
E^(i), E-bar, X and the optimizer state must be within 1e-4 relative
(Frobenius), and X after T steps within 1e-3; nothing is carried over or
widened from step to step.

Strict mode (handoff=False): no adoption at all; every bar is the same 1e-4
(and 1e-3 on X_T), so it only passes where every selected column is
well separated from the unselected ones.

bf16 storage (store="bf16"): both sides take the bf16 gradients torch's
conversion makes and store each residual rounded to bf16, the GPU from its
fp32 residual, the oracle from its fp64 one; where the two straddle a
rounding boundary the stored values are adjacent bf16 numbers, both correct,
and an element far below the matrix's scale (a near-cancellation) can sit
several bf16 steps away when the fp32 residual's own error exceeds its bf16
step.  So every element of E^(i) must be within one bf16 step (2^-7 of its
magnitude) plus 1e-5 of the largest |G| + |E| of the oracle's (about ten
times the fp32 path's elementwise error); at most 10% of the elements may
differ at all (a wrong rounding rule moves about half of them); E^(i) and
E-bar as a whole must agree to the format's unit roundoff 2^-9 (relative
Frobenius) instead of 1e-4; every other bar is unchanged; and the oracle then
continues from the GPU's stored buffers (a hand-off of E, as of U)."""
from __future__ import annotations

import numpy as np

from oracle.method import Oracle, oriented_to_mn
from synth import gradient_batch, planted_matrix

# per-step and end-of-trajectory bars (relative Frobenius)
STEP_TOL = 1e-4
FINAL_TOL = 1e-3
MARGIN = 1e-4        # selection margin below which either choice of J is correct
ORTH_TOL = 1e-5
SIGMA_TOL = 1e-5
ENERGY_TOL = 1e-5
GAP_FULL = 1e-2      # relative eigengap at r from which the projector bar is STEP_TOL
GAP_CLOSED = 1e-3    # below it the top-r projector is not determined by the data
BF16_ABS = 1e-5      # bf16 storage: elementwise E allowance beyond one bf16 step, times max |G| + |E|
BF16_TOL = 2.0 ** -9  # bf16 storage: relative bar of E and E-bar (the format's unit roundoff)
BF16_FLIPS = 0.1     # bf16 storage: largest fraction of E elements that may differ
ENERGY_TOL_CLOSED = 5e-4


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


def eigengap(sigma, r, sigma_next=None):
    """(sigma_r^2 - sigma_{r+1}^2) / sigma_1^2 (inf when r covers sigma);
    sigma_next stands for sigma_{r+1} when sigma holds only the top r."""
    s = np.asarray(sigma, dtype=np.float64)
    if s[0] <= 0:
        return np.inf
    if r >= len(s):
        if sigma_next is None:
            return np.inf
        return float((s[r - 1] ** 2 - sigma_next ** 2) / s[0] ** 2)
    return float((s[r - 1] ** 2 - s[r] ** 2) / s[0] ** 2)


def projector_bar(gap):
    return STEP_TOL if gap >= GAP_FULL else STEP_TOL * GAP_FULL / max(gap, 1e-300)


def refresh_rows(wl, d, r):
    """Rows of U^T a refresh defines: the top block only when tau = 1 and the
    library takes its subspace-iteration route (r < d, r <= 256)."""
    return r if (wl.tau == 1 and r < d and r <= 256) else d


class Handoff:
    """The oracle's hand-off hooks (oracle.method.Oracle.step): check the
    GPU's refresh and continue from its basis; take its J at margin-rule
    steps only."""

    def __init__(self, comp, wl, recs):
        self.comp, self.wl, self.recs = comp, wl, recs

    def basis(self, l, t, out):
        m, n = self.wl.shapes[l]
        d = min(m, n)
        r = min(self.wl.rank, d)
        rows = refresh_rows(self.wl, d, r)
        rec = self.recs[l]
        ut = self.comp.Ut(l).double().cpu().numpy()[:rows]
        rec["orth"] = float(np.abs(ut @ ut.T - np.eye(rows)).max())
        assert rec["orth"] < ORTH_TOL, (t, l, rec)
        sig_o = out["sigma"]
        sg = self.comp.sigma(l).double().cpu().numpy()
        k = min(len(sig_o), rows, r + 4)
        s1 = max(float(sig_o[0]), 1e-300)
        rec["sigma"] = float(np.abs(sg[:k] - sig_o[:k]).max() / s1)
        assert rec["sigma"] < SIGMA_TOL, (t, l, rec)
        mbar = out["mbar"]
        fro2 = float(np.sum(mbar * mbar))
        pg = ut[:r].T
        po = out["U"][:, :r]
        gap = eigengap(sig_o, r, out.get("sigma_next")) if r < d else np.inf
        rec["gap"] = gap
        if fro2 > 0 and r < d:
            tail = fro2 - float(np.sum((pg.T @ mbar) ** 2))
            tail_o = fro2 - float(np.sum(np.asarray(sig_o[:r]) ** 2))
            rec["energy"] = abs(tail - tail_o) / fro2
            bar = ENERGY_TOL if gap >= GAP_CLOSED else ENERGY_TOL_CLOSED
            assert rec["energy"] < bar, (t, l, rec)
        rec["proj"] = rel(pg @ pg.T, po @ po.T)
        if gap >= GAP_CLOSED:
            rec["proj_bar"] = projector_bar(gap)
            assert rec["proj"] < rec["proj_bar"], f"t={t} mat={l}: refresh projector rel {rec['proj']:.3e} ({rec})"
        else:
            rec["proj_unpinned"] = True
        return ut.T

    def selection(self, l, t, out, j_oracle):
        m, n = self.wl.shapes[l]
        d = min(m, n)
        r = min(self.wl.rank, d)
        rec = self.recs[l]
        jg = np.sort(self.comp.J(l).cpu().numpy())
        margin = selection_margin(out["score"], r)
        rec["margin"] = margin
        if margin < MARGIN:
            rec["j_handoff"] = True
            return jg
        assert np.array_equal(jg, j_oracle), f"t={t} mat={l}: J {jg} != {j_oracle} (margin {margin:.2e})"
        return j_oracle


def bf16_steps_apart(a, b):
    """Distance in bf16 steps between two arrays of bf16 values (as floats):
    the difference of their order-preserving integer codes (+0 and -0 equal)."""
    def code(x):
        u = (np.asarray(x, dtype=np.float64).astype(np.float32).view(np.uint32) >> 16).astype(np.int64)
        return np.where(u & 0x8000, -(u & 0x7FFF), u)
    return np.abs(code(a) - code(b))


def run_parity(glr, wl, steps=None, refresh="compressed", select="approx", cold_start=False,
               max_sweeps=30, tol=1e-6, check=None, handoff=True, ef=True, store="fp32"):
    """Runs both paths; returns a list of per-step dicts of relative errors.
    Raises AssertionError at the first step over the bars."""
    import torch

    T = wl.steps if steps is None else steps
    comp = glr.GreedyLore(wl.shapes, wl.workers, wl.rank, wl.tau, opt=wl.opt, lr=wl.lr,
                          beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps, refresh=refresh,
                          select=select, seed=wl.seed, max_sweeps=max_sweeps, tol=tol,
                          cold_start=cold_start, ef=ef, store=store)
    orc = Oracle.from_workload(wl, refresh=refresh, select=select, ef=ef, store=store)
    b16 = store == "bf16"
    galore = wl.opt == "galore_adam"
    planted = [planted_matrix(wl, l) for l in range(len(wl.shapes))]
    X = [torch.zeros(m, n, dtype=torch.float32, device="cuda") for (m, n) in wl.shapes]
    log = []
    for t in range(T):
        grads = [gradient_batch(wl, l, t, planted[l]) for l in range(len(wl.shapes))]
        G = [torch.from_numpy(g).cuda() for g in grads]
        if b16:
            G = [g.to(torch.bfloat16) for g in G]
        comp.step(X, G, t)
        torch.cuda.synchronize()
        st = comp.sync_status()
        assert st == 0, f"t={t}: device status {glr.STATUS_NAMES.get(st, st)}"
        recs = [{"t": t, "mat": l} for l in range(len(wl.shapes))]
        res = orc.step(grads, t, handoff=Handoff(comp, wl, recs) if handoff else None)
        for l, o in enumerate(res):
            m, n = wl.shapes[l]
            d = min(m, n)
            r = min(wl.rank, d)
            rec = recs[l]
            rec["refresh"] = o["refresh"]
            jg = comp.J(l).cpu().numpy()
            rows = refresh_rows(wl, d, r)
            ut = comp.Ut(l).double().cpu().numpy()[:rows]
            pg = ut[jg].T
            po = o["P"]
            if not handoff:
                rec["orth"] = float(np.abs(ut @ ut.T - np.eye(rows)).max())
                assert rec["orth"] < ORTH_TOL, (t, l, rec)
                if o["refresh"]:
                    sg = comp.sigma(l).double().cpu().numpy()
                    k = min(len(o["sigma"]), rows, r + 4)
                    rec["sigma"] = float(np.abs(sg[:k] - o["sigma"][:k]).max() / max(o["sigma"][0], 1e-300))
                    assert rec["sigma"] < SIGMA_TOL, (t, l, rec)
                elif r < d:
                    rec["margin"] = selection_margin(o["score"], r)
                    assert rec["margin"] >= MARGIN, f"t={t} mat={l}: selection margin {rec['margin']:.2e}"
                    assert np.array_equal(np.sort(jg), o["J"]), f"t={t} mat={l}: J {jg} != {o['J']}"
                rec["proj"] = rel(pg @ pg.T, po @ po.T)
                assert rec["proj"] < STEP_TOL, f"t={t} mat={l}: proj rel {rec['proj']:.3e} ({rec})"
            else:
                # the oracle continued from the GPU's basis: the selected
                # projectors coincide unless J differs
                rec["proj_sel"] = rel(pg @ pg.T, po @ po.T)
                assert rec["proj_sel"] < STEP_TOL, (t, l, rec)
            mi = np.abs(np.asarray(grads[l], dtype=np.float64)).max() + np.abs(o["E"]).max()
            e_o = oriented_to_mn(o["E"], m, n)
            e_g = comp.E(l).double().cpu().numpy()
            rec["E"] = rel(e_g, e_o, floor=1e-3 * mi * np.sqrt(e_o.size))
            if b16:
                apart = bf16_steps_apart(e_g, e_o)
                rec["E_steps"] = int(apart.max())
                rec["E_flips"] = int(np.count_nonzero(apart))
                bar = 2.0 ** -7 * np.maximum(np.abs(e_g), np.abs(e_o)) + BF16_ABS * mi
                rec["E_elem"] = float((np.abs(e_g - e_o) / bar).max())
                assert rec["E_elem"] <= 1.0, f"t={t} mat={l}: E element off by {rec['E_elem']:.2f} of its bar"
                assert rec["E_flips"] <= BF16_FLIPS * e_o.size, (t, l, rec)
                # the oracle continues from the GPU's stored buffers
                orc.states[l].e = np.swapaxes(e_g, -1, -2).copy() if m > n else e_g.copy()
            rec["X"] = rel(X[l].double().cpu().numpy(), o["X"])
            if galore:
                # Algorithm 5's moments, r x D (oriented) at the start of S1 / S2
                rD = o["g1"].size
                rec["S1"] = rel(comp.S1(l).flatten()[:rD].double().cpu().numpy(), o["g1"].ravel())
                rec["S2"] = rel(comp.S2(l).flatten()[:rD].double().cpu().numpy(), o["g2"].ravel())
            else:
                rec["S1"] = rel(comp.S1(l).double().cpu().numpy(), o["s1"])
                if o["s2"] is not None:
                    rec["S2"] = rel(comp.S2(l).double().cpu().numpy(), o["s2"])
            rec["Ebar"] = rel(comp.Ebar(l).double().cpu().numpy(), e_o.mean(axis=0),
                              floor=1e-3 * mi * np.sqrt(m * n))
            for key in ("E", "X", "S1", "S2", "Ebar"):
                if key in rec:
                    bar = BF16_TOL if (b16 and key in ("E", "Ebar")) else STEP_TOL
                    assert rec[key] < bar, f"t={t} mat={l}: {key} rel {rec[key]:.3e} ({rec})"
            if check is not None:
                check(comp, o, t, l, rec)
            log.append(rec)
    for l in range(len(wl.shapes)):
        final = rel(X[l].double().cpu().numpy(), orc.states[l].x)
        log.append({"final_X": final, "mat": l})
        assert final < FINAL_TOL, f"mat {l}: X after {T} steps rel {final:.3e} (bar {FINAL_TOL:.0e})"
    summarize(wl.name, log)
    return log


def summarize(name, log):
    """Prints the largest value of every compared quantity (and the smallest
    eigengap and selection margin, and how many J hand-offs took place)."""
    keys = ("proj", "proj_sel", "E", "Ebar", "X", "S1", "S2", "orth", "sigma", "energy", "final_X", "E_steps",
            "E_flips", "E_elem")
    pinned = [r for r in log if not r.get("proj_unpinned")]
    out = {k: max(r[k] for r in (pinned if k == "proj" else log) if k in r)
           for k in keys if any(k in r for r in (pinned if k == "proj" else log))}
    gaps = [r["gap"] for r in log if "gap" in r and np.isfinite(r["gap"])]
    if gaps:
        out["min_gap"] = min(gaps)
    margins = [r["margin"] for r in log if "margin" in r and np.isfinite(r["margin"])]
    if margins:
        out["min_margin"] = min(margins)
    out["j_handoffs"] = sum(1 for r in log if r.get("j_handoff"))
    out["closed_gap_refreshes"] = sum(1 for r in log if r.get("proj_unpinned"))
    print(f"[parity] {name} max " + " ".join(f"{k}={v:.2e}" if isinstance(v, float) else f"{k}={v}"
                                             for k, v in out.items()), flush=True)
    return out
