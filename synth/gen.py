"""Seeded synthetic gradients for the GreedyLore compression path.

Every gradient is  G_t^(i) = U_s diag(s) V_s^T + nu * Z_t^(i):  a planted
low-rank part shared by all workers and all steps, plus fresh i.i.d. N(0, 1)
noise per (step t, worker i).  U_s and V_s are Haar-distributed (QR of a
Gaussian matrix with the signs fixed so that diag(R) > 0).  The paper trains on
real model gradients (LLaMA / RoBERTa 2-D weights, reshaped ResNet conv kernels,
Experiments section); these planted-spectrum matrices stand in for them with the
same shapes.

Streams are independent per (workload, matrix, 'planted') and per
(workload, matrix, t): a step can be regenerated on its own.

This module draws inputs only; it holds none of the method's arithmetic.
"""
from __future__ import annotations

import zlib
from dataclasses import dataclass, field

import numpy as np

_PLANTED_TAG = 0x5EED0001
_NOISE_TAG = 0x5EED0002
_SHAPE_TAG = 0x5EED0003


@dataclass(frozen=True)
class Workload:
    """One experiment: a set of layer matrices, N simulated workers, rank r,
    refresh period tau, T steps and the optimizer."""

    name: str
    shapes: tuple            # ((m, n), ...) in the caller's layout
    workers: int             # N
    rank: int                # r
    tau: int                 # refresh period
    steps: int               # T
    opt: str                 # "msgd" | "adam"
    lr: float
    beta1: float             # MSGD momentum beta, or Adam beta1
    beta2: float = 0.999
    eps: float = 1e-8
    seed: int = 0
    recipe: str = "geometric"
    params: tuple = field(default_factory=tuple)   # recipe parameters

    @property
    def wid(self) -> int:
        return zlib.crc32(self.name.encode()) & 0x7FFFFFFF

    def dims(self, mat: int):
        m, n = self.shapes[mat]
        return min(m, n), max(m, n)


# ----------------------------------------------------------------------------
# spectrum recipes: return (s, nu) for matrix `mat` of the workload
# ----------------------------------------------------------------------------

def _spectrum(wl: Workload, mat: int):
    d, D = wl.dims(mat)
    p = dict(wl.params)
    rec = wl.recipe
    if rec == "cfg1":
        # s_k = 10 * 0.7^k for k < 8, then 0.05 for the rest of min(m, n)
        k = np.arange(d)
        s = np.where(k < 8, 10.0 * 0.7 ** k, 0.05)
        return s, 0.01
    if rec == "decay":
        # planted rank `rank` with s_k = top * decay^k; optional division of
        # s_k for k >= split by `div` (a spectral gap at index split)
        rank = min(p["rank"], d)
        k = np.arange(rank)
        s = p.get("top", 10.0) * p["decay"] ** k
        if "split" in p:
            s = np.where(k >= p["split"], s / p["div"], s)
        return s, p["nu"]
    if rec == "powerlaw":
        # s_k = 1 / (k + 1) over planted rank `rank`; optional gap at `split`;
        # nu puts the worker-mean noise edge at s[-1] / 2
        rank = min(p["rank"], d)
        k = np.arange(rank)
        s = 1.0 / (k + 1.0)
        if "split" in p:
            s = np.where(k >= p["split"], s / p["div"], s)
        edge = s[-1] / 2.0
        nu = edge * np.sqrt(wl.workers) / (np.sqrt(d) + np.sqrt(D))
        return s, float(nu)
    if rec == "conv":
        # i.i.d. N(0, 1) gradients plus a planted part of rank len(weights),
        # s = weights * (sqrt(d) + sqrt(D))
        w = np.asarray(p["weights"], dtype=np.float64)
        w = w[: min(len(w), d)]
        return w * (np.sqrt(d) + np.sqrt(D)), 1.0
    if rec == "cfg5":
        # s_k = 10^(1 - k/255) for k < 256, 1/3 for 256 <= k < 512;
        # nu = 1 / (6 (sqrt(d) + sqrt(D)))
        rank = min(512, d)
        k = np.arange(rank)
        s = np.where(k < 256, 10.0 ** (1.0 - k / 255.0), 1.0 / 3.0)
        return s, 1.0 / (6.0 * (np.sqrt(d) + np.sqrt(D)))
    if rec == "geometric":
        # generic small-test recipe: s_k = top * decay^k over planted rank,
        # gap factor `div` at index `split` (defaults to the workload rank)
        rank = min(p.get("rank", d), d)
        k = np.arange(rank)
        s = p.get("top", 5.0) * p.get("decay", 0.85) ** k
        split = p.get("split", wl.rank)
        s = np.where(k >= split, s / p.get("div", 3.0), s)
        return s, p.get("nu", 1e-3)
    if rec == "lowrank":
        # exactly rank-`rank` gradients, no noise (exact-compression cases)
        rank = min(p["rank"], d)
        k = np.arange(rank)
        return 3.0 * 0.8 ** k, 0.0
    if rec == "zero":
        return np.zeros(0), 0.0
    raise ValueError(f"unknown recipe {rec!r}")


# ----------------------------------------------------------------------------
# generators
# ----------------------------------------------------------------------------

def _haar(rng: np.random.Generator, n: int, k: int) -> np.ndarray:
    """n x k with orthonormal columns: QR of a Gaussian, signs fixed."""
    if k == 0:
        return np.zeros((n, 0))
    a = rng.standard_normal((n, k))
    q, r = np.linalg.qr(a)
    sg = np.sign(np.diag(r))
    sg[sg == 0] = 1.0
    return q * sg


def planted_factors(wl: Workload, mat: int):
    """(U_s, s, V_s, nu) for matrix `mat`, float64; U_s is m x k, V_s is n x k."""
    m, n = wl.shapes[mat]
    s, nu = _spectrum(wl, mat)
    k = len(s)
    rng = np.random.default_rng([wl.seed, wl.wid, mat, _PLANTED_TAG])
    us = _haar(rng, m, k)
    vs = _haar(rng, n, k)
    return us, np.asarray(s, dtype=np.float64), vs, float(nu)


def noise_level(wl: Workload, mat: int) -> float:
    """nu, the standard deviation of the per-step Gaussian noise."""
    return float(_spectrum(wl, mat)[1])


def planted_matrix(wl: Workload, mat: int) -> np.ndarray:
    us, s, vs, _ = planted_factors(wl, mat)
    return (us * s) @ vs.T


def noise_rng(wl: Workload, mat: int, t: int) -> np.random.Generator:
    return np.random.default_rng([wl.seed, wl.wid, mat, int(t), _NOISE_TAG])


def gradient_batch(wl: Workload, mat: int, t: int, planted: np.ndarray | None = None) -> np.ndarray:
    """N x m x n float32 gradients of matrix `mat` at step t."""
    m, n = wl.shapes[mat]
    if planted is None:
        planted = planted_matrix(wl, mat)
    nu = _spectrum(wl, mat)[1]
    out = np.empty((wl.workers, m, n), dtype=np.float32)
    rng = noise_rng(wl, mat, t)
    for i in range(wl.workers):
        g = planted + nu * rng.standard_normal((m, n)) if nu != 0.0 else planted.copy()
        out[i] = g.astype(np.float32)
    return out


# ----------------------------------------------------------------------------
# the workloads
# ----------------------------------------------------------------------------

def _conv_shapes(seed: int, count: int):
    rng = np.random.default_rng([seed, _SHAPE_TAG])
    ds = rng.choice([64, 128, 256, 512], size=count)
    Ds = rng.choice([576, 1152, 2304], size=count)
    return tuple((int(a), int(b)) for a, b in zip(ds, Ds))


def _mk():
    w = {}

    def add(wl):
        w[wl.name] = wl

    # One matrix 256 x 128 (right-projected), N = 4, r = 4, tau = 5, T = 20
    add(Workload("one_256x128", ((256, 128),), 4, 4, 5, 20, "msgd", 0.01, 0.9,
                 recipe="cfg1"))
    # One layer 4096 x 4096, N = 8, r = 64, tau = 10, T = 50, MSGD
    add(Workload("layer_4096", ((4096, 4096),), 8, 64, 10, 50, "msgd", 0.01, 0.9,
                 recipe="decay", params=(("rank", 128), ("decay", 0.9), ("nu", 1e-3))))
    add(Workload("layer_4096_gap", ((4096, 4096),), 8, 64, 10, 50, "msgd", 0.01, 0.9,
                 recipe="decay",
                 params=(("rank", 128), ("decay", 0.9), ("nu", 5e-5), ("split", 64), ("div", 3.0))))
    # Transformer block: 4 x 4096^2 attention, 2 x 11008 x 4096 (gate/up),
    # 1 x 4096 x 11008 (down); N = 8, r = 128, Adam, tau = 10, T = 20
    blk = ((4096, 4096),) * 4 + ((11008, 4096), (11008, 4096), (4096, 11008))
    add(Workload("block_4096", blk, 8, 128, 10, 20, "adam", 1e-3, 0.9,
                 recipe="powerlaw", params=(("rank", 256),)))
    add(Workload("block_4096_gap", blk, 8, 128, 10, 20, "adam", 1e-3, 0.9,
                 recipe="powerlaw", params=(("rank", 256), ("split", 128), ("div", 3.0))))
    # 50 conv-shaped matrices, N = 16, r = 8, tau = 20, T = 100, MSGD
    add(Workload("conv_50", _conv_shapes(0, 50), 16, 8, 20, 100, "msgd", 0.01, 0.9,
                 recipe="conv", params=(("weights", (4.0, 3.5, 3.0, 2.5)),)))
    add(Workload("conv_50_gap", _conv_shapes(0, 50), 16, 8, 20, 100, "msgd", 0.01, 0.9,
                 recipe="conv", params=(("weights", tuple(np.linspace(4.0, 2.0, 8))),)))
    # One large matrix 8192 x 28672, N = 4, r = 256, tau = 1, T = 10, Adam
    add(Workload("large_8192x28672", ((8192, 28672),), 4, 256, 1, 10, "adam", 1e-3, 0.9,
                 recipe="cfg5"))

    # ---- the four-block tournament off the 4096 shape: 256 seats holding 194
    # blocks (62 padding seats, a ragged last block, right-oriented), and 64
    # seats with a ragged last block; gapped at r for the fp64 projector check
    add(Workload("seats256_right", ((3300, 3100),), 4, 48, 2, 3, "msgd", 0.01, 0.9,
                 recipe="decay",
                 params=(("rank", 96), ("decay", 0.95), ("nu", 5e-5), ("split", 48), ("div", 3.0))))
    add(Workload("seats64_left", ((1012, 1100),), 4, 32, 2, 3, "adam", 1e-3, 0.9,
                 recipe="decay",
                 params=(("rank", 64), ("decay", 0.95), ("nu", 5e-5), ("split", 32), ("div", 3.0))))

    # ---- the largest full-basis refresh: d = 8192 (the LDS sort limit), pairs
    # on 512 seats (511 rounds a sweep); gapped at r
    add(Workload("max_8192", ((8192, 8256),), 2, 32, 2, 3, "msgd", 0.01, 0.9,
                 recipe="decay",
                 params=(("rank", 64), ("decay", 0.95), ("nu", 5e-5), ("split", 32), ("div", 3.0))))

    # ---- the largest rank: r = 1024 of d = 1100 (four 256-row projection
    # tiles, the wide residual), gapped at r
    add(Workload("max_rank", ((1100, 1300),), 2, 1024, 2, 3, "msgd", 0.01, 0.9,
                 recipe="decay",
                 params=(("rank", 1100), ("decay", 0.998), ("nu", 5e-5), ("split", 1024), ("div", 3.0))))

    # ---- small parity cases: several tiles, ragged tails, both orientations
    add(Workload("tiny_left", ((40, 72),), 3, 5, 4, 10, "msgd", 0.05, 0.9,
                 recipe="geometric", params=(("rank", 12), ("nu", 1e-3))))
    add(Workload("ragged_right", ((200, 72),), 3, 6, 3, 8, "adam", 1e-3, 0.9,
                 recipe="geometric", params=(("rank", 16), ("nu", 5e-4))))
    add(Workload("mixed_small", ((96, 160), (170, 66), (33, 33), (1, 37), (5, 9)),
                 4, 4, 3, 7, "adam", 2e-3, 0.9,
                 recipe="geometric", params=(("rank", 8), ("nu", 1e-3))))
    add(Workload("single_worker", ((64, 96),), 1, 6, 3, 7, "adam", 1e-3, 0.9,
                 recipe="geometric", params=(("rank", 12), ("nu", 1e-3))))
    add(Workload("mid_left", ((256, 600),), 4, 16, 4, 9, "msgd", 0.01, 0.9,
                 recipe="geometric", params=(("rank", 40), ("nu", 2e-4))))
    add(Workload("lowrank_exact", ((48, 100), (90, 30)), 2, 6, 3, 6, "msgd", 0.01, 0.9,
                 recipe="lowrank", params=(("rank", 4),)))
    add(Workload("zero_grad", ((32, 64),), 2, 4, 2, 4, "adam", 1e-3, 0.9,
                 recipe="zero"))
    # ranks above 128: the wide-rank residual/optimizer pass, ragged tiles,
    # both orientations and both optimizers (and tau = 1 with such a rank)
    add(Workload("wide_left", ((300, 700),), 3, 150, 3, 6, "msgd", 0.01, 0.9,
                 recipe="geometric", params=(("rank", 200), ("decay", 0.985), ("nu", 1e-4))))
    add(Workload("wide_right", ((650, 290),), 2, 140, 2, 5, "adam", 1e-3, 0.9,
                 recipe="geometric", params=(("rank", 180), ("decay", 0.985), ("nu", 1e-4))))
    # 64 < r <= 128: the projection's two 64-row rank tiles in the XCD order
    # (ragged last column tile, a tile count that is not a multiple of 8)
    add(Workload("two_tiles_left", ((300, 900),), 3, 100, 3, 6, "msgd", 0.01, 0.9,
                 recipe="geometric", params=(("rank", 140), ("decay", 0.985), ("nu", 1e-4))))
    add(Workload("two_tiles_right", ((900, 300),), 3, 100, 3, 6, "msgd", 0.01, 0.9,
                 recipe="geometric", params=(("rank", 140), ("decay", 0.985), ("nu", 1e-4))))
    # (gap factor 10 at r: error feedback lifts the discarded directions by
    # about their own size per step, so the gap stays open over the 4 steps)
    # (MSGD: Adam's first step X = -lr sign-like(Ghat) turns the ~1e-8
    # rounding of the elements with |Ghat| near 1e-8 into O(lr) differences,
    # and 234 000 elements hold a few such)
    add(Workload("tau1_wide", ((260, 900),), 2, 136, 1, 4, "msgd", 0.01, 0.9,
                 recipe="geometric", params=(("rank", 180), ("decay", 0.985), ("nu", 1e-4), ("div", 10.0))))
    # tau = 1: every step a refresh, only the top-r block of U is used
    add(Workload("tau1_left", ((64, 300),), 3, 8, 1, 6, "adam", 1e-3, 0.9,
                 recipe="geometric", params=(("rank", 16), ("nu", 1e-3))))
    add(Workload("tau1_right", ((500, 96),), 2, 12, 1, 5, "msgd", 0.01, 0.9,
                 recipe="geometric", params=(("rank", 24), ("nu", 5e-4))))
    add(Workload("tau1_k40", ((200, 1000),), 2, 40, 1, 4, "adam", 1e-3, 0.9,
                 recipe="geometric", params=(("rank", 60), ("decay", 0.93), ("nu", 1e-4))))
    return w


WORKLOADS = _mk()


def get_workload(name: str, **override) -> Workload:
    wl = WORKLOADS[name]
    if override:
        d = dict(wl.__dict__)
        d.update(override)
        wl = Workload(**d)
    return wl
