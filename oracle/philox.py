"""Philox4x32-10 and Box-Muller normals for the random vectors of Approx-Top-r.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

The paper draws v_j ~ N(0, I_n) for j in [m] with a seed shared by all nodes
(Section V-C, eq:random-v) and fixes nothing else.  Both this oracle and the
GPU path implement the same counter-based generator from its published
definition, Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw,
"Parallel random numbers: as easy as 1, 2, 3", SC'11):

  * one round maps counter (x0, x1, x2, x3) under key (k0, k1) to
        (hi(B*x2) ^ x1 ^ k0,  lo(B*x2),  hi(A*x0) ^ x3 ^ k1,  lo(A*x0))
    with the 32-bit multipliers A = 0xD2511F53, B = 0xCD9E8D57;
  * the key is advanced by the Weyl increments (0x9E3779B9, 0xBB67AE85)
    between rounds.

Stream layout (this build's reading of the paper's "synchronised seed"):
  key     = (seed mod 2^32, seed >> 32)
  counter = (c, j, l, t mod 2^32) with c = b // 4 for element b of v_j,
            l = matrix index, t = step.
  The four output words (x0, x1, x2, x3) give v_j[4c], v_j[4c+1] by
  Box-Muller on (x0, x1) and v_j[4c+2], v_j[4c+3] on (x2, x3).
  Uniform map: u(x) = (x >> 9) * 2^-23 + 2^-24, which lies in (0, 1) and is
  exact in fp32.
  Box-Muller (Box & Muller 1958): rho = sqrt(-2 ln u_a),
  z0 = rho cos(2 pi u_b), z1 = rho sin(2 pi u_b).
The oracle evaluates Box-Muller in fp64 and rounds to fp32.

Pins: known-answer vectors of the published generator and distribution tests
(tests/test_oracle_rng.py).
"""
from __future__ import annotations

import numpy as np

MUL_A = np.uint64(0xD2511F53)
MUL_B = np.uint64(0xCD9E8D57)
WEYL_0 = 0x9E3779B9
WEYL_1 = 0xBB67AE85
MASK32 = np.uint64(0xFFFFFFFF)


def philox4x32_10(ctr, key):
    """Philox4x32-10 over arrays.

    ctr: uint32 array of shape (..., 4); key: (k0, k1) python ints or uint32
    arrays broadcastable to ctr[..., 0].  Returns uint32 array (..., 4).
    """
    c = np.asarray(ctr, dtype=np.uint64)
    x0, x1, x2, x3 = (c[..., i].copy() for i in range(4))
    k0 = np.asarray(key[0], dtype=np.uint64) & MASK32
    k1 = np.asarray(key[1], dtype=np.uint64) & MASK32
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + np.uint64(WEYL_0)) & MASK32
            k1 = (k1 + np.uint64(WEYL_1)) & MASK32
        pa = MUL_A * x0          # < 2^64: fits uint64 exactly
        pb = MUL_B * x2
        hi_a, lo_a = pa >> np.uint64(32), pa & MASK32
        hi_b, lo_b = pb >> np.uint64(32), pb & MASK32
        x0, x1, x2, x3 = (hi_b ^ x1 ^ k0) & MASK32, lo_b, (hi_a ^ x3 ^ k1) & MASK32, lo_a
    return np.stack([x0, x1, x2, x3], axis=-1).astype(np.uint32)


def uniform01(x):
    """u(x) = (x >> 9) * 2^-23 + 2^-24 (exact in fp32 and fp64)."""
    x = np.asarray(x, dtype=np.uint32)
    return (x >> np.uint32(9)).astype(np.float64) * 2.0 ** -23 + 2.0 ** -24


def box_muller(xa, xb):
    """Two N(0,1) values from two 32-bit words, fp64 evaluation."""
    ua = uniform01(xa)
    ub = uniform01(xb)
    rho = np.sqrt(-2.0 * np.log(ua))
    ang = 2.0 * np.pi * ub
    return rho * np.cos(ang), rho * np.sin(ang)


def seed_key(seed: int):
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return seed & 0xFFFFFFFF, seed >> 32


def gaussian_vectors(seed: int, t: int, mat: int, rows, length: int) -> np.ndarray:
    """v_j in R^length for each j in `rows`, as float32 (len(rows) x length).

    Element b of v_j comes from counter (b // 4, j, mat, t mod 2^32).
    """
    rows = np.asarray(rows, dtype=np.uint64)
    nblk = (length + 3) // 4
    cc = np.arange(nblk, dtype=np.uint64)
    ctr = np.empty((len(rows), nblk, 4), dtype=np.uint64)
    ctr[..., 0] = cc[None, :]
    ctr[..., 1] = rows[:, None]
    ctr[..., 2] = np.uint64(mat)
    ctr[..., 3] = np.uint64(int(t) & 0xFFFFFFFF)
    x = philox4x32_10(ctr, seed_key(seed))
    z0, z1 = box_muller(x[..., 0], x[..., 1])
    z2, z3 = box_muller(x[..., 2], x[..., 3])
    v = np.stack([z0, z1, z2, z3], axis=-1).reshape(len(rows), nblk * 4)
    return v[:, :length].astype(np.float32)
