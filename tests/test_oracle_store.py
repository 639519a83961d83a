"""Pins for the oracle's bf16 storage mode (store="bf16": G^(i) and E^(i)
held in bfloat16; the paper fixes no precision, so the mode is a reading of
its own): the stored buffers are bf16 bit patterns, each residual is rounded
once with the bf16 unit roundoff as its error bound, the next step is formed
from the stored buffers, the gradient rounding agrees with torch's own
float-to-bfloat16 conversion, Proposition 3 survives the rounding within its
bound, and the column-restricted step follows the full one in the mode."""
import numpy as np
import pytest
import torch

from oracle.method import ColumnOracle, Oracle, compress
from synth import get_workload, gradient_batch, planted_matrix

U_BF16 = 2.0 ** -8          # unit roundoff of an 8-significant-bit format


def _torch_bf16(a):
    """bf16 values of `a` by torch's conversion (round to nearest even), as fp64."""
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16).to(
        torch.float64).numpy()


def _grads(wl, t, planted):
    return [gradient_batch(wl, l, t, planted[l]) for l in range(len(wl.shapes))]


@pytest.mark.parametrize("name", ["tiny_left", "ragged_right", "mixed_small"])
def test_stored_buffers_are_bf16_bit_patterns(name):
    wl = get_workload(name)
    orc = Oracle.from_workload(wl, store="bf16")
    planted = [planted_matrix(wl, l) for l in range(len(wl.shapes))]
    for t in range(wl.steps):
        for o in orc.step(_grads(wl, t, planted), t):
            e = o["E"]
            e32 = e.astype(np.float32)
            assert np.array_equal(e32.astype(np.float64), e)          # exact in binary32
            assert not np.any(e32.view(np.uint32) & 0xFFFF)            # and its lower half is zero


@pytest.mark.parametrize("name", ["tiny_left", "ragged_right"])
def test_each_residual_is_rounded_once(name):
    # fed the same bf16 gradients, the fp32 and bf16 modes agree up to the
    # first residual; the stored residual is then within the bf16 unit
    # roundoff of the fp32 mode's (plus the binary32 step in between), and
    # the rounding is not a no-op
    wl = get_workload(name)
    planted = [planted_matrix(wl, l) for l in range(len(wl.shapes))]
    g = [_torch_bf16(x) for x in _grads(wl, 0, planted)]
    o32 = Oracle.from_workload(wl).step(g, 0)
    o16 = Oracle.from_workload(wl, store="bf16").step(g, 0)
    for a, b in zip(o32, o16):
        assert np.array_equal(a["P"], b["P"])
        e, f = a["E"], b["E"]
        assert np.all(np.abs(f - e) <= (U_BF16 + 2.0 ** -23) * np.abs(e))
        assert np.count_nonzero(f != e) > 0.9 * e.size
        # Q, Rbar, Ghat and X are formed before the rounding: unchanged
        for k in ("Q", "Rbar", "ghat", "X"):
            assert np.array_equal(a[k], b[k]), k


def test_next_step_reads_the_stored_buffers():
    # Mbar at step t + 1 is the mean of the rounded gradients plus the stored
    # (rounded) error buffers of step t
    wl = get_workload("ragged_right")
    orc = Oracle.from_workload(wl, store="bf16")
    planted = [planted_matrix(wl, 0)]
    prev = None
    for t in range(5):
        g = _grads(wl, t, planted)
        o = orc.step(g, t)[0]
        if prev is not None:
            gb = np.swapaxes(_torch_bf16(g[0]), 1, 2)                  # 200 x 72: oriented
            want = (gb + prev).mean(axis=0)
            assert np.allclose(o["mbar"], want, rtol=0, atol=1e-15 * np.abs(want).max())
        prev = o["E"]


def test_gradient_rounding_matches_torch():
    # the oracle rounds what it is given; torch-rounded input gives the same
    # trajectory bit for bit (so the two roundings agree on every element)
    wl = get_workload("tiny_left")
    planted = [planted_matrix(wl, 0)]
    a = Oracle.from_workload(wl, store="bf16")
    b = Oracle.from_workload(wl, store="bf16")
    for t in range(wl.steps):
        g = _grads(wl, t, planted)
        oa = a.step(g, t)[0]
        ob = b.step([_torch_bf16(g[0])], t)[0]
        for k in ("E", "X", "s1", "J", "mbar"):
            assert np.array_equal(oa[k], ob[k]), (t, k)


@pytest.mark.parametrize("opt", ["msgd", "adam"])
def test_prop3_with_rounded_buffers(opt):
    # one worker, exact top-r selection: Proposition 3 bounds the residual of
    # the compressed matrix, ||M - P P^T M||^2 <= (1 - r/d) ||M||^2; the stored
    # buffer adds at most the unit roundoff per element
    wl = get_workload("tiny_left", workers=1, opt=opt)
    orc = Oracle.from_workload(wl, store="bf16", select="exact")
    planted = [planted_matrix(wl, 0)]
    d, r = 40, wl.rank
    for t in range(wl.steps):
        o = orc.step(_grads(wl, t, planted), t)[0]
        m = o["mbar"]                                                 # N = 1: Mbar = M
        assert np.sum((m - compress(o["P"], m)) ** 2) <= (1 - r / d) * np.sum(m ** 2) * (1 + 1e-12)
        assert np.sum(o["E"] ** 2) <= (1 - r / d) * np.sum(m ** 2) * (1 + U_BF16) ** 2


@pytest.mark.parametrize("name", ["mid_left", "ragged_right"])
def test_column_oracle_follows_the_full_oracle_in_bf16(name):
    wl = get_workload(name, steps=6)
    full = Oracle.from_workload(wl, store="bf16")
    m, n = wl.shapes[0]
    D = max(m, n)
    cols = np.array([0, 5, D // 2, D - 1])
    col = ColumnOracle(wl.shapes[0], cols, wl.workers, opt=wl.opt, lr=wl.lr, beta1=wl.beta1,
                       beta2=wl.beta2, eps=wl.eps, store="bf16")
    planted = planted_matrix(wl, 0)
    for t in range(wl.steps):
        g = gradient_batch(wl, 0, t, planted)
        o = full.step([g], t)[0]
        go = np.swapaxes(g, 1, 2) if m > n else g
        c = col.step(go[:, :, cols], o["P"], o["refresh"])
        # the stored residuals are rounded from values that agree to ~1e-16:
        # equal except where a value sits on a rounding boundary
        e, f = c["E"], o["E"][:, :, cols]
        assert np.count_nonzero(e != f) <= 2
        assert np.all(np.abs(e - f) <= 2.0 ** -7 * np.abs(f) + 1e-300)
        tr = (lambda a: a.T) if m > n else (lambda a: a)
        assert np.linalg.norm(c["X"] - tr(o["X"])[:, cols]) <= 1e-6 * np.linalg.norm(o["X"][:, :])
