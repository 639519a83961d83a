"""glr_create_static (the workspace in the library's static device scratch
array, for callers that cannot allocate) against glr_create with a caller
workspace: the same steps on the same inputs give the same E, X and optimizer
state, over two handles in a row on one device, the second with a smaller
input; a second live handle on the device and a workspace beyond the array
are refused."""
import ctypes

import numpy as np
import pytest

from synth import get_workload, gradient_batch, planted_matrix
from tests.parity import STEP_TOL, rel

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[no-alloc]", *a, flush=True)


def _static_run(glr, wl, grads):
    """The steps through glr_create_static; returns (E, X, S1) per matrix and
    the handle's status after every step."""
    import torch
    lib = glr.load()
    cfg, _keep = glr.make_config(wl.shapes, wl.workers, wl.rank, wl.tau, opt=wl.opt, lr=wl.lr,
                                 beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps, seed=wl.seed)
    sb, wb = glr.workspace_bytes(cfg)
    assert wb <= glr.STATIC_SCRATCH_BYTES
    state = torch.empty(sb + 256, dtype=torch.uint8, device="cuda")
    s0 = (-state.data_ptr()) % 256
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    h = ctypes.c_void_p()
    st = lib.glr_create_static(ctypes.byref(cfg), ctypes.c_void_p(state.data_ptr() + s0), sb, stream,
                               ctypes.byref(h))
    assert st == 0, lib.glr_last_error(None).decode()
    try:
        # a second handle on the same device would share the array: refused
        h2 = ctypes.c_void_p()
        assert lib.glr_create_static(ctypes.byref(cfg), ctypes.c_void_p(state.data_ptr() + s0), sb, stream,
                                     ctypes.byref(h2)) == 4
        X = [torch.zeros(m, n, device="cuda") for m, n in wl.shapes]
        n = len(wl.shapes)
        for t, G in enumerate(grads):
            xs = (ctypes.c_void_p * n)(*[x.data_ptr() for x in X])
            gs = (ctypes.c_void_p * n)(*[g.data_ptr() for g in G])
            assert lib.glr_step(h, xs, gs, t, stream) == 0, lib.glr_last_error(h).decode()
            assert lib.glr_sync_status(h, stream) == 0, lib.glr_last_error(h).decode()
        torch.cuda.synchronize()
        out = []
        for l in range(n):
            L = glr.state_layout(cfg, l)
            blob = state[s0:s0 + sb]
            e = blob[L.off_E:L.off_E + wl.workers * L.m * L.n * 4].view(torch.float32)
            s1 = blob[L.off_S1:L.off_S1 + L.m * L.n * 4].view(torch.float32)
            out.append((e.double().cpu().numpy(), X[l].double().cpu().numpy(), s1.double().cpu().numpy()))
        return out
    finally:
        assert lib.glr_destroy(h) == 0


def _caller_run(glr, wl, grads):
    import torch
    comp = glr.GreedyLore(wl.shapes, wl.workers, wl.rank, wl.tau, opt=wl.opt, lr=wl.lr, beta1=wl.beta1,
                          beta2=wl.beta2, eps=wl.eps, seed=wl.seed)
    X = [torch.zeros(m, n, device="cuda") for m, n in wl.shapes]
    for t, G in enumerate(grads):
        comp.step(X, G, t)
        assert comp.sync_status() == 0
    torch.cuda.synchronize()
    return [(comp.E(l).double().flatten().cpu().numpy(), X[l].double().cpu().numpy(),
             comp.S1(l).double().flatten().cpu().numpy()) for l in range(len(wl.shapes))]


def _grads(wl, steps):
    import torch
    planted = [planted_matrix(wl, l) for l in range(len(wl.shapes))]
    return [[torch.from_numpy(gradient_batch(wl, l, t, planted[l])).cuda() for l in range(len(wl.shapes))]
            for t in range(steps)]


def test_static_scratch_matches_the_caller_workspace_twice_in_a_row(gpu_lib):
    # mid_left (256 x 600) then tiny_left (40 x 72): the second handle reuses
    # the array the first one left behind
    for name in ("mid_left", "tiny_left"):
        wl = get_workload(name)
        steps = min(wl.steps, 2 * wl.tau + 1)
        _say(name, "steps", steps)
        grads = _grads(wl, steps)
        a = _static_run(gpu_lib, wl, grads)
        b = _caller_run(gpu_lib, wl, grads)
        for l, ((ea, xa, sa), (eb, xb, sb)) in enumerate(zip(a, b)):
            errs = (rel(ea, eb), rel(xa, xb), rel(sa, sb))
            same = np.array_equal(ea, eb) and np.array_equal(xa, xb) and np.array_equal(sa, sb)
            _say(name, "mat", l, "rel E, X, S1", errs, "bitwise" if same else "")
            assert max(errs) < STEP_TOL


def test_static_scratch_with_several_matrices(gpu_lib):
    # five matrices (the joint refresh of several matrices) in the array
    wl = get_workload("mixed_small")
    _say("mixed_small")
    grads = _grads(wl, wl.steps)
    a = _static_run(gpu_lib, wl, grads)
    b = _caller_run(gpu_lib, wl, grads)
    for (ea, xa, sa), (eb, xb, sb) in zip(a, b):
        assert max(rel(ea, eb), rel(xa, xb), rel(sa, sb)) < STEP_TOL


def test_static_scratch_refuses_a_workspace_beyond_the_array(gpu_lib):
    lib = gpu_lib.load()
    cfg, _keep = gpu_lib.make_config([(4096, 4096)], 8, 64, 10)
    assert gpu_lib.workspace_bytes(cfg)[1] > gpu_lib.STATIC_SCRATCH_BYTES
    h = ctypes.c_void_p()
    assert lib.glr_create_static(ctypes.byref(cfg), ctypes.c_void_p(0x100000), 1 << 30, None,
                                 ctypes.byref(h)) == 3
    assert "static scratch" in lib.glr_last_error(None).decode()
