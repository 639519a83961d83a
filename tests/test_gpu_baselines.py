"""GPU parity of the paper's baseline modes against the oracle's same modes:
the Lazy-SVD operator and Algorithm 1 (Section IV), Proposition 1 on the
device, Appendix C's trajectory exactly in fp32, and the distributed
Adam-type GaLore of Algorithm 5 (Appendix E)."""
import numpy as np
import pytest

from synth import get_workload
from tests.parity import rel, run_parity

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[baselines]", *a, flush=True)


@pytest.mark.parametrize("name", ["tiny_left", "ragged_right"])
def test_algorithm1_lazy_svd_parity(gpu_lib, name):
    # Lazy-SVD projection, no error feedback, Ghat = the mean gradient at
    # refresh steps: Algorithm 1 step by step against the oracle
    _say(name, "algorithm 1")

    def check(comp, o, t, l, rec):
        assert float(comp.E(l).abs().max()) == 0.0 and float(comp.Ebar(l).abs().max()) == 0.0
        assert np.array_equal(np.sort(comp.J(l).cpu().numpy()), np.arange(min(get_workload(name).rank, 40)))

    run_parity(gpu_lib, get_workload(name), select="lazy", refresh="full", ef=False, check=check)


def test_lazy_svd_with_error_feedback_parity(gpu_lib):
    _say("mid_left lazy + EF")
    run_parity(gpu_lib, get_workload("mid_left"), select="lazy")


@pytest.mark.parametrize("name", ["tiny_left", "ragged_right", "mixed_small"])
def test_galore_adam_parity(gpu_lib, name):
    # Algorithm 5: subspace Adam moments (reset at every refresh), X -= lr P Rhat
    _say(name, "galore adam")
    run_parity(gpu_lib, get_workload(name, opt="galore_adam"))


def test_prop1_lazy_svd_nullifies_error_feedback_on_the_device(gpu_lib):
    # with P kept between refreshes the runs with and without error feedback
    # take the same steps (C(G + E) = C(G)), while E differs
    import torch
    from synth import gradient_batch, planted_matrix
    wl = get_workload("mid_left", tau=5)
    _say("mid_left prop 1")
    a = gpu_lib.GreedyLore(wl.shapes, wl.workers, wl.rank, wl.tau, opt=wl.opt, lr=wl.lr, select="lazy")
    b = gpu_lib.GreedyLore(wl.shapes, wl.workers, wl.rank, wl.tau, opt=wl.opt, lr=wl.lr, select="lazy", ef=False)
    Xa = [torch.zeros(*wl.shapes[0], device="cuda")]
    Xb = [torch.zeros(*wl.shapes[0], device="cuda")]
    planted = planted_matrix(wl, 0)
    for t in range(5):
        G = [torch.from_numpy(gradient_batch(wl, 0, t, planted)).cuda()]
        a.step(Xa, G, t)
        b.step(Xb, G, t)
        torch.cuda.synchronize()
        assert a.sync_status() == 0 and b.sync_status() == 0
        r = rel(Xa[0].double().cpu().numpy(), Xb[0].double().cpu().numpy())
        assert r < 1e-5, (t, r)
        if t > 0:
            assert float(a.E(0).abs().max()) > 0 and float(b.E(0).abs().max()) == 0


@pytest.mark.parametrize("ef", [True, False])
def test_appendix_c_trajectory_exact_in_fp32(gpu_lib, ef):
    # f(diag(x, y)) = L x^2 / 2 + L y^2 / 4 from diag(1, 1); the refresh at
    # t = 0 picks P = e1 and keeps it (Lazy-SVD); plain gradient descent
    # (MSGD with beta 0), gamma = 1 / (2L): x_k = 2^-k and y_k = 1 exactly,
    # down to the smallest normal fp32 value, and no NaN after it
    import torch
    L = 4.0
    comp = gpu_lib.GreedyLore([(2, 2)], 1, 1, 10 ** 6, opt="msgd", lr=1.0 / (2 * L), beta1=0.0,
                              select="lazy", ef=ef)
    X = [torch.eye(2, device="cuda")]
    for k in range(1, 131):
        x = X[0].cpu()
        G = torch.diag(torch.tensor([L * float(x[0, 0]), L / 2 * float(x[1, 1])], dtype=torch.float32))
        comp.step(X, [G[None].contiguous().cuda()], k - 1)
        torch.cuda.synchronize()
        xk = X[0].cpu()
        assert torch.isfinite(xk).all()
        if k <= 126:
            assert float(xk[0, 0]) == 2.0 ** -k, (k, float(xk[0, 0]))
        assert float(xk[1, 1]) == 1.0 and float(xk[0, 1]) == 0.0 and float(xk[1, 0]) == 0.0
    assert comp.sync_status() == 0
