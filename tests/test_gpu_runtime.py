"""GPU runtime contract through the C ABI: the device status word (non-finite
input under GLR_CHECK_FINITE), the step-order contract, resuming from a copy
of the state blob, and bitwise determinism of repeated runs."""
import numpy as np
import pytest

from synth import get_workload, gradient_batch, planted_matrix

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[runtime]", *a, flush=True)


def _inputs(wl, steps):
    import torch
    planted = [planted_matrix(wl, l) for l in range(len(wl.shapes))]
    return [[torch.from_numpy(gradient_batch(wl, l, t, planted[l])).cuda() for l in range(len(wl.shapes))]
            for t in range(steps)]


def _make(glr, wl, **kw):
    return glr.GreedyLore(wl.shapes, wl.workers, wl.rank, wl.tau, opt=wl.opt, lr=wl.lr, beta1=wl.beta1,
                          seed=wl.seed, **kw)


def _zeros(wl):
    import torch
    return [torch.zeros(m, n, device="cuda") for m, n in wl.shapes]


def _blob(comp):
    return comp.state[comp._s0: comp._s0 + comp.state_bytes]


@pytest.mark.parametrize("store", ["fp32", "bf16"])
def test_nonfinite_gradient_is_reported_and_state_marked_suspect(gpu_lib, store):
    import torch
    wl = get_workload("one_256x128")
    _say("one_256x128 check_finite", store)
    comp = _make(gpu_lib, wl, check_finite=True, store=store)
    X = _zeros(wl)
    G = _inputs(wl, 2)
    if store == "bf16":
        G = [[g.to(torch.bfloat16) for g in gt] for gt in G]
    comp.step(X, G[0], 0)
    assert comp.sync_status() == gpu_lib.GLR_OK
    bad = G[1][0].clone()
    bad[1, 3, 5] = float("nan")
    comp.step(X, [bad], 1)
    assert comp.sync_status() == 6          # GLR_ERR_NONFINITE
    with pytest.raises(gpu_lib.GlrError) as ei:
        comp.step(X, G[1], 2)
    assert ei.value.status == 4             # GLR_ERR_STATE until the caller resumes
    comp.resume(2)
    comp.step(X, G[1], 2)
    assert comp.sync_status() == gpu_lib.GLR_OK
    torch.cuda.synchronize()


def test_step_order_contract(gpu_lib):
    import torch
    wl = get_workload("one_256x128")
    _say("one_256x128 order")
    comp = _make(gpu_lib, wl)
    X = _zeros(wl)
    G = _inputs(wl, 3)
    with pytest.raises(gpu_lib.GlrError) as ei:
        comp.step(X, G[1], 1)               # must start at t = 0
    assert ei.value.status == 4
    comp.step(X, G[0], 0)
    torch.cuda.synchronize()
    x0 = X[0].clone()
    e0 = comp.E(0).clone()
    with pytest.raises(gpu_lib.GlrError):
        comp.step(X, G[2], 2)               # skips t = 1: rejected before any launch
    torch.cuda.synchronize()
    assert torch.equal(X[0], x0) and torch.equal(comp.E(0), e0)
    assert comp.next_step() == 1
    comp.step(X, G[1], 1)
    assert comp.sync_status() == gpu_lib.GLR_OK


@pytest.mark.parametrize("name", ["one_256x128", "tau1_left"])
def test_resume_from_a_copied_state_matches_the_uninterrupted_run(gpu_lib, name):
    import torch
    wl = get_workload(name)
    T = min(wl.steps, 7)
    cut = 3
    _say(name, "resume at", cut, "of", T)
    G = _inputs(wl, T)
    a = _make(gpu_lib, wl)
    Xa = _zeros(wl)
    for t in range(T):
        a.step(Xa, G[t], t)
    b = _make(gpu_lib, wl)
    Xb = _zeros(wl)
    for t in range(cut):
        b.step(Xb, G[t], t)
    torch.cuda.synchronize()
    c = _make(gpu_lib, wl)
    _blob(c).copy_(_blob(b))
    c.resume(cut)
    Xc = [x.clone() for x in Xb]
    del b
    for t in range(cut, T):
        c.step(Xc, G[t], t)
    torch.cuda.synchronize()
    assert a.sync_status() == gpu_lib.GLR_OK and c.sync_status() == gpu_lib.GLR_OK
    for l in range(len(wl.shapes)):
        assert torch.equal(Xa[l], Xc[l]), f"mat {l}: X differs after resume"
        assert torch.equal(a.E(l), c.E(l)), f"mat {l}: E differs after resume"


@pytest.mark.parametrize("name", ["mid_left", "tau1_right"])
def test_repeated_runs_are_bitwise_identical(gpu_lib, name):
    import torch
    wl = get_workload(name)
    T = min(wl.steps, wl.tau + 2)
    _say(name, "determinism over", T, "steps")
    G = _inputs(wl, T)
    runs = []
    for _ in range(2):
        comp = _make(gpu_lib, wl)
        X = _zeros(wl)
        for t in range(T):
            comp.step(X, G[t], t)
        torch.cuda.synchronize()
        runs.append((comp, X))
    (c1, x1), (c2, x2) = runs
    for l in range(len(wl.shapes)):
        assert torch.equal(x1[l], x2[l])
        assert torch.equal(c1.E(l), c2.E(l))
        assert torch.equal(c1.Ut(l), c2.Ut(l))
        assert torch.equal(c1.J(l), c2.J(l))


def test_concurrent_lanes_match_the_one_stream_order(gpu_lib, monkeypatch):
    # several matrices run on up to four streams at once; each matrix's result
    # must be bitwise that of running all of them in order on one stream
    import torch
    wl = get_workload("mixed_small")
    T = min(wl.steps, wl.tau + 2)
    _say("mixed_small lanes vs one stream over", T, "steps,", len(wl.shapes), "matrices")
    G = _inputs(wl, T)
    runs = []
    for lanes in ("1", None):
        if lanes is None:
            monkeypatch.delenv("GLR_LANES", raising=False)
        else:
            monkeypatch.setenv("GLR_LANES", lanes)
        comp = _make(gpu_lib, wl)
        X = _zeros(wl)
        for t in range(T):
            comp.step(X, G[t], t)
        assert comp.sync_status() == gpu_lib.GLR_OK
        runs.append((comp, X))
    (c1, x1), (c2, x2) = runs
    for l in range(len(wl.shapes)):
        assert torch.equal(x1[l], x2[l]), f"mat {l}: X differs"
        assert torch.equal(c1.E(l), c2.E(l)), f"mat {l}: E differs"
        assert torch.equal(c1.Ut(l), c2.Ut(l)), f"mat {l}: U differs"
        assert torch.equal(c1.J(l), c2.J(l)), f"mat {l}: J differs"


@pytest.mark.parametrize("name,override", [
    ("mixed_small", {}),
    # twelve of the conv layers, pairs of 16-row blocks, refreshed at t = 0 and 3
    ("conv_50", {"tau": 3}),
    # three matrices with d in [1009, 1024]: groups of four blocks, different sweep counts
    ("seats64_left", {"shapes": ((1012, 1100), (1100, 1020), (1016, 1030)), "tau": 2}),
])
def test_joint_refresh_matches_the_per_matrix_sweeps(gpu_lib, monkeypatch, name, override):
    # a refresh step of several matrices sweeps all of them in shared launches;
    # every matrix must end bitwise where its own sweeps take it
    import torch
    wl = get_workload(name, **override)
    if name == "conv_50":
        wl = get_workload(name, shapes=wl.shapes[:12], **override)
    T = min(wl.steps, wl.tau + 2)
    _say(name, "joint vs per-matrix refresh over", T, "steps,", len(wl.shapes), "matrices")
    G = _inputs(wl, T)
    runs = []
    for joint in ("0", None):
        if joint is None:
            monkeypatch.delenv("GLR_JAC_JOINT", raising=False)
        else:
            monkeypatch.setenv("GLR_JAC_JOINT", joint)
        comp = _make(gpu_lib, wl)
        X = _zeros(wl)
        for t in range(T):
            comp.step(X, G[t], t)
        assert comp.sync_status() == gpu_lib.GLR_OK
        runs.append((comp, X))
    (c1, x1), (c2, x2) = runs
    for l in range(len(wl.shapes)):
        assert torch.equal(x1[l], x2[l]), f"mat {l}: X differs"
        assert torch.equal(c1.E(l), c2.E(l)), f"mat {l}: E differs"
        assert torch.equal(c1.Ut(l), c2.Ut(l)), f"mat {l}: U differs"
        assert torch.equal(c1.sigma(l), c2.sigma(l)), f"mat {l}: sigma differs"
        assert torch.equal(c1.J(l), c2.J(l)), f"mat {l}: J differs"
        assert torch.equal(c1.info(l), c2.info(l)), f"mat {l}: sweep record differs"


_RIGHT_TRIO = {"shapes": ((1100, 1012), (1030, 1016), (700, 96)), "tau": 3, "steps": 6}
# ranks in the projection's middle tiers: 64 x 64 tiles with fp64 partial
# sums (32 < r <= 64) and one 128 x 64 rank tile over 1024-term slices
# (64 < r <= 128)
_RIGHT_TRIO_R48 = {"shapes": ((1100, 1012), (1030, 1016), (700, 300)), "tau": 3, "steps": 6, "rank": 48}
_RIGHT_TRIO_R100 = {"shapes": ((1100, 1012), (1030, 1016), (700, 300)), "tau": 3, "steps": 6, "rank": 100}


@pytest.mark.parametrize("name,override,select,store", [
    ("conv_50", {"tau": 3}, "approx", "fp32"),             # twelve conv layers, d < n, MSGD
    ("seats64_left", _RIGHT_TRIO, "approx", "fp32"),       # d = n < m, Adam
    ("seats64_left", _RIGHT_TRIO, "exact", "fp32"),
    ("seats64_left", _RIGHT_TRIO, "approx_bf16", "fp32"),
    ("conv_50", {"tau": 3}, "approx", "bf16"),             # bf16 gradients and error buffers
    ("seats64_left", _RIGHT_TRIO, "approx", "bf16"),
    ("seats64_left", _RIGHT_TRIO_R48, "approx", "fp32"),
    ("seats64_left", _RIGHT_TRIO_R100, "approx", "fp32"),
])
def test_grouped_selection_steps_match_the_per_matrix_launches(gpu_lib, monkeypatch, name, override, select,
                                                               store):
    # a selection step of several matrices launches each kernel once for all
    # of them; every matrix must end bitwise where its own launches take it
    import torch
    wl = get_workload(name, **override)
    if name == "conv_50":
        wl = get_workload(name, shapes=wl.shapes[:12], **override)
    T = min(wl.steps, wl.tau + 3)
    _say(name, select, store, "grouped vs per-matrix selection over", T, "steps,", len(wl.shapes), "matrices")
    G = _inputs(wl, T)
    if store == "bf16":
        G = [[g.to(torch.bfloat16) for g in gt] for gt in G]
    runs = []
    for grouped in ("0", None):
        if grouped is None:
            monkeypatch.delenv("GLR_GROUPED", raising=False)
        else:
            monkeypatch.setenv("GLR_GROUPED", grouped)
        comp = _make(gpu_lib, wl, select=select, store=store)
        X = _zeros(wl)
        for t in range(T):
            comp.step(X, G[t], t)
        assert comp.sync_status() == gpu_lib.GLR_OK
        runs.append((comp, X))
    (c1, x1), (c2, x2) = runs
    for l in range(len(wl.shapes)):
        assert torch.equal(x1[l], x2[l]), f"mat {l}: X differs"
        assert torch.equal(c1.E(l), c2.E(l)), f"mat {l}: E differs"
        assert torch.equal(c1.Ut(l), c2.Ut(l)), f"mat {l}: U differs"
        assert torch.equal(c1.J(l), c2.J(l)), f"mat {l}: J differs"


@pytest.mark.parametrize("store", ["fp32", "bf16"])
def test_state_read_and_write_through_the_abi_resume_the_run(gpu_lib, store):
    # glr_read_state into host tensors after 3 steps of one handle, then
    # glr_write_state of those tensors into a fresh handle (a restore), which
    # continues bitwise like the uninterrupted run (E in the storage type)
    import torch
    wl = get_workload("ragged_right")
    T, cut = 6, 3
    _say("ragged_right read/write state at", cut, store)
    G = _inputs(wl, T)
    edt = torch.bfloat16 if store == "bf16" else torch.float32
    if store == "bf16":
        G = [[g.to(torch.bfloat16) for g in gt] for gt in G]
    a = gpu_lib.GreedyLore(wl.shapes, wl.workers, wl.rank, wl.tau, opt=wl.opt, lr=wl.lr, beta1=wl.beta1,
                           seed=wl.seed, store=store)
    Xa = _zeros(wl)
    for t in range(T):
        a.step(Xa, G[t], t)
    b = gpu_lib.GreedyLore(wl.shapes, wl.workers, wl.rank, wl.tau, opt=wl.opt, lr=wl.lr, beta1=wl.beta1,
                           seed=wl.seed, store=store)
    Xb = _zeros(wl)
    for t in range(cut):
        b.step(Xb, G[t], t)
    L = b.layouts[0]
    m, n, d, D, r, N = L.m, L.n, L.d, L.D, L.r, wl.workers
    host = {"E": torch.empty(N, m, n, dtype=edt), "Ebar": torch.empty(m, n), "Ut": torch.empty(d, d),
            "sigma": torch.empty(d), "J": torch.empty(r, dtype=torch.int32), "score": torch.empty(d),
            "S1": torch.empty(m, n), "S2": torch.empty(m, n), "Rbar": torch.empty(r, D),
            "info": torch.empty(64, dtype=torch.int32)}
    b.read_state(0, **host)
    torch.cuda.synchronize()
    assert torch.equal(host["E"], b.E(0).cpu()) and torch.equal(host["Ut"], b.Ut(0).cpu())
    assert torch.equal(host["S2"], b.S2(0).cpu()) and torch.equal(host["J"], b.J(0).cpu())
    c = gpu_lib.GreedyLore(wl.shapes, wl.workers, wl.rank, wl.tau, opt=wl.opt, lr=wl.lr, beta1=wl.beta1,
                           seed=wl.seed, store=store)
    c.write_state(0, **host)
    c.resume(cut)
    Xc = [x.clone() for x in Xb]
    for t in range(cut, T):
        c.step(Xc, G[t], t)
    torch.cuda.synchronize()
    assert a.sync_status() == gpu_lib.GLR_OK and c.sync_status() == gpu_lib.GLR_OK
    assert torch.equal(Xa[0], Xc[0]) and torch.equal(a.E(0), c.E(0)) and torch.equal(a.S2(0), c.S2(0))


def test_state_copy_rejects_s2_without_adam(gpu_lib):
    import torch
    wl = get_workload("one_256x128")
    comp = _make(gpu_lib, wl)
    with pytest.raises(gpu_lib.GlrError) as ei:
        comp.read_state(0, S2=torch.empty(256, 128))
    assert ei.value.status == 1
    with pytest.raises(gpu_lib.GlrError):
        comp.read_state(3, E=torch.empty(4, 256, 128))


def test_refresh_step_only_enqueues(gpu_lib):
    # a refresh of a 4096 x 4096 layer takes ~0.1 s on the device; glr_step
    # returns before it completes (no host wait per sweep), and the result is
    # there once the stream is
    import torch
    wl = get_workload("layer_4096", workers=2)
    _say("layer_4096 N=2 enqueue-only refresh")
    comp = gpu_lib.GreedyLore(wl.shapes, wl.workers, wl.rank, wl.tau, opt=wl.opt, lr=wl.lr, seed=wl.seed)
    X = _zeros(wl)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)
    planted = torch.from_numpy(planted_matrix(wl, 0).astype(np.float32)).cuda()
    G = [torch.randn((2, 4096, 4096), generator=gen, device="cuda").mul_(1e-3).add_(planted)]
    torch.cuda.synchronize()
    ev = torch.cuda.Event()
    comp.step(X, G, 0)
    ev.record()
    pending = not ev.query()
    torch.cuda.synchronize()
    assert pending, "glr_step waited for the refresh to complete"
    its, conv, _ = comp.sweep_history(0)
    assert conv and its > 1
    assert comp.sync_status() == gpu_lib.GLR_OK


@pytest.mark.parametrize("name,tau,store", [("zero_grad", 2, "fp32"), ("zero_grad", 1, "fp32"),
                                            ("lowrank_exact", 3, "fp32"), ("lowrank_exact", 1, "fp32"),
                                            ("zero_grad", 2, "bf16"), ("zero_grad", 1, "bf16")])
def test_zero_and_rank_deficient_gradients(gpu_lib, name, tau, store):
    # all-zero gradients, and exactly rank-4 gradients with r = 6 (< the
    # oversampled tau = 1 block): the full-basis and the tau = 1 refresh both
    # stay finite and orthonormal, and compress exactly (E = 0), as the
    # oracle does; X and the optimizer state follow the oracle
    import torch
    from oracle.method import Oracle
    from tests.parity import rel
    # (bf16 storage with zero gradients only: a rank-4 matrix rounded to bf16
    # is full rank at the 2^-9 level)
    wl = get_workload(name, tau=tau)
    _say(name, "tau", tau, store)
    comp = gpu_lib.GreedyLore(wl.shapes, wl.workers, wl.rank, wl.tau, opt=wl.opt, lr=wl.lr, beta1=wl.beta1,
                              seed=wl.seed, store=store)
    orc = Oracle.from_workload(wl, store=store)
    gdt = torch.bfloat16 if store == "bf16" else torch.float32
    planted = [planted_matrix(wl, l) for l in range(len(wl.shapes))]
    X = _zeros(wl)
    for t in range(wl.steps):
        grads = [gradient_batch(wl, l, t, planted[l]) for l in range(len(wl.shapes))]
        comp.step(X, [torch.from_numpy(g).cuda().to(gdt) for g in grads], t)
        torch.cuda.synchronize()
        st = comp.sync_status()
        assert st == gpu_lib.GLR_OK, f"t={t}: status {gpu_lib.STATUS_NAMES.get(st, st)}"
        res = orc.step(grads, t)
        for l, o in enumerate(res):
            m, n = wl.shapes[l]
            d = min(m, n)
            rows = min(wl.rank, d) if tau == 1 and wl.rank < d else d
            ut = comp.Ut(l)[:rows].double()
            assert torch.isfinite(ut).all() and torch.isfinite(X[l]).all()
            orth = float((ut @ ut.T - torch.eye(rows, dtype=torch.float64, device="cuda")).abs().max())
            assert orth < 1e-5, (t, l, orth)
            scale = max(float(np.abs(grads[l]).max()), 1e-30)
            assert float(comp.E(l).abs().max()) <= 1e-5 * scale, (t, l)
            # the oracle compresses the fp32 gradients, which are rank 4 only
            # up to their rounding (2^-24 relative)
            assert np.abs(o["E"]).max() <= 1e-6 * scale
            if np.any(o["X"]):
                assert rel(X[l].double().cpu().numpy(), o["X"]) < 1e-4
            else:
                assert not bool(X[l].any())
