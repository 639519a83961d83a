"""The DDP communication hook on the GPU: a small convolution + MLP model
trained under DistributedDataParallel (one rank, RCCL) with GreedyLoreHook;
every compressed parameter's trajectory is replayed by the oracle on the
gradients the hook received (one worker, the parameter's own seed), with the
hand-off of tests/parity.py, at the per-step and end-of-run bars."""
import socket
from datetime import timedelta

import numpy as np
import pytest

from oracle.method import Oracle, oriented_to_mn
from synth.gen import Workload
from tests.parity import FINAL_TOL, STEP_TOL, Handoff, rel, summarize

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[ddp]", *a, flush=True)


def _free_port():
    with socket.socket() as s:
        s.bind(("127.0.0.1", 0))
        return s.getsockname()[1]


@pytest.fixture(scope="module")
def process_group(gpu_lib):
    import torch.distributed as dist
    dist.init_process_group("nccl", init_method=f"tcp://127.0.0.1:{_free_port()}", rank=0,
                            world_size=1, timeout=timedelta(seconds=60))
    yield dist
    dist.destroy_process_group()


def _model(torch):
    nn = torch.nn
    F = torch.nn.functional

    class Net(nn.Module):
        def __init__(self):
            super().__init__()
            self.conv = nn.Conv2d(3, 8, 3, padding=1)   # 8 x 27
            self.fc1 = nn.Linear(512, 64)               # 64 x 512 (left)
            self.fc2 = nn.Linear(64, 96)                # 96 x 64 (right)
            self.fc3 = nn.Linear(96, 10)                # 10 x 96

        def forward(self, x):
            x = F.relu(self.conv(x)).flatten(1)
            return self.fc3(F.relu(self.fc2(F.relu(self.fc1(x)))))

    return Net()


@pytest.mark.parametrize("opt,lr", [("msgd", 0.05), ("adam", 1e-3)])
def test_ddp_hook_trajectories_match_the_oracle(gpu_lib, process_group, opt, lr):
    import torch
    from torch.nn.parallel import DistributedDataParallel as DDP
    from paper_2507_08784_amd.ddp import GreedyLoreHook, matrix_shape

    _say(opt)
    rank, tau, steps, seed = 4, 3, 7, 5
    torch.manual_seed(0)
    model = _model(torch).cuda()
    params = list(model.parameters())
    hook = GreedyLoreHook(params, rank=rank, tau=tau, seed=seed, opt=opt, lr=lr, beta1=0.9)
    ddp = DDP(model, device_ids=[0], bucket_cap_mb=0.05)
    hook.register(ddp)
    sgd = torch.optim.SGD(hook.other_parameters(), lr=0.05)
    comp_params = hook.compressed_parameters()
    assert [tuple(p.shape) for p in comp_params] == [(8, 3, 3, 3), (64, 512), (96, 64), (10, 96)]
    index = {p.data_ptr(): i for i, p in enumerate(params)}

    seen = {}
    handles = [p.register_hook(lambda g, k=k: seen.__setitem__(k, g.detach().to("cpu", copy=True)))
               for k, p in enumerate(comp_params)]
    oracles, wls = [], []
    for p in comp_params:
        m, n = matrix_shape(p)
        orc = Oracle(shapes=((m, n),), workers=1, rank=rank, tau=tau, opt=opt, lr=lr, beta1=0.9,
                     seed=seed + index[p.data_ptr()])
        orc.states[0].x = p.detach().double().cpu().numpy().reshape(m, n).copy()
        oracles.append(orc)
        wls.append(Workload(name="ddp", shapes=((m, n),), workers=1, rank=rank, tau=tau, steps=steps,
                            opt=opt, lr=lr, beta1=0.9, seed=seed + index[p.data_ptr()]))
    gen = torch.Generator().manual_seed(1)
    log = []
    for t in range(steps):
        x = torch.randn(16, 3, 8, 8, generator=gen).cuda()
        y = torch.randint(0, 10, (16,), generator=gen).cuda()
        sgd.zero_grad(set_to_none=True)
        loss = torch.nn.functional.cross_entropy(ddp(x), y)
        loss.backward()
        sgd.step()
        torch.cuda.synchronize()
        hook.check_status()
        for k, p in enumerate(comp_params):
            m, n = matrix_shape(p)
            assert hook.steps_done(p) == t + 1
            assert float(p.grad.abs().max()) == 0.0     # the hook took the gradient
            comp = hook.compressor(p)
            g = seen[k].double().numpy().reshape(1, m, n)
            rec = {"t": t, "mat": k}
            o = oracles[k].step([g], t, handoff=Handoff(comp, wls[k], [rec]))[0]
            rec["X"] = rel(p.detach().double().cpu().numpy().reshape(m, n), o["X"])
            mi = np.abs(g).max() + np.abs(o["E"]).max()
            e_o = oriented_to_mn(o["E"], m, n)
            rec["E"] = rel(comp.E(0).double().cpu().numpy(), e_o, floor=1e-3 * mi * np.sqrt(e_o.size))
            rec["S1"] = rel(comp.S1(0).double().cpu().numpy(), o["s1"])
            if o["s2"] is not None:
                rec["S2"] = rel(comp.S2(0).double().cpu().numpy(), o["s2"])
            for key in ("X", "E", "S1", "S2"):
                if key in rec:
                    assert rec[key] < STEP_TOL, f"t={t} param {k}: {key} rel {rec[key]:.3e} ({rec})"
            log.append(rec)
    for h in handles:
        h.remove()
    for k, p in enumerate(comp_params):
        m, n = matrix_shape(p)
        final = rel(p.detach().double().cpu().numpy().reshape(m, n), oracles[k].states[0].x)
        log.append({"final_X": final, "mat": k})
        assert final < FINAL_TOL
    summarize(f"ddp_{opt}", log)


def test_ddp_hook_leaves_the_other_parameters_to_the_optimizer(gpu_lib, process_group):
    # the biases keep DDP's (one-rank) gradient, the one a plain backward
    # gives, while the compressed weights are moved by the hook and left with
    # a zero gradient
    import torch
    from torch.nn.parallel import DistributedDataParallel as DDP
    from paper_2507_08784_amd.ddp import GreedyLoreHook

    _say("other parameters")
    torch.manual_seed(0)
    ref = _model(torch).cuda()
    model = _model(torch).cuda()
    model.load_state_dict(ref.state_dict())
    hook = GreedyLoreHook(model.parameters(), rank=4, tau=3, opt="msgd", lr=0.05)
    ddp = DDP(model, device_ids=[0], bucket_cap_mb=0.05)
    hook.register(ddp)
    assert len(hook.other_parameters()) == 4
    x = torch.randn(16, 3, 8, 8, device="cuda")
    y = torch.randint(0, 10, (16,), device="cuda")
    torch.nn.functional.cross_entropy(ddp(x), y).backward()
    torch.nn.functional.cross_entropy(ref(x), y).backward()
    torch.cuda.synchronize()
    hook.check_status()
    for (name, p), (_, q) in zip(model.named_parameters(), ref.named_parameters()):
        if name.endswith("bias"):
            # the same products (the convolution's reductions may differ in order)
            assert torch.allclose(p.grad, q.grad, rtol=1e-5, atol=1e-7), name
        else:
            assert float(p.grad.abs().max()) == 0.0, name
            assert not torch.equal(p.detach(), q.detach()), name
