"""PyTorch DistributedDataParallel communication hook driving the GreedyLore
step (the paper deploys GreedyLore as a DDP communication hook: Section I,
contributions; Section VII, experimental setup).

When DDP hands the hook a bucket of ready gradients, every compressed
parameter in it (two or more dimensions, viewed as m x n with
m = shape[0], n = the product of the rest, as the paper reshapes
convolution kernels, and min(m, n) > rank) runs one GreedyLore step in the
library: error feedback, the semi-lazy subspace, projection, residual and
the optimizer update of the parameter itself (Algorithm 4 with the MSGD or
Adam rule of Section III).  Its slot in the bucket is then zeroed, so DDP
writes a zero gradient back; the remaining parameters keep their gradients
for the caller's own optimizer (`other_parameters()`).

The work runs on a side stream of default priority that first waits for
everything queued before the hook, so the compression of one bucket
overlaps the backward pass of the earlier layers; the returned future
carries that stream, and DDP's wait orders the next use of the parameters
after it.

One process, one worker: the library averages workers that share one GPU,
and a process group of more than one rank would need the all-reduces of the
projections instead, which this library does not issue, so such a group is
refused.  Each compressed parameter has a handle of its own (one matrix,
its own seed), so DDP's rebuilding of buckets after the first iteration
changes nothing in the per-parameter trajectories.
"""
from __future__ import annotations

from . import GreedyLore, STATUS_NAMES, GlrError


def matrix_shape(p):
    """(m, n) under which a parameter of two or more dimensions is
    compressed: m = shape[0], n = the product of the other dimensions."""
    if p.dim() < 2:
        return None
    m = int(p.shape[0])
    return m, (int(p.numel()) // m if m else 0)


def compressible(p, rank):
    """Whether the hook compresses p: a matrix view exists and its smaller
    side exceeds the rank (at or below it the compression would be exact)."""
    s = matrix_shape(p)
    return s is not None and min(s) > rank


class _Param:
    """One compressed parameter: its handle, the matrix view of its data and
    the next step index."""

    def __init__(self, torch, p, shape, seed, stream, kw):
        m, n = shape
        self.p = p
        self.shape = shape
        self.X = p.data.view(m, n)
        self.comp = GreedyLore([shape], 1, device=p.device, seed=seed, stream=stream, **kw)
        self.stage = None
        self.t = 0
        self.torch = torch

    def step(self, g):
        m, n = self.shape
        g = g.view(1, m, n)
        if g.data_ptr() % 256:
            # a bucket slot starts wherever the previous parameter ended: the
            # library takes 256-byte aligned buffers, so stage the gradient
            if self.stage is None:
                self.stage = self.torch.empty(1, m, n, dtype=self.torch.float32, device=g.device)
            self.stage.copy_(g)
            g = self.stage
        self.comp.step([self.X], [g], self.t)
        self.t += 1


class GreedyLoreHook:
    """GreedyLore as a DDP communication hook.

        hook = GreedyLoreHook(model.parameters(), rank=4, tau=10, opt="adam", lr=1e-3)
        ddp = DistributedDataParallel(model, device_ids=[0])
        hook.register(ddp)
        opt = torch.optim.AdamW(hook.other_parameters(), lr=1e-3)

    The compressed parameters are updated by the hook during backward; the
    caller's optimizer steps the others.  Keyword arguments after `rank` and
    `tau` are those of `GreedyLore` (opt, lr, beta1, beta2, eps, refresh,
    select, max_sweeps, tol, check_finite, cold_start, ef); parameter i (in
    the order given) uses seed `seed + i`."""

    def __init__(self, parameters, rank, tau, seed=0, process_group=None, **kw):
        import torch
        import torch.distributed as dist

        self.torch = torch
        world = dist.get_world_size(process_group) if dist.is_initialized() else 1
        if world != 1:
            raise NotImplementedError(
                f"GreedyLoreHook averages the workers of one process on its GPU; a process group of "
                f"{world} ranks would need the all-reduces of the projections, which this library does not issue")
        self.rank, self.tau, self.kw = int(rank), int(tau), dict(kw)
        self.params = list(parameters)
        self._plan = {}      # data_ptr -> (index, p, (m, n))
        self.others = []
        for i, p in enumerate(self.params):
            if not compressible(p, self.rank):
                self.others.append(p)
                continue
            if not p.is_cuda:
                raise ValueError(f"parameter {i}: GreedyLore runs on the GPU only (got {p.device})")
            if p.dtype != torch.float32 or not p.is_contiguous():
                raise ValueError(f"parameter {i}: compressed parameters must be contiguous float32")
            if p.data_ptr() % 256:
                raise ValueError(f"parameter {i}: its storage must be 256-byte aligned")
            self._plan[p.data_ptr()] = (i, p, matrix_shape(p))
        self.seed = int(seed)
        self._live = {}      # data_ptr -> _Param, created at the first bucket holding it
        self.stream = None
        self.device = None
        if self._plan:
            self.device = next(iter(self._plan.values()))[1].device
            self.stream = torch.cuda.Stream(device=self.device)

    # ------------------------------------------------------------------ API
    def other_parameters(self):
        """The parameters the hook does not compress (for the caller's optimizer)."""
        return list(self.others)

    def compressed_parameters(self):
        return [p for (_, p, _) in self._plan.values()]

    def register(self, ddp):
        """Registers the hook on a DistributedDataParallel module (DDP takes a
        plain function: `greedylore_hook` with this object as its state)."""
        ddp.register_comm_hook(self, greedylore_hook)
        return self

    def compressor(self, p):
        """(GreedyLore handle, matrix index 0) of a compressed parameter, once
        its first step has run; None before."""
        ent = self._live.get(p.data_ptr())
        return None if ent is None else ent.comp

    def steps_done(self, p):
        ent = self._live.get(p.data_ptr())
        return 0 if ent is None else ent.t

    def check_status(self):
        """Waits for the hook's work and raises GlrError on the first handle
        whose device status is not GLR_OK (non-finite gradient, breakdown,
        non-convergence)."""
        for ent in self._live.values():
            st = ent.comp.sync_status()
            if st != 0:
                i = self._plan[ent.p.data_ptr()][0]
                raise GlrError(st, f"parameter {i}: {STATUS_NAMES.get(st, st)}")

    # ----------------------------------------------------------------- hook
    def _entry(self, p):
        key = p.data_ptr()
        ent = self._live.get(key)
        if ent is None:
            i, param, shape = self._plan[key]
            ent = _Param(self.torch, param, shape, self.seed + i, self.stream, dict(rank=self.rank, tau=self.tau, **self.kw))
            self._live[key] = ent
        return ent

    def run_bucket(self, bucket):
        """One bucket: the compressed parameters' steps on the side stream;
        returns the future DDP waits on."""
        torch = self.torch
        buf = bucket.buffer()
        todo = [(p, g) for p, g in zip(bucket.parameters(), bucket.gradients()) if p.data_ptr() in self._plan]
        if not todo:
            fut = torch.futures.Future(devices=[buf.device])
            fut.set_result(buf)
            return fut
        side = self.stream
        side.wait_stream(torch.cuda.current_stream(self.device))
        buf.record_stream(side)
        with torch.cuda.stream(side):
            for p, g in todo:
                self._entry(p).step(g)
                g.zero_()
            fut = torch.futures.Future(devices=[self.device])
            fut.set_result(buf)
        return fut


def greedylore_hook(state, bucket):
    """The DDP communication hook function; `state` is a GreedyLoreHook."""
    return state.run_bucket(bucket)
