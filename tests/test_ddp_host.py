"""Host-side checks of the DDP communication hook: which parameters it
compresses and under which matrix view, and its refusals (CPU parameters,
process groups of more than one rank), on the CPU with gloo."""
import os
import socket

import pytest
import torch

from paper_2507_08784_amd.ddp import GreedyLoreHook, compressible, matrix_shape


def test_matrix_views_follow_the_reshaping_of_convolution_kernels():
    assert matrix_shape(torch.empty(8, 3, 3, 3)) == (8, 27)
    assert matrix_shape(torch.empty(64, 512)) == (64, 512)
    assert matrix_shape(torch.empty(5)) is None
    assert matrix_shape(torch.empty(0, 4)) == (0, 0)


def test_only_matrices_wider_than_the_rank_are_compressed():
    assert compressible(torch.empty(10, 96), 4)
    assert not compressible(torch.empty(4, 96), 4)      # min side = rank: exact anyway
    assert not compressible(torch.empty(96), 4)
    assert compressible(torch.empty(8, 3, 3, 3), 4)
    assert not compressible(torch.empty(8, 1, 2, 2), 4)  # 8 x 4


def test_cpu_parameters_are_refused():
    lin = torch.nn.Linear(32, 16)
    with pytest.raises(ValueError, match="GPU only"):
        GreedyLoreHook(lin.parameters(), rank=4, tau=2)


def test_parameters_it_does_not_compress_need_no_gpu():
    # vectors and thin matrices stay with the caller's optimizer
    ps = [torch.nn.Parameter(torch.zeros(16)), torch.nn.Parameter(torch.zeros(3, 40))]
    hook = GreedyLoreHook(ps, rank=4, tau=2)
    assert hook.other_parameters() == ps and hook.compressed_parameters() == []


def _two_ranks(rank, port, q):
    import torch.distributed as dist
    os.environ["MASTER_ADDR"] = "127.0.0.1"
    os.environ["MASTER_PORT"] = str(port)
    dist.init_process_group("gloo", rank=rank, world_size=2)
    try:
        GreedyLoreHook([torch.nn.Parameter(torch.zeros(16, 32))], rank=4, tau=2)
        q.put((rank, "accepted"))
    except NotImplementedError as e:
        q.put((rank, "refused" if "2 ranks" in str(e) else str(e)))
    finally:
        dist.destroy_process_group()


def test_a_group_of_two_ranks_is_refused():
    import torch.multiprocessing as mp
    with socket.socket() as s:
        s.bind(("127.0.0.1", 0))
        port = s.getsockname()[1]
    ctx = mp.get_context("spawn")
    q = ctx.Queue()
    procs = [ctx.Process(target=_two_ranks, args=(r, port, q)) for r in range(2)]
    for p in procs:
        p.start()
    for p in procs:
        p.join(120)
    out = sorted(q.get(timeout=5) for _ in range(2))
    assert out == [(0, "refused"), (1, "refused")]
