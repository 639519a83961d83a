"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every symbol include/greedylore.h declares, validates configurations and
computes a consistent, aligned state layout."""
import ctypes
import os
import re

import pytest

import paper_2507_08784_amd as glr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "greedylore.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(glr_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = glr.load()
    names = _declared()
    assert set(names) == set(glr.EXPORTED)
    for name in names:
        assert hasattr(lib, name), name


def _cfg(**kw):
    args = dict(shapes=[(256, 128)], workers=4, rank=4, tau=5)
    args.update(kw)
    return glr.make_config(**args)


def _status(cfg):
    return glr.load().glr_validate_config(ctypes.byref(cfg))


def test_valid_config():
    cfg, _keep = _cfg()
    assert _status(cfg) == glr.GLR_OK


@pytest.mark.parametrize("kw,code", [
    (dict(workers=0), 1), (dict(rank=0), 1), (dict(tau=0), 1), (dict(opt=7), 1),
    (dict(lr=0.0), 1), (dict(lr=float("nan")), 1), (dict(beta1=1.0), 1), (dict(beta1=-0.1), 1),
    (dict(opt="adam", beta2=1.0), 1), (dict(opt="adam", eps=0.0), 1), (dict(refresh=5), 1),
    (dict(select=4), 1), (dict(opt="galore_adam", refresh="full"), 1), (dict(max_sweeps=0), 1), (dict(tol=0.0), 1), (dict(tol=1.0), 1),
    (dict(flags=0x80), 1), (dict(opt="galore_adam", flags=glr.STORE_BF16), 1),
    (dict(shapes=[(0, 5)]), 2), (dict(shapes=[(5, -1)]), 2),
    (dict(shapes=[(9000, 9000)]), 2), (dict(shapes=[(2000, 3000)], rank=2000), 2),
    (dict(shapes=[(8192, 1 << 17)]), 2),   # m n = 2^30: beyond 32-bit byte offsets
])
def test_invalid_configs_are_rejected(kw, code):
    cfg, _keep = _cfg(**kw)
    assert _status(cfg) == code
    assert glr.load().glr_last_error(None).decode()


def test_null_config_and_outputs():
    lib = glr.load()
    assert lib.glr_validate_config(None) == 1
    cfg, _keep = _cfg()
    assert lib.glr_workspace_bytes(ctypes.byref(cfg), None, None) == 1
    assert lib.glr_state_layout(ctypes.byref(cfg), 0, None) == 1
    out = glr.MatLayout()
    assert lib.glr_state_layout(ctypes.byref(cfg), 3, ctypes.byref(out)) == 1


def test_create_rejects_bad_buffers_without_touching_the_device():
    lib = glr.load()
    cfg, _keep = _cfg()
    h = ctypes.c_void_p()
    sb, wb = glr.workspace_bytes(cfg)
    # NULL buffers, misaligned buffers and undersized buffers fail before any HIP call
    assert lib.glr_create(ctypes.byref(cfg), None, sb, None, wb, None, ctypes.byref(h)) == 1
    assert lib.glr_create(ctypes.byref(cfg), ctypes.c_void_p(0x1000 + 4), sb, ctypes.c_void_p(0x2000),
                          wb, None, ctypes.byref(h)) == 1
    assert lib.glr_create(ctypes.byref(cfg), ctypes.c_void_p(0x1000), sb - 4, ctypes.c_void_p(0x2000),
                          wb, None, ctypes.byref(h)) == 3
    assert h.value is None


def test_step_and_status_reject_null_handle():
    lib = glr.load()
    assert lib.glr_step(None, None, None, 0, None) == 1
    assert lib.glr_step_bf16(None, None, None, 0, None) == 1
    assert lib.glr_sync_status(None, None) == 1
    assert lib.glr_resume(None, 0) == 1
    assert lib.glr_destroy(None) == 0
    assert lib.glr_status_string(4) == b"invalid state"


@pytest.mark.parametrize("opt,store", [("msgd", "fp32"), ("adam", "fp32"), ("adam", "bf16")])
def test_layout_is_aligned_disjoint_and_sized(opt, store):
    shapes = [(96, 160), (170, 66), (1, 37), (4096, 11008)]
    esz = 2 if store == "bf16" else 4
    cfg, _keep = glr.make_config(shapes, workers=3, rank=8, tau=4, opt=opt,
                                 flags=glr.STORE_BF16 if store == "bf16" else 0)
    sb, wb = glr.workspace_bytes(cfg)
    spans = [(0, 256)]
    for i, (m, n) in enumerate(shapes):
        L = glr.state_layout(cfg, i)
        d, D = min(m, n), max(m, n)
        assert (L.m, L.n, L.d, L.D, L.right, L.r) == (m, n, d, D, int(m > n), min(8, d))
        parts = [(L.off_E, 3 * m * n * esz), (L.off_Ebar, m * n * 4), (L.off_U, d * d * 4),
                 (L.off_sigma, d * 4), (L.off_J, L.r * 4), (L.off_score, d * 4),
                 (L.off_S1, m * n * 4), (L.off_Rbar, L.r * D * 4), (L.off_info, 256)]
        if opt == "adam":
            parts.append((L.off_S2, m * n * 4))
        else:
            assert L.off_S2 == 0
        for off, size in parts:
            assert off % 256 == 0
            spans.append((off, off + size))
    spans.sort()
    for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
        assert a1 <= b0
    assert spans[-1][1] <= sb
    assert wb > 0


def test_workspace_holds_a_region_per_matrix():
    # matrices running at the same time (concurrent streams, the joint sweeps
    # of a refresh, the grouped launches of a selection step) never share
    # scratch: the workspace of several matrices holds each one's own region
    shapes = [(512, 576), (256, 2304), (1012, 1100), (130, 70)]
    cfg, _keep = glr.make_config(shapes, 4, 8, 5)
    _, total = glr.workspace_bytes(cfg)
    alone = []
    for s in shapes:
        c1, _k1 = glr.make_config([s], 4, 8, 5)
        alone.append(glr.workspace_bytes(c1)[1])
    # each configuration also carries a few KiB of per-matrix launch tables
    slack = 4096
    assert total >= sum(alone) - slack * len(shapes)
    # one region per matrix, sized by that matrix: not a copy of the largest
    # matrix's region per stream
    assert total <= sum(alone)
    # and a matrix's region does not depend on the others
    c2, _k2 = glr.make_config(shapes + [(4096, 4096)], 4, 8, 5)
    c3, _k3 = glr.make_config([(4096, 4096)], 4, 8, 5)
    assert glr.workspace_bytes(c2)[1] >= total + glr.workspace_bytes(c3)[1] - slack


def test_state_copies_reject_bad_arguments_without_touching_the_device():
    lib = glr.load()
    view = glr.StateView()
    assert lib.glr_read_state(None, 0, ctypes.byref(view), None) == 1
    assert lib.glr_write_state(None, 0, ctypes.byref(view), None) == 1
    assert lib.glr_status_string(8) == b"orthonormalisation breakdown"
    assert glr.STATUS_NAMES[8] == "GLR_ERR_BREAKDOWN"
    assert [f[0] for f in glr.StateView._fields_] == list(glr.STATE_PARTS)
