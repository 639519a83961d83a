"""GreedyLore compression step on MI355X (gfx950): Python binding of the
C-ABI library libgreedylore.so (include/greedylore.h).

This module only marshals arguments: every step of the method runs in the
library's HIP kernels.  PyTorch provides device memory and the stream.  There
is no CPU fallback: if the library was not built, load() raises.

    import paper_2507_08784_amd as glr
    comp = glr.GreedyLore(shapes=[(4096, 4096)], workers=8, rank=64, tau=10)
    comp.step([X], [G], t)          # G: N x m x n fp32 on cuda, X: m x n fp32

With store="bf16" the gradients and error buffers are bfloat16 (G passed as
torch.bfloat16 tensors; X stays fp32).

`paper_2507_08784_amd.ddp.GreedyLoreHook` drives the same step from a
DistributedDataParallel communication hook.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgreedylore.so")

GLR_OK = 0
STATUS_NAMES = {
    0: "GLR_OK", 1: "GLR_ERR_INVALID_ARG", 2: "GLR_ERR_SHAPE", 3: "GLR_ERR_BUFFER_TOO_SMALL",
    4: "GLR_ERR_STATE", 5: "GLR_ERR_DEVICE", 6: "GLR_ERR_NONFINITE", 7: "GLR_ERR_NOT_CONVERGED",
    8: "GLR_ERR_BREAKDOWN",
}
CHECK_FINITE = 0x1
COLD_START = 0x2
NO_EF = 0x4
STORE_BF16 = 0x8
EXPORTED = (
    "glr_validate_config", "glr_workspace_bytes", "glr_state_layout", "glr_create", "glr_step",
    "glr_sync_status", "glr_resume", "glr_next_step", "glr_destroy", "glr_status_string",
    "glr_last_error", "glr_profile_enable", "glr_profile_reset", "glr_profile_query",
    "glr_read_state", "glr_write_state", "glr_create_static", "glr_step_bf16",
)
STATIC_SCRATCH_BYTES = 64 << 20
STATE_PARTS = ("E", "Ebar", "Ut", "sigma", "J", "score", "S1", "S2", "Rbar", "info")
PROF_GROUPS = ("ef_mean", "select", "topr", "proj", "rbar", "resid_opt", "full_refresh",
               "jac_init", "jac_update", "jac_finish", "refresh", "sub_iter", "jac_solve",
               "rr_update", "rr_solve", "sub_z", "sub_p", "sub_orth", "sub_chol")


class GlrError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class Shape(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int64), ("n", ctypes.c_int64)]


class Config(ctypes.Structure):
    _fields_ = [
        ("num_mats", ctypes.c_int32), ("shapes", ctypes.POINTER(Shape)),
        ("num_workers", ctypes.c_int32), ("rank", ctypes.c_int32), ("tau", ctypes.c_int32),
        ("opt", ctypes.c_int32), ("lr", ctypes.c_float), ("beta1", ctypes.c_float),
        ("beta2", ctypes.c_float), ("eps", ctypes.c_float), ("refresh", ctypes.c_int32),
        ("select", ctypes.c_int32), ("seed", ctypes.c_uint64), ("max_sweeps", ctypes.c_int32),
        ("tol", ctypes.c_float), ("flags", ctypes.c_uint32),
    ]


class MatLayout(ctypes.Structure):
    _fields_ = [
        ("m", ctypes.c_int64), ("n", ctypes.c_int64), ("d", ctypes.c_int64), ("D", ctypes.c_int64),
        ("right", ctypes.c_int32), ("r", ctypes.c_int32),
        ("off_E", ctypes.c_uint64), ("off_Ebar", ctypes.c_uint64), ("off_U", ctypes.c_uint64),
        ("off_sigma", ctypes.c_uint64), ("off_J", ctypes.c_uint64), ("off_score", ctypes.c_uint64),
        ("off_S1", ctypes.c_uint64), ("off_S2", ctypes.c_uint64), ("off_Rbar", ctypes.c_uint64),
        ("off_info", ctypes.c_uint64),
    ]


class StateView(ctypes.Structure):
    _fields_ = [(name, ctypes.c_void_p) for name in STATE_PARTS]


_lib = None


def load():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2507_08784_amd.build` "
            "(the GreedyLore path has no CPU fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
    sig = {
        "glr_validate_config": (I32, [P(Config)]),
        "glr_workspace_bytes": (I32, [P(Config), P(ctypes.c_size_t), P(ctypes.c_size_t)]),
        "glr_state_layout": (I32, [P(Config), I32, P(MatLayout)]),
        "glr_create": (I32, [P(Config), VP, ctypes.c_size_t, VP, ctypes.c_size_t, VP, P(VP)]),
        "glr_step": (I32, [VP, P(VP), P(VP), I64, VP]),
        "glr_step_bf16": (I32, [VP, P(VP), P(VP), I64, VP]),
        "glr_sync_status": (I32, [VP, VP]),
        "glr_resume": (I32, [VP, I64]),
        "glr_next_step": (I32, [VP, P(I64)]),
        "glr_destroy": (I32, [VP]),
        "glr_status_string": (ctypes.c_char_p, [I32]),
        "glr_last_error": (ctypes.c_char_p, [VP]),
        "glr_profile_enable": (I32, [VP, I32]),
        "glr_profile_reset": (I32, [VP]),
        "glr_profile_query": (I32, [VP, I32, P(ctypes.c_double), P(I64)]),
        "glr_read_state": (I32, [VP, I32, P(StateView), VP]),
        "glr_create_static": (I32, [P(Config), VP, ctypes.c_size_t, VP, P(VP)]),
        "glr_write_state": (I32, [VP, I32, P(StateView), VP]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def make_config(shapes, workers, rank, tau, opt="msgd", lr=0.01, beta1=0.9, beta2=0.999,
                eps=1e-8, refresh="compressed", select="approx", seed=0, max_sweeps=30,
                tol=1e-6, flags=0):
    """(Config, keep-alive shape array) for the C ABI."""
    arr = (Shape * len(shapes))(*[Shape(int(m), int(n)) for m, n in shapes])
    cfg = Config(
        num_mats=len(shapes), shapes=ctypes.cast(arr, ctypes.POINTER(Shape)), num_workers=workers,
        rank=rank, tau=tau, opt={"msgd": 0, "adam": 1, "galore_adam": 2}[opt] if isinstance(opt, str) else opt,
        lr=lr, beta1=beta1, beta2=beta2, eps=eps,
        refresh={"compressed": 0, "full": 1}[refresh] if isinstance(refresh, str) else refresh,
        select={"approx": 0, "exact": 1, "approx_bf16": 2, "lazy": 3}[select] if isinstance(select, str) else select,
        seed=seed, max_sweeps=max_sweeps, tol=tol, flags=flags)
    return cfg, arr


def _check(status, handle=None):
    if status != GLR_OK:
        lib = load()
        msg = lib.glr_last_error(handle).decode()
        raise GlrError(status, msg)


def workspace_bytes(cfg):
    lib = load()
    s, w = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib.glr_workspace_bytes(ctypes.byref(cfg), ctypes.byref(s), ctypes.byref(w)))
    return s.value, w.value


def state_layout(cfg, mat):
    lib = load()
    out = MatLayout()
    _check(lib.glr_state_layout(ctypes.byref(cfg), mat, ctypes.byref(out)))
    return out


class GreedyLore:
    """One GreedyLore compressor over a set of layer matrices, N simulated
    workers on the current GPU.  Owns (as torch tensors) the state blob and
    the workspace the C library works in."""

    def __init__(self, shapes, workers, rank, tau, opt="msgd", lr=0.01, beta1=0.9, beta2=0.999,
                 eps=1e-8, refresh="compressed", select="approx", seed=0, max_sweeps=30,
                 tol=1e-6, check_finite=False, cold_start=False, ef=True, store="fp32", device="cuda",
                 stream=None):
        import torch
        self.lib = load()
        self.torch = torch
        self.shapes = [tuple(int(x) for x in s) for s in shapes]
        self.workers = workers
        self.opt = opt
        if store not in ("fp32", "bf16"):
            raise ValueError(f"store must be 'fp32' or 'bf16', not {store!r}")
        self.store = store
        self.gdtype = torch.bfloat16 if store == "bf16" else torch.float32
        flags = ((CHECK_FINITE if check_finite else 0) | (COLD_START if cold_start else 0) | (0 if ef else NO_EF)
                 | (STORE_BF16 if store == "bf16" else 0))
        self.cfg, self._shape_arr = make_config(self.shapes, workers, rank, tau, opt, lr, beta1,
                                                beta2, eps, refresh, select, seed, max_sweeps,
                                                tol, flags)
        sb, wb = workspace_bytes(self.cfg)
        self.device = torch.device(device)
        if self.device.index is None:
            self.device = torch.device(self.device.type, torch.cuda.current_device())
        self.state = torch.empty(sb + 256, dtype=torch.uint8, device=self.device)
        self.work = torch.empty(wb + 256, dtype=torch.uint8, device=self.device)
        self._s0 = (-self.state.data_ptr()) % 256
        self._w0 = (-self.work.data_ptr()) % 256
        self.state_bytes, self.ws_bytes = sb, wb
        self.layouts = [state_layout(self.cfg, i) for i in range(len(self.shapes))]
        self.stream = stream
        h = ctypes.c_void_p()
        _check(self.lib.glr_create(ctypes.byref(self.cfg), self.state.data_ptr() + self._s0, sb,
                                   self.work.data_ptr() + self._w0, wb, self._stream_ptr(),
                                   ctypes.byref(h)))
        self.handle = h

    def _stream_ptr(self):
        s = self.stream if self.stream is not None else self.torch.cuda.current_stream(self.device)
        return ctypes.c_void_p(s.cuda_stream)

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and h.value:
            self.lib.glr_destroy(h)
            self.handle = None

    # ------------------------------------------------------------------ calls
    def step(self, X, G, t):
        """One step t on every matrix: X[l] (m x n, fp32) is updated in place,
        G[l] holds the N worker gradients (N x m x n) on this GPU, fp32 (bf16
        with store="bf16")."""
        n = len(self.shapes)
        xs = (ctypes.c_void_p * n)(*[x.data_ptr() for x in X])
        gs = (ctypes.c_void_p * n)(*[g.data_ptr() for g in G])
        for l, ((m, nn), x, g) in enumerate(zip(self.shapes, X, G)):
            if x.dtype != self.torch.float32 or g.dtype != self.gdtype:
                raise TypeError(f"matrix {l}: X must be float32 and G {self.gdtype}")
            if tuple(x.shape) != (m, nn) or tuple(g.shape) != (self.workers, m, nn):
                raise ValueError(f"matrix {l}: X must be {m}x{nn}, G {self.workers}x{m}x{nn}")
            if not (x.is_contiguous() and g.is_contiguous()):
                raise ValueError(f"matrix {l}: X and G must be contiguous")
            if x.device != self.device or g.device != self.device:
                raise ValueError(f"matrix {l}: X and G must live on {self.device}")
        fn = self.lib.glr_step_bf16 if self.store == "bf16" else self.lib.glr_step
        _check(fn(self.handle, xs, gs, int(t), self._stream_ptr()), self.handle)

    def sync_status(self):
        return self.lib.glr_sync_status(self.handle, self._stream_ptr())

    def check_status(self):
        _check(self.sync_status(), self.handle)

    def resume(self, next_t):
        _check(self.lib.glr_resume(self.handle, int(next_t)), self.handle)

    def _state_view(self, parts):
        bad = set(parts) - set(STATE_PARTS)
        if bad:
            raise ValueError(f"unknown state parts {sorted(bad)}")
        return StateView(**{k: ctypes.c_void_p(int(v.data_ptr()) if hasattr(v, "data_ptr") else int(v))
                            for k, v in parts.items()})

    def read_state(self, mat, **parts):
        """Enqueues stream-ordered copies of matrix `mat`'s state parts into
        the given tensors (host or device, contiguous, of the part's size):
        read_state(0, E=t1, Ut=t2)."""
        for k, v in parts.items():
            if not v.is_contiguous():
                raise ValueError(f"{k}: destination must be contiguous")
        view = self._state_view(parts)
        _check(self.lib.glr_read_state(self.handle, int(mat), ctypes.byref(view), self._stream_ptr()),
               self.handle)

    def write_state(self, mat, **parts):
        """Enqueues copies of the given tensors into matrix `mat`'s state and
        marks the state valid (a hand-off or a restore)."""
        for k, v in parts.items():
            if not v.is_contiguous():
                raise ValueError(f"{k}: source must be contiguous")
        view = self._state_view(parts)
        _check(self.lib.glr_write_state(self.handle, int(mat), ctypes.byref(view), self._stream_ptr()),
               self.handle)

    def next_step(self):
        t = ctypes.c_int64()
        _check(self.lib.glr_next_step(self.handle, ctypes.byref(t)), self.handle)
        return t.value

    def profile(self, on=True):
        _check(self.lib.glr_profile_enable(self.handle, 1 if on else 0), self.handle)

    def profile_reset(self):
        _check(self.lib.glr_profile_reset(self.handle), self.handle)

    def profile_query(self):
        """{group: (total_ms, launches)} since the last reset."""
        out = {}
        for i, name in enumerate(PROF_GROUPS):
            ms, n = ctypes.c_double(), ctypes.c_int64()
            _check(self.lib.glr_profile_query(self.handle, i, ctypes.byref(ms), ctypes.byref(n)),
                   self.handle)
            out[name] = (ms.value, n.value)
        return out

    # ------------------------------------------------------------ state views
    def _view(self, off, count, dtype):
        torch = self.torch
        esz = torch.empty((), dtype=dtype).element_size()
        b = self.state[self._s0 + off: self._s0 + off + count * esz]
        return b.view(dtype)

    def E(self, mat):
        """N x m x n error buffers (bf16 with store="bf16")."""
        L = self.layouts[mat]
        return self._view(L.off_E, self.workers * L.m * L.n, self.gdtype).view(self.workers, L.m, L.n)

    def Ebar(self, mat):
        L = self.layouts[mat]
        return self._view(L.off_Ebar, L.m * L.n, self.torch.float32).view(L.m, L.n)

    def Ut(self, mat):
        """d x d; row j holds u_j, the j-th column of U."""
        L = self.layouts[mat]
        return self._view(L.off_U, L.d * L.d, self.torch.float32).view(L.d, L.d)

    def sigma(self, mat):
        L = self.layouts[mat]
        return self._view(L.off_sigma, L.d, self.torch.float32)

    def J(self, mat):
        L = self.layouts[mat]
        return self._view(L.off_J, L.r, self.torch.int32)

    def score(self, mat):
        L = self.layouts[mat]
        return self._view(L.off_score, L.d, self.torch.float32)

    def S1(self, mat):
        L = self.layouts[mat]
        return self._view(L.off_S1, L.m * L.n, self.torch.float32).view(L.m, L.n)

    def S2(self, mat):
        L = self.layouts[mat]
        if not L.off_S2:
            return None
        return self._view(L.off_S2, L.m * L.n, self.torch.float32).view(L.m, L.n)

    def Rbar(self, mat):
        L = self.layouts[mat]
        return self._view(L.off_Rbar, L.r * L.D, self.torch.float32).view(L.r, L.D)

    def info(self, mat):
        L = self.layouts[mat]
        return self._view(L.off_info, 64, self.torch.int32)

    def sweep_history(self, mat):
        """(sweeps, converged, [largest pair off-norm of each sweep])."""
        inf = self.info(mat).cpu()
        n = int(inf[0])
        hist = inf[2:2 + min(n, 60)].view(self.torch.float32).tolist()
        return n, bool(inf[1]), hist

    def sub_info(self, mat):
        """tau = 1 refresh: (block iterations run, relative gain of the energy
        the leading r rows capture over the last iteration)."""
        inf = self.info(mat).cpu()
        return int(inf[62]), float(inf[63:64].view(self.torch.float32)[0])

    def P(self, mat):
        """d x r: the selected columns of U (P = U[:, J])."""
        return self.Ut(mat)[self.J(mat).long()].T
