"""ctypes binding of ``libmlp2.so`` (the C ABI in ``include/mlp2.h``).

Argument marshalling only: every step of the computation runs in the HIP
kernels of the library.  PyTorch supplies device memory and the stream.  When
the compiled library is missing, ``load()`` raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libmlp2.so")
TRACE_LIB_PATH = os.path.join(PKG, "libmlp2_trace.so")

ACT_IDENTITY, ACT_GELU_TANH, ACT_SWIGLU = 0, 1, 2
DTYPE_BF16 = 0
MODE_SEQUENTIAL, MODE_TILE_PIPELINED, MODE_WORKQUEUE, MODE_STAGE1, MODE_STAGE2, MODE_SENTINEL = 0, 1, 2, 3, 4, 5
MODES = {"sequential": MODE_SEQUENTIAL, "tile_pipelined": MODE_TILE_PIPELINED, "workqueue": MODE_WORKQUEUE,
         "stage1": MODE_STAGE1, "stage2": MODE_STAGE2, "sentinel": MODE_SENTINEL}
ORDER_AUTO, ORDER_COLUMN_FIRST, ORDER_ROW_FIRST, ORDER_REVERSED, ORDER_SHUFFLED, ORDER_BANDED = 0, 1, 2, 3, 4, 5
OPT_SPIN_LIMIT, OPT_DROP_SIGNAL, OPT_ORDER, OPT_GRID = 1, 2, 3, 4

OK = 0
ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_ALIGNMENT, ERR_HIP, ERR_TIMEOUT, ERR_DEVICE = -1, -2, -3, -4, -5, -6

# Every symbol include/mlp2.h declares.
EXPORTS = (
    "mlp2_plan",
    "mlp2_plan_ex",
    "mlp2_run",
    "mlp2_destroy",
    "mlp2_last_error",
    "mlp2_strerror",
    "mlp2_check",
    "mlp2_plan_info",
    "mlp2_intermediate",
    "mlp2_set_option",
    "mlp2_trace_attach",
    "mlp2_chain_plan",
    "mlp2_chain_run",
    "mlp2_chain_check",
    "mlp2_chain_set_spin_limit",
    "mlp2_chain_destroy",
    "mlp2_chain_grid",
    "mlp2_chain_trace_attach",
    "mlp2_run_noalloc",
)


class Tuning(ctypes.Structure):
    _fields_ = [
        ("bm", ctypes.c_int),
        ("bn1", ctypes.c_int),
        ("splitk1", ctypes.c_int),
        ("bn2", ctypes.c_int),
        ("splitk2", ctypes.c_int),
        ("grid", ctypes.c_int),
        ("order", ctypes.c_int),
        ("stages", ctypes.c_int),
        ("row_group", ctypes.c_int),
        ("waves", ctypes.c_int),
        ("lag", ctypes.c_int),
        ("p1", ctypes.c_int),
        ("bk", ctypes.c_int),
        ("weights_nt", ctypes.c_int),
    ]


class Info(ctypes.Structure):
    _fields_ = [
        ("M", ctypes.c_int64),
        ("H", ctypes.c_int64),
        ("F", ctypes.c_int64),
        ("act", ctypes.c_int),
        ("bm", ctypes.c_int),
        ("bn1", ctypes.c_int),
        ("splitk1", ctypes.c_int),
        ("bn2", ctypes.c_int),
        ("splitk2", ctypes.c_int),
        ("bk", ctypes.c_int),
        ("row_blocks", ctypes.c_int),
        ("col_blocks1", ctypes.c_int),
        ("col_blocks2", ctypes.c_int),
        ("items1", ctypes.c_int),
        ("items2", ctypes.c_int),
        ("grid_pipelined", ctypes.c_int),
        ("occupancy", ctypes.c_int),
        ("num_cus", ctypes.c_int),
        ("order", ctypes.c_int),
        ("workspace_bytes", ctypes.c_int64),
        ("spin_limit", ctypes.c_uint32),
        ("stages", ctypes.c_int),
        ("grid_gemm1", ctypes.c_int),
        ("grid_gemm2", ctypes.c_int),
        ("row_group", ctypes.c_int),
        ("waves", ctypes.c_int),
        ("lag", ctypes.c_int),
        ("p1", ctypes.c_int),
        ("weights_nt", ctypes.c_int),
    ]


class Mlp2Error(RuntimeError):
    def __init__(self, code: int, what: str):
        self.code = code
        super().__init__(f"{what}: {strerror(code)} ({code})")


_lib = None


def load(path: str | None = None) -> ctypes.CDLL:
    """Load the compiled library (raises if it was not built).

    The first call loads the product library ``libmlp2.so`` unless ``path``
    names another build (the timing-trace tool passes ``TRACE_LIB_PATH``);
    later calls without a path return the loaded one.  A process holds one
    library: asking for a different path after the first load raises.
    """
    global _lib
    if _lib is not None:
        if path is not None and os.path.abspath(_lib._name) != os.path.abspath(path):
            raise RuntimeError(f"{_lib._name} is already loaded; cannot also load {path}")
        return _lib
    if path is None:
        path = LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2607_07862_amd.build`")
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    lib.mlp2_plan.restype = P
    lib.mlp2_plan.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int, ctypes.c_int]
    lib.mlp2_plan_ex.restype = P
    lib.mlp2_plan_ex.argtypes = lib.mlp2_plan.argtypes + [ctypes.POINTER(Tuning)]
    lib.mlp2_run.restype = ctypes.c_int
    lib.mlp2_run.argtypes = [P, P, P, P, P, P, ctypes.c_int]
    lib.mlp2_destroy.restype = None
    lib.mlp2_destroy.argtypes = [P]
    lib.mlp2_last_error.restype = ctypes.c_int
    lib.mlp2_last_error.argtypes = []
    lib.mlp2_strerror.restype = ctypes.c_char_p
    lib.mlp2_strerror.argtypes = [ctypes.c_int]
    lib.mlp2_check.restype = ctypes.c_int
    lib.mlp2_check.argtypes = [P]
    lib.mlp2_plan_info.restype = ctypes.c_int
    lib.mlp2_plan_info.argtypes = [P, ctypes.POINTER(Info)]
    lib.mlp2_intermediate.restype = P
    lib.mlp2_intermediate.argtypes = [P]
    lib.mlp2_set_option.restype = ctypes.c_int
    lib.mlp2_set_option.argtypes = [P, ctypes.c_int, ctypes.c_int64]
    lib.mlp2_trace_attach.restype = ctypes.c_int
    lib.mlp2_trace_attach.argtypes = [P, P, ctypes.c_int]
    lib.mlp2_chain_plan.restype = P
    lib.mlp2_chain_plan.argtypes = [ctypes.c_int64, ctypes.c_int, ctypes.POINTER(ctypes.c_int64), ctypes.c_int, ctypes.c_int]
    lib.mlp2_chain_run.restype = ctypes.c_int
    lib.mlp2_chain_run.argtypes = [P, P, ctypes.POINTER(P), P, P, ctypes.c_int]
    lib.mlp2_chain_check.restype = ctypes.c_int
    lib.mlp2_chain_check.argtypes = [P]
    lib.mlp2_chain_set_spin_limit.restype = ctypes.c_int
    lib.mlp2_chain_set_spin_limit.argtypes = [P, ctypes.c_int64]
    lib.mlp2_chain_grid.restype = ctypes.c_int
    lib.mlp2_chain_grid.argtypes = [P]
    lib.mlp2_chain_trace_attach.restype = ctypes.c_int
    lib.mlp2_chain_trace_attach.argtypes = [P, P, ctypes.c_int]
    lib.mlp2_chain_destroy.restype = None
    lib.mlp2_chain_destroy.argtypes = [P]
    lib.mlp2_run_noalloc.restype = ctypes.c_int
    lib.mlp2_run_noalloc.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                                     P, P, P, P, P, ctypes.c_int]
    _lib = lib
    return lib


def loaded_path() -> str | None:
    """Path of the library this process has loaded, or None."""
    return None if _lib is None else _lib._name


def strerror(code: int) -> str:
    return load().mlp2_strerror(int(code)).decode()


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _check_tensor(t, name, numel, device):
    import torch

    if t.dtype != torch.bfloat16:
        raise TypeError(f"{name} must be bfloat16")
    if not t.is_cuda or t.device != device:
        raise ValueError(f"{name} must live on {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() != numel:
        raise ValueError(f"{name} must hold {numel} elements, has {t.numel()}")


class Plan:
    """A plan for ``Y[M,H] = act(X[M,H] @ W1) @ W2`` on the current device."""

    def __init__(self, M: int, H: int, F: int, act: int, tuning: dict | None = None):
        import torch

        self.lib = load()
        self.M, self.H, self.F, self.act = int(M), int(H), int(F), int(act)
        self.device = torch.device("cuda", torch.cuda.current_device())
        if tuning:
            t = Tuning()
            for k, v in tuning.items():
                setattr(t, k, int(v))
            h = self.lib.mlp2_plan_ex(self.M, self.H, self.F, self.act, DTYPE_BF16, ctypes.byref(t))
        else:
            h = self.lib.mlp2_plan(self.M, self.H, self.F, self.act, DTYPE_BF16)
        if not h:
            raise Mlp2Error(self.lib.mlp2_last_error(), "mlp2_plan")
        self.handle = ctypes.c_void_p(h)

    def close(self):
        if getattr(self, "handle", None):
            self.lib.mlp2_destroy(self.handle)
            self.handle = None

    def __del__(self):  # pragma: no cover - best effort
        try:
            self.close()
        except Exception:
            pass

    def run(self, X, W1, W2, Y, mode, stream=None) -> None:
        """Enqueue one evaluation on ``stream`` (default: torch's current stream)."""
        import torch

        n1 = 2 if self.act == ACT_SWIGLU else 1
        _check_tensor(X, "X", self.M * self.H, self.device)
        _check_tensor(W1, "W1", n1 * self.H * self.F, self.device)
        _check_tensor(W2, "W2", self.F * self.H, self.device)
        _check_tensor(Y, "Y", self.M * self.H, self.device)
        mode = MODES.get(mode, mode)
        if stream is None:
            stream = torch.cuda.current_stream(self.device)
        sp = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
        rc = self.lib.mlp2_run(self.handle, _ptr(X), _ptr(W1), _ptr(W2), _ptr(Y), sp, int(mode))
        if rc != OK:
            raise Mlp2Error(rc, "mlp2_run")

    def run_raw(self, X: int, W1: int, W2: int, Y: int, stream: int, mode: int) -> int:
        """The C call with raw integers (no checks here), returning its status."""
        return self.lib.mlp2_run(self.handle, X, W1, W2, Y, stream, mode)

    def check(self) -> int:
        return self.lib.mlp2_check(self.handle)

    def info(self) -> dict:
        i = Info()
        rc = self.lib.mlp2_plan_info(self.handle, ctypes.byref(i))
        if rc != OK:
            raise Mlp2Error(rc, "mlp2_plan_info")
        return {f: getattr(i, f) for f, _ in Info._fields_}

    def set_option(self, key: int, value: int) -> None:
        rc = self.lib.mlp2_set_option(self.handle, int(key), int(value))
        if rc != OK:
            raise Mlp2Error(rc, "mlp2_set_option")

    def attach_trace(self, buffer, records_per_group: int) -> None:
        """Attach a device uint64/int64 tensor as the timing-trace buffer (trace builds only)."""
        rc = self.lib.mlp2_trace_attach(self.handle, _ptr(buffer), int(records_per_group))
        if rc != OK:
            raise Mlp2Error(rc, "mlp2_trace_attach")

    def intermediate_ptr(self) -> int:
        return int(self.lib.mlp2_intermediate(self.handle) or 0)

    def intermediate(self):
        """A copy of the plan's bf16 Z as a torch tensor [row_blocks*bm, F] (synchronises)."""
        import torch

        info = self.info()
        rows = info["row_blocks"] * info["bm"]
        out = torch.empty(rows, self.F, dtype=torch.bfloat16, device=self.device)
        torch.cuda.synchronize(self.device)
        _hip_memcpy_d2d(out.data_ptr(), self.intermediate_ptr(), rows * self.F * 2)
        return out


_hip = None


def _hip_memcpy_d2d(dst: int, src: int, nbytes: int) -> None:
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipMemcpy.restype = ctypes.c_int
        _hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    rc = _hip.hipMemcpy(dst, src, nbytes, 3)  # hipMemcpyDeviceToDevice
    if rc != 0:
        raise RuntimeError(f"hipMemcpy failed ({rc})")


def run_noalloc(X, W1, W2, Y, act: int, mode, stream=None) -> None:
    """``mlp2_run_noalloc``: one evaluation with the library's static device
    workspace (no allocation; shapes from X [M,H] and W1 [H,F] / [2,H,F])."""
    import torch

    lib = load()
    M, H = int(X.shape[0]), int(X.shape[1])
    F = int(W1.shape[-1])
    n1 = 2 if act == ACT_SWIGLU else 1
    dev = X.device
    _check_tensor(X, "X", M * H, dev)
    _check_tensor(W1, "W1", n1 * H * F, dev)
    _check_tensor(W2, "W2", F * H, dev)
    _check_tensor(Y, "Y", M * H, dev)
    mode = MODES.get(mode, mode)
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    sp = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    rc = lib.mlp2_run_noalloc(M, H, F, int(act), DTYPE_BF16, _ptr(X), _ptr(W1), _ptr(W2), _ptr(Y), sp, int(mode))
    if rc != OK:
        raise Mlp2Error(rc, "mlp2_run_noalloc")


class ChainPlan:
    """A plan for the GEMM chain ``Z_l = act(Z_{l-1} @ W_l)``, ``Y = Z_{L-1} @ W_L`` (dims = [D_0, ..., D_L])."""

    def __init__(self, M: int, dims, act: int):
        import torch

        self.lib = load()
        self.M, self.dims, self.act = int(M), [int(d) for d in dims], int(act)
        self.L = len(self.dims) - 1
        self.device = torch.device("cuda", torch.cuda.current_device())
        arr = (ctypes.c_int64 * len(self.dims))(*self.dims)
        h = self.lib.mlp2_chain_plan(self.M, self.L, arr, self.act, DTYPE_BF16)
        if not h:
            raise Mlp2Error(self.lib.mlp2_last_error(), "mlp2_chain_plan")
        self.handle = ctypes.c_void_p(h)

    def close(self):
        if getattr(self, "handle", None):
            self.lib.mlp2_chain_destroy(self.handle)
            self.handle = None

    def __del__(self):  # pragma: no cover - best effort
        try:
            self.close()
        except Exception:
            pass

    def run(self, X, Ws, Y, mode, stream=None) -> None:
        """Enqueue one evaluation on ``stream`` (default: torch's current stream)."""
        import torch

        if len(Ws) != self.L:
            raise ValueError(f"expected {self.L} weights")
        _check_tensor(X, "X", self.M * self.dims[0], self.device)
        for l, W in enumerate(Ws):
            _check_tensor(W, f"W{l + 1}", self.dims[l] * self.dims[l + 1], self.device)
        _check_tensor(Y, "Y", self.M * self.dims[-1], self.device)
        mode = MODES.get(mode, mode)
        if stream is None:
            stream = torch.cuda.current_stream(self.device)
        sp = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
        ptrs = (ctypes.c_void_p * self.L)(*[_ptr(W) for W in Ws])
        rc = self.lib.mlp2_chain_run(self.handle, _ptr(X), ptrs, _ptr(Y), sp, int(mode))
        if rc != OK:
            raise Mlp2Error(rc, "mlp2_chain_run")

    def check(self) -> int:
        return self.lib.mlp2_chain_check(self.handle)

    def grid(self) -> int:
        return int(self.lib.mlp2_chain_grid(self.handle))

    def attach_trace(self, buffer, records_per_group: int) -> None:
        """Attach a device int64 tensor as the timing-trace buffer (trace builds only)."""
        rc = self.lib.mlp2_chain_trace_attach(self.handle, _ptr(buffer), int(records_per_group))
        if rc != OK:
            raise Mlp2Error(rc, "mlp2_chain_trace_attach")

    def set_spin_limit(self, polls: int) -> None:
        rc = self.lib.mlp2_chain_set_spin_limit(self.handle, int(polls))
        if rc != OK:
            raise Mlp2Error(rc, "mlp2_chain_set_spin_limit")
