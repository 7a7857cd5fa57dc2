"""ctypes binding of liblssvm.so (C ABI in include/lssvm.h).

Argument marshalling only: every step of the path runs in the HIP library.
PyTorch provides device memory and the current stream. There is no CPU
fallback: without the built library every call raises.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "liblssvm.so")

F64, F32 = 0, 1
LINEAR, POLY, RBF = 0, 1, 2
OK, NOT_CONVERGED, EINVAL, ENONFINITE, EBADLABEL, EBREAKDOWN, EHIP = 0, 1, -1, -2, -3, -4, -5
STOP_EPS, STOP_MAX_ITER, STOP_STALL, STOP_BREAKDOWN = 0, 1, 2, 3
KERNELS = {"linear": LINEAR, "poly": POLY, "polynomial": POLY, "rbf": RBF}
STATUS_NAMES = {OK: "OK", NOT_CONVERGED: "NOT_CONVERGED", EINVAL: "EINVAL",
                ENONFINITE: "ENONFINITE", EBADLABEL: "EBADLABEL", EBREAKDOWN: "EBREAKDOWN",
                EHIP: "EHIP"}


class Params(ctypes.Structure):
    _fields_ = [("gamma", ctypes.c_double), ("coef0", ctypes.c_double),
                ("degree", ctypes.c_int32)]


class Info(ctypes.Structure):
    _fields_ = [("iterations", ctypes.c_int64), ("n_matvec", ctypes.c_int64),
                ("rel_residual", ctypes.c_double), ("true_rel_residual", ctypes.c_double),
                ("t_setup_ms", ctypes.c_double), ("t_cg_ms", ctypes.c_double),
                ("t_total_ms", ctypes.c_double), ("compute_true_residual", ctypes.c_int32),
                ("warm_start", ctypes.c_int32),
                ("residual_history", ctypes.POINTER(ctypes.c_double)),
                ("history_capacity", ctypes.c_int64), ("time_matvec", ctypes.c_int32),
                ("stop_reason", ctypes.c_int32), ("t_matvec_ms", ctypes.c_double),
                ("n_matvec_timed", ctypes.c_int64),
                ("matvec_times", ctypes.POINTER(ctypes.c_double)),
                ("matvec_times_capacity", ctypes.c_int64)]


class LssvmError(RuntimeError):
    """A failed call: ``code`` is the library's status, ``info`` (training only)
    what the call's report recorded before it failed (iterations, ...)."""

    def __init__(self, code: int, msg: str, info: dict | None = None):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code
        self.info = info or {}


_lib = None

_SIGS = {
    "lssvm_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32]),
    "lssvm_predict_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int64, ctypes.c_int64,
                                                        ctypes.c_int64, ctypes.c_int32]),
    "lssvm_train": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                   ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                   ctypes.POINTER(Params), ctypes.c_double, ctypes.c_double,
                                   ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t,
                                   ctypes.c_void_p, ctypes.POINTER(ctypes.c_double),
                                   ctypes.POINTER(Info), ctypes.c_void_p]),
    "lssvm_predict": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_double,
                                     ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                     ctypes.c_int32, ctypes.POINTER(Params), ctypes.c_void_p,
                                     ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t,
                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "lssvm_matvec": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                    ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(Params),
                                    ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "lssvm_cg_step_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int64]),
    "lssvm_cg_step_noalloc": (ctypes.c_int, [ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                             ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                             ctypes.c_void_p]),
    "lssvm_host_contexts": (ctypes.c_int64, []),
    "lssvm_cg_step": (ctypes.c_int, [ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "lssvm_mfma_peak_workspace_bytes": (ctypes.c_size_t, []),
    "lssvm_mfma_peak": (ctypes.c_int, [ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t,
                                       ctypes.POINTER(ctypes.c_double), ctypes.c_void_p]),
    "lssvm_last_error": (ctypes.c_char_p, []),
    # host file IO (include/lssvm_io.h)
    "lssvm_libsvm_scan": (ctypes.c_int, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_int64),
                                         ctypes.POINTER(ctypes.c_int64), ctypes.c_int32]),
    "lssvm_libsvm_read": (ctypes.c_int, [ctypes.c_char_p, ctypes.c_int32, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                         ctypes.c_int32]),
    "lssvm_libsvm_write": (ctypes.c_int, [ctypes.c_char_p, ctypes.c_int32, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                          ctypes.c_int32]),
    "lssvm_model_write": (ctypes.c_int, [ctypes.c_char_p, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.POINTER(Params), ctypes.c_double,
                                         ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.c_int64, ctypes.c_int64, ctypes.c_int32]),
    "lssvm_model_scan": (ctypes.c_int, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_int32),
                                        ctypes.POINTER(Params), ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_int64),
                                        ctypes.POINTER(ctypes.c_int64)]),
    "lssvm_model_read": (ctypes.c_int, [ctypes.c_char_p, ctypes.c_int32, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                        ctypes.c_int64, ctypes.c_int32]),
    "lssvm_tile_size": (ctypes.c_int32, [ctypes.c_int32]),
    "lssvm_tile_plan": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                       ctypes.c_int32, ctypes.POINTER(ctypes.c_int64)]),
}


def lib() -> ctypes.CDLL:
    """The loaded HIP library; raises if it has not been built.

    torch is imported first: it ships its own HIP runtime, and the library's
    libamdhip64 dependency must resolve to that same copy (two HIP runtimes in
    one process do not share the device)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2202_12674_amd.build` (no CPU fallback exists)")
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def last_error() -> str:
    return lib().lssvm_last_error().decode()


def _check(code: int, allow_not_converged: bool = False, info: dict | None = None) -> int:
    if code < 0 or (code == NOT_CONVERGED and not allow_not_converged):
        raise LssvmError(code, last_error(), info)
    return code


# ------------------------------------------------------------ torch layer ---

def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float64:
        return F64
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}; use float64 or float32")


def _dev_ptr(t, name: str):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _matrix(t, name: str):
    """(rows, columns) of a 2-D tensor, else TypeError / ValueError."""
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if t.dim() != 2:
        raise ValueError(f"{name} must be 2-D (points x features), not {tuple(t.shape)}")
    return t.shape


def _expect(t, name: str, shape: tuple, like, like_name: str = "X") -> None:
    """Refuse t unless it has the given shape and the dtype and device of
    `like`: a vector shorter than the sizes passed to the library would be read
    or written past its end on the device, so this runs before any call."""
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if tuple(t.shape) != tuple(shape) or t.dtype != like.dtype or t.device != like.device:
        raise ValueError(f"{name} must have shape {tuple(shape)} and the dtype and device of "
                         f"{like_name}, not {tuple(t.shape)} {t.dtype} on {t.device}")


def _workspace(ws, device):
    torch = _torch()
    if not isinstance(ws, torch.Tensor) or ws.device != device:
        raise ValueError(f"workspace must be a tensor on {device}")
    return ws


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def _stream(device):
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _params(kernel: str, gamma: float, coef0: float, degree: int):
    if kernel not in KERNELS:
        raise ValueError(f"unknown kernel {kernel!r}")
    return KERNELS[kernel], Params(float(gamma), float(coef0), int(degree))


def workspace_bytes(n: int, d: int, dtype) -> int:
    torch = _torch()
    code = F64 if dtype == torch.float64 else F32
    return int(lib().lssvm_workspace_bytes(n, d, code))


def predict_workspace_bytes(n: int, n_test: int, d: int, dtype) -> int:
    torch = _torch()
    code = F64 if dtype == torch.float64 else F32
    return int(lib().lssvm_predict_workspace_bytes(n, n_test, d, code))


def alloc_workspace(nbytes: int, device):
    torch = _torch()
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


@dataclasses.dataclass
class TrainResult:
    alpha: object            # torch tensor (n,), dtype of X
    b: float
    status: int
    converged: bool
    iterations: int
    n_matvec: int
    rel_residual: float
    true_rel_residual: float
    t_setup_ms: float
    t_cg_ms: float
    t_total_ms: float
    history: list
    stalled: bool = False     # NOT_CONVERGED because CG stopped making progress
    t_matvec_ms: float = 0.0
    n_matvec_timed: int = 0
    matvec_times: list = dataclasses.field(default_factory=list)   # ms per timed product


def train(X, y, kernel: str = "linear", gamma: float = 1.0, coef0: float = 0.0,
          degree: int = 1, C: float = 1.0, eps: float = 1e-8, max_iter: int = 0,
          workspace=None, true_residual: bool = False, history: int = 0,
          raise_not_converged: bool = False, time_matvec: bool = False,
          alpha0=None, matvec_times: int = 0) -> TrainResult:
    """lssvm_train on device tensors X (n x d) and y (n,), same float dtype.

    alpha0 (device tensor, n values): start CG from its first n - 1 entries
    (a previous solution or a saved iterate) instead of zero. With
    time_matvec, matvec_times > 0 returns the duration of each of the first
    that many products as well as their sum."""
    torch = _torch()
    n, d = _matrix(X, "X")
    dt = _dtype_code(X)
    _expect(y, "y", (n,), X)
    if alpha0 is not None:
        _expect(alpha0, "alpha0", (n,), X)
    k, kp = _params(kernel, gamma, coef0, degree)
    if workspace is None:
        workspace = alloc_workspace(lib().lssvm_workspace_bytes(n, d, dt), X.device)
    _workspace(workspace, X.device)
    _dev_ptr(X, "X")
    alpha = torch.empty(n, dtype=X.dtype, device=X.device)
    b = ctypes.c_double(0.0)
    info = Info()
    if alpha0 is not None:
        alpha.copy_(alpha0)
        info.warm_start = 1
    info.compute_true_residual = 1 if true_residual else 0
    info.time_matvec = 1 if time_matvec else 0
    hist = (ctypes.c_double * history)() if history > 0 else None
    if hist is not None:
        info.residual_history = ctypes.cast(hist, ctypes.POINTER(ctypes.c_double))
        info.history_capacity = history
    times = (ctypes.c_double * matvec_times)() if matvec_times > 0 else None
    if times is not None:
        info.matvec_times = ctypes.cast(times, ctypes.POINTER(ctypes.c_double))
        info.matvec_times_capacity = matvec_times
    code = lib().lssvm_train(_dev_ptr(X, "X"), _dev_ptr(y, "y"), n, d, dt, k, ctypes.byref(kp),
                             float(C), float(eps), int(max_iter), _dev_ptr(workspace, "workspace"),
                             _nbytes(workspace), _dev_ptr(alpha, "alpha"), ctypes.byref(b),
                             ctypes.byref(info), _stream(X.device))
    _check(code, allow_not_converged=not raise_not_converged,
           info={"iterations": info.iterations, "n_matvec": info.n_matvec,
                 "rel_residual": info.rel_residual, "stop_reason": info.stop_reason})
    stalled = info.stop_reason == STOP_STALL
    return TrainResult(alpha, b.value, code, code == OK, info.iterations, info.n_matvec,
                       info.rel_residual, info.true_rel_residual, info.t_setup_ms, info.t_cg_ms,
                       info.t_total_ms,
                       list(hist[:min(history, info.iterations)]) if hist is not None else [],
                       stalled, info.t_matvec_ms, info.n_matvec_timed,
                       list(times[:min(matvec_times, info.n_matvec_timed)])
                       if times is not None else [])


def predict(X_train, alpha, b: float, X_test, kernel: str = "linear", gamma: float = 1.0,
            coef0: float = 0.0, degree: int = 1, workspace=None, want_labels: bool = True):
    """lssvm_predict: (scores, labels) for the rows of X_test."""
    torch = _torch()
    n, d = _matrix(X_train, "X_train")
    nt, dx = _matrix(X_test, "X_test")
    dt = _dtype_code(X_train)
    _expect(alpha, "alpha", (n,), X_train, "X_train")
    _expect(X_test, "X_test", (nt, d), X_train, "X_train")
    k, kp = _params(kernel, gamma, coef0, degree)
    if workspace is None:
        workspace = alloc_workspace(lib().lssvm_predict_workspace_bytes(n, nt, d, dt),
                                    X_train.device)
    _workspace(workspace, X_train.device)
    _dev_ptr(X_train, "X_train")
    scores = torch.empty(nt, dtype=X_train.dtype, device=X_train.device)
    labels = torch.empty(nt, dtype=torch.int32, device=X_train.device) if want_labels else None
    code = lib().lssvm_predict(_dev_ptr(X_train, "X_train"), _dev_ptr(alpha, "alpha"), float(b),
                               n, d, dt, k, ctypes.byref(kp), _dev_ptr(X_test, "X_test"), nt,
                               _dev_ptr(workspace, "workspace"), _nbytes(workspace),
                               _dev_ptr(scores, "scores"),
                               _dev_ptr(labels, "labels") if labels is not None else None,
                               _stream(X_train.device))
    _check(code)
    return scores, labels


def matvec(X, p, kernel: str = "linear", gamma: float = 1.0, coef0: float = 0.0,
           degree: int = 1, C: float = 1.0, workspace=None, out=None):
    """lssvm_matvec: out = Q~ p for the reduced system of the points X."""
    torch = _torch()
    n, d = _matrix(X, "X")
    dt = _dtype_code(X)
    _expect(p, "p", (n - 1,), X)
    if out is not None:
        _expect(out, "out", (n - 1,), X)
    k, kp = _params(kernel, gamma, coef0, degree)
    if workspace is None:
        workspace = alloc_workspace(lib().lssvm_workspace_bytes(n, d, dt), X.device)
    _workspace(workspace, X.device)
    _dev_ptr(X, "X")
    if out is None:
        out = torch.empty(n - 1, dtype=X.dtype, device=X.device)
    code = lib().lssvm_matvec(_dev_ptr(X, "X"), n, d, dt, k, ctypes.byref(kp), float(C),
                              _dev_ptr(p, "p"), _dev_ptr(out, "out"),
                              _dev_ptr(workspace, "workspace"), _nbytes(workspace),
                              _stream(X.device))
    _check(code)
    return out


def cg_step(x, r, d, q, scalars, workspace=None):
    """lssvm_cg_step: one CG iteration in place on fp64 device vectors given
    q = A d; scalars (4 fp64 on the device) carries r^T r in and
    (r^T r, d^T q, step, beta) out. Nothing is read back."""
    torch = _torch()
    N = x.numel()
    for t, nm in ((x, "x"), (r, "r"), (d, "d"), (q, "q"), (scalars, "scalars")):
        if t.dtype != torch.float64:
            raise TypeError(f"{nm} must be float64")
    if not (r.numel() == d.numel() == q.numel() == N) or scalars.numel() < 4:
        raise ValueError("x, r, d, q need equal lengths and scalars 4 entries")
    if any(t.device != x.device for t in (r, d, q, scalars)):
        raise ValueError("x, r, d, q and scalars must be on one device")
    if workspace is None:
        workspace = alloc_workspace(lib().lssvm_cg_step_workspace_bytes(N), x.device)
    _workspace(workspace, x.device)
    _check(lib().lssvm_cg_step(N, _dev_ptr(x, "x"), _dev_ptr(r, "r"), _dev_ptr(d, "d"),
                               _dev_ptr(q, "q"), _dev_ptr(scalars, "scalars"),
                               _dev_ptr(workspace, "workspace"), _nbytes(workspace),
                               _stream(x.device)))


def cg_step_noalloc(x, r, d, q, scalars):
    """lssvm_cg_step_noalloc: lssvm_cg_step in the library's own fixed device
    array (no workspace, nothing allocated). Calls on one device must not
    overlap."""
    torch = _torch()
    N = x.numel()
    for t, nm in ((x, "x"), (r, "r"), (d, "d"), (q, "q"), (scalars, "scalars")):
        if t.dtype != torch.float64:
            raise TypeError(f"{nm} must be float64")
    if not (r.numel() == d.numel() == q.numel() == N) or scalars.numel() < 4:
        raise ValueError("x, r, d, q need equal lengths and scalars 4 entries")
    if any(t.device != x.device for t in (r, d, q, scalars)):
        raise ValueError("x, r, d, q and scalars must be on one device")
    with torch.cuda.device(x.device):
        _check(lib().lssvm_cg_step_noalloc(N, _dev_ptr(x, "x"), _dev_ptr(r, "r"),
                                           _dev_ptr(d, "d"), _dev_ptr(q, "q"),
                                           _dev_ptr(scalars, "scalars"), _stream(x.device)))


def tile_plan(n: int, d: int, dtype: str, kernel: str) -> tuple:
    """lssvm_tile_plan: (workgroups per tile, tiles of the finer-split last
    round, workgroups per such tile) of the implicit product for n points of
    d features; dtype "f64" or "f32", kernel "linear", "poly" or "rbf"."""
    plan = (ctypes.c_int64 * 3)()
    _check(lib().lssvm_tile_plan(int(n), int(d), {"f64": 0, "f32": 1}[dtype],
                                 {"linear": 0, "poly": 1, "rbf": 2}[kernel], plan))
    return tuple(int(v) for v in plan)


def host_contexts() -> int:
    """lssvm_host_contexts: host contexts the library holds."""
    return int(lib().lssvm_host_contexts())


def mfma_peak(dtype, device) -> float:
    """lssvm_mfma_peak: sustained TFLOP/s of the tile kernel's matrix-core
    instruction for dtype (torch.float32 or torch.float64) on device."""
    torch = _torch()
    code = F64 if dtype == torch.float64 else F32
    ws = alloc_workspace(lib().lssvm_mfma_peak_workspace_bytes(), device)
    out = ctypes.c_double(0.0)
    _check(lib().lssvm_mfma_peak(code, _dev_ptr(ws, "workspace"), _nbytes(ws), ctypes.byref(out),
                                 _stream(device)))
    return out.value
