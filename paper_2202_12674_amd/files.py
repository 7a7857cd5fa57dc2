"""LIBSVM-format data and model files through the C ABI of include/lssvm_io.h.

Argument marshalling only: parsing and formatting run in liblssvm.so on the
host, multi-threaded. Arrays are NumPy host arrays (C-contiguous float64 or
float32); copy them to the device for training.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

import numpy as np

from ._binding import F32, F64, KERNELS, Params, _check, lib

KERNEL_NAMES = {0: "linear", 1: "poly", 2: "rbf"}


def _code(dtype) -> int:
    dt = np.dtype(dtype)
    if dt == np.float64:
        return F64
    if dt == np.float32:
        return F32
    raise TypeError(f"unsupported dtype {dt}; use float64 or float32")


def _path(path) -> bytes:
    return os.fsencode(path)


def _host(a, dtype, name):
    if not isinstance(a, np.ndarray) or a.dtype != np.dtype(dtype) or not a.flags.c_contiguous:
        raise TypeError(f"{name} must be a C-contiguous {np.dtype(dtype)} NumPy array")
    return ctypes.c_void_p(a.ctypes.data if a.size else 0)


def scan(path):
    """(n, d): number of points and largest feature index of a data file."""
    n, d = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().lssvm_libsvm_scan(_path(path), ctypes.byref(n), ctypes.byref(d), 0))
    return n.value, d.value


def read(path, dtype=np.float64, d: int | None = None, threads: int = 0, out=None):
    """(X, y) of a data file: X dense (n x d, absent features 0), y labels.

    `out`, if given, is a callable (n, d) -> (X, y) returning the arrays to
    fill (for instance views of pinned host memory for a fast upload)."""
    n, dmax = scan(path)
    d = dmax if d is None else int(d)
    if out is not None:
        X, y = out(n, d)
    else:
        X = np.empty((n, d), dtype=dtype)
        y = np.empty(n, dtype=dtype)
    if X.shape != (n, d) or y.shape != (n,):
        raise ValueError(f"out returned arrays of shapes {X.shape}, {y.shape}; need ({n}, {d})")
    _check(lib().lssvm_libsvm_read(_path(path), _code(dtype), _host(X, dtype, "X"),
                                   _host(y, dtype, "y"), n, d, threads))
    return X, y


def write(path, X, y, threads: int = 0) -> None:
    """Write points X (n x d) with labels y (n,) as a data file."""
    n, d = X.shape
    _check(lib().lssvm_libsvm_write(_path(path), _code(X.dtype), _host(X, X.dtype, "X"),
                                    _host(y, X.dtype, "y"), n, d, threads))


@dataclasses.dataclass
class Model:
    kernel: str
    gamma: float
    coef0: float
    degree: int
    b: float
    X: np.ndarray        # support vectors (n x d), label +1 first
    alpha: np.ndarray    # weights of f(x) = sum alpha_i k(x_i, x) + b
    y: np.ndarray        # labels of the support vectors


def write_model(path, X, y, alpha, b: float, kernel: str = "linear", gamma: float = 1.0,
                coef0: float = 0.0, degree: int = 1, threads: int = 0) -> None:
    """Write a trained model: every training point is a support vector."""
    n, d = X.shape
    if kernel not in KERNELS:
        raise ValueError(f"unknown kernel {kernel!r}")
    kp = Params(float(gamma), float(coef0), int(degree))
    dt = X.dtype
    _check(lib().lssvm_model_write(_path(path), _code(dt), KERNELS[kernel], ctypes.byref(kp),
                                   float(b), _host(alpha, dt, "alpha"), _host(X, dt, "X"),
                                   _host(y, dt, "y"), n, d, threads))


def read_model(path, dtype=np.float64, threads: int = 0) -> Model:
    """Read a model file written by write_model (or LIBSVM, labels 1 and -1)."""
    k = ctypes.c_int32()
    kp = Params()
    b = ctypes.c_double()
    n, d = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().lssvm_model_scan(_path(path), ctypes.byref(k), ctypes.byref(kp), ctypes.byref(b),
                                  ctypes.byref(n), ctypes.byref(d)))
    X = np.empty((n.value, d.value), dtype=dtype)
    alpha = np.empty(n.value, dtype=dtype)
    y = np.empty(n.value, dtype=dtype)
    _check(lib().lssvm_model_read(_path(path), _code(dtype), _host(X, dtype, "X"),
                                  _host(alpha, dtype, "alpha"), _host(y, dtype, "y"), n.value,
                                  d.value, threads))
    return Model(KERNEL_NAMES[k.value], kp.gamma, kp.coef0, kp.degree, b.value, X, alpha, y)
