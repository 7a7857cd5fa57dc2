"""C-ABI checks that need no GPU: the library loads, exports every function
declared in include/lssvm.h, sizes workspaces, and rejects bad arguments on
the host before any GPU work (so these paths run here without a device)."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

import paper_2202_12674_amd as P
from paper_2202_12674_amd import _binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lssvm.h")

FAKE = ctypes.c_void_p(4096)          # never dereferenced: validation fails first
ALIGNED_WS = ctypes.c_void_p(1 << 20)


def header_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(lssvm_[a-z_]+)\s*\(", txt)))


def test_library_exports_every_declared_function():
    L = P.lib()
    names = header_functions()
    assert {"lssvm_train", "lssvm_predict", "lssvm_matvec", "lssvm_workspace_bytes",
            "lssvm_predict_workspace_bytes", "lssvm_last_error", "lssvm_tile_size"} <= set(names)
    for nm in names:
        assert hasattr(L, nm), nm


def test_workspace_sizes():
    L = P.lib()
    assert L.lssvm_workspace_bytes(0, 4, 0) == 0
    assert L.lssvm_workspace_bytes(4, 0, 0) == 0
    assert L.lssvm_workspace_bytes(4, 4, 7) == 0
    small = L.lssvm_workspace_bytes(256, 64, 0)
    assert small > 256 * 64 * 8
    # fp32 layout of 32768 x 4096 points alone is 512 MiB
    assert L.lssvm_workspace_bytes(32768, 4096, 1) >= 32768 * 4096 * 4
    assert L.lssvm_workspace_bytes(1, 1, 1) > 0
    assert L.lssvm_predict_workspace_bytes(100, 0, 3, 0) == 0
    assert L.lssvm_predict_workspace_bytes(100, 10, 3, 1) > 100 * 3 * 4
    assert L.lssvm_tile_size(0) in (64, 128, 256) and L.lssvm_tile_size(1) in (64, 128, 256)
    assert L.lssvm_tile_size(5) == 0


def test_workspace_sizes_at_the_supported_limits():
    # 2^22 points and 2^21 features are the largest sizes the entry points
    # accept; beyond them the size queries answer 0 instead of a wrapped size
    L = P.lib()
    big, wide = 1 << 22, 1 << 21
    for dt in (0, 1):
        assert L.lssvm_workspace_bytes(big, 1, dt) > big * 8
        assert L.lssvm_workspace_bytes(2, wide, dt) > 2 * wide * 4
        assert L.lssvm_workspace_bytes(big + 1, 1, dt) == 0
        assert L.lssvm_workspace_bytes(2, wide + 1, dt) == 0
        assert L.lssvm_workspace_bytes(1 << 62, 1 << 40, dt) == 0
        assert L.lssvm_predict_workspace_bytes(big, big, 1, dt) > 2 * big * 4
        assert L.lssvm_predict_workspace_bytes(big + 1, 1, 1, dt) == 0
        assert L.lssvm_predict_workspace_bytes(2, big + 1, 1, dt) == 0
        assert L.lssvm_predict_workspace_bytes(2, 1, wide + 1, dt) == 0


def test_workspace_grows_with_the_points_not_their_square():
    """A product's row sums take two 64-bit words per row (fixed-point
    accumulators), not a partial slot per tile column: at 2^20 points of 16
    features the training workspace is the points' own layout (2^20 x 64 x 4
    bytes, features padded to two blocks) plus about a fifth of a GiB (the
    tile visit order, n^2 / 8192 bytes, is the only quadratic term). A slot
    per tile column would have been n^2 / 16 bytes = 64 GiB."""
    L = P.lib()
    n = 1 << 20
    ws = L.lssvm_workspace_bytes(n, 16, 1)
    layout = n * 64 * 4
    assert ws < 4 << 30
    assert ws - layout < (n * n // 16) // 200
    assert L.lssvm_workspace_bytes(2 * n, 16, 1) < 3 * ws


def test_tile_plan():
    """The launch plan of the implicit product: pinned for the five benchmark
    workloads, the paper-sized linear problem and the smallest workload, and
    for every shape split widths that leave an even number of feature blocks
    per workgroup (on the small problems whose CG iterations are single
    launches, n <= 1025 without a split last round, the linear kernel's tiles
    split as far as one round of workgroups allows, down to one block each),
    a tail exactly the tiles after the last full round, and at most one round
    of workgroups in a tail launch; EINVAL (plan untouched) outside the
    range."""
    L = P.lib()
    plan = (ctypes.c_int64 * 3)(-5, -5, -5)
    for args in [(1, 64, 0, 0), (256, 0, 0, 0), (256, 64, 9, 0), (256, 64, 0, 3),
                 ((1 << 22) + 1, 64, 0, 0), (256, (1 << 21) + 1, 1, 0)]:
        assert L.lssvm_tile_plan(*args, plan) == B.EINVAL, args
        assert list(plan) == [-5, -5, -5]
    assert L.lssvm_tile_plan(256, 64, 0, 0, None) == B.EINVAL
    pins = {("f64", "linear", 4096, 1024): (1, 16, 32),
            ("f64", "linear", 16384, 4096): (1, 64, 8),
            ("f64", "rbf", 16384, 2048): (1, 64, 8),
            ("f32", "poly", 32768, 4096): (1, 128, 4),
            ("f32", "rbf", 65536, 1024): (1, 0, 1),
            ("f32", "rbf", 32768, 256): (1, 128, 4),
            ("f64", "linear", 256, 64): (4, 0, 4)}
    for (dtype, kernel, n, d), want in pins.items():
        assert P.tile_plan(n, d, dtype, kernel) == want, (dtype, kernel, n, d)
    for dtype in ("f64", "f32"):
        bk = 16 if dtype == "f64" else 32
        for kernel in ("linear", "poly", "rbf"):
            for n in (2, 129, 600, 1000, 2000, 3000, 4096, 6000, 8192, 12000, 40000):
                for d in (1, 7, 64, 100, 256, 1024, 4096):
                    S, Q, T = P.tile_plan(n, d, dtype, kernel)
                    nkb = -(-d // (2 * bk)) * 2
                    nT = -(-(n - 1) // 128)
                    W = nT * (nT + 1) // 2
                    where = (dtype, kernel, n, d, S, Q, T)
                    small = kernel == "linear" and n <= 1025 and Q == 0
                    assert S in (1, 2, 4, 8, 16), where
                    if small and S == nkb:
                        assert S > 1 and W * S <= 512, where   # one feature block each
                    else:
                        assert nkb % (2 * S) == 0, where       # an even count each
                    if small and S < nkb:
                        # as split as the blocks and one round of workgroups allow
                        assert (S == 16 or W * 2 * S > 512
                                or (nkb % (4 * S) != 0 and nkb != 2 * S)), where
                    assert T in (1, 2, 4, 8, 16, 32, 64) and (nkb % (2 * T) == 0 or T == S == nkb), where
                    if kernel != "linear":
                        assert S == 1, where
                    if Q == 0:
                        assert T == S, where
                        continue
                    assert T > S and Q * T <= 512, where
                    if kernel == "linear":
                        full = W * S // 512
                        assert full >= 1 and Q == W - full * (512 // S), where
                    else:
                        assert Q == W % 512 and 4 <= T <= 16, where


def _train(n=10, d=3, dtype=0, kernel=0, params=None, C=1.0, eps=1e-3, max_iter=0,
           ws=ALIGNED_WS, ws_bytes=1 << 40, X=FAKE, y=FAKE, alpha=FAKE, b=True, info=None):
    L = P.lib()
    bb = ctypes.c_double(0)
    kp = ctypes.byref(params) if params is not None else None
    return L.lssvm_train(X, y, n, d, dtype, kernel, kp, C, eps, max_iter, ws, ws_bytes, alpha,
                         ctypes.byref(bb) if b else None, info, None)


@pytest.mark.parametrize("kw,msg", [
    (dict(X=None), "NULL"), (dict(y=None), "NULL"), (dict(alpha=None), "NULL"),
    (dict(b=False), "NULL"), (dict(n=0), "n must"), (dict(d=0), "d must"),
    (dict(dtype=2), "dtype"), (dict(kernel=3), "kernel"),
    (dict(kernel=1), "parameters required"),
    (dict(kernel=1, params=B.Params(0.0, 1.0, 3)), "gamma"),
    (dict(kernel=2, params=B.Params(-1.0, 0.0, 1)), "gamma"),
    (dict(kernel=1, params=B.Params(1.0, 1.0, 0)), "degree"),
    (dict(kernel=1, params=B.Params(1.0, float("nan"), 2)), "coef0"),
    (dict(C=0.0), "C must"), (dict(C=float("inf")), "C must"), (dict(C=-1.0), "C must"),
    (dict(eps=0.0), "eps"), (dict(eps=1.0), "eps"), (dict(eps=float("nan")), "eps"),
    (dict(max_iter=-1), "max_iter"),
    (dict(ws=None), "workspace is NULL"), (dict(ws=ctypes.c_void_p(4100)), "aligned"),
    (dict(ws_bytes=16), "too small"),
    (dict(n=1 << 23), "too large"), (dict(d=1 << 22), "too large"),
])
def test_train_rejects_bad_arguments(kw, msg):
    code = _train(**kw)
    assert code == B.EINVAL
    assert msg in P.last_error()


def test_train_history_without_buffer():
    info = B.Info()
    info.history_capacity = 5
    assert _train(info=ctypes.byref(info)) == B.EINVAL
    assert "history" in P.last_error()
    info = B.Info()
    info.matvec_times_capacity = 5
    assert _train(info=ctypes.byref(info)) == B.EINVAL
    assert "matvec_times" in P.last_error()


def test_info_layout_matches_header():
    """The binding's lssvm_info mirrors the header field for field."""
    txt = open(HEADER).read()
    body = re.search(r"typedef struct lssvm_info \{(.*?)\} lssvm_info;", txt, re.S).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    names = re.findall(r"(\w+)\s*;", body)
    assert names == [f[0] for f in B.Info._fields_]


def test_predict_rejects_bad_arguments():
    L = P.lib()
    kp = B.Params(1.0, 0.0, 1)

    def call(**kw):
        a = dict(Xtr=FAKE, alpha=FAKE, b=0.0, n=10, d=3, dt=0, k=0, X_test=FAKE, nt=5,
                 ws=ALIGNED_WS, wsb=1 << 40, scores=FAKE)
        a.update(kw)
        return L.lssvm_predict(a["Xtr"], a["alpha"], a["b"], a["n"], a["d"], a["dt"], a["k"],
                               ctypes.byref(kp), a["X_test"], a["nt"], a["ws"], a["wsb"],
                               a["scores"], None, None)

    assert call(Xtr=None) == B.EINVAL
    assert call(scores=None) == B.EINVAL
    assert call(nt=0) == B.EINVAL and "n_test" in P.last_error()
    assert call(b=float("nan")) == B.EINVAL
    assert call(wsb=8) == B.EINVAL and "too small" in P.last_error()
    assert call(dt=9) == B.EINVAL


def test_matvec_rejects_bad_arguments():
    L = P.lib()
    kp = B.Params(1.0, 0.0, 1)

    def call(n=10, d=3, C=1.0, p=FAKE, wsb=1 << 40, k=0):
        return L.lssvm_matvec(FAKE, n, d, 0, k, ctypes.byref(kp), C, p, FAKE, ALIGNED_WS, wsb,
                              None)

    assert call(n=1) == B.EINVAL and "n must be >= 2" in P.last_error()
    assert call(C=0.0) == B.EINVAL
    assert call(p=None) == B.EINVAL
    assert call(wsb=1) == B.EINVAL
    assert call(k=7) == B.EINVAL


def test_binding_refuses_cpu_tensors():
    import torch
    X = torch.zeros(4, 2, dtype=torch.float64)
    y = torch.ones(4, dtype=torch.float64)
    with pytest.raises((TypeError, RuntimeError)):
        P.train(X, y, workspace=torch.zeros(1 << 16, dtype=torch.uint8))


def test_binding_checks_shapes_before_the_device():
    # Sizes the library is given come from X; a shorter p, out, alpha or
    # X_test would be read or written past its end on the device, so the
    # binding refuses them before any call (CPU tensors reach these checks).
    import torch
    f64, f32 = torch.float64, torch.float32
    X = torch.zeros(6, 3, dtype=f64)
    ws = torch.zeros(256, dtype=torch.uint8)
    with pytest.raises(ValueError, match="p must have shape"):
        P.matvec(X, torch.zeros(4, dtype=f64), workspace=ws)
    with pytest.raises(ValueError, match="p must have shape"):
        P.matvec(X, torch.zeros(5, dtype=f32), workspace=ws)
    with pytest.raises(ValueError, match="out must have shape"):
        P.matvec(X, torch.zeros(5, dtype=f64), workspace=ws, out=torch.zeros(4, dtype=f64))
    with pytest.raises(ValueError, match="2-D"):
        P.matvec(torch.zeros(6, dtype=f64), torch.zeros(5, dtype=f64), workspace=ws)
    with pytest.raises(ValueError, match="y must have shape"):
        P.train(X, torch.ones(5, dtype=f64), workspace=ws)
    with pytest.raises(ValueError, match="y must have shape"):
        P.train(X, torch.ones(6, dtype=f32), workspace=ws)
    with pytest.raises(ValueError, match="alpha0 must have shape"):
        P.train(X, torch.ones(6, dtype=f64), workspace=ws, alpha0=torch.zeros(5, dtype=f64))
    with pytest.raises(ValueError, match="alpha must have shape"):
        P.predict(X, torch.zeros(5, dtype=f64), 0.0, torch.zeros(2, 3, dtype=f64), workspace=ws)
    with pytest.raises(ValueError, match="X_test must have shape"):
        P.predict(X, torch.zeros(6, dtype=f64), 0.0, torch.zeros(2, 4, dtype=f64), workspace=ws)
    with pytest.raises(ValueError, match="X_test must have shape"):
        P.predict(X, torch.zeros(6, dtype=f64), 0.0, torch.zeros(2, 3, dtype=f32), workspace=ws)
    with pytest.raises(TypeError):
        P.matvec(X.to(torch.int32), torch.zeros(5, dtype=torch.int32), workspace=ws)
    # well-shaped CPU tensors pass the shape checks and stop at the device check
    with pytest.raises(TypeError, match="GPU tensor"):
        P.matvec(X, torch.zeros(5, dtype=f64), workspace=ws)
    with pytest.raises(TypeError, match="GPU tensor"):
        P.predict(X, torch.zeros(6, dtype=f64), 0.0, torch.zeros(2, 3, dtype=f64), workspace=ws)


def test_last_error_is_thread_local():
    import threading
    _train(n=0)
    seen = {}

    def other():
        seen["msg"] = P.last_error()

    t = threading.Thread(target=other)
    t.start()
    t.join()
    assert seen["msg"] == ""
    assert "n must" in P.last_error()


def test_cg_step_rejects_bad_arguments():
    L = P.lib()
    assert L.lssvm_cg_step_workspace_bytes(0) == 0
    assert L.lssvm_cg_step_workspace_bytes(1 << 35) == 0
    small = L.lssvm_cg_step_workspace_bytes(1000)
    assert 0 < small < L.lssvm_cg_step_workspace_bytes(1 << 30)
    v = [ctypes.c_void_p(4096 * k) for k in range(1, 6)]
    N = 100

    def call(N=N, x=v[0], r=v[1], d=v[2], q=v[3], sc=v[4], ws=ALIGNED_WS, wsb=1 << 20):
        return L.lssvm_cg_step(N, x, r, d, q, sc, ws, wsb, None)

    assert call(x=None) == B.EINVAL and "NULL" in P.last_error()
    assert call(sc=None) == B.EINVAL
    assert call(N=0) == B.EINVAL and "N must" in P.last_error()
    assert call(N=1 << 35) == B.EINVAL
    assert call(q=v[0]) == B.EINVAL and "overlap" in P.last_error()
    assert call(r=ctypes.c_void_p(4096 + 8 * 50)) == B.EINVAL     # r inside x
    assert call(ws=None) == B.EINVAL
    assert call(wsb=8) == B.EINVAL and "too small" in P.last_error()


def test_cg_step_noalloc_rejects_bad_arguments():
    """The no-workspace step checks its arguments on the host, before it looks
    up its device array (so these run without a GPU)."""
    L = P.lib()
    buf = (ctypes.c_double * 64)()
    p = ctypes.cast(buf, ctypes.c_void_p)
    q = ctypes.c_void_p(ctypes.addressof(buf) + 8 * 16)
    assert L.lssvm_cg_step_noalloc(0, p, p, p, p, p, None) == -1
    assert L.lssvm_cg_step_noalloc((1 << 34) + 1, p, p, p, p, p, None) == -1
    assert L.lssvm_cg_step_noalloc(4, None, p, q, p, p, None) == -1
    assert L.lssvm_cg_step_noalloc(16, p, q, p, q, p, None) == -1
    assert "overlap" in P.last_error()


def test_host_contexts_without_a_call():
    assert P.lib().lssvm_host_contexts() >= 0


def test_mfma_peak_rejects_bad_arguments():
    L = P.lib()
    assert L.lssvm_mfma_peak_workspace_bytes() >= 512 * 256 * 8
    out = ctypes.c_double()
    assert L.lssvm_mfma_peak(3, ALIGNED_WS, 1 << 30, ctypes.byref(out), None) == B.EINVAL
    assert L.lssvm_mfma_peak(1, None, 1 << 30, ctypes.byref(out), None) == B.EINVAL
    assert L.lssvm_mfma_peak(1, ctypes.c_void_p(4100), 1 << 30, ctypes.byref(out), None) \
        == B.EINVAL and "aligned" in P.last_error()
    assert L.lssvm_mfma_peak(1, ALIGNED_WS, 1024, ctypes.byref(out), None) == B.EINVAL
    assert "too small" in P.last_error()
    assert L.lssvm_mfma_peak(0, ALIGNED_WS, 1 << 30, None, None) == B.EINVAL
