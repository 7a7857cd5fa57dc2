"""GPU: lssvm_cg_step_noalloc (the CG vector step in the library's own fixed
device array, for callers that cannot allocate) against lssvm_cg_step with a
caller workspace: bit-identical vectors and scalars on two calls in a row, the
second on a shorter vector, plus its argument checks."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2202_12674_amd as P
    P.lib()
    return torch, torch.device("cuda:0")


def _state(torch, dev, N, seed):
    rng = np.random.default_rng(seed)
    x, r, d = (rng.standard_normal(N) for _ in range(3))
    q = d * rng.uniform(0.5, 2.0, N)            # d^T q > 0
    t = [torch.from_numpy(a).to(dev) for a in (x, r, d, q)]
    sc = torch.tensor([float(r @ r), 0.0, 0.0, 0.0], dtype=torch.float64, device=dev)
    return t, sc


def test_noalloc_step_equals_workspace_step(torch_dev):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    for N, seed in ((300_001, 1), (1000, 2)):     # the second call on a shorter vector
        (x1, r1, d1, q1), s1 = _state(torch, dev, N, seed)
        (x2, r2, d2, q2), s2 = _state(torch, dev, N, seed)
        P.cg_step(x1, r1, d1, q1, s1)
        P.cg_step_noalloc(x2, r2, d2, q2, s2)
        torch.cuda.synchronize()
        for a, b in ((x1, x2), (r1, r2), (d1, d2), (s1, s2)):
            assert torch.equal(a, b), N
        assert torch.equal(q1, q2)
        assert float(s2[1]) > 0.0 and np.isfinite(s2.cpu().numpy()).all()


def test_noalloc_step_chained_on_a_stream(torch_dev):
    """Steps queued back to back on one stream, nothing read in between, keep
    matching the workspace entry point."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    n = 257
    rng = np.random.default_rng(4)
    M = rng.standard_normal((n, n))
    A = torch.from_numpy(M @ M.T / n + np.eye(n)).to(dev)
    b = torch.from_numpy(rng.standard_normal(n)).to(dev)
    runs = []
    for fn in (P.cg_step, P.cg_step_noalloc):
        x = torch.zeros(n, dtype=torch.float64, device=dev)
        r, d = b.clone(), b.clone()
        q = torch.empty_like(b)
        sc = torch.tensor([float(b @ b), 0, 0, 0], dtype=torch.float64, device=dev)
        for _ in range(12):
            torch.matmul(A, d, out=q)
            fn(x, r, d, q, sc)
        torch.cuda.synchronize()
        runs.append((x.clone(), sc.clone()))
    assert torch.equal(runs[0][0], runs[1][0]) and torch.equal(runs[0][1], runs[1][1])


def test_noalloc_step_rejects_bad_arguments(torch_dev):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    L = P.lib()
    v = torch.zeros(16, dtype=torch.float64, device=dev)
    p = ctypes.c_void_p(v.data_ptr())
    q = ctypes.c_void_p(v.data_ptr() + 8 * 8)
    assert L.lssvm_cg_step_noalloc(0, p, p, p, p, p, None) == -1
    assert L.lssvm_cg_step_noalloc((1 << 34) + 1, p, p, p, p, p, None) == -1
    assert L.lssvm_cg_step_noalloc(4, p, None, p, p, p, None) == -1
    assert L.lssvm_cg_step_noalloc(8, p, q, p, q, p, None) == -1   # aliased vectors
    assert "overlap" in P.last_error()
