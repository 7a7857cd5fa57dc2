"""GPU: lssvm_cg_step (one CG iteration's vector work, Sec. III-B) against
the oracle's cg_step, chained into a solve, on breakdown; and the matrix-core
loop probe."""
from __future__ import annotations

import numpy as np
import pytest

import oracle as O
import synthdata as S
from gpu_common import (GOLDEN, TOL_ALPHA, TOL_MV, SPLIT_SHAPES, TAIL_SHAPES, check_train,  # noqa: F401
                        data_of, golden, golden_tight, kw_of, labels_match, log, oracle_ref,
                        random_cases, random_large_cases, rel_err, small_cfg, spec_of,
                        to_dev)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("N", [1, 255, 256, 1000, 65537, 600_001, 1 << 22])
def test_cg_step_matches_oracle(torch_dev, N):
    """One step on random vectors, including lengths past the block cap
    of the vector kernels (grid-stride regime)."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    log(f"[cg_step] N={N}")
    rng = np.random.default_rng(N)
    x, r, d = (rng.standard_normal(N) for _ in range(3))
    q = d * rng.uniform(0.5, 2.0, N)            # d^T q > 0
    rr = float(r @ r)
    xo, ro, do, rro, go, ao, bo = O.cg_step(x, r, d, q, rr)
    t = [to_dev(torch, dev, a) for a in (x, r, d, q)]
    sc = torch.tensor([rr, 0.0, 0.0, 0.0], dtype=torch.float64, device=dev)
    P.cg_step(*t, sc)
    torch.cuda.synchronize()
    got = sc.cpu().numpy()
    for name, a, ref in (("x", t[0], xo), ("r", t[1], ro), ("d", t[2], do)):
        e = rel_err(a.cpu().numpy(), ref)
        assert e <= 1e-12, (name, e)
    np.testing.assert_array_equal(t[3].cpu().numpy(), q)          # q is only read
    for k, ref in enumerate((rro, go, ao, bo)):
        assert abs(got[k] - ref) <= 1e-12 * max(abs(ref), 1e-300), (k, got[k], ref)


def test_cg_step_chained_solves_spd_system(torch_dev):
    """Steps chained on the stream with q = A d from a plain fp64 product
    reach the oracle CG iterate and, run to convergence, the direct solve."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    rng = np.random.default_rng(4)
    n = 300
    M = rng.standard_normal((n, n))
    A = M @ M.T / n + np.eye(n)
    b = rng.standard_normal(n)
    Ad = to_dev(torch, dev, A)
    x = torch.zeros(n, dtype=torch.float64, device=dev)
    r = to_dev(torch, dev, b)
    d = r.clone()
    q = torch.empty_like(r)
    sc = torch.tensor([float(b @ b), 0, 0, 0], dtype=torch.float64, device=dev)
    ws = P.alloc_workspace(P.lib().lssvm_cg_step_workspace_bytes(n), dev)
    xo, ro, do, rro = np.zeros(n), b.copy(), b.copy(), float(b @ b)
    for k in range(15):              # well above rounding level: r^T r ~ 1e-13 r0^T r0
        torch.matmul(Ad, d, out=q)
        qo = A @ do
        P.cg_step(x, r, d, q, sc, workspace=ws)
        xo, ro, do, rro, *_ = O.cg_step(xo, ro, do, qo, rro)
    torch.cuda.synchronize()
    assert rel_err(x.cpu().numpy(), xo) <= 1e-9
    assert abs(sc[0].item() - rro) <= 1e-6 * rro
    for k in range(25):
        torch.matmul(Ad, d, out=q)
        P.cg_step(x, r, d, q, sc, workspace=ws)
    torch.cuda.synchronize()
    np.testing.assert_allclose(x.cpu().numpy(), np.linalg.solve(A, b), rtol=1e-10, atol=1e-12)


def test_cg_step_breakdown_keeps_vectors(torch_dev):
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    n = 5000
    x = torch.ones(n, dtype=torch.float64, device=dev)
    r = torch.full((n,), 2.0, dtype=torch.float64, device=dev)
    d = torch.ones(n, dtype=torch.float64, device=dev)
    q = -torch.ones(n, dtype=torch.float64, device=dev)          # d^T q < 0
    sc = torch.tensor([7.0, 0, 0, 0], dtype=torch.float64, device=dev)
    P.cg_step(x, r, d, q, sc)
    torch.cuda.synchronize()
    assert torch.all(x == 1.0) and torch.all(r == 2.0) and torch.all(d == 1.0)
    got = sc.cpu().numpy()
    assert got[0] == 7.0 and got[1] == -float(n) and got[3] == 0.0


@pytest.mark.parametrize("dtype,published", [("float32", 157.3), ("float64", 78.6)])
def test_mfma_peak_probe_is_plausible(torch_dev, dtype, published):
    """The measured matrix-core loop rate lies near the published peak (one
    resident round of back-to-back MFMAs sustains ~99% of it on gfx950) and
    not above it (a probe that lost its work would report far more)."""
    torch, dev = torch_dev
    import paper_2202_12674_amd as P
    tf = P.mfma_peak(getattr(torch, dtype), dev)
    log(f"[mfma peak] {dtype}: {tf:.1f} TFLOP/s (published {published})")
    assert 0.9 * published < tf < 1.02 * published
