"""GPU: the library loaded through the file-IO module in a fresh process,
before anything else imported torch, still reaches the device (torch's HIP
runtime must be the one the library binds to). Runs in a child process so
that the order of loading is the one under test."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import sys
sys.path.insert(0, sys.argv[1])
from paper_2202_12674_amd import files            # loads the library first
files.lib() if hasattr(files, "lib") else None
import paper_2202_12674_amd as P
P.lib()
import torch
assert torch.cuda.is_available()
X = torch.randn(64, 8, dtype=torch.float64, device="cuda")
y = torch.where(X[:, 0] > 0, 1.0, -1.0).to(torch.float64)
r = P.train(X, y, kernel="rbf", gamma=0.1, eps=1e-8)
print("ok", r.iterations)
"""


def test_library_loaded_before_torch_reaches_the_device():
    print("[load order] child process", flush=True)
    r = subprocess.run([sys.executable, "-c", CHILD, ROOT], capture_output=True, text=True,
                       timeout=240)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("ok")
