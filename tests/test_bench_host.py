"""Host-side parts of bench.py that need no GPU: the multi-GPU refusal, the
comment-blind kernel hash that ties committed counter runs to the code, the
traffic record's lookup and the CPU baseline's record on a tiny workload."""
from __future__ import annotations

import importlib.util
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_code_only_ignores_comments_and_layout():
    b = _bench()
    a = "int a = 1; // one\n/* two\n lines */ int b = 2;\n"
    assert b.code_only(a) == b.code_only("int  a = 1;\n\nint b = 2;")
    assert b.code_only(a) != b.code_only("int a = 1; int b = 3;")
    h = b.kernel_source_hash()
    assert len(h) == 16 and h == b.kernel_source_hash()


def test_traffic_record_matches_the_kernel_hash():
    b = _bench()
    assert b.traffic_record("no_such_workload") is None
    rec = b.traffic_record("poly_f32_32768x4096")
    # present exactly when the committed counter run was taken on this code
    import json
    with open(os.path.join(ROOT, "profiles", "k_tiles_poly_f32_32768x4096_traffic.json")) as fh:
        stored = json.load(fh)
    if stored["kernel_source_hash"] == b.kernel_source_hash():
        assert rec == stored["hbm_bytes_per_product"] and rec > 0
    else:
        assert rec is None


def test_cpu_baseline_record():
    b = _bench()
    sys.path.insert(0, ROOT)
    import synthdata as S
    cfg = S.Config("rbf_f64_300x20", "f64", "rbf", 300, 20, mu=1.0, inf_frac=0.5,
                   flip_frac=0.05, C=1.0, eps=1e-8, gamma=0.05)
    X, _, _ = S.make_train(cfg)
    rec = b.cpu_baseline(cfg, X, budget_s=0.5)
    assert rec["kind"] == "oracle" and rec["unit"] == "GFLOP/s" and rec["value"] > 0
    assert rec["cores"] >= 1 and "299 of 299 rows" in rec["sample"]
    host = rec["host"]
    assert host["cpus_available"] == len(os.sched_getaffinity(0))
    assert host["blas"] is None or isinstance(host["blas"], str)
    assert np.isfinite(rec["value"])
