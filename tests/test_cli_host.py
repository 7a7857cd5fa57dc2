"""Command-line tools (lssvm-train, lssvm-predict): the paths that end before
any GPU work — usage errors, unreadable or empty inputs, malformed models, and
prediction of an empty test file."""
from __future__ import annotations

import os
import subprocess

import pytest

import paper_2202_12674_amd as P  # noqa: F401  (the package builds the tools with the library)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BIN = os.path.join(ROOT, "paper_2202_12674_amd", "bin")
TRAIN = os.path.join(BIN, "lssvm-train")
PREDICT = os.path.join(BIN, "lssvm-predict")

MODEL = ("svm_type c_svc\nkernel_type rbf\ngamma 0.5\nnr_class 2\ntotal_sv 2\nrho 0.1\n"
         "label 1 -1\nnr_sv 1 1\nSV\n0.5 1:1 2:-1\n-0.5 1:-1\n")


def run(*args):
    if not os.path.exists(TRAIN) or not os.path.exists(PREDICT):
        pytest.skip("tools not built")
    return subprocess.run(list(args), capture_output=True, text=True, timeout=60)


@pytest.mark.parametrize("argv", [
    [], ["-t", "3", "f"], ["-t", "x", "f"], ["-c", "0", "f"], ["-c", "-1", "f"],
    ["-e", "0", "f"], ["-e", "1", "f"], ["-g", "0", "f"], ["-g", "-2", "f"], ["-d", "0", "f"],
    ["-p", "16", "f"], ["-i", "-1", "f"], ["-T", "-1", "f"], ["-z", "1", "f"], ["-c"],
    ["a", "b", "c"], ["-cc", "1", "f"],
])
def test_train_usage_errors(argv):
    r = run(TRAIN, *argv)
    assert r.returncode == 2 and "Usage: lssvm-train" in r.stderr


def test_train_unreadable_and_empty(tmp_path):
    r = run(TRAIN, str(tmp_path / "missing.libsvm"))
    assert r.returncode == 1 and "cannot open" in r.stderr
    empty = tmp_path / "empty.libsvm"
    empty.write_text("\n\n")
    r = run(TRAIN, str(empty))
    assert r.returncode == 1 and "no data points" in r.stderr
    bad = tmp_path / "bad.libsvm"
    bad.write_text("1 1:1\n-1 2:1 1:3\n")
    r = run(TRAIN, str(bad))
    # the full parse runs into pinned host memory, so without a device the
    # allocation fails first; with one, the parse names line 2
    assert r.returncode == 1 and (":2:" in r.stderr or "host allocation" in r.stderr)


@pytest.mark.parametrize("argv", [[], ["a", "b"], ["-p", "8", "a", "b", "c"], ["-x", "a", "b", "c"],
                                  ["a", "b", "c", "d"]])
def test_predict_usage_errors(argv):
    r = run(PREDICT, *argv)
    assert r.returncode == 2 and "Usage: lssvm-predict" in r.stderr


def test_predict_bad_model_and_empty_test(tmp_path):
    test = tmp_path / "t.libsvm"
    test.write_text("")
    model = tmp_path / "m.model"
    model.write_text(MODEL.replace("nr_class 2", "nr_class 3"))
    r = run(PREDICT, str(test), str(model), str(tmp_path / "out"))
    assert r.returncode == 1 and "nr_class" in r.stderr
    model.write_text(MODEL)
    out = tmp_path / "out"
    r = run(PREDICT, str(test), str(model), str(out))   # no test points: no device work
    assert r.returncode == 0, r.stderr
    assert out.read_text() == ""
    r = run(PREDICT, str(tmp_path / "missing"), str(model), str(out))
    assert r.returncode == 1 and "cannot open" in r.stderr
