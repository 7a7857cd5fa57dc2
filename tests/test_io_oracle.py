"""Pins of the plain-Python LIBSVM-format reader in oracle/libsvm_format.py.

The expected values here come from the format's definition written out by
hand (tests/golden/libsvm_small.txt, tests/golden/model_small.txt) and from
exact rational arithmetic on float32 neighbours, never from the reader's own
code paths.
"""
from __future__ import annotations

import decimal
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import libsvm_format as L
import oracle as O

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

# Dense content of libsvm_small.txt, written out from the file by hand: five
# points (lines 1, 3, 4, 6, 7; lines 2 and 5 are blank), largest index 5.
SMALL_X = np.array([
    [0.5, 0.0, -0.25, 0.0, 0.0],
    [0.0, 100.0, 0.0, 7.0, 0.0],
    [0.0, 0.0, 0.0, 0.0, 0.0],
    [0.0, 0.0, -0.0, 0.0, 0.25],
    [1.0, -3.0, 0.0, 0.0, 4.0],
])
SMALL_Y = np.array([1.0, -1.0, 1.0, -1.0, 1.0])


def _exact_decimal(fr: Fraction) -> str:
    """Exact decimal text of a dyadic rational."""
    with decimal.localcontext() as ctx:
        ctx.prec = 2000
        return format(decimal.Decimal(fr.numerator) / decimal.Decimal(fr.denominator), "f")


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_golden_small_file(dtype):
    X, y = L.read_data(os.path.join(GOLDEN, "libsvm_small.txt"), dtype)
    assert X.dtype == dtype and X.shape == (5, 5)
    np.testing.assert_array_equal(X, SMALL_X.astype(dtype))
    np.testing.assert_array_equal(y, SMALL_Y.astype(dtype))
    assert np.signbit(X[3, 2])          # "-0" keeps its sign
    X7, _ = L.read_data(os.path.join(GOLDEN, "libsvm_small.txt"), dtype, d=7)
    np.testing.assert_array_equal(X7[:, :5], SMALL_X)
    assert not X7[:, 5:].any()


def test_f32_ties_and_near_ties_follow_round_to_nearest_even():
    rng = np.random.default_rng(7)
    bits = rng.integers(0x00800000, 0x7F000000, size=200, dtype=np.int64).astype(np.uint32)
    for a in bits.view(np.float32):
        b = np.nextafter(a, np.float32(np.inf))
        mid = (Fraction(float(a)) + Fraction(float(b))) / 2
        even = a if int(a.view(np.uint32)) % 2 == 0 else b
        tiny = Fraction(float(b) - float(a)) / 10**12
        assert L.parse_number(_exact_decimal(mid), np.float32) == even
        assert L.parse_number(_exact_decimal(mid + tiny), np.float32) == b
        assert L.parse_number(_exact_decimal(mid - tiny), np.float32) == a
        assert L.parse_number("-" + _exact_decimal(mid + tiny), np.float32) == -b


def test_f32_rounds_once_not_through_float64():
    # 1 + 2^-24 is the midpoint of 1 and 1 + 2^-23; a decimal 1e-28 above it
    # rounds to the upper neighbour, while rounding to float64 first would land
    # on the midpoint and then tie to 1.0
    assert L.parse_number("1.0000000596046447753906250001", np.float32) == np.float32(1 + 2**-23)
    assert L.parse_number("1.000000059604644775390625", np.float32) == np.float32(1.0)


def test_f32_overflow_and_subnormal_limits():
    big = Fraction(2) ** 128 - Fraction(2) ** 103      # max float32 + half an ulp
    assert np.isposinf(L.parse_number(_exact_decimal(big), np.float32))
    below = big - Fraction(1)
    assert L.parse_number(_exact_decimal(below), np.float32) == np.finfo(np.float32).max
    tiny = Fraction(1, 2**149)                         # smallest subnormal
    assert L.parse_number(_exact_decimal(tiny), np.float32) == np.float32(2.0**-149)
    assert L.parse_number(_exact_decimal(tiny / 2), np.float32) == 0.0      # tie to even 0
    assert L.parse_number(_exact_decimal(tiny / 2 + tiny / 1000), np.float32) == \
        np.float32(2.0**-149)
    assert np.signbit(L.parse_number("-1e-60", np.float32))


def test_f64_midpoints():
    mid = Fraction(1) + Fraction(1, 2**53)
    assert L.parse_number(_exact_decimal(mid), np.float64) == 1.0
    assert L.parse_number(_exact_decimal(mid + Fraction(1, 2**80)), np.float64) == 1 + 2**-52


@pytest.mark.parametrize("tok", ["1", "-2.5", "+3", ".5", "5.", "1e3", "1E-3", "-1.5e+2",
                                 "inf", "-Infinity", "NaN"])
def test_number_grammar_accepts(tok):
    L.parse_number(tok, np.float64)


@pytest.mark.parametrize("tok", ["", ".", "e3", "1e", "--1", "+-1", "1_0", "0x10", "1,5", "i"])
def test_number_grammar_rejects(tok):
    with pytest.raises(ValueError):
        L.parse_number(tok, np.float64)


@pytest.mark.parametrize("text,line", [
    ("1 1:1\n1 2:1 2:3\n", 2),             # repeated index
    ("1 3:1 2:1\n", 1),                    # decreasing
    ("1 1:1\n\n1 0:4\n", 3),               # index 0
    ("1 1:\n", 1), ("1 1:x\n", 1), ("x 1:1\n", 1), ("1 1 :2\n", 1), ("1 1:2:3\n", 1),
    ("1 +1:2\n", 1),
])
def test_malformed_lines_name_their_line(tmp_path, text, line):
    p = tmp_path / "bad.txt"
    p.write_text(text)
    with pytest.raises(L.FormatError) as e:
        L.read_data(p)
    assert e.value.line == line


def test_index_beyond_given_d(tmp_path):
    p = tmp_path / "d.txt"
    p.write_text("1 1:1\n-1 4:2\n")
    with pytest.raises(L.FormatError) as e:
        L.read_data(p, d=3)
    assert e.value.line == 2


def test_golden_model_and_libsvm_decision():
    model, X, coef, y = L.read_model(os.path.join(GOLDEN, "model_small.txt"))
    assert model["kernel_type"] == "linear" and model["rho"] == 0.5
    assert model["label"] == [1, -1] and model["nr_sv"] == [2, 1]
    np.testing.assert_array_equal(X, [[1, 2, 0], [0, -1, 4], [2, 0, 1]])
    np.testing.assert_array_equal(coef, [0.25, 0.5, -0.75])
    np.testing.assert_array_equal(y, [1, 1, -1])
    # decision values worked out by hand: k = (3,3,3), (1,0,2), (0,4,1)
    Xt = np.array([[1.0, 1.0, 1.0], [1.0, 0.0, 0.0], [0.0, 0.0, 1.0]])
    dec, lab = L.libsvm_decision(model, X, coef, Xt)
    np.testing.assert_array_equal(dec, [-0.5, -1.75, 0.75])
    np.testing.assert_array_equal(lab, [-1, -1, 1])


@pytest.mark.parametrize("kernel,kt", [("linear", "linear"), ("poly", "polynomial"),
                                       ("rbf", "rbf")])
def test_libsvm_decision_is_the_lssvm_decision(kernel, kt):
    """A model with coef = alpha, rho = -b and labels (1, -1) makes LIBSVM's
    decision value the LS-SVM f(x) (Eq. (10), alpha carrying the sign)."""
    rng = np.random.default_rng(3)
    X = rng.uniform(-1, 1, (40, 6))
    alpha = rng.standard_normal(40)
    b = 0.37
    Xt = rng.uniform(-1, 1, (25, 6))
    spec = O.KernelSpec(kernel, gamma=0.3, coef0=0.5, degree=3)
    model = {"kernel_type": kt, "gamma": 0.3, "coef0": 0.5, "degree": 3, "rho": -b,
             "label": [1, -1]}
    dec, lab = L.libsvm_decision(model, X, alpha, Xt)
    f, lab_o = O.predict(X, alpha, b, Xt, spec)
    np.testing.assert_allclose(dec, f, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(lab, lab_o)
