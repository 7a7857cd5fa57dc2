"""Plain-Python reader of LIBSVM-format data and model files (test infrastructure).

THIS IS TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT. Only the test suite may
import it. It shares no code with the native reader and writer and never
calls them.

The paper's training reads its data from LIBSVM-format files and writes the
learned support vectors and weights to a model file (Sec. III, the four
training steps; Sec. IV-E, "read" and "write"). The formats, as read here:

* data line: "<label> <index>:<value> ...", tokens separated by spaces, tabs
  or carriage returns, indices 1-based and strictly increasing, absent
  features 0, blank lines skipped;
* a number is an optional sign, then digits with an optional fraction and
  exponent, or inf / infinity / nan (any case);
* a value becomes the dtype element nearest to the exact decimal, ties to
  even (rounded once: for float32 the exact decimal is compared with the
  float32 neighbours, not rounded to float64 first);
* model file: "key value" header lines up to a line "SV", then one line per
  support vector "<coef> <index>:<value> ...". LIBSVM's binary decision value
  is sum_i coef_i k(sv_i, x) - rho, and it predicts the first listed label
  when that value is positive, the second otherwise.

Pins (tests/test_io_oracle.py): hand-written files whose dense content is
written out in the test, exact ties and near-ties of float32 rounding checked
with rational arithmetic, the float32 overflow threshold, and the LIBSVM
decision value of a written model checked against the oracle's f(x).
"""
from __future__ import annotations

import decimal
import re

import numpy as np

__all__ = ["FormatError", "parse_number", "read_data", "read_model", "libsvm_decision",
           "format_number"]

_NUMBER = r"[+-]?(?:(?:[0-9]+\.?[0-9]*|\.[0-9]+)(?:[eE][+-]?[0-9]+)?|inf(?:inity)?|nan)"
_NUMBER_RE = re.compile(_NUMBER, re.IGNORECASE)
_FEATURE_RE = re.compile(r"([0-9]+):(" + _NUMBER + r")", re.IGNORECASE)
_SEP_RE = re.compile(r"[ \t\r]+")

# values at or above max + half an ulp (= 2^128 - 2^103) round to infinity
_F32_OVERFLOW = decimal.Decimal(2**128 - 2**103)   # exact integer


class FormatError(ValueError):
    def __init__(self, line: int, what: str):
        super().__init__(f"line {line}: {what}")
        self.line = line


def _round_to_f32(tok: str) -> np.float32:
    """The float32 nearest to the exact decimal `tok`, ties to even."""
    with decimal.localcontext() as ctx:
        ctx.prec = 2000                  # exact for any float32 and short decimal
        exact = decimal.Decimal(tok)
        if exact.is_nan():
            return np.float32("nan")
        if exact.is_infinite() or abs(exact) >= _F32_OVERFLOW:
            return np.float32(np.copysign(np.inf, float(exact)))
        with np.errstate(over="ignore"):
            start = np.float32(float(exact))  # within one float32 step of the answer
            cands = {start, np.nextafter(start, np.float32(np.inf)),
                     np.nextafter(start, np.float32(-np.inf))}
        cands = [c for c in cands if np.isfinite(c)]
        best = None
        for c in cands:
            dist = abs(decimal.Decimal(float(c)) - exact)
            even = int(c.view(np.uint32)) & 1 == 0
            key = (dist, not even)
            if best is None or key < best[0]:
                best = (key, c)
        r = best[1]
        if r == 0 and exact.is_signed():
            r = np.float32(-0.0)
        return np.float32(r)


def parse_number(tok: str, dtype) -> np.floating:
    """One number token as dtype (float64 through Python's correctly rounded
    float(), float32 by exact comparison with its neighbours)."""
    if not _NUMBER_RE.fullmatch(tok):
        raise ValueError(f"not a number: {tok!r}")
    if np.dtype(dtype) == np.float32:
        return _round_to_f32(tok)
    return np.float64(float(tok))


def _lines(path):
    with open(path, "rb") as fh:
        text = fh.read().decode("latin-1")
    lines = text.split("\n")
    if lines and lines[-1] == "":
        lines.pop()
    return lines


def _parse_rows(lines, first_lineno, dtype):
    """(head, [(index, value), ...]) per non-blank line."""
    rows = []
    for k, line in enumerate(lines):
        lineno = first_lineno + k
        toks = [t for t in _SEP_RE.split(line) if t]
        if not toks:
            continue
        try:
            head = parse_number(toks[0], dtype)
        except ValueError:
            raise FormatError(lineno, "the first token is not a number") from None
        feats, prev = [], 0
        for t in toks[1:]:
            m = _FEATURE_RE.fullmatch(t)
            if not m:
                raise FormatError(lineno, f"bad feature token {t!r}")
            idx = int(m.group(1))
            if idx < 1 or idx <= prev:
                raise FormatError(lineno, "feature indices must start at 1 and increase")
            feats.append((idx, parse_number(m.group(2), dtype)))
            prev = idx
        rows.append((head, feats, lineno))
    return rows


def _dense(rows, d, dtype):
    if d is None:
        d = max((f[-1][0] for _, f, _ in rows if f), default=0)
    X = np.zeros((len(rows), d), dtype=dtype)
    heads = np.empty(len(rows), dtype=dtype)
    for i, (h, feats, lineno) in enumerate(rows):
        if feats and feats[-1][0] > d:
            raise FormatError(lineno, f"feature index {feats[-1][0]} exceeds d = {d}")
        heads[i] = h
        for idx, v in feats:
            X[i, idx - 1] = v
    return X, heads


def read_data(path, dtype=np.float64, d=None):
    """(X, y) of a data file, X dense n x d (d = largest index unless given)."""
    rows = _parse_rows(_lines(path), 1, dtype)
    return _dense(rows, d, dtype)


def read_model(path, dtype=np.float64):
    """Header dict plus support vectors X, coefficients coef and labels y."""
    lines = _lines(path)
    header = {}
    for k, line in enumerate(lines):
        toks = [t for t in _SEP_RE.split(line) if t]
        if not toks:
            continue
        if toks == ["SV"]:
            sv_start = k + 1
            break
        header[toks[0]] = toks[1:]
    else:
        raise FormatError(len(lines), "no SV section")
    rows = _parse_rows(lines[sv_start:], sv_start + 1, dtype)
    X, coef = _dense(rows, None, dtype)
    labels = [int(t) for t in header["label"]]
    nr_sv = [int(t) for t in header["nr_sv"]]
    if sum(nr_sv) != len(rows) or int(header["total_sv"][0]) != len(rows):
        raise FormatError(sv_start, "support vector count does not match the header")
    y = np.array([labels[0]] * nr_sv[0] + [labels[1]] * nr_sv[1], dtype=dtype)
    model = {
        "svm_type": header["svm_type"][0],
        "kernel_type": header["kernel_type"][0],
        "degree": int(header["degree"][0]) if "degree" in header else None,
        "gamma": float(header["gamma"][0]) if "gamma" in header else None,
        "coef0": float(header["coef0"][0]) if "coef0" in header else None,
        "nr_class": int(header["nr_class"][0]),
        "total_sv": int(header["total_sv"][0]),
        "rho": float(header["rho"][0]),
        "label": labels,
        "nr_sv": nr_sv,
    }
    return model, X, coef, y


def libsvm_decision(model, X_sv, coef, X_test):
    """LIBSVM's binary decision values sum_i coef_i k(sv_i, x) - rho and labels,
    with its kernels: u.v, (gamma u.v + coef0)^degree, exp(-gamma |u - v|^2)."""
    A = np.asarray(X_test, dtype=np.float64)
    S = np.asarray(X_sv, dtype=np.float64)
    kt = model["kernel_type"]
    if kt == "linear":
        K = A @ S.T
    elif kt == "polynomial":
        K = (model["gamma"] * (A @ S.T) + model["coef0"]) ** model["degree"]
    elif kt == "rbf":
        sq = ((A[:, None, :] - S[None, :, :]) ** 2).sum(axis=2)
        K = np.exp(-model["gamma"] * sq)
    else:
        raise ValueError(kt)
    dec = K @ np.asarray(coef, dtype=np.float64) - model["rho"]
    lab = np.where(dec > 0, model["label"][0], model["label"][1])
    return dec, lab


def format_number(v) -> str:
    """Shortest decimal text that reads back to v (float64 or float32)."""
    if isinstance(v, np.float32):
        return np.format_float_positional(v, unique=True, trim="-") \
            if 1e-4 <= abs(v) < 1e16 or v == 0 or not np.isfinite(v) \
            else np.format_float_scientific(v, unique=True, trim="-")
    return repr(float(v))
