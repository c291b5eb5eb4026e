"""Pins for the oracle's canonical fp32 primitives: summation order, exp, log,
quantization rounding and the length penalty."""
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


@pytest.mark.parametrize("row", _rows("canon_sum_order.txt"), ids=lambda r: r[0])
def test_canon_sum_worked_examples(row):
    _, n, x0, rest, expected = row
    x = np.full(int(n), np.float32(float(rest)), np.float32)
    x[0] = np.float32(float(x0))
    assert oracle.canon_sum(x) == np.float32(float(expected))


def _vocab_cases():
    path = os.path.join(os.path.dirname(__file__), "golden", "canon_vocab_sum_order.txt")
    rows = []
    for line in open(path):
        line = line.strip()
        if line and not line.startswith("#"):
            rows.append(line.split())
    return rows


@pytest.mark.parametrize("row", _vocab_cases(), ids=lambda r: r[0])
def test_canon_vocab_sum_worked_examples(row):
    """The vocabulary sum of the beam search's log-sum-exp (reading R2b)
    against hand-derived values; each case also differs from the wave64 order."""
    _, n, default, entries, expected = row
    x = np.full(int(n), np.float32(float(default)), np.float32)
    for e in entries.split(","):
        i, v = e.split(":")
        x[int(i)] = np.float32(float(v))
    assert oracle.canon_vocab_sum(x) == np.float32(float(expected))
    assert oracle.canon_sum(x) != np.float32(float(expected))


def test_canon_vocab_sum_exact_on_integers_and_error_bound():
    rng = np.random.default_rng(3)
    for n in (1, 5, 2048, 2051, 32000, 32768):
        xi = rng.integers(-1000, 1000, size=n).astype(np.float32)
        assert oracle.canon_vocab_sum(xi) == np.float32(xi.astype(np.int64).sum())
        x = rng.standard_normal(n).astype(np.float32)
        exact = math.fsum(float(v) for v in x)
        depth = -(-n // 2048) * 4 + 6 + 3  # terms per partial, halving, tree
        bound = depth * 2.0 ** -24 * float(np.abs(x).sum())
        assert abs(float(oracle.canon_vocab_sum(x)) - exact) <= bound
    assert oracle.canon_vocab_sum(np.zeros(0, np.float32)) == 0.0


def test_canon_sum_exact_on_integers_and_error_bound():
    rng = np.random.default_rng(1)
    for n in (1, 7, 63, 64, 65, 256, 1000, 32000):
        xi = rng.integers(-1000, 1000, size=n).astype(np.float32)  # exact partial sums
        assert oracle.canon_sum(xi) == np.float32(xi.astype(np.int64).sum())
        x = rng.standard_normal(n).astype(np.float32)
        exact = math.fsum(float(v) for v in x)
        # each term passes through at most ceil(n/64) + 6 roundings
        depth = -(-n // 64) + 6
        bound = depth * 2.0 ** -24 * float(np.abs(x).sum())
        assert abs(float(oracle.canon_sum(x)) - exact) <= bound


def test_canon_sum_empty_and_signed_zero():
    assert oracle.canon_sum(np.zeros(0, np.float32)) == 0.0
    s = oracle.canon_sum(np.array([-0.0], np.float32))
    assert s == 0.0 and not np.signbit(s)  # partials start at +0


def _ulp_err(y, exact):
    e32 = exact.astype(np.float32)
    return np.abs(y.astype(np.float64) - exact) / np.spacing(np.abs(e32)).astype(np.float64)


def test_exp_sweep_ulp():
    # every 61st fp32 value in [-87, 0]: ~9e6 points... sampled to 1.7e7/61
    lo = np.float32(-87.0).view(np.uint32)
    bits = np.arange(0, lo + 1, 61, dtype=np.uint32) | np.uint32(0x80000000)
    x = bits.view(np.float32)
    x = x[x >= -87.0]
    y = oracle.exp_array(x)
    err = _ulp_err(y, np.exp(x.astype(np.float64)))
    assert err.max() <= 2.0, err.max()


def test_exp_special_values():
    assert oracle.exp(0.0) == 1.0
    assert oracle.exp(-0.0) == 1.0
    assert oracle.exp(-87.5) == 0.0
    assert oracle.exp(-1000.0) == 0.0
    # near x = k ln2 the result is 2^k up to the rounding of x itself
    for k in range(-120, 1, 7):
        x = np.float32(k * math.log(2))
        y = oracle.exp(x)
        assert abs(y / 2.0 ** k - 1.0) <= abs(float(x) - k * math.log(2)) + 3e-7
    x = np.linspace(-20, 0, 200001, dtype=np.float32)
    y = oracle.exp_array(x)
    assert np.all(np.diff(y) >= 0)  # monotone on a dense grid


def test_log_sweep_ulp():
    one = np.float32(1.0).view(np.uint32)
    top = np.float32(1e6).view(np.uint32)
    bits = np.arange(one, top, 37, dtype=np.uint32)
    x = bits.view(np.float32)
    y = oracle.log_array(x)
    exact = np.log(x.astype(np.float64))
    nz = exact != 0
    err = _ulp_err(y[nz], exact[nz])
    # the series in f = (m - 1)/(m + 1) carries the rounding of m + 1 and of the
    # division: up to ~3 ulp just above 1, well under 1 ulp elsewhere
    assert err.max() <= 3.0, err.max()
    assert np.percentile(err, 99) <= 1.0
    # below 1 as well
    bits = np.arange(np.float32(1e-30).view(np.uint32), one, 997, dtype=np.uint32)
    x = bits.view(np.float32)
    err = _ulp_err(oracle.log_array(x), np.log(x.astype(np.float64)))
    assert err.max() <= 3.0, err.max()


def test_log_special_values():
    assert oracle.log(1.0) == 0.0
    for k in range(-100, 101, 9):
        y = oracle.log(np.float32(2.0) ** k)
        assert abs(y - k * math.log(2)) <= 1e-6 * max(1.0, abs(k))
    assert abs(oracle.log(math.e) - 1.0) < 2e-7


@pytest.mark.parametrize("row", _rows("quantize_ties.txt"), ids=lambda r: r[0])
def test_quantize_tie_table(row):
    y, expected = float(row[0]), int(row[1])
    assert oracle.quantize(np.float32(y), 1.0) == expected


def test_quantize_roundtrip_all_codes():
    # a code times its scale quantizes back to itself (255 codes, several scales)
    for s in (0.02, 0.031496062, 1.0 / 127, 3.7e-3, 0.25):
        inv = np.float32(1.0 / s)
        for c in range(-127, 128):
            assert oracle.quantize(np.float32(c) * np.float32(s), inv) == c


def test_quantize_vs_float64():
    rng = np.random.default_rng(3)
    y = (rng.standard_normal(20000) * 60).astype(np.float32)
    inv = np.float32(1.0 / 0.7)
    q = np.array([oracle.quantize(v, inv) for v in y])
    prod = (y * inv).astype(np.float64)  # the fp32 product, as the oracle forms it
    ref = np.clip(np.round(prod), -127, 127)  # numpy rounds half to even
    assert np.array_equal(q, ref)
    ref64 = np.clip(np.round(y.astype(np.float64) / 0.7), -127, 127)
    assert np.abs(q - ref64).max() <= 1  # differs only right at .5 boundaries


def test_length_penalty_closed_form():
    for L in (1, 2, 7, 30, 64, 80):
        for a in (0.0, 0.6, 1.0):
            v = oracle.length_penalty(L, a)
            a32 = float(np.float32(a))  # alpha travels as fp32
            assert v == np.float32(((5.0 + L) / 6.0) ** a32)
    assert oracle.length_penalty(1, 0.6) == 1.0  # ((5 + 1) / 6)^a = 1


@pytest.mark.parametrize("row", _rows("canon_sum_squares.txt"), ids=lambda r: r[0])
def test_canon_sum_squares_worked_examples(row):
    # the variance sum accumulates each square with one fused multiply-add
    n, x0, xm, xl, expected = int(row[1]), float(row[2]), float(row[3]), float(row[4]), float(row[5])
    x = np.full(n, xm, np.float32)
    x[0], x[-1] = x0, xl
    assert oracle.canon_sum_squares(x) == np.float32(expected)


def test_length_penalty_exact_values():
    # ((5 + L) / 6)^alpha at points where the closed form is known exactly
    for L, a, v in ((1, 0.6, 1.0), (7, 1.0, 2.0), (13, 1.0, 3.0), (19, 0.5, 2.0), (31, 0.5, math.sqrt(6.0)),
                    (91, 0.25, 2.0), (187, 0.2, 2.0), (40, 0.0, 1.0)):
        assert oracle.length_penalty(L, a) == np.float32(v), (L, a)
    # 2^0.6 = exp(0.6 ln 2) = 1.51571656651039808...: L = 7 gives base 2
    assert oracle.length_penalty(7, 0.6) == np.float32(1.5157165665103981)
    # monotone in L for alpha > 0
    vals = [oracle.length_penalty(L, 0.6) for L in range(1, 100)]
    assert all(b > a for a, b in zip(vals, vals[1:]))
