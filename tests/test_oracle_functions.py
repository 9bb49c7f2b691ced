"""Pins of the oracle's benchmark functions (Problem.evaluate) and argmin.

Each function is pinned by closed forms at points where its value is known
analytically: optima, integer lattices where cos(2 pi k) = 1, half-integers
where cos(pi k) = -1, and small hand-worked vectors chosen so that a dropped
term, a wrong sign, a wrong index offset or a swapped neighbour changes the
value.  The argmin is pinned by brute force over all orderings of small
arrays with ties, signed zeros, infinities and NaNs.
"""
import itertools
import math

import numpy as np
import pytest

S, A, R, G, RB, SW = range(6)
E = math.e


def ev(ref, fn, rows):
    return ref.evaluate(fn, np.asarray(rows, dtype=np.float32))


def close(got, want, rel=2e-7, abs_=0.0):
    return abs(float(got) - want) <= max(rel * abs(want), abs_)


# ---------------- Sphere ----------------

def test_sphere_closed_forms(ref):
    assert ev(ref, S, np.zeros((1, 17)))[0] == 0.0
    assert ev(ref, S, np.full((1, 7), 3.0))[0] == 63.0
    k = np.array([[1, -2, 3, -4, 5]], np.float32)
    assert ev(ref, S, k)[0] == 55.0
    assert ev(ref, S, [[0.5] * 4])[0] == 1.0


# ---------------- Ackley ----------------

def ackley_lattice(k_abs_rms):
    # cos(2 pi k) = 1 for integer k: the second term is exp(1)
    return -20.0 * math.exp(-0.2 * k_abs_rms) - E + 20.0 + E


def test_ackley_optimum(ref):
    assert abs(ev(ref, A, np.zeros((1, 30)))[0]) <= 1e-15


@pytest.mark.parametrize("k", [1, 2, -3, 7])
def test_ackley_integer_lattice(ref, k):
    D = 11
    assert close(ev(ref, A, np.full((1, D), k))[0], ackley_lattice(abs(k)))


def test_ackley_mean_not_sum(ref):
    # x = (1, 0): mean x^2 = 1/2, mean cos = 1
    assert close(ev(ref, A, [[1.0, 0.0]])[0], 20.0 - 20.0 * math.exp(-0.2 * math.sqrt(0.5)))
    # x = (0.5, 0): mean x^2 = 1/8, mean cos = (-1 + 1)/2 = 0
    want = -20.0 * math.exp(-0.2 * math.sqrt(0.125)) - 1.0 + 20.0 + E
    assert close(ev(ref, A, [[0.5, 0.0]])[0], want)
    # all half-integers: mean cos = -1
    want = -20.0 * math.exp(-0.2 * 0.5) - math.exp(-1.0) + 20.0 + E
    assert close(ev(ref, A, np.full((1, 6), -0.5))[0], want)


# ---------------- Rastrigin ----------------

def test_rastrigin_closed_forms(ref):
    assert ev(ref, R, np.zeros((1, 13)))[0] == 0.0
    k = np.array([[1, -2, 3, 0, -5, 4]], np.float32)
    assert close(ev(ref, R, k)[0], float((k.astype(np.int64) ** 2).sum()), abs_=1e-9)
    # half-integers: each term 0.25 + 10 + 10 (A + x^2 - A cos(pi) ...)
    D = 9
    assert close(ev(ref, R, np.full((1, D), 0.5))[0], 20.25 * D)


def test_rastrigin_equals_the_textbook_sum(ref):
    """The oracle sums x^2 + 2A sin^2(pi x); the textbook form A D + sum(x^2 -
    A cos 2 pi x), computed here in fp64 with numpy's cosine, is the same
    function (it cancels, so compare within its own rounding scale)."""
    rng = np.random.default_rng(7)
    X = rng.uniform(-5.12, 5.12, size=(64, 301)).astype(np.float32)
    x = X.astype(np.float64)
    textbook = 10.0 * x.shape[1] + (x * x - 10.0 * np.cos(2.0 * np.pi * x)).sum(1)
    got = np.array([ref.lib().evox_ref_eval_row_f64(R, ref._ptr(np.ascontiguousarray(X[i])), X.shape[1])
                    for i in range(X.shape[0])])
    assert np.all(np.abs(got - textbook) <= 1e-12 * (20.0 * x.shape[1] + (x * x).sum(1)))


def test_rastrigin_near_the_optimum_is_relative_accurate(ref):
    """Near x = 0 each term is x^2 + 2A (pi x)^2 (1 - (pi x)^2 / 3 + ...): the
    fp32 value is within a few ulp of that expansion however small F is."""
    x = (np.arange(1, 41, dtype=np.float64) * 1e-4 * np.array([1, -1] * 20)).astype(np.float32)
    xd = x.astype(np.float64)
    y = np.pi * xd
    want = float((xd * xd + 20.0 * y * y * (1.0 - y * y / 3.0 + 2.0 * y ** 4 / 45.0)).sum())
    got = float(ev(ref, R, x[None, :])[0])
    assert abs(got - want) <= 2e-7 * want
    assert got > 0.0


# ---------------- Griewank ----------------

def test_griewank_optimum(ref):
    assert ev(ref, G, np.zeros((1, 50)))[0] == 0.0


@pytest.mark.parametrize("a", [0.75, 3.0, -10.5, 123.25])
def test_griewank_one_dimension_is_textbook(ref, a):
    assert close(ev(ref, G, [[a]])[0], 1.0 + a * a / 4000.0 - math.cos(a), abs_=1e-7)


def test_griewank_index_starts_at_one(ref):
    a = 2.5
    # only the second coordinate is nonzero: divisor sqrt(2)
    want = 1.0 + a * a / 4000.0 - math.cos(a / math.sqrt(2.0))
    assert close(ev(ref, G, [[0.0, a]])[0], want, abs_=1e-7)
    want3 = 1.0 + a * a / 4000.0 - math.cos(a / math.sqrt(3.0))
    assert close(ev(ref, G, [[0.0, 0.0, a]])[0], want3, abs_=1e-7)


def test_griewank_product_not_sum(ref):
    # cos(pi/2 * sqrt(i)/sqrt(i)) style zero: coordinate 1 = pi/2 makes the
    # product (nearly) zero whatever the others are
    x = np.array([[math.pi / 2, 1.0, 2.0]], np.float32)
    want = 1.0 + float((x.astype(np.float64) ** 2).sum()) / 4000.0
    assert close(ev(ref, G, x)[0], want, abs_=1e-6)


# ---------------- Rosenbrock ----------------

def test_rosenbrock_closed_forms(ref):
    assert ev(ref, RB, np.ones((1, 1000)))[0] == 0.0
    assert ev(ref, RB, np.zeros((1, 8)))[0] == 7.0
    assert ev(ref, RB, [[0.0]])[0] == 0.0          # D = 1: no pair
    assert ev(ref, RB, [[-1.0, 1.0]])[0] == 4.0
    assert ev(ref, RB, [[2.0, 4.0]])[0] == 1.0
    assert ev(ref, RB, [[2.0, 1.0]])[0] == 901.0   # 100 (1 - 4)^2 + (1 - 2)^2
    assert ev(ref, RB, [[1.0, 1.0, 2.0]])[0] == 100.0  # last pair counted


# ---------------- Schwefel ----------------

def test_schwefel_closed_forms(ref):
    D = 10
    assert close(ev(ref, SW, np.zeros((1, D)))[0], 418.9829 * D)
    # sqrt(x) = pi/2: sin = 1, the term equals x
    x = (math.pi / 2) ** 2
    assert close(ev(ref, SW, np.full((1, D), x))[0], 418.9829 * D - x * D, rel=1e-6)
    # odd in x: negative coordinates add instead of subtract
    assert close(ev(ref, SW, np.full((1, D), -x))[0], 418.9829 * D + x * D, rel=1e-6)
    # the known minimiser 420.9687: value ~ 1.27e-5 per dimension
    f = ref.eval_row_f64(SW, np.full(D, 420.9687, np.float32))
    assert 0.0 <= f / D < 1e-4


# ---------------- evaluation over rows / pitch ----------------

def test_evaluate_rows_are_independent(ref):
    rng = np.random.default_rng(5)
    X = rng.uniform(-3, 3, size=(9, 13)).astype(np.float32)
    for fn in range(6):
        whole = ref.evaluate(fn, X)
        single = np.array([ref.evaluate(fn, X[i:i + 1])[0] for i in range(9)])
        assert np.array_equal(whole, single)
        assert np.array_equal(whole, np.array([np.float32(ref.eval_row_f64(fn, X[i]))
                                               for i in range(9)]))


# ---------------- argmin ----------------

def brute_argmin(f):
    """Rank (class, value, index): class 0 for numbers, 1 for NaN."""
    keys = [((1, 0.0) if math.isnan(v) else (0, float(v)), i) for i, v in enumerate(f)]
    return min(keys)[1]


@pytest.mark.parametrize("vals", [
    [3.0, 1.0, 2.0, 1.0],
    [0.0, -0.0, 0.0],
    [-0.0, 0.0],
    [float("nan"), float("inf"), 5.0],
    [float("nan"), float("nan")],
    [float("inf"), float("inf"), float("nan")],
    [float("-inf"), 1.0, float("-inf")],
])
def test_argmin_all_orderings(ref, vals):
    for perm in set(itertools.permutations(range(len(vals)))):
        f = np.array([vals[p] for p in perm], np.float32)
        assert ref.argmin(f) == brute_argmin(f), f


def test_argmin_random_with_ties(ref):
    rng = np.random.default_rng(9)
    for _ in range(200):
        n = int(rng.integers(1, 60))
        f = rng.integers(-3, 4, size=n).astype(np.float32)
        f[rng.random(n) < 0.1] = np.nan
        assert ref.argmin(f) == brute_argmin(f)
