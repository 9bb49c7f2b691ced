"""Pins of the oracle's CSO generation.

The permutation is pinned against a library sort of rocRAND's Philox keys
and, at N = 4, by a chi-square test over all 24 orderings.  Degenerate
parameters expose the loser update (v = 0, x_l = 0, x_w = 1, phi = 0 gives
v_l = R2 exactly, R2 recomputed from rocRAND).  A two-particle generation is
worked by hand, and invariants (winners untouched, exactly floor(N/2)
losers, the best never gets worse, resumption) are checked on random runs.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

from conftest import u01_exact

GRIEWANK = 3


def keys_from_rocrand(rocrand_philox, seed, t, N):
    rows = [(seed, i // 4, 0, t, 4) for i in range(N)]
    words = rocrand_philox(rows)
    return np.array([words[i, i % 4] for i in range(N)], dtype=np.uint32)


@pytest.mark.parametrize("N,t", [(1, 0), (2, 3), (17, 0), (1000, 7)])
def test_perm_is_sorted_rocrand_keys(ref, rocrand_philox, N, t):
    seed = 99
    keys = keys_from_rocrand(rocrand_philox, seed, t, N)
    want = np.lexsort((np.arange(N), keys))      # by key, then by index
    got = ref.perm(seed, t, N)
    assert np.array_equal(got, want)
    assert np.array_equal(np.sort(got), np.arange(N))


def test_perm_uniform_over_24_orderings(ref):
    counts = {}
    n = 0
    for seed in range(60):
        for t in range(40):
            key = tuple(ref.perm(seed, t, 4).tolist())
            counts[key] = counts.get(key, 0) + 1
            n += 1
    assert len(counts) == 24
    expected = n / 24
    chi2 = sum((c - expected) ** 2 / expected for c in counts.values())
    # 23 degrees of freedom: P(chi2 > 49.7) ~ 0.001
    assert chi2 < 49.7, chi2


def test_colmean_exact(ref):
    rng = np.random.default_rng(4)
    X = rng.uniform(-600, 600, size=(501, 7)).astype(np.float32)
    got = ref.colmean(X)
    for j in range(7):
        exact = sum(Fraction(float(v)) for v in X[:, j]) / X.shape[0]
        want = np.float32(float(exact))
        assert abs(int(got[j].view(np.int32)) - int(want.view(np.int32))) <= 1
    Y = np.array([[1.0, 2.0], [2.0, 2.0], [4.0, -3.0]], np.float32)
    assert ref.colmean(Y).tolist() == [np.float32(7 / 3), np.float32(1 / 3)]


def fresh(ref, N, D, seed=5, fn=GRIEWANK, **kw):
    P = ref.make_params(fn, N, D, -600.0, 600.0, seed=seed, **kw)
    return ref.CSO(P)


def test_loser_velocity_equals_r2(ref, rocrand_philox):
    N, D, seed = 12, 6, 31
    s = fresh(ref, N, D, seed=seed, phi=0.0)
    winners_side = np.arange(N) % 2 == 0
    s.x[:] = np.where(winners_side[:, None], 1.0, 0.0).astype(np.float32)
    s.fit[:] = np.where(winners_side, 0.0, 1.0).astype(np.float32)
    s.v[:] = 0.0
    perm = ref.perm(seed, 0, N)
    f0 = s.fit.copy()
    s.step(1)
    for k in range(N // 2):
        a, b = perm[2 * k], perm[2 * k + 1]
        w, l = (b, a) if f0[b] < f0[a] else (a, b)
        rows = [(seed, 3 * (j // 4) + 1, l, 0, 3) for j in range(D)]
        words = rocrand_philox(rows)
        R2 = u01_exact([words[j, j % 4] for j in range(D)])
        gap = np.float32(1.0) if winners_side[w] and not winners_side[l] else np.float32(0.0)
        assert np.array_equal(s.v[l], (R2 * gap).astype(np.float32)), (k, w, l)
        assert np.array_equal(s.x[w], np.full(D, 1.0 if winners_side[w] else 0.0, np.float32))


def test_hand_worked_generation(ref, rocrand_philox):
    seed, phi = 8, 0.25
    s = fresh(ref, 2, 1, seed=seed, fn=0, phi=phi)    # Sphere
    s.x[:] = [[0.0], [1.0]]
    s.v[:] = [[0.0], [0.5]]
    s.fit[:] = [0.0, 1.0]
    s.step(1)
    # particle 1 loses whatever the order; mean = 0.5
    rows = [(seed, k, 1, 0, 3) for k in range(3)]
    words = rocrand_philox(rows)
    R1, R2, R3 = (u01_exact([words[k, 0]])[0] for k in range(3))
    t0 = np.float32(R1 * np.float32(0.5))
    t1 = np.float32(np.float64(R2) * -1.0 + np.float64(t0))      # fma(R2, 0 - 1, t0)
    c = np.float32(np.float32(phi) * R3)
    vn = np.float32(np.float64(c) * -0.5 + np.float64(t1))       # fma(c, 0.5 - 1, t1)
    assert s.v[1, 0] == vn
    assert s.x[1, 0] == np.float32(np.float32(1.0) + vn)
    assert s.fit[1] == np.float32(float(s.x[1, 0]) ** 2)
    assert s.x[0, 0] == 0.0 and s.v[0, 0] == 0.0 and s.fit[0] == 0.0
    assert s.best_idx == 0 and s.best_fit == 0.0


@pytest.mark.parametrize("N", [2, 9, 64])
def test_winners_untouched_and_loser_count(ref, N):
    s = fresh(ref, N, 5, v_lo=-1.0, v_hi=1.0)
    for _ in range(6):
        x0, v0, f0 = s.x.copy(), s.v.copy(), s.fit.copy()
        s.step(1)
        losers = s.loser.astype(bool)
        assert losers.sum() == N // 2
        assert np.array_equal(s.x[~losers], x0[~losers])
        assert np.array_equal(s.v[~losers], v0[~losers])
        assert np.array_equal(s.fit[~losers], f0[~losers])
        assert np.array_equal(ref.evaluate(GRIEWANK, s.x), s.fit)


def test_best_never_worse(ref):
    s = fresh(ref, 40, 8)
    prev = s.fit.min()
    for _ in range(30):
        s.step(1)
        assert s.best_fit <= prev and s.best_fit == s.fit.min()
        assert s.best_idx == int(np.argmin(s.fit))
        prev = s.best_fit


def test_converges_on_griewank(ref):
    s = fresh(ref, 200, 10, seed=3)
    start = s.fit.min()
    s.step(150)
    assert s.best_fit < 0.05 * start


def test_resume_is_bit_exact(ref):
    a, b = fresh(ref, 31, 6), fresh(ref, 31, 6)
    a.step(9)
    b.step(4)
    b.step(5)
    for name in ("x", "v", "fit"):
        assert np.array_equal(getattr(a, name), getattr(b, name)), name
    assert (a.best_fit, a.best_idx, a.t) == (b.best_fit, b.best_idx, b.t)


def test_argsort_is_a_stable_sort(ref):
    """The sort under the pairing, pinned to numpy's stable argsort, on keys
    with heavy ties, all-equal keys, extremes and random words."""
    rng = np.random.default_rng(77)
    cases = [rng.integers(0, 16, size=5000), np.full(3000, 7), np.array([2**32 - 1, 0, 2**32 - 1, 0, 5]),
             rng.integers(0, 2**32, size=20000, dtype=np.uint64), np.arange(100)[::-1], np.zeros(0)]
    for keys in cases:
        keys = np.asarray(keys, dtype=np.uint32)
        assert np.array_equal(ref.argsort_u32(keys), np.argsort(keys, kind="stable"))


# ---- the neighbourhood version (the loser learns from its ring neighbourhood's mean) ----

def test_ring_mean_hand_worked(ref):
    X = np.array([[0.0], [3.0], [6.0], [9.0]], np.float32)
    assert ref.ring_mean(X)[:, 0].tolist() == [4.0, 3.0, 6.0, 5.0]     # (9+0+3)/3, (0+3+6)/3, ...
    Y = np.array([[1.0, 2.0], [2.0, 2.0], [4.0, -3.0]], np.float32)     # N = 3: every ring is the swarm
    assert np.array_equal(ref.ring_mean(Y), np.repeat(ref.colmean(Y)[None], 3, axis=0))


def test_three_individuals_local_equals_global(ref):
    a = fresh(ref, 3, 9, seed=12, cso_local=0)
    b = fresh(ref, 3, 9, seed=12, cso_local=1)
    for _ in range(6):
        a.step(1)
        b.step(1)
        assert np.array_equal(a.x, b.x) and np.array_equal(a.v, b.v) and np.array_equal(a.fit, b.fit)


def test_loser_learns_from_its_ring_mean(ref, rocrand_philox):
    """v = 0: v_l' = R2 (x_w - x_l) + phi R3 (m_l - x_l), so m_l is decoded from
    the update with rocRAND's words and must be the mean of rows l - 1, l, l + 1
    (wrapping), which here is far from the swarm mean."""
    N, D, seed, phi = 10, 3, 13, 0.5
    s = fresh(ref, N, D, seed=seed, phi=phi, cso_local=1)
    x0 = (np.arange(N, dtype=np.float32)[:, None] ** 2 * np.array([1.0, -2.0, 0.5], np.float32)).astype(np.float32)
    s.x[:] = x0
    s.v[:] = 0.0
    s.fit[:] = np.arange(N, dtype=np.float32)[::-1]
    perm = ref.perm(seed, 0, N)
    f0 = s.fit.copy()
    s.step(1)
    ring = (np.roll(x0, 1, 0).astype(np.float64) + x0 + np.roll(x0, -1, 0)) / 3
    glob = x0.astype(np.float64).mean(0)
    for k in range(N // 2):
        a, b = perm[2 * k], perm[2 * k + 1]
        w, l = (b, a) if f0[b] < f0[a] else (a, b)
        words = rocrand_philox([(seed, 3 * (j // 4) + q, l, 0, 3) for j in range(D) for q in (1, 2)])
        R2 = u01_exact([words[2 * j, j % 4] for j in range(D)]).astype(np.float64)
        R3 = u01_exact([words[2 * j + 1, j % 4] for j in range(D)]).astype(np.float64)
        xl, xw = x0[l].astype(np.float64), x0[w].astype(np.float64)
        m = xl + (s.v[l].astype(np.float64) - R2 * (xw - xl)) / (np.float32(phi) * R3)
        scale = np.abs(xl) + np.abs(xw) + np.abs(ring[l]) + 1
        assert np.all(np.abs(m - ring[l]) <= 1e-5 * scale / (phi * R3)), (l, m, ring[l])
        assert np.any(np.abs(m - glob) > 1e-2 * scale), l


def test_local_version_converges_and_resumes(ref):
    a = fresh(ref, 40, 10, seed=14, cso_local=1)
    b = fresh(ref, 40, 10, seed=14, cso_local=1)
    f0 = a.best_fit if a.t else float(a.fit.min())
    a.step(200)
    for n in (1, 99, 100):
        b.step(n)
    assert np.array_equal(a.x, b.x) and np.array_equal(a.fit, b.fit)
    assert a.best_fit < 0.5 * f0
