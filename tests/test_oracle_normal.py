"""Pins of the oracle's normal initial population (stream 5, Box-Muller).

The deviates are checked against what does not depend on the oracle's own
code: rocRAND's Philox words through the inverse of the Box-Muller map (the
radius and angle of each pair give back u1 and u2), the normal distribution
(Kolmogorov-Smirnov), the chi-square law of a pair's squared radius, the
bound that u1 >= 2^-24 puts on |z|, and the independence of an element's
value from the matrix shape.
"""
import math

import numpy as np
from scipy import stats

from conftest import u01_exact


def test_pairs_invert_to_rocrand_words(ref, rocrand_philox):
    seed = 0x5EED_0000_0004
    cells = [(i, c) for i in (0, 1, 7, 1000, 65535) for c in (0, 1, 5, 250)]
    words = rocrand_philox([(seed, c, i, 0, 5) for i, c in cells])
    for (i, c), w in zip(cells, words):
        for q in (0, 1):
            z0 = ref.normal01(seed, i, 4 * c + 2 * q)
            z1 = ref.normal01(seed, i, 4 * c + 2 * q + 1)
            u1 = float(u01_exact([w[2 * q]])[0]) + 2.0 ** -24     # (a >> 8 + 1) 2^-24
            u2 = float(u01_exact([w[2 * q + 1]])[0])
            r2 = z0 * z0 + z1 * z1
            assert math.isclose(r2, -2.0 * math.log(u1), rel_tol=1e-12, abs_tol=1e-14)
            if r2 > 1e-20:
                ang = math.atan2(z1, z0) % (2.0 * math.pi)
                d = abs(ang - 2.0 * math.pi * u2)
                assert min(d, 2.0 * math.pi - d) < 1e-9, (i, c, q)


def test_marginals_are_standard_normal(ref):
    X = ref.init_normal(11, 4000, 64, 0.0, 1.0).astype(np.float64)
    for pos in range(4):            # every position within a Philox call
        z = X[:, pos::4].ravel()
        assert stats.kstest(z, "norm").pvalue > 1e-3, pos
    z = X.ravel()
    assert abs(z.mean()) < 0.01 and abs(z.std() - 1.0) < 0.01


def test_pair_radius_is_chi_square_two(ref):
    X = ref.init_normal(12, 3000, 32, 0.0, 1.0).astype(np.float64)
    r2 = X[:, 0::2] ** 2 + X[:, 1::2] ** 2
    assert stats.kstest(r2.ravel(), "chi2", args=(2,)).pvalue > 1e-3
    # different pairs of one call are independent: no correlation of radii
    a = X[:, 0::4] ** 2 + X[:, 1::4] ** 2
    b = X[:, 2::4] ** 2 + X[:, 3::4] ** 2
    assert abs(np.corrcoef(a.ravel(), b.ravel())[0, 1]) < 0.02


def test_deviates_are_bounded(ref):
    zmax = math.sqrt(-2.0 * math.log(2.0 ** -24))
    X = ref.init_normal(13, 2000, 100, 0.0, 1.0)
    assert np.all(np.isfinite(X)) and np.abs(X).max() <= zmax


def test_shape_independence_and_affine_map(ref):
    A = ref.init_normal(14, 50, 37, 0.0, 1.0)
    B = ref.init_normal(14, 80, 64, 0.0, 1.0)
    assert np.array_equal(A, B[:50, :37])
    C = ref.init_normal(14, 50, 37, 1.0, 0.5)
    Z = np.array([[ref.normal01(14, i, j) for j in range(37)] for i in range(50)])
    assert np.array_equal(C, (1.0 + 0.5 * Z).astype(np.float32))


def test_normal_state_init(ref):
    P = ref.make_params(4, 30, 20, -2.0, 2.0, seed=21, x_init=1, x_mu=1.0, x_sigma=0.5)
    s = ref.PSO(P)
    assert np.array_equal(s.x, ref.init_normal(21, 30, 20, 1.0, 0.5))
    assert np.array_equal(s.p, s.x) and np.all(s.v == 0)
    c = ref.CSO(ref.make_params(4, 30, 20, -2.0, 2.0, seed=21, x_init=1, x_mu=1.0, x_sigma=0.5))
    assert np.array_equal(c.x, s.x)
