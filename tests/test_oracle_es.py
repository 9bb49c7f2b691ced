"""Pins of the oracle's OpenES generation (Salimans et al., 2017).

The perturbations are tied to rocRAND's Philox words through the inverse of
the Box-Muller map (with the generation in the counter); the ranks to numpy's
lexicographic sort; the rank-gradient-update chain to a closed form (center
at the Sphere optimum: the two samples of a pair tie, so every pair has rank
difference one and the step is a known sum of perturbations); the estimate to
the descent direction on Sphere (statistically); plus convergence, resumption
and the shape of the first center.
"""
import math

import numpy as np

from conftest import u01_exact

SPHERE = 0


def params(ref, N, D, seed=3, **kw):
    return ref.make_params(SPHERE, N, D, -5.0, 5.0, seed=seed, **kw)


def test_perturbations_invert_to_rocrand_words(ref, rocrand_philox):
    seed = 0xE5
    cells = [(t, k, c) for t in (0, 3, 2**32 - 1) for k in (0, 9, 5000) for c in (0, 7)]
    words = rocrand_philox([(seed, c, k, t, 7) for t, k, c in cells])
    for (t, k, c), w in zip(cells, words):
        for q in (0, 1):
            z0 = ref.es_eps(seed, t, k, 4 * c + 2 * q)
            z1 = ref.es_eps(seed, t, k, 4 * c + 2 * q + 1)
            u1 = float(u01_exact([w[2 * q]])[0]) + 2.0 ** -24
            u2 = float(u01_exact([w[2 * q + 1]])[0])
            assert math.isclose(z0 * z0 + z1 * z1, -2.0 * math.log(u1), rel_tol=1e-12, abs_tol=1e-14)
            if z0 * z0 + z1 * z1 > 1e-20:
                d = abs(math.atan2(z1, z0) % (2 * math.pi) - 2 * math.pi * u2)
                assert min(d, 2 * math.pi - d) < 1e-9


def test_ranks_are_the_argmin_order(ref):
    s = ref.ES(params(ref, 300, 7, seed=4))
    s.step(2)
    order = np.lexsort((np.arange(300), s.fit))       # by fitness, then index
    want = np.empty(300, np.int64)
    want[order] = np.arange(300)
    assert np.array_equal(s.rank, want)
    assert s.best_idx == order[0] and s.best_fit == s.fit[order[0]]


def test_step_at_the_optimum_is_a_sum_of_perturbations(ref):
    """theta = 0 on Sphere: f(+sigma eps) = f(-sigma eps) exactly, so the
    lower index of each pair ranks just before the other, u_{2k} - u_{2k+1}
    = -1/(N - 1), and theta_j becomes lr sum_k eps_kj / (N (N - 1) sigma)."""
    N, D, sigma, lr, seed = 40, 9, 0.25, 0.5, 6
    s = ref.ES(params(ref, N, D, seed=seed, es_sigma=sigma, es_lr=lr))
    s.theta[:] = 0.0
    s.step(1)
    assert np.all(s.rank[0::2] + 1 == s.rank[1::2])
    eps = np.array([[ref.es_eps(seed, 0, k, j) for j in range(D)] for k in range(N // 2)])
    g = -eps.sum(0) / (N - 1) / (N * sigma)
    want = (-np.float32(lr) * g.astype(np.float32)).astype(np.float32)
    assert np.array_equal(s.theta, want)


def test_estimate_points_downhill_on_sphere(ref):
    D = 64
    s = ref.ES(params(ref, 2000, D, seed=8, es_sigma=0.05, es_lr=1.0))
    theta0 = s.theta.astype(np.float64).copy()
    s.step(1)
    step = s.theta.astype(np.float64) - theta0                 # = -lr g
    cos = step @ (-2.0 * theta0) / (np.linalg.norm(step) * np.linalg.norm(theta0) * 2.0)
    assert cos > 0.5


def test_convergence_and_resume(ref):
    a = ref.ES(params(ref, 100, 20, seed=2, es_sigma=0.1, es_lr=0.05))
    b = ref.ES(params(ref, 100, 20, seed=2, es_sigma=0.1, es_lr=0.05))
    f0 = float((a.theta.astype(np.float64) ** 2).sum())
    a.step(150)
    for n in (1, 49, 100):
        b.step(n)
    assert np.array_equal(a.theta, b.theta) and np.array_equal(a.fit, b.fit)
    assert float((a.theta.astype(np.float64) ** 2).sum()) < 1e-3 * f0


def test_first_center_is_row_zero_of_the_uniform_population(ref):
    s = ref.ES(params(ref, 10, 33, seed=5))
    assert np.array_equal(s.theta, ref.init_uniform(5, 0, 1, 33, -5.0, 5.0)[0])


def test_odd_population_rejected(ref):
    import pytest
    with pytest.raises(ValueError):
        ref.ES(params(ref, 9, 5))
