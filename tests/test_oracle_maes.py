"""Pins of the oracle's MA-ES generation (the matrix-adaptation form of
CMA-ES, Beyer and Sendhoff 2017, with Hansen's default constants).

The deviates are tied to rocRAND's Philox words (stream 9) through the
inverse of the Box-Muller map; chi_D to the exact expected length of a
standard normal vector (gamma functions); the sampling to the covariance
M M^T of the steps; the whole generation to the invariances the method has
by construction -- rotating the search space (a transposed operand or a
product in the wrong order breaks it), trading step size against the scale
of M (bit-exact with a power of two), and the unbiasedness of the
adaptation under neutral selection (sigma = 0 makes every sample tie, so
the parents are the first mu by index: E[M'] = M and the path keeps a
standard normal law exactly when it starts in it -- a dropped term or a
wrong coefficient shifts one of them); the step-size rule to its direction
(shrinks at the optimum, grows on a slope); plus the row-restricted update,
the rank-mu form of the matrix update, convergence and resumption.
"""
import math

import numpy as np
import pytest
from scipy import special, stats

from conftest import u01_exact

SPHERE = 0


def params(ref, N, D, seed=3, **kw):
    return ref.make_params(SPHERE, N, D, -5.0, 5.0, seed=seed, **kw)


def test_deviates_invert_to_rocrand_words(ref, rocrand_philox):
    seed = 0x3AE5
    cells = [(t, k, c) for t in (0, 6, 2**32 - 3) for k in (0, 17, 16383) for c in (0, 9)]
    words = rocrand_philox([(seed, c, k, t, 9) for t, k, c in cells])
    for (t, k, c), w in zip(cells, words):
        for q in (0, 1):
            z0 = ref.maes_z(seed, t, k, 4 * c + 2 * q)
            z1 = ref.maes_z(seed, t, k, 4 * c + 2 * q + 1)
            u1 = float(u01_exact([w[2 * q]])[0]) + 2.0 ** -24
            u2 = float(u01_exact([w[2 * q + 1]])[0])
            assert math.isclose(z0 * z0 + z1 * z1, -2.0 * math.log(u1), rel_tol=1e-12, abs_tol=1e-14)
            if z0 * z0 + z1 * z1 > 1e-20:
                d = abs(math.atan2(z1, z0) % (2 * math.pi) - 2 * math.pi * u2)
                assert min(d, 2 * math.pi - d) < 1e-9


@pytest.mark.parametrize("D", [1, 2, 3, 10, 100, 16384])
def test_chi_is_the_expected_normal_length(ref, D):
    exact = math.sqrt(2.0) * math.exp(special.gammaln((D + 1) / 2.0) - special.gammaln(D / 2.0))
    chi = ref.maes_consts(10, D)[2]["chi"]
    assert abs(chi / exact - 1.0) < 2e-2 / D ** 2        # the approximation error falls as D^-2


@pytest.mark.parametrize("N,D", [(2, 1), (3, 5), (10, 10), (100, 16384), (4096, 2000)])
def test_constants_are_in_range(ref, N, D):
    mu, w, c = ref.maes_consts(N, D)
    assert mu == N // 2 and w.size == mu
    assert np.all(w > 0) and np.all(np.diff(w) < 0) and abs(w.sum() - 1.0) < 1e-12
    assert 1.0 <= c["mu_eff"] <= mu + 1e-12
    assert 0 < c["c_s"] < 1 and c["d_s"] >= 1.0
    assert 0 < c["c_1"] and 0 <= c["c_w"] <= 1 - c["c_1"]


def random_state(ref, N, D, seed, sigma=0.3):
    rng = np.random.default_rng(seed)
    m = ref.MAES(params(ref, N, D, seed=seed, es_sigma=sigma))
    m.y[:] = rng.uniform(-2, 2, D)
    m.M[:] = (np.eye(D) + 0.3 * rng.standard_normal((D, D))).astype(np.float32)
    m.s[:] = rng.standard_normal(D)
    return m, rng


def test_rotation_invariance(ref):
    """Sphere is rotation invariant, so the state (R y, sigma, R M, s) sees
    the same fitness as (y, sigma, M, s) and must move to (R y', sigma',
    R M', s')."""
    N, D = 16, 8
    a, rng = random_state(ref, N, D, 5)
    R = np.linalg.qr(rng.standard_normal((D, D)))[0]
    b = ref.MAES(params(ref, N, D, seed=5, es_sigma=0.3))
    b.y[:] = R @ a.y.astype(np.float64)
    b.M[:] = R @ a.M.astype(np.float64)
    b.s[:] = a.s
    a.step(1)
    b.step(1)
    assert np.array_equal(a.rank, b.rank)
    assert np.allclose(b.y, R @ a.y.astype(np.float64), rtol=0, atol=1e-5)
    assert np.allclose(b.M, R @ a.M.astype(np.float64), rtol=0, atol=1e-5)
    assert np.allclose(b.s, a.s, rtol=1e-6, atol=1e-6)
    assert math.isclose(b.sigma[0], a.sigma[0], rel_tol=1e-6)


def test_step_size_against_matrix_scale_is_exact(ref):
    """(y, 4 sigma, M / 4, s) draws the same points as (y, sigma, M, s)
    (scaling by a power of two is exact), so y' and s' agree bit for bit,
    M' is the same quarter and sigma' the same four times."""
    N, D = 12, 7
    a, _ = random_state(ref, N, D, 6)
    b = ref.MAES(params(ref, N, D, seed=6))
    b.y[:], b.s[:] = a.y, a.s
    b.M[:] = a.M / 4
    b.sigma[:] = a.sigma * 4
    for _ in range(3):
        a.step(1)
        b.step(1)
        assert np.array_equal(a.fit, b.fit) and np.array_equal(a.y, b.y) and np.array_equal(a.s, b.s)
        assert np.array_equal(b.M, a.M / 4) and b.sigma[0] == a.sigma[0] * 4


def neutral_runs(ref, N, D, runs):
    """One generation from M = I, sigma = 0 and s ~ N(0, I) per seed: every
    sample ties, the parents are samples 0..mu-1 (an index, independent of
    z), so M' = T is one draw of the adaptation under neutral selection."""
    Ts, s1 = [], []
    for seed in range(runs):
        m = ref.MAES(params(ref, N, D, seed=seed, es_sigma=0.0))
        m.s[:] = np.random.default_rng(10_000 + seed).standard_normal(D)
        y0 = m.y.copy()
        m.step(1)
        assert np.array_equal(m.y, y0) and m.sigma[0] == 0.0
        assert np.array_equal(m.rank, np.arange(N))
        Ts.append(m.M.astype(np.float64))
        s1.append(m.s.astype(np.float64))
    return np.array(Ts), np.array(s1)


def test_neutral_selection_is_unbiased(ref):
    N, D, runs = 8, 3, 3000
    T, s1 = neutral_runs(ref, N, D, runs)
    mean, se = T.mean(0), T.std(0, ddof=1) / math.sqrt(runs)
    assert np.all(np.abs(mean - np.eye(D)) < 5 * se + 1e-7), (mean, se)
    # the path stays standard normal: s' = (1 - c_s) s + sqrt(mu_eff c_s (2 - c_s)) <z>_w
    assert stats.kstest(s1.ravel(), "norm").pvalue > 1e-3
    assert abs(s1.var() - 1.0) < 0.05


def test_steps_have_covariance_m_mt(ref):
    N, D = 4000, 4
    m, rng = random_state(ref, N, D, 7)
    A = m.M.astype(np.float64)
    m.step(1, keep_d=True)
    C = np.cov(m.d.astype(np.float64).T)
    want = A @ A.T
    scale = np.sqrt(np.outer(np.diag(want), np.diag(want)))
    assert np.all(np.abs(C - want) < 6 * scale / math.sqrt(N)), (C, want)


def test_step_size_direction(ref):
    # at the optimum the parents are the shortest steps: |s| falls, sigma shrinks
    m = ref.MAES(params(ref, 20, 10, seed=8, es_sigma=1.0))
    m.y[:] = 0.0
    sig0 = m.sigma[0]
    m.step(5)
    assert m.sigma[0] < sig0
    # far away with a small step the fitness is nearly linear: steps line up, sigma grows
    m = ref.MAES(params(ref, 20, 10, seed=9, es_sigma=1e-3))
    m.y[:] = 1000.0
    sig0 = m.sigma[0]
    m.step(5)
    assert m.sigma[0] > 2 * sig0


def test_row_restricted_update(ref):
    N, D = 10, 9
    a, _ = random_state(ref, N, D, 11)
    b = ref.MAES(params(ref, N, D, seed=11))
    b.y[:], b.M[:], b.s[:], b.sigma[:] = a.y, a.M, a.s, a.sigma
    M0 = a.M.copy()
    rows = [0, 4, 8]
    a.step(1)
    b.step(1, rows=rows)
    assert np.array_equal(b.M[rows], a.M[rows])
    others = [i for i in range(D) if i not in rows]
    assert np.array_equal(b.M[others], M0[others])
    assert np.array_equal(a.y, b.y) and np.array_equal(a.s, b.s) and a.sigma[0] == b.sigma[0]


def test_matrix_update_in_rank_mu_form(ref):
    """M T = (1 - (c_1 + c_w)/2) M + c_1/2 (M s') s'^T + c_w/2 sum_i w_i d_i z_i^T
    over the parents, with d_i = M z_i the steps already drawn."""
    N, D, seed = 14, 6, 12
    m, _ = random_state(ref, N, D, seed)
    M0 = m.M.astype(np.float64)
    m.step(1, keep_d=True)
    mu, w, c = ref.maes_consts(N, D)
    order = np.argsort(m.rank)
    z = np.array([[np.float32(ref.maes_z(seed, 0, k, j)) for j in range(D)] for k in range(N)], np.float64)
    s1 = m.s.astype(np.float64)
    want = (1 - (c["c_1"] + c["c_w"]) / 2) * M0 + c["c_1"] / 2 * np.outer(M0 @ s1, s1)
    for r in range(mu):
        k = order[r]
        want += c["c_w"] / 2 * w[r] * np.outer(M0 @ z[k], z[k])
    assert np.allclose(m.M, want, rtol=1e-6, atol=1e-6)
    assert np.allclose(m.d[order[:mu]], (M0 @ z[order[:mu]].T).T, rtol=1e-6, atol=1e-6)


def test_convergence_and_resume(ref):
    a = ref.MAES(params(ref, 12, 8, seed=2, es_sigma=1.0))
    b = ref.MAES(params(ref, 12, 8, seed=2, es_sigma=1.0))
    f0 = float((a.y.astype(np.float64) ** 2).sum())
    a.step(150)
    for n in (1, 49, 100):
        b.step(n)
    for u, v in ((a.y, b.y), (a.M, b.M), (a.s, b.s), (a.sigma, b.sigma)):
        assert np.array_equal(u, v)
    assert float((a.y.astype(np.float64) ** 2).sum()) < 1e-8 * f0


def test_initial_state(ref):
    m = ref.MAES(params(ref, 10, 33, seed=5, es_sigma=0.7))
    assert np.array_equal(m.y, ref.init_uniform(5, 0, 1, 33, -5.0, 5.0)[0])
    assert m.sigma[0] == np.float32(0.7) and np.array_equal(m.M, np.eye(33, dtype=np.float32))
    assert not m.s.any()


def test_bad_sizes_rejected(ref):
    with pytest.raises(ValueError):
        ref.MAES(params(ref, 1, 5))
