"""Pins of the oracle's PGPE generation (Sehnke et al., 2010, symmetric
sampling).

The deviates are tied to rocRAND's Philox words (stream 8, the generation in
the counter) by inverting the Box-Muller map; the samples to mu +- sigma z
through a decodable case (one dimension, Sphere: each sample's fitness gives
back its perturbation); the sigma update to its clip (a huge sigma learning
rate moves every sigma by exactly the allowed fraction) and to its direction
at the optimum (where wider perturbations are worse, sigma shrinks); the
center step at the optimum to a closed form; plus convergence and resumption.
"""
import math

import numpy as np

from conftest import u01_exact

SPHERE = 0


def params(ref, N, D, seed=3, **kw):
    return ref.make_params(SPHERE, N, D, -5.0, 5.0, seed=seed, **kw)


def test_deviates_invert_to_rocrand_words(ref, rocrand_philox):
    seed = 0x96E
    cells = [(t, k, c) for t in (0, 5, 2**32 - 2) for k in (0, 3, 8191) for c in (0, 11)]
    words = rocrand_philox([(seed, c, k, t, 8) for t, k, c in cells])
    for (t, k, c), w in zip(cells, words):
        for q in (0, 1):
            z0 = ref.pgpe_z(seed, t, k, 4 * c + 2 * q)
            z1 = ref.pgpe_z(seed, t, k, 4 * c + 2 * q + 1)
            u1 = float(u01_exact([w[2 * q]])[0]) + 2.0 ** -24
            u2 = float(u01_exact([w[2 * q + 1]])[0])
            assert math.isclose(z0 * z0 + z1 * z1, -2.0 * math.log(u1), rel_tol=1e-12, abs_tol=1e-14)
            if z0 * z0 + z1 * z1 > 1e-20:
                d = abs(math.atan2(z1, z0) % (2 * math.pi) - 2 * math.pi * u2)
                assert min(d, 2 * math.pi - d) < 1e-9


def test_samples_are_center_plus_minus_scaled_deviates(ref):
    """D = 1 on Sphere: f(x) = x^2, so sqrt(f) recovers |mu +- sigma z|."""
    N, seed, mu, sig = 20, 4, 3.0, 0.5
    s = ref.PGPE(params(ref, N, 1, seed=seed, es_sigma=sig))
    s.mu[:] = mu
    s.step(1)
    for k in range(N // 2):
        z = np.float32(ref.pgpe_z(seed, 0, k, 0))
        xp = np.float32(np.float32(mu) + np.float32(sig) * z)
        xm = np.float32(np.float32(mu) - np.float32(sig) * z)
        assert s.fit[2 * k] == np.float32(float(xp) ** 2) and s.fit[2 * k + 1] == np.float32(float(xm) ** 2)


def test_sigma_change_is_clipped(ref):
    s = ref.PGPE(params(ref, 40, 6, seed=5, es_sigma=0.3, pgpe_sigma_lr=1e6, pgpe_max_change=0.2))
    s0 = s.sigma.copy()
    s.step(1)
    cap = (np.float32(0.2) * s0).astype(np.float32)
    d = (s.sigma - s0).astype(np.float32)
    assert np.all((d == cap) | (d == -cap))


def test_sigma_shrinks_at_the_optimum(ref):
    s = ref.PGPE(params(ref, 400, 8, seed=6, es_sigma=0.5, pgpe_sigma_lr=0.05))
    s.mu[:] = 0.0
    s0 = s.sigma.copy()
    s.step(1)
    assert np.all(s.sigma < s0)


def test_center_step_at_the_optimum(ref):
    """mu = 0 on Sphere: the two samples of a pair tie, the lower index ranks
    first, so u_{2k} - u_{2k+1} = -1/(N - 1) and the center moves to
    lr / (H (N - 1)) * sum_k sigma_j z_kj / 2."""
    N, D, sig, lr, seed = 30, 5, 0.25, 0.5, 7
    s = ref.PGPE(params(ref, N, D, seed=seed, es_sigma=sig, es_lr=lr))
    s.mu[:] = 0.0
    s.step(1)
    assert np.all(s.rank[0::2] + 1 == s.rank[1::2])
    z = np.array([[np.float32(ref.pgpe_z(seed, 0, k, j)) for j in range(D)] for k in range(N // 2)],
                 dtype=np.float64)
    g = (0.5 * (-1.0 / (N - 1)) * np.float64(np.float32(sig)) * z).sum(0) / (N // 2)
    want = (-np.float32(lr) * g.astype(np.float32)).astype(np.float32)
    assert np.array_equal(s.mu, want)


def test_convergence_and_resume(ref):
    kw = dict(es_sigma=1.0, es_lr=0.5, pgpe_sigma_lr=0.1)
    a = ref.PGPE(params(ref, 100, 20, seed=2, **kw))
    b = ref.PGPE(params(ref, 100, 20, seed=2, **kw))
    f0 = float((a.mu.astype(np.float64) ** 2).sum())
    a.step(200)
    for n in (1, 99, 100):
        b.step(n)
    assert np.array_equal(a.mu, b.mu) and np.array_equal(a.sigma, b.sigma)
    assert float((a.mu.astype(np.float64) ** 2).sum()) < 1e-2 * f0
