"""Pins of the oracle's NSGA-II on DTLZ1 (Deb, Pratap, Agarwal, Meyarivan 2002;
Deb, Thiele, Laumanns, Zitzler 2002).

DTLZ1 is tied to its closed forms (the objectives sum to (1 + g)/2 for any
x, so to 1/2 on the Pareto set; g at the corners; a hand-worked point);
non-dominated sorting to the three properties that characterise the fronts
(no dominance inside a front, every point of front k + 1 dominated from
front k, front 0 the brute-force non-dominated set) on inputs with ties and
duplicates, and to a chain and an antichain; crowding to a hand-worked
front and to its invariance under scaling an objective; the tournaments to
rocRAND's Philox words; the crossover to the conservation of the parents'
sum, to the words that decide which variables cross, and to the published
density of its spread factor; the mutation to its closed-form end points;
the generation to elitism, the size of the survivor set, convergence and
resumption.
"""
import math

import numpy as np
import pytest
from scipy import integrate, stats

from conftest import u01_exact


def test_dtlz1_objectives_sum_to_half_one_plus_g(ref):
    rng = np.random.default_rng(1)
    for M in (2, 3, 5):
        for _ in range(20):
            x = rng.random(12).astype(np.float32)
            f = ref.dtlz1_f64(x, M)
            d = x[M - 1:].astype(np.float64) - 0.5
            g = 100 * (d.size + (d * d - np.cos(20 * math.pi * d)).sum())
            assert math.isclose(f.sum(), 0.5 * (1 + g), rel_tol=1e-12)
            assert np.all(f >= 0)


def test_dtlz1_pareto_set_and_corners(ref):
    rng = np.random.default_rng(2)
    for M in (2, 3, 4):
        x = rng.random(10).astype(np.float32)
        x[M - 1:] = 0.5
        assert math.isclose(ref.dtlz1_f64(x, M).sum(), 0.5, rel_tol=1e-12)
        # every distance variable 0: each term is 1/4 - cos(10 pi) = -3/4, g = 25 k
        x[M - 1:] = 0.0
        k = 10 - M + 1
        assert math.isclose(ref.dtlz1_f64(x, M).sum(), 0.5 * (1 + 25 * k), rel_tol=1e-12)


def test_dtlz1_hand_worked_point(ref):
    # D = 3, M = 2, x = (1/4, 0, 0): g = 100 (2 + 2 (1/4 - 1)) = 50
    f = ref.dtlz1_f64(np.array([0.25, 0.0, 0.0], np.float32), 2)
    assert np.allclose(f, [0.5 * 51 * 0.25, 0.5 * 51 * 0.75], rtol=1e-12)


def check_fronts(F, front):
    n = F.shape[0]
    dom = lambda a, b: np.all(F[a] <= F[b]) and np.any(F[a] < F[b])
    nf = front.max() + 1
    assert set(front.tolist()) == set(range(nf))
    for i in range(n):
        for j in range(n):
            if front[i] == front[j]:
                assert not dom(i, j)
    for i in range(n):
        if front[i] > 0:
            assert any(dom(j, i) for j in range(n) if front[j] == front[i] - 1)
    nd = [i for i in range(n) if not any(dom(j, i) for j in range(n))]
    assert sorted(nd) == sorted(np.nonzero(front == 0)[0].tolist())


@pytest.mark.parametrize("seed", range(6))
def test_fronts_have_their_defining_properties(ref, seed):
    rng = np.random.default_rng(seed)
    n, M = 60, 2 + seed % 3
    F = rng.integers(0, 6, size=(n, M)).astype(np.float32)     # many ties and duplicates
    check_fronts(F, ref.nds(F))


def test_chain_and_antichain(ref):
    F = np.array([[i, i] for i in range(7)], np.float32)[::-1].copy()
    assert np.array_equal(ref.nds(F), np.arange(7)[::-1])
    G = np.array([[i, 6 - i] for i in range(7)], np.float32)
    assert np.array_equal(ref.nds(G), np.zeros(7))


def test_crowding_hand_worked(ref):
    F = np.array([[0, 4], [1, 2], [2, 1], [4, 0]], np.float32)
    c = ref.crowding(F, np.zeros(4, np.int32))
    # f0: (1,2) gets (2 - 0)/4, (2,1) gets (4 - 1)/4; f1 the mirror image
    assert np.isinf(c[0]) and np.isinf(c[3])
    assert c[1] == 0.5 + 0.75 and c[2] == 0.75 + 0.5


def test_crowding_breaks_ties_by_index(ref):
    """A = (0, 3), B = (1, 1), C = (1, 1), D = (3, 0): in both objectives B
    (lower index) sorts before its duplicate C, so B gets (1 - 0)/3 twice and
    C (3 - 1)/3 twice."""
    F = np.array([[0, 3], [1, 1], [1, 1], [3, 0]], np.float32)
    c = ref.crowding(F, np.zeros(4, np.int32))
    assert np.isinf(c[0]) and np.isinf(c[3])
    assert c[1] == 1 / 3 + 1 / 3 and c[2] == 2 / 3 + 2 / 3


def test_crowding_small_fronts_and_scaling(ref):
    rng = np.random.default_rng(3)
    F = rng.random((40, 3)).astype(np.float32)
    front = ref.nds(F)
    c = ref.crowding(F, front)
    for k in range(front.max() + 1):
        if (front == k).sum() <= 2:
            assert np.all(np.isinf(c[front == k]))
    G = F.copy()
    G[:, 1] *= 4.0                        # exact in fp32: ranges and gaps scale alike
    assert np.array_equal(ref.nds(G), front)
    assert np.allclose(ref.crowding(G, front), c, rtol=1e-12)


def test_tournaments_follow_rocrand_words(ref, rocrand_philox):
    rng = np.random.default_rng(4)
    N, seed = 37, 99
    front = rng.integers(0, 4, N).astype(np.int32)
    crowd = rng.random(N)
    crowd[rng.random(N) < 0.2] = np.inf
    for t, p in [(t, p) for t in range(8) for p in range(18)]:
        w = rocrand_philox([(seed, 0, p, t, 10)])[0]
        c = [(int(x) * N) >> 32 for x in w]

        def win(a, b):
            if front[a] != front[b]:
                return a if front[a] < front[b] else b
            if crowd[a] != crowd[b]:
                return a if crowd[a] > crowd[b] else b
            return min(a, b)
        assert ref.nsga2_parents(seed, t, p, N, front, crowd) == (win(c[0], c[1]), win(c[2], c[3]))


def test_crossover_conserves_and_follows_words(ref, rocrand_philox):
    D, seed, t, p = 64, 5, 2, 3
    P = ref.nsga2_params(10, D, 3, eta_c=20.0, eta_m=20.0, seed=seed)
    rng = np.random.default_rng(5)
    a = rng.uniform(0.2, 0.8, D).astype(np.float32)
    b = rng.uniform(0.2, 0.8, D).astype(np.float32)
    c0, c1 = ref.nsga2_offspring(P, t, p, a, b)
    w = rocrand_philox([(seed, j, p, t, 11) for j in range(D)])
    mutated = (u01_exact(w[:, 2]) < 1.0 / D) | (u01_exact(w[:, 3]) < 1.0 / D)
    crossed = u01_exact(w[:, 1]) < 0.5
    keep = ~mutated & ~crossed
    assert np.array_equal(c0[keep], a[keep]) and np.array_equal(c1[keep], b[keep])
    both = ~mutated & crossed
    s = c0[both].astype(np.float64) + c1[both] - a[both] - b[both]
    assert np.all(np.abs(s) <= 2 * np.spacing(np.float32(1.0)))


def test_spread_factor_has_the_published_density(ref):
    """SBX spread beta: density (eta+1)/2 beta^eta on [0, 1] and
    (eta+1)/2 beta^-(eta+2) above 1 (Deb and Agrawal 1995); its sign is a fair
    coin.  beta = (c0 - c1) / (a - b) for crossed, unclipped variables."""
    eta, D = 3.0, 4096
    P = ref.nsga2_params(10, D, 3, eta_c=eta, eta_m=20.0, seed=6)
    a = np.full(D, 0.49, np.float32)
    b = np.full(D, 0.51, np.float32)
    betas = []
    for p in range(4):
        c0, c1 = ref.nsga2_offspring(P, 0, p, a, b)
        beta = (c0.astype(np.float64) - c1) / (a.astype(np.float64) - b)
        inside = (c0 > 0) & (c0 < 1) & (c1 > 0) & (c1 < 1) & (np.abs(beta - 1) > 1e-3)
        betas.append(beta[inside])
    beta = np.concatenate(betas)

    def cdf_abs(x):
        x = np.asarray(x, np.float64)
        return np.where(x <= 1, 0.5 * x ** (eta + 1), 1 - 0.5 * x ** -(eta + 1))
    assert stats.kstest(np.abs(beta), cdf_abs).pvalue > 1e-3
    assert abs((beta > 0).mean() - 0.5) < 0.03
    assert math.isclose(integrate.quad(lambda x: 0.5 * (eta + 1) * x ** eta, 0, 1)[0] +
                        integrate.quad(lambda x: 0.5 * (eta + 1) * x ** -(eta + 2), 1, np.inf)[0], 1.0,
                        rel_tol=1e-9)


def test_polynomial_mutation_end_points(ref):
    for x in (0.0, 0.2, 0.5, 0.9, 1.0):
        assert ref.poly_mutate(x, 0.5, 20.0) == pytest.approx(x, abs=1e-15)
        assert ref.poly_mutate(x, 0.0, 20.0) == pytest.approx(0.0, abs=1e-15)
        assert ref.poly_mutate(x, 1.0, 20.0) == pytest.approx(1.0, abs=1e-15)    # the limit u -> 1
    us = np.linspace(0.0, 0.999, 200)
    ys = [ref.poly_mutate(0.3, u, 20.0) for u in us]
    assert np.all(np.diff(ys) >= 0)


def test_generation_is_elitist_and_fills(ref):
    P = ref.nsga2_params(60, 10, 3, seed=7)
    s = ref.NSGA2(P)
    for _ in range(5):
        F0 = s.F[s.front == 0].copy()
        s.step(1)
        assert s.X.shape == (60, 10) and np.all((s.X >= 0) & (s.X <= 1))
        assert np.array_equal(s.F, ref.dtlz1(s.X, 3))
        for f in F0:   # every old non-dominated point survives or is dominated by a survivor
            kept = np.any(np.all(s.F == f, axis=1))
            assert kept or any(ref.dominates(g, f) for g in s.F)
        # the survivors' fronts are those of the merged population: re-sorting
        # them alone keeps front 0 (a subset of the merged front 0) non-dominated
        assert np.array_equal(ref.nds(s.F) == 0, ref.nds(s.F) == 0)
        assert np.all(ref.nds(s.F)[s.front == 0] == 0)


def rebuild_generation(ref, s):
    """The merged population of the next generation of state s, from the
    pinned parts: tournaments, offspring, DTLZ1, fronts, crowding."""
    P, N, M = s.P, s.P.N, s.P.M
    Q = np.zeros((N, P.D), np.float32)
    for p in range(N // 2):
        a, b = ref.nsga2_parents(P.seed, s.t, p, N, s.front, s.crowd)
        Q[2 * p], Q[2 * p + 1] = ref.nsga2_offspring(P, s.t, p, s.X[a], s.X[b])
    XR = np.concatenate([s.X, Q])
    FR = np.concatenate([s.F, ref.dtlz1(Q, M)])
    fr = ref.nds(FR)
    return XR, FR, fr, ref.crowding(FR, fr)


def expected_survivors(fr, cr, N):
    """Whole fronts before the first one that does not fit; from that one,
    the members of largest crowding distance, lower index first on ties.
    Also whether the cut falls between equal distances."""
    sizes = np.bincount(fr)
    k = int(np.nonzero(np.cumsum(sizes) > N)[0][0])
    keep = fr < k
    left = N - keep.sum()
    order = sorted(np.nonzero(fr == k)[0].tolist(), key=lambda i: (-cr[i], i))
    keep[order[:left]] = True
    tie = 0 < left < len(order) and cr[order[left - 1]] == cr[order[left]]
    return keep, tie


def test_truncation_keeps_the_least_crowded_out(ref):
    """Survivors as the rule says, in their merged order with their merged
    fronts and distances; over small populations (fronts of one or two
    points, so many infinite distances) the cut must have fallen between
    equal distances at least once."""
    ties = 0
    for seed in range(12):
        s = ref.NSGA2(ref.nsga2_params(8, 4, 3, seed=seed))
        for _ in range(4):
            XR, FR, fr, cr = rebuild_generation(ref, s)
            keep, tie = expected_survivors(fr, cr, 8)
            ties += tie
            s.step(1)
            assert np.array_equal(s.X, XR[keep]) and np.array_equal(s.F, FR[keep])
            assert np.array_equal(s.front, fr[keep]) and np.array_equal(s.crowd, cr[keep])
    assert ties > 0


def test_convergence_and_resume(ref):
    P = ref.nsga2_params(40, 8, 3, seed=8)
    a, b = ref.NSGA2(P), ref.NSGA2(P)
    g0 = float(a.F.sum(1).mean())
    a.step(60)
    for n in (1, 19, 40):
        b.step(n)
    for u, v in ((a.X, b.X), (a.F, b.F), (a.front, b.front), (a.crowd, b.crowd)):
        assert np.array_equal(u, v)
    assert float(a.F.sum(1).mean()) < 0.05 * g0


def test_bad_sizes_rejected(ref):
    with pytest.raises(ValueError):
        ref.NSGA2(ref.nsga2_params(7, 5, 3))
    with pytest.raises(ValueError):
        ref.NSGA2(ref.nsga2_params(8, 2, 3))
