"""Pins of the oracle's DE/rand/1/bin generation (Storn & Price, 1997).

The partner choice is checked for what the method requires (three partners,
mutually distinct and distinct from the target, every ordered choice equally
likely) and tied to rocRAND's Philox words through a decodable population;
the crossover mask is exposed the same way and compared with the words; the
generation is checked against a hand-worked four-individual case, invariants
(greedy selection never worsens a target, the best never worsens, rows are
the old row or a trial), the all-equal degenerate case and resumption.
"""
import itertools

import numpy as np
from scipy import stats

from conftest import u01_exact

SPHERE = 0


def params(ref, N, D, seed=3, **kw):
    return ref.make_params(SPHERE, N, D, -5.0, 5.0, seed=seed, **kw)


def test_partners_are_distinct_and_in_range(ref):
    for N in (4, 5, 7, 100, 2**20):
        for t in range(3):
            for i in list(range(min(N, 30))) + [N - 1]:
                r1, r2, r3, jr = ref.de_choices(5, t, i, N, 17)
                assert len({i, r1, r2, r3}) == 4, (N, t, i)
                assert all(0 <= r < N for r in (r1, r2, r3)) and 0 <= jr < 17


def test_partner_triples_are_uniform(ref):
    N, i = 5, 2
    others = [k for k in range(N) if k != i]
    triples = list(itertools.permutations(others, 3))       # 24 ordered choices
    counts = dict.fromkeys(triples, 0)
    for seed in range(40):
        for t in range(120):
            counts[ref.de_choices(seed, t, i, N, 1)[:3]] += 1
    obs = np.array(list(counts.values()))
    assert stats.chisquare(obs).pvalue > 1e-3


def kth_free(a, taken, N):
    """The a-th (from 0) index of 0..N-1 not in taken (a list comprehension,
    not the oracle's stepping)."""
    return [k for k in range(N) if k not in taken][a]


def test_partners_follow_rocrand_words(ref, rocrand_philox):
    seed, N, D = 77, 9, 13
    cells = [(t, i) for t in (0, 1, 40) for i in range(N)]
    words = rocrand_philox([(seed, 0, i, t, 6) for t, i in cells])
    for (t, i), w in zip(cells, words):
        taken = [i]
        want = []
        for k in range(3):
            a = (int(w[k]) * (N - 1 - k)) >> 32
            r = kth_free(a, taken, N)
            want.append(r)
            taken.append(r)
        want.append((int(w[3]) * D) >> 32)
        assert ref.de_choices(seed, t, i, N, D) == tuple(want), (t, i)


def test_generation_exposes_partners_and_mask(ref, rocrand_philox):
    """Rows x_k = 10^k (exact in fp32) and every trial accepted (targets'
    fitness set to +inf): with F = 1 the trial's mutant elements equal
    10^r1 + 10^r2 - 10^r3, which names the partners; elements not taken
    from the mutant keep 10^i, which names the crossover mask."""
    N, D, seed, cr = 6, 24, 11, 0.5
    s = ref.DE(params(ref, N, D, seed=seed, de_f=1.0, de_cr=cr))
    s.x[:] = (10.0 ** np.arange(N, dtype=np.float64))[:, None].astype(np.float32)
    s.fit[:] = np.inf
    x0 = s.x.copy()
    s.step(1)
    for i in range(N):
        r1, r2, r3, jr = ref.de_choices(seed, 0, i, N, D)
        mutant = np.float32(10.0 ** r1 + 10.0 ** r2 - 10.0 ** r3)
        w = rocrand_philox([(seed, 1 + q, i, 0, 6) for q in range(D // 4)]).reshape(-1)
        take = (u01_exact(w) <= np.float32(cr)) | (np.arange(D) == jr)
        assert np.array_equal(s.x[i], np.where(take, mutant, x0[i, 0])), i


def test_hand_worked_generation(ref):
    """Four individuals on Sphere in one dimension: every partner triple is a
    permutation of the other three, the single element is always j_rand, so
    the trial is x_r1 + F (x_r2 - x_r3) and replaces the target iff better."""
    N, D, seed, F = 4, 1, 4, 0.5
    s = ref.DE(params(ref, N, D, seed=seed, de_f=F, de_cr=0.0))
    x0 = np.array([[3.0], [-1.0], [0.5], [2.0]], np.float32)
    s.x[:] = x0
    s.fit[:] = (x0[:, 0].astype(np.float64) ** 2).astype(np.float32)
    f0 = s.fit.copy()
    s.step(1)
    for i in range(N):
        r1, r2, r3, jr = ref.de_choices(seed, 0, i, N, D)
        assert jr == 0
        trial = np.float32(np.float32(x0[r1, 0]) + np.float32(F) * np.float32(x0[r2, 0] - x0[r3, 0]))
        ft = np.float32(float(trial) ** 2)
        want = trial if ft < f0[i] else x0[i, 0]
        assert s.x[i, 0] == want and s.fit[i] == min(ft, f0[i]), i


def test_invariants(ref):
    N, D = 40, 8
    s = ref.DE(params(ref, N, D, seed=9))
    best = s.best_fit
    for _ in range(20):
        x0, f0 = s.x.copy(), s.fit.copy()
        s.step(1)
        assert np.all(s.fit <= f0)
        kept = ~s.accepted.astype(bool)
        assert np.array_equal(s.x[kept], x0[kept]) and np.array_equal(s.fit[kept], f0[kept])
        assert np.all(s.fit[~kept] < f0[~kept])
        assert np.allclose(s.fit, ref.evaluate(SPHERE, s.x), rtol=0, atol=0)
        assert s.best_fit <= best and s.best_fit == s.fit.min()
        best = s.best_fit


def test_all_equal_population_is_a_fixed_point(ref):
    s = ref.DE(params(ref, 10, 5, seed=1))
    s.x[:] = 1.25
    s.fit[:] = ref.evaluate(SPHERE, s.x)
    s.step(3)
    assert np.all(s.x == 1.25) and not s.accepted.any()


def test_resume_and_convergence(ref):
    a = ref.DE(params(ref, 30, 6, seed=2))
    b = ref.DE(params(ref, 30, 6, seed=2))
    f0 = a.best_fit
    a.step(60)
    for n in (7, 23, 30):
        b.step(n)
    assert np.array_equal(a.x, b.x) and np.array_equal(a.fit, b.fit)
    assert a.best_fit < 1e-2 * f0


def test_small_population_rejected(ref):
    import pytest
    with pytest.raises(ValueError):
        ref.DE(params(ref, 3, 5))
