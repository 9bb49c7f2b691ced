"""Pins of the oracle's PSO generation.

Degenerate parameters expose each ingredient of the update separately:
  * w = 0, c1 = 1, c2 = 0, x = 0, p = 1  ->  v = r1 exactly,
  * w = 0, c1 = 0, c2 = 1, x = 0, g = 1  ->  v = r2 exactly,
  * w = 1, c1 = c2 = 0                   ->  x_t = x_0 + v_0 + ... (fp32 adds),
  * w = 1/2, c1 = c2 = 0                 ->  v_t = v_0 / 2^t,
with r1, r2 recomputed here from rocRAND's Philox through the stated counter
layout, so that the draw addressing, the u01 map and the update are pinned
against something outside the oracle.  A two-particle generation is worked
by hand, and invariants of the method (personal bests never get worse, the
global best is the best personal best, resumption at any generation) are
checked on random runs.
"""
import numpy as np
import pytest

from conftest import u01_exact

SPHERE = 0


def draws(rocrand_philox, seed, N, D, K, k, t, stream):
    rows = [(seed, K * (j // 4) + k, i, t, stream) for i in range(N) for j in range(D)]
    words = rocrand_philox(rows)
    return u01_exact([words[e, (e % D) % 4] for e in range(N * D)]).reshape(N, D)


def fresh(ref, N, D, seed=3, **kw):
    P = ref.make_params(SPHERE, N, D, -1.0, 1.0, seed=seed, **kw)
    return ref.PSO(P)


@pytest.mark.parametrize("t0", [0, 5])
def test_velocity_equals_r1(ref, rocrand_philox, t0):
    N, D, seed = 3, 6, 77
    s = fresh(ref, N, D, seed=seed, w=0.0, c1=1.0, c2=0.0)
    s.t = t0
    s.x[:] = 0.0
    s.p[:] = 1.0
    s.v[:] = 123.0                      # multiplied by w = 0
    s.pf[:] = -np.inf                   # nothing improves: p stays 1
    s.step(1)
    r1 = draws(rocrand_philox, seed, N, D, 2, 0, t0, 2)
    assert np.array_equal(s.v, r1)
    assert np.array_equal(s.x, r1)


def test_velocity_equals_r2(ref, rocrand_philox):
    N, D, seed = 2, 9, 5
    s = fresh(ref, N, D, seed=seed, w=0.0, c1=0.0, c2=1.0)
    s.x[:] = 0.0
    s.p[:] = 1.0                        # g is the best personal best = ones
    s.pf[:] = -np.inf
    s.step(1)
    r2 = draws(rocrand_philox, seed, N, D, 2, 1, 0, 2)
    assert np.array_equal(s.v, r2)


def test_inertia_only_is_sequential_adds(ref):
    s = fresh(ref, 4, 5, w=1.0, c1=0.0, c2=0.0, v_lo=-1.0, v_hi=1.0)
    x0, v0 = s.x.copy(), s.v.copy()
    s.step(7)
    want = x0.copy()
    for _ in range(7):
        want = (want + v0).astype(np.float32)
    assert np.array_equal(s.x, want)
    assert np.array_equal(s.v, v0)


def test_inertia_halving(ref):
    s = fresh(ref, 3, 4, w=0.5, c1=0.0, c2=0.0, v_lo=-1.0, v_hi=1.0)
    v0 = s.v.copy()
    s.step(5)
    assert np.array_equal(s.v, (v0 / 32.0).astype(np.float32))


def test_hand_worked_generation(ref, rocrand_philox):
    # two particles in one dimension on Sphere, w = 0.5, c1 = c2 = 1
    seed = 21
    s = fresh(ref, 2, 1, seed=seed, w=0.5, c1=1.0, c2=1.0)
    s.x[:] = [[1.0], [2.0]]
    s.p[:] = s.x
    s.v[:] = [[0.5], [0.0]]
    s.step(1)
    # f = (1, 4): both improve from +inf; particle 0 is the global best
    assert s.pf.tolist() == [1.0, 4.0] and s.gi == 0 and s.gf == 1.0
    assert s.g.tolist() == [1.0]
    r2 = draws(rocrand_philox, seed, 2, 1, 2, 1, 0, 2)
    # particle 0: p - x = g - x = 0  ->  v = 0.5 * 0.5
    assert s.v[0, 0] == 0.25 and s.x[0, 0] == 1.25
    # particle 1: p - x = 0, g - x = -1  ->  v = -r2
    assert s.v[1, 0] == -r2[1, 0]
    assert s.x[1, 0] == np.float32(2.0) - r2[1, 0]


def test_velocity_clamp(ref):
    s = fresh(ref, 5, 8, w=1.0, c1=0.0, c2=0.0, vmax=0.25, v_lo=-1.0, v_hi=1.0)
    v0 = s.v.copy()
    s.step(1)
    assert np.array_equal(s.v, np.clip(v0, -0.25, 0.25))


def test_position_clamp(ref):
    s = fresh(ref, 5, 8, w=1.0, c1=0.0, c2=0.0, v_lo=-3.0, v_hi=3.0, clamp_x=1)
    x0, v0 = s.x.copy(), s.v.copy()
    s.step(1)
    assert np.array_equal(s.x, np.clip((x0 + v0).astype(np.float32), -1.0, 1.0))


def test_single_particle_global_is_personal(ref):
    P = ref.make_params(2, 1, 6, -5.12, 5.12, seed=8)
    s = ref.PSO(P)
    for _ in range(10):
        s.step(1)
        assert s.gi == 0 and s.gf == s.pf[0]
        assert np.array_equal(s.g, s.p[0])


@pytest.mark.parametrize("fn", range(6))
def test_invariants_random_run(ref, fn):
    P = ref.make_params(fn, 24, 7, -4.0, 4.0, v_lo=-0.5, v_hi=0.5, seed=fn + 100)
    s = ref.PSO(P)
    prev_pf = np.full(24, np.inf, np.float32)
    prev_gf = np.inf
    for _ in range(15):
        s.step(1)
        assert np.all(s.pf <= prev_pf)
        assert s.gf <= prev_gf
        assert s.gf == s.pf.min() and s.gi == int(np.argmin(s.pf))
        assert np.array_equal(s.g, s.p[s.gi])
        assert np.array_equal(ref.evaluate(fn, s.p), s.pf)
        prev_pf, prev_gf = s.pf.copy(), s.gf


def test_sphere_converges(ref):
    P = ref.make_params(SPHERE, 100, 10, -32.0, 32.0, seed=0)
    s = ref.PSO(P)
    s.step(1)
    first = s.gf
    s.step(99)
    assert s.gf < 1e-2 * first


def test_resume_is_bit_exact(ref):
    P = ref.make_params(1, 16, 9, -32.768, 32.768, v_lo=-1.0, v_hi=1.0, seed=1)
    a, b = ref.PSO(P), ref.PSO(P)
    a.step(12)
    b.step(5)
    b.step(7)
    for name in ("x", "v", "p", "pf", "g"):
        assert np.array_equal(getattr(a, name), getattr(b, name)), name
    assert (a.gf, a.gi, a.t) == (b.gf, b.gi, b.t)
