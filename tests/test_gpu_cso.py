"""GPU parity of the CSO generation against the oracle.

The pairing permutation is integer work and must match exactly; the loser
update is bit-exact given the same swarm mean; the mean itself is an fp64 sum
in a different order on each side and must agree to 1 ulp; so that every
generation is compared bit for bit, the single-generation tests give the
GPU the oracle's mean before each step (parity.cso_lockstep); fitness within
the fitness tolerance; the reported best index exactly.
"""
import numpy as np
import pytest
import torch

from parity import assert_fitness, cso_lockstep, index_ok, ulp_diff

pytestmark = pytest.mark.gpu


def pair(evox, ref, fn, N, D, seed, lb, ub, **kw):
    g = evox.Swarm(evox.make_params(evox.CSO, fn, N, D, lb, ub, seed=seed, **kw))
    r = ref.CSO(ref.make_params(fn, N, D, lb, ub, seed=seed, **kw))
    return g, r


def host(t, D):
    return t[..., :D].cpu().numpy()


def compare(g, r, fn, what):
    D = r.P.D
    x, v, f = host(g.x, D), host(g.v, D), g.fit.cpu().numpy()
    bad = np.nonzero((x != r.x).any(1))[0]
    assert bad.size == 0, f"{what}: x differs in rows {bad[:8]}"
    assert np.array_equal(v, r.v), f"{what}: v differs"
    assert_fitness(fn, r.x, f, r.fit, f"{what}: fit")
    bf, bi = g.best()
    if r.t > 0:
        assert index_ok(fn, r.x, r.fit, bi, r.best_idx), f"{what}: best {bi} vs {r.best_idx}"
        assert bi == r.best_idx, f"{what}: best index {bi} vs {r.best_idx} (tolerance tie)"


def test_init_matches(evox_gpu, ref):
    g, r = pair(evox_gpu, ref, 3, 101, 100, 3, -600.0, 600.0)
    torch.cuda.synchronize()
    assert np.array_equal(host(g.x, 100), r.x)
    assert np.all(host(g.v, 100) == 0)
    assert_fitness(3, r.x, g.fit.cpu().numpy(), r.fit, "init fit")
    assert ulp_diff(host(g.xbar, 100), ref.colmean(r.x)).max() <= 1
    bf, bi = g.best()
    assert index_ok(3, r.x, r.fit, bi, ref.argmin(r.fit))


CASES = [
    dict(fn=3, N=1000, D=100, seed=3, lb=-600.0, ub=600.0, gens=20),
    dict(fn=0, N=101, D=10, seed=0, lb=-32.0, ub=32.0, gens=40),
    dict(fn=1, N=64, D=37, seed=1, lb=-32.768, ub=32.768, v_lo=-1.0, v_hi=1.0, gens=20),
    dict(fn=2, N=33, D=257, seed=2, lb=-5.12, ub=5.12, gens=15),
    dict(fn=4, N=12, D=1001, seed=4, lb=-2.0, ub=2.0, gens=10),
    dict(fn=5, N=7, D=3, seed=5, lb=-500.0, ub=500.0, clamp_x=1, gens=30),
    dict(fn=4, N=5, D=2050, seed=6, lb=-2.0, ub=2.0, gens=6),
    dict(fn=0, N=2, D=1, seed=8, lb=-1.0, ub=1.0, gens=10),
    # several superbuckets in the pairing sort (pairs that straddle two of
    # them), odd and even populations
    dict(fn=0, N=5001, D=4, seed=13, lb=-5.0, ub=5.0, gens=12),
    dict(fn=3, N=70_001, D=20, seed=14, lb=-600.0, ub=600.0, gens=6),
    dict(fn=2, N=131_072, D=8, seed=15, lb=-5.12, ub=5.12, gens=4),
]


@pytest.mark.parametrize("case", CASES, ids=[f"fn{c['fn']}-{c['N']}x{c['D']}" for c in CASES])
def test_generations_match_oracle(evox_gpu, ref, case):
    c = dict(case)
    gens = c.pop("gens")
    print(f"cso {c} gens={gens}", flush=True)
    g, r = pair(evox_gpu, ref, **c)
    for t in range(gens):
        cso_lockstep(ref, g, r, f"generation {t}")
        compare(g, r, c["fn"], f"generation {t}")
    assert g.t == r.t == gens


def test_winners_untouched_and_losers_counted(evox_gpu, ref):
    g, _ = pair(evox_gpu, ref, 3, 999, 20, 5, -600.0, 600.0, v_lo=-1.0, v_hi=1.0)
    x0, v0, f0 = g.x.clone(), g.v.clone(), g.fit.clone()
    g.step(1)
    changed = (g.x != x0).any(1) | (g.v != v0).any(1)
    assert int(changed.sum()) <= 999 // 2
    assert int(changed.sum()) >= 999 // 2 - 5       # a loser may by chance not move
    same = ~changed
    assert torch.equal(g.fit[same & (g.fit == f0)], f0[same & (g.fit == f0)])


def test_multi_generation_call_equals_single_steps(evox_gpu, ref):
    kw = dict(fn=3, N=500, D=30, seed=12, lb=-600.0, ub=600.0)
    a, _ = pair(evox_gpu, ref, **kw)
    b, _ = pair(evox_gpu, ref, **kw)
    a.step(20)
    for n in (3, 9, 8):
        b.step(n)
    for name in ("x", "v", "fit", "xbar"):
        assert torch.equal(getattr(a, name), getattr(b, name)), name
    assert a.best() == b.best()


def test_loser_velocity_exposes_r2(evox_gpu, ref):
    N, D, seed = 40, 9, 31
    g, r = pair(evox_gpu, ref, 0, N, D, seed, -1.0, 1.0, phi=0.0)
    side = (np.arange(N) % 2 == 0)
    xs = np.where(side[:, None], 1.0, 0.0).astype(np.float32) * np.ones((N, D), np.float32)
    fs = np.where(side, 0.0, 1.0).astype(np.float32)
    g.x[:, :D] = torch.from_numpy(xs).cuda()
    g.v.zero_()
    g.fit.copy_(torch.from_numpy(fs).cuda())
    g.refresh(refit=False)
    r.x[:] = xs
    r.v[:] = 0.0
    r.fit[:] = fs
    g.step(1)
    r.step(1)
    assert np.array_equal(host(g.v, D), r.v)
    assert np.array_equal(host(g.x, D), r.x)


def test_refresh_after_external_edit(evox_gpu, ref):
    g, r = pair(evox_gpu, ref, 2, 64, 16, 2, -5.12, 5.12)
    rng = np.random.default_rng(0)
    X = rng.uniform(-1, 1, size=(64, 16)).astype(np.float32)
    g.x[:, :16] = torch.from_numpy(X).cuda()
    g.refresh(refit=True)
    r.x[:] = X
    r.fit[:] = ref.evaluate(2, X)
    assert_fitness(2, X, g.fit.cpu().numpy(), r.fit, "refit")
    assert ulp_diff(host(g.xbar, 16), ref.colmean(X)).max() <= 1


@pytest.mark.parametrize("D,ldx", [(100, 100), (100, 128), (37, 40), (70, 96), (257, 288), (64, 64)])
def test_pitched_states_match_oracle(evox_gpu, ref, D, ldx):
    """Any 4-multiple pitch gives the same generations; padding stays zero."""
    N, fn, gens = 301, 3, 6
    print(f"cso pitched D={D} ldx={ldx}", flush=True)
    g = evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.CSO, fn, N, D, -600.0, 600.0, seed=9, ldx=ldx))
    r = ref.CSO(ref.make_params(fn, N, D, -600.0, 600.0, seed=9))
    assert g.P.ldx == ldx and g.x.shape[1] == ldx
    for t in range(gens):
        cso_lockstep(ref, g, r, f"generation {t}")
        compare(g, r, fn, f"generation {t}")
        for name in ("x", "v", "xbar"):
            pad = getattr(g, name)[..., D:]
            assert int((pad != 0).sum()) == 0, f"{name} padding written at generation {t}"


def test_default_pitch_is_dense(evox_gpu, ref):
    g = evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.CSO, 3, 64, 100, -600.0, 600.0, seed=3))
    assert g.P.ldx == 100
    g = evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.CSO, 3, 64, 37, -600.0, 600.0, seed=3))
    assert g.P.ldx == 40


LOCAL_CASES = [
    dict(fn=3, N=1000, D=100, seed=3, lb=-600.0, ub=600.0, gens=15),
    dict(fn=1, N=64, D=37, seed=1, lb=-32.768, ub=32.768, v_lo=-1.0, v_hi=1.0, gens=15),
    dict(fn=2, N=33, D=257, seed=2, lb=-5.12, ub=5.12, clamp_x=1, gens=10),
    dict(fn=0, N=3, D=5, seed=7, lb=-1.0, ub=1.0, gens=10),
    dict(fn=0, N=2, D=1, seed=8, lb=-1.0, ub=1.0, gens=10),
]


@pytest.mark.parametrize("case", LOCAL_CASES, ids=[f"fn{c['fn']}-{c['N']}x{c['D']}" for c in LOCAL_CASES])
def test_neighbourhood_version_matches_oracle(evox_gpu, ref, case):
    """The ring means are computed in the oracle's fp64 order, so rows and
    velocities match bit for bit generation after generation."""
    c = dict(case)
    gens = c.pop("gens")
    print(f"cso local {c} gens={gens}", flush=True)
    g, r = pair(evox_gpu, ref, cso_local=1, **c)
    for t in range(gens):
        g.step(1)
        r.step(1)
        compare(g, r, c["fn"], f"generation {t}")
    assert g.t == r.t


def test_neighbourhood_version_several_generations_per_call(evox_gpu, ref):
    """Calls of 2, 3 and 4 generations: the positions alternate between the
    caller's x and the second buffer inside a call, and an odd count ends
    with the copy back into x; rows, velocities and padding must be exact."""
    c = dict(fn=3, N=501, D=29, seed=5, lb=-600.0, ub=600.0)
    print(f"cso local multi {c}", flush=True)
    g, r = pair(evox_gpu, ref, cso_local=1, **c)
    for n in (2, 3, 4):
        g.step(n)
        r.step(n)
        compare(g, r, c["fn"], f"after a call of {n}")
        assert not g.x[:, c["D"]:].any(), "padding columns must stay zero"


def test_neighbourhood_version_equals_swarm_version_at_three(evox_gpu, ref):
    a, _ = pair(evox_gpu, ref, 0, 3, 9, 12, -5.0, 5.0)
    b, _ = pair(evox_gpu, ref, 0, 3, 9, 12, -5.0, 5.0, cso_local=1)
    a.step(8)
    b.step(8)
    for name in ("x", "v", "fit"):
        assert torch.equal(getattr(a, name), getattr(b, name)), name


def test_neighbourhood_flag_only_for_cso(evox_gpu):
    import paper_2301_12457_amd as ev
    with pytest.raises(ev.EvoxError):
        ev.Swarm(ev.make_params(ev.PSO, 0, 10, 5, -1.0, 1.0, cso_local=1))
    with pytest.raises(ev.EvoxError):
        ev.Swarm(ev.make_params(ev.CSO, 0, 10, 5, -1.0, 1.0, cso_local=2))
