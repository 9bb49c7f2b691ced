"""GPU parity of the DE/rand/1/bin generation against the oracle.

Partner choice, crossover and mutant are exact integer / fp32 work, so the
population must match bit for bit; fitness within the fitness tolerance; the
best index exactly.  Odd and even generation counts cover the return of the
population from the second buffer.
"""
import numpy as np
import pytest
import torch

from parity import assert_fitness, index_ok

pytestmark = pytest.mark.gpu


def pair(evox, ref, fn, N, D, seed, lb, ub, ldx=None, **kw):
    g = evox.Swarm(evox.make_params(evox.DE, fn, N, D, lb, ub, seed=seed, ldx=ldx, **kw))
    r = ref.DE(ref.make_params(fn, N, D, lb, ub, seed=seed, **kw))
    return g, r


def compare(g, r, fn, what):
    D = r.P.D
    x = g.x[:, :D].cpu().numpy()
    bad = np.nonzero((x != r.x).any(1))[0]
    assert bad.size == 0, f"{what}: x differs in rows {bad[:8]}"
    assert_fitness(fn, r.x, g.fit.cpu().numpy(), r.fit, f"{what}: fit")
    bf, bi = g.best()
    assert index_ok(fn, r.x, r.fit, bi, r.best_idx), f"{what}: best {bi} vs {r.best_idx}"
    assert bi == r.best_idx, f"{what}: best index {bi} vs {r.best_idx} (tolerance tie)"
    if g.P.ldx > D:
        assert int((g.x[:, D:] != 0).sum()) == 0, f"{what}: padding written"


CASES = [
    dict(fn=0, N=100, D=10, seed=0, lb=-32.0, ub=32.0, gens=30),
    dict(fn=1, N=64, D=37, seed=1, lb=-32.768, ub=32.768, gens=15),
    dict(fn=2, N=33, D=257, seed=2, lb=-5.12, ub=5.12, gens=10, de_f=0.8, de_cr=0.3),
    dict(fn=3, N=200, D=100, seed=3, lb=-600.0, ub=600.0, gens=12),
    dict(fn=4, N=12, D=1001, seed=4, lb=-2.0, ub=2.0, gens=7),
    dict(fn=5, N=7, D=3, seed=5, lb=-500.0, ub=500.0, gens=25, de_cr=1.0),
    dict(fn=4, N=5, D=2050, seed=6, lb=-2.0, ub=2.0, gens=4),
    dict(fn=0, N=4, D=1, seed=8, lb=-1.0, ub=1.0, gens=20, de_cr=0.0),
]


@pytest.mark.parametrize("case", CASES, ids=[f"fn{c['fn']}-{c['N']}x{c['D']}" for c in CASES])
def test_generations_match_oracle(evox_gpu, ref, case):
    c = dict(case)
    gens = c.pop("gens")
    print(f"de {c} gens={gens}", flush=True)
    g, r = pair(evox_gpu, ref, **c)
    assert np.array_equal(g.x[:, :c["D"]].cpu().numpy(), r.x)
    assert_fitness(c["fn"], r.x, g.fit.cpu().numpy(), r.fit, "init fit")
    for t in range(gens):
        g.step(1)
        r.step(1)
        compare(g, r, c["fn"], f"generation {t}")
    assert g.t == r.t == gens


@pytest.mark.parametrize("D,ldx", [(37, 40), (10, 64), (1000, 1024), (100, 128)])
def test_pitched_states(evox_gpu, ref, D, ldx):
    g, r = pair(evox_gpu, ref, 2, 50, D, 12, -5.12, 5.12, ldx=ldx)
    assert g.P.ldx == ldx
    g.step(3)
    r.step(3)
    compare(g, r, 2, f"D {D} ldx {ldx}")


def test_multi_generation_call_equals_single_steps(evox_gpu, ref):
    kw = dict(fn=1, N=300, D=30, seed=12, lb=-32.768, ub=32.768)
    a, r = pair(evox_gpu, ref, **kw)
    b, _ = pair(evox_gpu, ref, **kw)
    a.step(21)
    for n in (1, 4, 9, 7):
        b.step(n)
    assert torch.equal(a.x, b.x) and torch.equal(a.fit, b.fit)
    assert a.best() == b.best()
    r.step(21)
    compare(a, r, 1, "21 generations in one call")


def test_greedy_selection_invariants(evox_gpu, ref):
    g, _ = pair(evox_gpu, ref, 0, 500, 20, 21, -5.0, 5.0)
    for _ in range(10):
        f0, x0 = g.fit.clone(), g.x.clone()
        g.step(1)
        assert torch.all(g.fit <= f0)
        kept = g.fit == f0
        assert torch.equal(g.x[kept], x0[kept])
    bf, bi = g.best()
    assert bf == float(g.fit.min()) and g.fit[bi] == bf


def test_normal_init(evox_gpu, ref):
    from parity import normal_tol
    g, r = pair(evox_gpu, ref, 4, 64, 40, 9, -2.0, 2.0, x_init=1, x_mu=1.0, x_sigma=0.5)
    x = g.x[:, :40].cpu().numpy().astype(np.float64)
    assert np.all(np.abs(x - r.x) <= normal_tol(r.x, 1.0, 0.5))


def test_rejects_small_population(evox_gpu):
    with pytest.raises(evox_gpu.EvoxError):
        evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.DE, 0, 3, 5, -1.0, 1.0))
