"""GPU parity of the OpenES generation against the oracle, in lockstep.

The perturbations are Box-Muller deviates: fp32 with the device logf and
hardware cosine on the GPU, fp64 in the oracle, so the samples differ in the
last bits (by at most sigma 1e-6 max(1, |z|) + 1 ulp, the bound of the normal
population) and nothing downstream is bit-exact.  Each generation therefore
starts both sides from the oracle's center (inputs flow from the oracle to the
GPU only) and checks: sample fitness within twice the fitness tolerance (the
second half covers the sample difference, 1e-6 relative against the 1e-5 of
the tolerance); the ranks equal wherever the oracle's fitness has no
tolerance tie between neighbours; the new center within the bound that the
perturbation difference puts on the gradient:
    |theta_gpu - theta_ref| <= lr (3e-6 / sigma + 2 ulp(g)) + 2 ulp(theta).
"""
import numpy as np
import pytest
import torch

from parity import tol

pytestmark = pytest.mark.gpu


def pair(evox, ref, fn, N, D, seed, lb, ub, **kw):
    g = evox.Swarm(evox.make_params(evox.ES, fn, N, D, lb, ub, seed=seed, **kw))
    r = ref.ES(ref.make_params(fn, N, D, lb, ub, seed=seed, **kw))
    return g, r


def ranks(f):
    order = np.lexsort((np.arange(f.size), f))
    out = np.empty(f.size, np.int64)
    out[order] = np.arange(f.size)
    return out


def lockstep(evox, ref, g, r, fn, what):
    D = r.P.D
    g.x[:D] = torch.from_numpy(r.theta).cuda()
    theta0 = r.theta.astype(np.float64).copy()
    g.step(1)
    r.step(1)
    f_gpu, f_ref = g.fit.cpu().numpy().astype(np.float64), r.fit.astype(np.float64)
    # the samples themselves are not stored; the fitness scale S of the
    # tolerance is taken with the center's magnitude, which bounds theirs
    # to within sigma * 6 per element
    xs = np.abs(theta0) + 6.0 * r.P.es_sigma
    X = np.broadcast_to(xs, (f_ref.size, D))
    assert np.all(np.abs(f_gpu - f_ref) <= 2.0 * tol(fn, X, f_ref)), f"{what}: sample fitness"
    srt = np.sort(f_ref)
    gaps = np.diff(srt)
    if gaps.size == 0 or gaps.min() > 4.0 * tol(fn, X[:1], srt[:1]).max():
        assert np.array_equal(ranks(f_gpu.astype(np.float32)), r.rank), f"{what}: ranks"
    th_gpu = g.x[:D].cpu().numpy().astype(np.float64)
    th_ref = r.theta.astype(np.float64)
    lr, sigma = r.P.es_lr, r.P.es_sigma
    gref = np.abs(theta0 - th_ref) / lr
    ulp = lambda v: np.spacing(np.abs(v).astype(np.float32)).astype(np.float64)
    bound = lr * (3e-6 / sigma + 2.0 * ulp(gref)) + 2.0 * ulp(th_ref)
    bad = np.nonzero(np.abs(th_gpu - th_ref) > bound)[0]
    assert bad.size == 0, f"{what}: center off at {bad[:5]}, {th_gpu[bad[:3]]} vs {th_ref[bad[:3]]}"
    bf, bi = g.best()
    assert bi == r.best_idx or abs(f_ref[bi] - f_ref[r.best_idx]) <= 2 * tol(fn, X[:1], f_ref[[bi]]).max()


CASES = [
    dict(fn=0, N=200, D=50, seed=1, lb=-5.0, ub=5.0, es_sigma=0.1, es_lr=0.05, gens=6),
    dict(fn=2, N=64, D=257, seed=2, lb=-5.12, ub=5.12, es_sigma=0.2, es_lr=0.01, gens=4),
    dict(fn=1, N=1000, D=33, seed=3, lb=-32.768, ub=32.768, es_sigma=0.5, es_lr=0.1, gens=3),
    dict(fn=4, N=2, D=1001, seed=4, lb=-2.0, ub=2.0, es_sigma=0.01, es_lr=0.001, gens=3),
    dict(fn=0, N=16384, D=3, seed=5, lb=-1.0, ub=1.0, es_sigma=0.1, es_lr=0.1, gens=2),
]


@pytest.mark.parametrize("case", CASES, ids=[f"fn{c['fn']}-{c['N']}x{c['D']}" for c in CASES])
def test_lockstep_generations(evox_gpu, ref, case):
    c = dict(case)
    gens = c.pop("gens")
    print(f"es {c} gens={gens}", flush=True)
    g, r = pair(evox_gpu, ref, **c)
    assert np.array_equal(g.x[:c["D"]].cpu().numpy(), r.theta)      # first center, exact
    for t in range(gens):
        lockstep(evox_gpu, ref, g, r, c["fn"], f"generation {t}")


def test_free_running_descends_and_resumes(evox_gpu, ref):
    kw = dict(fn=0, N=256, D=40, seed=7, lb=-5.0, ub=5.0, es_sigma=0.1, es_lr=0.05)
    a, _ = pair(evox_gpu, ref, **kw)
    b, _ = pair(evox_gpu, ref, **kw)
    f0 = float((a.x[:40].double() ** 2).sum())
    a.step(100)
    for n in (1, 30, 69):
        b.step(n)
    assert torch.equal(a.x, b.x) and torch.equal(a.fit, b.fit)
    assert float((a.x[:40].double() ** 2).sum()) < 0.2 * f0
    bf, bi, center = a.best(with_x=True)
    assert bf == float(a.fit.min()) and a.fit[bi] == bf
    assert np.array_equal(center, a.x[:40].cpu().numpy())          # the solution is the center


def test_rejects_bad_population(evox_gpu):
    for N in (1, 7, 16386):
        with pytest.raises(evox_gpu.EvoxError):
            evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.ES, 0, N, 5, -1.0, 1.0))
