"""GPU parity of the PGPE generation against the oracle, in lockstep.

As for OpenES, the deviates are Box-Muller in fp32 on the GPU and fp64 in
the oracle (within 1e-6 max(1, |z|) <= 5.8e-6 of each other), so each
generation starts both sides from the oracle's center and deviations and
checks the sample fitness within twice the fitness tolerance, the ranks
away from tolerance ties, and the new center and deviations within the bound
the deviate difference puts on the gradients (sum_k |m_k| <= 1/2 and
sum_k |s_k| <= 1/2 over the pair weights; |d(z^2)| <= 2 |z| dz <= 6.7e-5):
    |mu_gpu - mu_ref|       <= lr (3e-6 sigma + 2 ulp(g_mu)) + 2 ulp(mu)
    |sigma_gpu - sigma_ref| <= sigma_lr (3.4e-5 sigma + 2 ulp(g_sigma)) + 2 ulp(sigma).
"""
import numpy as np
import pytest
import torch

from parity import tol

pytestmark = pytest.mark.gpu


def ulp(v):
    return np.spacing(np.abs(np.asarray(v)).astype(np.float32)).astype(np.float64)


def ranks(f):
    order = np.lexsort((np.arange(f.size), f))
    out = np.empty(f.size, np.int64)
    out[order] = np.arange(f.size)
    return out


CASES = [
    dict(fn=0, N=200, D=50, seed=1, lb=-5.0, ub=5.0, es_sigma=1.0, es_lr=0.5, pgpe_sigma_lr=0.1, gens=6),
    dict(fn=2, N=64, D=257, seed=2, lb=-5.12, ub=5.12, es_sigma=0.5, es_lr=0.1, pgpe_sigma_lr=0.05, gens=4),
    dict(fn=1, N=1000, D=33, seed=3, lb=-32.768, ub=32.768, es_sigma=2.0, es_lr=1.0, pgpe_sigma_lr=0.2,
         pgpe_max_change=0.1, gens=3),
    dict(fn=4, N=2, D=1001, seed=4, lb=-2.0, ub=2.0, es_sigma=0.05, es_lr=0.01, pgpe_sigma_lr=0.01, gens=3),
    dict(fn=0, N=8, D=32768, seed=5, lb=-1.0, ub=1.0, es_sigma=0.2, es_lr=0.1, pgpe_sigma_lr=0.1, gens=2),
]


@pytest.mark.parametrize("case", CASES, ids=[f"fn{c['fn']}-{c['N']}x{c['D']}" for c in CASES])
def test_lockstep_generations(evox_gpu, ref, case):
    c = dict(case)
    gens = c.pop("gens")
    fn, N, D = c["fn"], c["N"], c["D"]
    print(f"pgpe {c} gens={gens}", flush=True)
    kw = {k: v for k, v in c.items() if k not in ("fn", "N", "D", "lb", "ub")}
    g = evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.PGPE, fn, N, D, c["lb"], c["ub"], **kw))
    r = ref.PGPE(ref.make_params(fn, N, D, c["lb"], c["ub"], **kw))
    assert np.array_equal(g.x[:D].cpu().numpy(), r.mu) and np.array_equal(g.v[:D].cpu().numpy(), r.sigma)
    lr, slr = r.P.es_lr, r.P.pgpe_sigma_lr
    for t in range(gens):
        g.x[:D] = torch.from_numpy(r.mu).cuda()
        g.v[:D] = torch.from_numpy(r.sigma).cuda()
        mu0, s0 = r.mu.astype(np.float64).copy(), r.sigma.astype(np.float64).copy()
        g.step(1)
        r.step(1)
        X = np.broadcast_to(np.abs(mu0) + 6.0 * s0, (N, D))
        f_gpu, f_ref = g.fit.cpu().numpy().astype(np.float64), r.fit.astype(np.float64)
        assert np.all(np.abs(f_gpu - f_ref) <= 2.0 * tol(fn, X, f_ref)), f"generation {t}: fitness"
        srt = np.sort(f_ref)
        if N < 3 or np.diff(srt).min() > 4.0 * tol(fn, X[:1], srt[:1]).max():
            assert np.array_equal(ranks(f_gpu.astype(np.float32)), r.rank), f"generation {t}: ranks"
        mu_g, s_g = g.x[:D].cpu().numpy().astype(np.float64), g.v[:D].cpu().numpy().astype(np.float64)
        gm = np.abs(mu0 - r.mu) / lr
        gs = np.abs(s0 - r.sigma) / slr
        bm = lr * (3e-6 * s0 + 2.0 * ulp(gm)) + 2.0 * ulp(r.mu)
        bs = slr * (3.4e-5 * s0 + 2.0 * ulp(gs)) + 2.0 * ulp(r.sigma)
        assert np.all(np.abs(mu_g - r.mu) <= bm), f"generation {t}: center"
        assert np.all(np.abs(s_g - r.sigma) <= bs), f"generation {t}: deviations"
        assert np.all(s_g >= (1.0 - r.P.pgpe_max_change) * s0 * (1 - 1e-6))


def test_free_running_descends_resumes_and_reports_center(evox_gpu):
    kw = dict(seed=7, es_sigma=1.0, es_lr=0.5, pgpe_sigma_lr=0.1)
    a = evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.PGPE, 0, 100, 20, -5.0, 5.0, **kw))
    b = evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.PGPE, 0, 100, 20, -5.0, 5.0, **kw))
    f0 = float((a.x[:20].double() ** 2).sum())
    a.step(200)
    for n in (1, 99, 100):
        b.step(n)
    assert torch.equal(a.x, b.x) and torch.equal(a.v, b.v) and torch.equal(a.fit, b.fit)
    assert float((a.x[:20].double() ** 2).sum()) < 1e-2 * f0
    bf, bi, center = a.best(with_x=True)
    assert bf == float(a.fit.min()) and np.array_equal(center, a.x[:20].cpu().numpy())


def test_padding_and_bad_population(evox_gpu):
    g = evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.PGPE, 0, 10, 5, -1.0, 1.0, ldx=8, es_sigma=0.3))
    g.step(3)
    assert torch.all(g.v[5:] == 0) and torch.all(g.x[5:] == 0) and torch.all(g.v[:5] > 0)
    with pytest.raises(evox_gpu.EvoxError):
        evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.PGPE, 0, 7, 5, -1.0, 1.0))
