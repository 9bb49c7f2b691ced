"""Rows at 1024 lanes per row group, the widest layouts: D just past each
step of the chunk count the kernels are compiled for (1, 2, 4 and 8 float4
chunks per lane) up to the largest D, for every algorithm, against the
oracle (PSO, CSO, DE bit for bit; ES in lockstep within its bound)."""
import numpy as np
import pytest
import torch

from parity import assert_fitness, cso_lockstep, tol

pytestmark = pytest.mark.gpu

WIDE_D = [4097, 8193, 16385, 32768]


@pytest.mark.parametrize("D", WIDE_D)
@pytest.mark.parametrize("fn", [1, 4])
def test_pso_wide(evox_gpu, ref, D, fn):
    print(f"pso wide fn={fn} D={D}", flush=True)
    kw = dict(seed=D + fn, v_lo=-0.5, v_hi=0.5, vmax=1.0)
    g = evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.PSO, fn, 6, D, -2.0, 2.0, **kw))
    r = ref.PSO(ref.make_params(fn, 6, D, -2.0, 2.0, **kw))
    g.step(4)
    r.step(4)
    assert np.array_equal(g.x[:, :D].cpu().numpy(), r.x)
    assert np.array_equal(g.v[:, :D].cpu().numpy(), r.v)
    assert_fitness(fn, r.p, g.pfit.cpu().numpy(), r.pf, f"pso D {D}")
    assert g.best()[1] == r.gi


@pytest.mark.parametrize("D", WIDE_D)
def test_cso_wide(evox_gpu, ref, D):
    print(f"cso wide D={D}", flush=True)
    g = evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.CSO, 3, 9, D, -600.0, 600.0, seed=D))
    r = ref.CSO(ref.make_params(3, 9, D, -600.0, 600.0, seed=D))
    for t in range(3):
        cso_lockstep(ref, g, r, f"cso D {D} generation {t}")
        assert np.array_equal(g.x[:, :D].cpu().numpy(), r.x), t
        assert np.array_equal(g.v[:, :D].cpu().numpy(), r.v), t
        assert_fitness(3, r.x, g.fit.cpu().numpy(), r.fit, f"cso D {D}")


@pytest.mark.parametrize("D", WIDE_D)
def test_de_wide(evox_gpu, ref, D):
    print(f"de wide D={D}", flush=True)
    g = evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.DE, 2, 8, D, -5.12, 5.12, seed=D))
    r = ref.DE(ref.make_params(2, 8, D, -5.12, 5.12, seed=D))
    g.step(3)
    r.step(3)
    assert np.array_equal(g.x[:, :D].cpu().numpy(), r.x)
    assert_fitness(2, r.x, g.fit.cpu().numpy(), r.fit, f"de D {D}")


@pytest.mark.parametrize("D", WIDE_D)
def test_es_wide(evox_gpu, ref, D):
    print(f"es wide D={D}", flush=True)
    kw = dict(seed=D, es_sigma=0.1, es_lr=0.01)
    g = evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.ES, 0, 8, D, -1.0, 1.0, **kw))
    r = ref.ES(ref.make_params(0, 8, D, -1.0, 1.0, **kw))
    assert np.array_equal(g.x[:D].cpu().numpy(), r.theta)
    theta0 = r.theta.astype(np.float64).copy()
    g.step(1)
    r.step(1)
    X = np.broadcast_to(np.abs(theta0) + 0.6, (8, D))
    f_gpu, f_ref = g.fit.cpu().numpy().astype(np.float64), r.fit.astype(np.float64)
    assert np.all(np.abs(f_gpu - f_ref) <= 2.0 * tol(0, X, f_ref))
    ulp = lambda v: np.spacing(np.abs(v).astype(np.float32)).astype(np.float64)
    gref = np.abs(theta0 - r.theta) / 0.01
    bound = 0.01 * (3e-6 / 0.1 + 2.0 * ulp(gref)) + 2.0 * ulp(r.theta)
    assert np.all(np.abs(g.x[:D].cpu().numpy().astype(np.float64) - r.theta) <= bound)
