"""GPU parity of the initial populations: the normal population of Philox
stream 5 (evox_fill_normal and x_init = 1 states) against the oracle's fp64
Box-Muller, within the bound derived in parity.normal_tol; and a normal-init
state, once given the oracle's positions, evolving bit for bit like it."""
import numpy as np
import pytest
import torch

from parity import normal_tol

pytestmark = pytest.mark.gpu


def assert_normal_close(x_gpu, x_ref, mu, sigma, what):
    err = np.abs(x_gpu.astype(np.float64) - x_ref.astype(np.float64))
    bound = normal_tol(x_ref, mu, sigma)
    bad = np.argwhere(err > bound)
    assert bad.size == 0, f"{what}: {len(bad)} elements off, e.g. {bad[:4].tolist()}"


@pytest.mark.parametrize("N,D,ldx,mu,sigma,seed", [(300, 37, 40, 1.0, 0.5, 5), (64, 100, 128, 0.0, 1.0, 0),
                                                   (5, 1, 4, -3.0, 2.0, 2**64 - 1),
                                                   (17, 1001, 1024, 1.0, 0.5, 4)])
def test_fill_normal_matches_oracle(evox_gpu, ref, N, D, ldx, mu, sigma, seed):
    print(f"fill_normal N={N} D={D} ldx={ldx}", flush=True)
    X = torch.full((N, ldx), 7.0, dtype=torch.float32, device="cuda")
    evox_gpu.evox_fill_normal(seed, N, D, ldx, mu, sigma, X)
    Xh = X.cpu().numpy()
    assert np.all(Xh[:, D:] == 0)
    assert_normal_close(Xh[:, :D], ref.init_normal(seed, N, D, mu, sigma), mu, sigma, "fill")


def test_fill_normal_full_size_sampled_rows(evox_gpu, ref):
    """The evaluation workload's population (1,048,576 x 1000, N(1, 0.5^2)):
    sampled rows against the oracle, moments of the whole matrix."""
    N, D, mu, sigma, seed = 1_048_576, 1000, 1.0, 0.5, 4
    X = torch.empty((N, D), dtype=torch.float32, device="cuda")
    evox_gpu.evox_fill_normal(seed, N, D, D, mu, sigma, X)
    rng = np.random.default_rng(7)
    rows = np.concatenate([[0, 1, N - 1], rng.integers(0, N, size=29)])
    got = X[torch.from_numpy(rows).cuda()].cpu().numpy()
    for k, i in enumerate(rows):
        z = np.array([ref.normal01(seed, int(i), j) for j in range(D)])
        want = (mu + sigma * z).astype(np.float32)
        assert_normal_close(got[k], want, mu, sigma, f"row {i}")
    m = X.double().mean().item()
    s = X.double().std().item()
    assert abs(m - mu) < 1e-3 and abs(s - sigma) < 1e-3


@pytest.mark.parametrize("algo", [0, 1])
def test_normal_state_init_and_lockstep(evox_gpu, ref, algo):
    N, D, fn, seed = 200, 30, 4, 23
    kw = dict(seed=seed, x_init=1, x_mu=1.0, x_sigma=0.5)
    g = evox_gpu.Swarm(evox_gpu.make_params(algo, fn, N, D, -2.0, 2.0, **kw))
    Ref = ref.PSO if algo == 0 else ref.CSO
    r = Ref(ref.make_params(fn, N, D, -2.0, 2.0, **kw))
    assert_normal_close(g.x[:, :D].cpu().numpy(), r.x, 1.0, 0.5, "state init")
    assert torch.all(g.v == 0)
    # from the oracle's positions on, the two evolve identically
    g.x[:, :D] = torch.from_numpy(r.x).cuda()
    if algo == 0:
        g.pbest[:, :D] = torch.from_numpy(r.x).cuda()
    else:
        g.refresh(refit=True)
        r.fit[:] = ref.evaluate(fn, r.x)
        if not np.array_equal(g.xbar[:D].cpu().numpy(), ref.colmean(r.x)):
            pytest.skip("swarm means differ by an ulp: no bit-exact lockstep")
    g.step(5)
    r.step(5)
    assert np.array_equal(g.x[:, :D].cpu().numpy(), r.x)
    assert np.array_equal(g.v[:, :D].cpu().numpy(), r.v)
