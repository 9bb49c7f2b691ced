"""GPU parity of NSGA-II on DTLZ1 against the oracle.

The sorting step (fronts and crowding distances) takes its decisions on the
same fp32 objectives as the oracle and sums the distances in the oracle's
order in fp64, so on identical inputs it must agree bit for bit.  A whole
generation differs from the oracle only where fp64 pow (the crossover and
mutation) or fp64 cos (DTLZ1, summed in another order) round differently,
which moves a child or an objective by at most an ulp after rounding to
fp32; each generation starts both sides from the oracle's state and
compares the survivors within that, and their fronts exactly.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def gpu_sort(evox, F):
    Fd = torch.from_numpy(np.ascontiguousarray(F, np.float32)).cuda()
    front = torch.empty(F.shape[0], dtype=torch.int32, device="cuda")
    crowd = torch.empty(F.shape[0], dtype=torch.float64, device="cuda")
    evox.evox_nsga2_sort(Fd, front, crowd)
    return front.cpu().numpy(), crowd.cpu().numpy()


def dtlz1_population(ref, n, D, M, seed):
    X = np.random.default_rng(seed).random((n, D)).astype(np.float32)
    return ref.dtlz1(X, M)


CASES = [("ties", 1, 2), ("ties", 5, 3), ("ties", 100, 2), ("ties", 1000, 3), ("ties", 3001, 4),
         ("dtlz1", 200, 3), ("dtlz1", 2048, 3), ("dtlz1", 1500, 5), ("dtlz1", 600, 8), ("line", 300, 2)]


@pytest.mark.parametrize("kind,n,M", CASES, ids=[f"{k}-{n}x{m}" for k, n, m in CASES])
def test_sort_matches_oracle_bit_for_bit(evox_gpu, ref, kind, n, M):
    print(f"nsga2 sort {kind} n={n} M={M}", flush=True)
    rng = np.random.default_rng(n + M)
    if kind == "ties":
        F = rng.integers(0, 8, size=(n, M)).astype(np.float32)
    elif kind == "dtlz1":
        F = dtlz1_population(ref, n, 12, M, n)
    else:                                   # a chain: n fronts of one point
        F = np.repeat(np.arange(n, dtype=np.float32)[::-1, None], M, axis=1).copy()
    front, crowd = gpu_sort(evox_gpu, F)
    want_front = ref.nds(F)
    assert np.array_equal(front, want_front)
    assert np.array_equal(crowd, ref.crowding(F, want_front))


def test_sort_full_merged_size(evox_gpu, ref):
    """2N = 32768 points of a DTLZ1 population (N = 16384, D = 100, M = 3):
    the fronts' defining properties on sampled points, and the crowding of
    sampled fronts against the oracle's crowding of that front alone."""
    n, M = 32768, 3
    F = dtlz1_population(ref, n, 100, M, 3)
    front, crowd = gpu_sort(evox_gpu, F)
    Fd = F.astype(np.float64)
    rng = np.random.default_rng(4)
    for i in rng.choice(n, 64, replace=False):
        dom = np.all(Fd <= Fd[i], axis=1) & np.any(Fd < Fd[i], axis=1)
        if front[i] == 0:
            assert not dom.any()
        else:
            assert dom[front == front[i] - 1].any()
        assert not dom[front == front[i]].any()
    for k in sorted(set([0, 1, int(front.max()) // 2, int(front.max())])):
        members = np.nonzero(front == k)[0]
        want = ref.crowding(F[members], np.zeros(members.size, np.int32))
        assert np.array_equal(crowd[members], want), k


def push(g, r):
    D = r.P.D
    g.x[:, :D] = torch.from_numpy(r.X).cuda()
    g.obj.copy_(torch.from_numpy(r.F).cuda())
    g.front.copy_(torch.from_numpy(r.front).cuda())
    g.crowd.copy_(torch.from_numpy(r.crowd).cuda())


def ulps(a, b):
    ai = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    bi = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    return np.abs(ai - bi)


GEN_CASES = [dict(N=8, D=4, M=3, seed=1, gens=5), dict(N=100, D=12, M=3, seed=2, gens=4),
             dict(N=64, D=30, M=2, seed=3, gens=4), dict(N=200, D=10, M=5, seed=4, gens=3),
             dict(N=1000, D=100, M=3, seed=5, gens=2)]


@pytest.mark.parametrize("case", GEN_CASES, ids=[f"{c['N']}x{c['D']}x{c['M']}" for c in GEN_CASES])
def test_lockstep_generations(evox_gpu, ref, case):
    c = dict(case)
    gens = c.pop("gens")
    print(f"nsga2 {c} gens={gens}", flush=True)
    P = evox_gpu.make_params(evox_gpu.NSGA2, 0, c["N"], c["D"], 0.0, 1.0, seed=c["seed"], n_obj=c["M"])
    g = evox_gpu.Swarm(P)
    r = ref.NSGA2(ref.nsga2_params(c["N"], c["D"], c["M"], seed=c["seed"]))
    D = c["D"]
    # the initial state: the uniform population, its objectives and sorting
    assert np.array_equal(g.x[:, :D].cpu().numpy(), r.X)
    assert np.all(ulps(g.obj.cpu().numpy(), r.F) <= 1)
    exact = 0
    for k in range(gens):
        push(g, r)
        g.step(1)
        r.step(1)
        X, F = g.x[:, :D].cpu().numpy(), g.obj.cpu().numpy()
        front, crowd = g.front.cpu().numpy(), g.crowd.cpu().numpy()
        assert np.all(ulps(X, r.X) <= 2), f"gen {k}: survivors' rows"
        assert np.all(ulps(F, r.F) <= 2), f"gen {k}: objectives"
        assert np.array_equal(front, r.front), f"gen {k}: fronts"
        same = np.isinf(crowd) == np.isinf(r.crowd)
        fin = ~np.isinf(r.crowd)
        assert same.all() and np.allclose(crowd[fin], r.crowd[fin], rtol=1e-5, atol=1e-12), f"gen {k}: crowding"
        exact += np.array_equal(X, r.X) and np.array_equal(F, r.F) and np.array_equal(crowd, r.crowd)
    print(f"  bit-exact generations: {exact} of {gens}", flush=True)


def test_free_run_converges_and_resumes(evox_gpu):
    import paper_2301_12457_amd as ev
    P = ev.make_params(ev.NSGA2, 0, 128, 12, 0.0, 1.0, seed=6, n_obj=3)
    a, b = ev.Swarm(P), ev.Swarm(P)
    s0 = float(a.obj.double().sum(1).mean())
    a.step(60)
    for n in (1, 19, 40):
        b.step(n)
    torch.cuda.synchronize()
    for u, v in ((a.x, b.x), (a.obj, b.obj), (a.front, b.front), (a.crowd, b.crowd)):
        assert torch.equal(u, v)
    assert float(a.obj.double().sum(1).mean()) < 0.05 * s0
    x = a.x[:, :12]
    assert bool(((x >= 0) & (x <= 1)).all())


def test_rejects_bad_arguments(evox_gpu):
    import paper_2301_12457_amd as ev
    for N, D, M in ((7, 10, 3), (2, 10, 3), (32770, 10, 3), (10, 2, 3), (10, 10, 9)):
        with pytest.raises(ev.EvoxError):
            ev.Swarm(ev.make_params(ev.NSGA2, 0, N, D, 0.0, 1.0, n_obj=M))
    L = ev.lib()
    assert L.evox_nsga2_sort_scratch_bytes(0, 3) == 0 and L.evox_nsga2_sort_scratch_bytes(10, 1) == 0
    s = ev.Swarm(ev.make_params(ev.NSGA2, 0, 8, 4, 0.0, 1.0, n_obj=3))
    with pytest.raises(ev.EvoxError):
        s.best()
