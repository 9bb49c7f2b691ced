"""GPU parity on seeded random shapes: PSO, CSO (both versions) and DE with
a random function, population, dimension, seed, generation count and
options, against the oracle.  Positions (and velocities, personal bests) must
match bit for bit; the one accepted difference is a PSO call whose final
global-best choice is a tolerance tie (two personal bests closer than the
fp32 evaluation error), which moves every row toward another gbest."""
import math
import random

import numpy as np
import pytest

from parity import cso_lockstep, tol

pytestmark = pytest.mark.gpu

BOUNDS = {0: (-32.0, 32.0), 1: (-32.768, 32.768), 2: (-5.12, 5.12), 3: (-600.0, 600.0), 4: (-2.048, 2.048),
          5: (-500.0, 500.0)}


def make_cases(seed, n, big):
    rng = random.Random(seed)
    cases = []
    for _ in range(n):
        algo = rng.choice(["pso", "pso", "cso", "cso_local", "de"])
        fn = rng.randrange(6)
        D = int(round(math.exp(rng.uniform(math.log(64) if big else 0.0, math.log(4100 if big else 2100)))))
        N = int(round(math.exp(rng.uniform(math.log(64 if big else 2), math.log(4000 if big else 3000)))))
        while N * D > (2_000_000 if big else 500_000):
            N = max(2, N // 2)
        if algo == "de":
            N = max(N, 4)
        kw = {}
        if algo == "pso" and rng.random() < 0.5:
            lb, ub = BOUNDS[fn]
            kw["vmax"] = 0.2 * (ub - lb)
        if rng.random() < 0.3:
            kw["clamp_x"] = 1
        if algo == "pso" and rng.random() < 0.5:
            kw["v_lo"], kw["v_hi"] = -1.0, 1.0
        cases.append(dict(algo=algo, fn=fn, N=N, D=D, seed=rng.randrange(1 << 30), gens=rng.randrange(1, 6), kw=kw))
    return cases


CASES = make_cases(2024, 40, False) + make_cases(2025, 20, True)


@pytest.mark.parametrize("c", CASES, ids=[f"{c['algo']}-fn{c['fn']}-{c['N']}x{c['D']}-g{c['gens']}" for c in CASES])
def test_random_shape_matches_oracle(evox_gpu, ref, c):
    ev = evox_gpu
    fn, N, D, seed, gens, kw = c["fn"], c["N"], c["D"], c["seed"], c["gens"], c["kw"]
    lb, ub = BOUNDS[fn]
    print(f"{c}", flush=True)
    if c["algo"] == "pso":
        g = ev.Swarm(ev.make_params(ev.PSO, fn, N, D, lb, ub, seed=seed, **kw))
        r = ref.PSO(ref.make_params(fn, N, D, lb, ub, seed=seed, **kw))
        g.step(gens)
        r.step(gens)
        x, v, p = (t[:, :D].cpu().numpy() for t in (g.x, g.v, g.pbest))
        if not (np.array_equal(x, r.x) and np.array_equal(v, r.v) and np.array_equal(p, r.p)):
            gf, gi = g.best()
            pf = r.pf.astype(np.float64)
            assert gi != r.gi and abs(pf[gi] - pf[r.gi]) <= float(tol(fn, r.p[[r.gi]], r.pf[[r.gi]])[0]), \
                "PSO state differs from the oracle without a tolerance tie of the final selection"
            assert np.array_equal(p, r.p), "personal bests differ"
    elif c["algo"] in ("cso", "cso_local"):
        local = c["algo"] == "cso_local"
        g = ev.Swarm(ev.make_params(ev.CSO, fn, N, D, lb, ub, seed=seed, cso_local=int(local), **kw))
        r = ref.CSO(ref.make_params(fn, N, D, lb, ub, seed=seed, cso_local=int(local), **kw))
        for t in range(gens):
            if local:
                g.step(1)
                r.step(1)
            else:
                cso_lockstep(ref, g, r, f"generation {t}")
        assert np.array_equal(g.x[:, :D].cpu().numpy(), r.x), "x"
        assert np.array_equal(g.v[:, :D].cpu().numpy(), r.v), "v"
    else:
        g = ev.Swarm(ev.make_params(ev.DE, fn, N, D, lb, ub, seed=seed, **kw))
        r = ref.DE(ref.make_params(fn, N, D, lb, ub, seed=seed, **kw))
        g.step(gens)
        r.step(gens)
        assert np.array_equal(g.x[:, :D].cpu().numpy(), r.x), "x"
