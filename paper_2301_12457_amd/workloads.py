"""The benchmark workloads and seeded synthetic inputs.

Holds none of the method's arithmetic: only the sizes and hyperparameters of
each workload and seeded generators of input matrices, shared by the tests
and the benchmark.  The populations of the PSO / CSO workloads are drawn by
the method itself (Philox streams 0 and 1 at creation); the evaluation-only
workload's population is the library's normal population (Philox stream 5,
evox_fill_normal) in the benchmark, and a matrix of the same distribution
generated here wherever the oracle must see the very same input (the oracle
never reads what the GPU path produced).

The shapes stand in for the paper's large-scale numerical experiments
(Sec. VII-A-1: population and dimension scaling on Sphere, populations up to
about a million): synthetic, seeded, no dataset.
"""
import math
from dataclasses import dataclass, field

PSO, CSO, DE, ES, PGPE, MAES, NSGA2, EVAL = "pso", "cso", "de", "es", "pgpe", "maes", "nsga2", "eval"


@dataclass(frozen=True)
class Workload:
    name: str
    algo: str
    fn: str
    N: int
    D: int
    gens: int
    seed: int
    lb: float = 0.0
    ub: float = 0.0
    v_lo: float = 0.0
    v_hi: float = 0.0
    w: float = 0.6
    c1: float = 1.5
    c2: float = 1.5
    phi: float = 0.1
    vmax: float = 0.0
    x_mu: float = 0.0      # evaluation-only input: x ~ N(x_mu, x_sigma^2)
    x_sigma: float = 0.0
    de_f: float = 0.5      # DE differential weight and crossover rate
    de_cr: float = 0.9
    es_sigma: float = 0.1  # OpenES perturbation scale (PGPE: initial deviation) and learning rate
    es_lr: float = 0.01
    pgpe_sigma_lr: float = 0.01
    pgpe_max_change: float = 0.2
    n_obj: int = 3
    cso_local: int = 0


WORKLOADS = {
    "pso_sphere_100x10": Workload("pso_sphere_100x10", PSO, "sphere", 100, 10, 100, 0,
                                  lb=-32.0, ub=32.0),
    "pso_ackley_1e4x1e3": Workload("pso_ackley_1e4x1e3", PSO, "ackley", 10_000, 1_000, 1_000, 1,
                                   lb=-32.768, ub=32.768, v_lo=-1.0, v_hi=1.0),
    "pso_rastrigin_1e5x1e3": Workload("pso_rastrigin_1e5x1e3", PSO, "rastrigin", 100_000, 1_000,
                                      200, 2, lb=-5.12, ub=5.12, vmax=0.2 * 10.24),
    "cso_griewank_1e6x100": Workload("cso_griewank_1e6x100", CSO, "griewank", 1_000_000, 100, 200,
                                     3, lb=-600.0, ub=600.0, phi=0.1),
    "cso_local_griewank_1e6x100": Workload("cso_local_griewank_1e6x100", CSO, "griewank", 1_000_000, 100,
                                           200, 3, lb=-600.0, ub=600.0, phi=0.1, cso_local=1),
    "de_sphere_1e5x1e3": Workload("de_sphere_1e5x1e3", DE, "sphere", 100_000, 1_000, 200, 5,
                                  lb=-32.0, ub=32.0),
    "es_sphere_1e4x1e4": Workload("es_sphere_1e4x1e4", ES, "sphere", 10_000, 10_000, 100, 6,
                                  lb=-5.0, ub=5.0, es_sigma=0.1, es_lr=0.05),
    "pgpe_sphere_1e4x1e4": Workload("pgpe_sphere_1e4x1e4", PGPE, "sphere", 10_000, 10_000, 100, 7,
                                    lb=-5.0, ub=5.0, es_sigma=1.0, es_lr=0.5, pgpe_sigma_lr=0.1),
    "maes_sphere_100x16384": Workload("maes_sphere_100x16384", MAES, "sphere", 100, 16_384, 20, 10,
                                      lb=-5.0, ub=5.0, es_sigma=1.0),
    "maes_sphere_4096x1830": Workload("maes_sphere_4096x1830", MAES, "sphere", 4096, 1830, 10, 12,
                                      lb=-5.0, ub=5.0, es_sigma=1.0),
    "nsga2_dtlz1_16384x100": Workload("nsga2_dtlz1_16384x100", NSGA2, "dtlz1", 16_384, 100, 10, 11,
                                      lb=0.0, ub=1.0, n_obj=3),
    "eval_rosenbrock_1m_x1e3": Workload("eval_rosenbrock_1m_x1e3", EVAL, "rosenbrock", 1_048_576,
                                        1_000, 1, 4, x_mu=1.0, x_sigma=0.5),
}


def normal_matrix_torch(N, D, mu, sigma, seed, device="cuda", ldx=None):
    """Seeded x ~ N(mu, sigma^2) of shape [N, ldx] (padding zero), made on the device."""
    import torch
    ldx = D if ldx is None else ldx
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    X = torch.zeros((N, ldx), dtype=torch.float32, device=device)
    X[:, :D].normal_(mu, sigma, generator=g)
    return X


def uniform_matrix_np(N, D, lo, hi, seed):
    import numpy as np
    rng = np.random.default_rng(seed)
    return rng.uniform(lo, hi, size=(N, D)).astype(np.float32)


def normal_matrix_np(N, D, mu, sigma, seed):
    import numpy as np
    rng = np.random.default_rng(seed)
    return rng.normal(mu, sigma, size=(N, D)).astype(np.float32)


def swarm_state_np(N, D, lb, ub, seed, spread, chunk=16384):
    """Seeded positions, velocities and personal bests shaped like a swarm
    part-way through a run: every individual near one common point
    c ~ U[lb, ub]^D, with s = spread * (ub - lb),
        x = c + s e1,   p = x + (s / 2) e2,   v = (s / 10) e3,
    e_k standard normal; float32 [N, D] each, drawn chunk by chunk so that
    large populations need no float64 temporaries."""
    import numpy as np
    rng = np.random.default_rng(seed)
    c = rng.uniform(lb, ub, size=D).astype(np.float32)
    s = np.float32(spread * (ub - lb))
    x = np.empty((N, D), np.float32)
    p = np.empty((N, D), np.float32)
    v = np.empty((N, D), np.float32)
    for a in range(0, N, chunk):
        b = min(N, a + chunk)
        x[a:b] = c + s * rng.standard_normal((b - a, D), dtype=np.float32)
        p[a:b] = x[a:b] + (s / 2) * rng.standard_normal((b - a, D), dtype=np.float32)
        v[a:b] = (s / 10) * rng.standard_normal((b - a, D), dtype=np.float32)
    return x, v, p
