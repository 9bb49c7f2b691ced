"""Achieved fitness accuracy per benchmark function at the benchmark shapes.

The GPU evaluates in fp32 (row reductions as lane partials and a butterfly);
the oracle in fp64, rounded once.  For each function, on inputs drawn like
the workload that uses it (full population size where the oracle finishes in
seconds), the test prints the largest plain relative error
|F_gpu - F_ref| / |F_ref| and the largest error as a fraction of the
tolerance, and asserts:
  - plain relative error <= 1e-5 for the functions with non-negative terms
    (Sphere, Rosenbrock, Rastrigin evaluated as sum x^2 + 20 sin^2(pi x)),
    also near their optima where F is small;
  - the scaled tolerance (tests/parity.py) for Ackley, Griewank and Schwefel,
    whose terms cancel at their optima.
"""
import numpy as np
import pytest
import torch

from parity import tol

pytestmark = pytest.mark.gpu

# (function, rows, D, input) -- input: ("uniform", lo, hi) or ("normal", mu, sigma)
CASES = [
    ("pso_rastrigin_1e5x1e3", 2, 100_000, 1000, ("uniform", -5.12, 5.12)),
    ("rastrigin_near_optimum", 2, 20_000, 1000, ("normal", 0.0, 1e-3)),
    ("pso_ackley_1e4x1e3", 1, 10_000, 1000, ("uniform", -32.768, 32.768)),
    ("cso_griewank_1e6x100", 3, 1_000_000, 100, ("uniform", -600.0, 600.0)),
    ("eval_rosenbrock_1m_x1e3 (262144 rows)", 4, 262_144, 1000, ("normal", 1.0, 0.5)),
    ("sphere_1e5x1e3", 0, 100_000, 1000, ("uniform", -32.0, 32.0)),
    ("sphere_near_optimum", 0, 20_000, 1000, ("normal", 0.0, 1e-4)),
    ("schwefel_1e5x1e3", 5, 100_000, 1000, ("uniform", -500.0, 500.0)),
]
PLAIN = {0, 2, 4}


def inputs(N, D, spec, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    X = torch.empty((N, D), dtype=torch.float32, device="cuda")
    if spec[0] == "uniform":
        X.uniform_(spec[1], spec[2], generator=g)
    else:
        X.normal_(spec[1], spec[2], generator=g)
    return X


@pytest.mark.parametrize("name,fn,N,D,spec", CASES, ids=[c[0].split()[0] for c in CASES])
def test_fitness_accuracy(evox_gpu, ref, name, fn, N, D, spec):
    X = inputs(N, D, spec, seed=fn * 101 + D)
    out = torch.empty(N, dtype=torch.float32, device="cuda")
    evox_gpu.evox_eval(fn, X, out)
    Xh = X.cpu().numpy()
    del X
    f_gpu = out.cpu().numpy().astype(np.float64)
    f_ref = ref.evaluate(fn, Xh).astype(np.float64)
    err = np.abs(f_gpu - f_ref)
    with np.errstate(divide="ignore", invalid="ignore"):
        plain = np.where(f_ref != 0, err / np.abs(f_ref), np.where(err == 0, 0.0, np.inf))
    of_tol = err / tol(fn, Xh, f_ref)
    print(f"accuracy {name}: max plain relative error {plain.max():.3e}, "
          f"max error / tolerance {of_tol.max():.3f}", flush=True)
    if fn in PLAIN:
        assert plain.max() <= 1e-5, f"{name}: plain relative error {plain.max():.3e}"
    assert of_tol.max() <= 1.0, f"{name}: {of_tol.max():.3f} of the tolerance"
