"""Tolerances and comparison helpers of the GPU-vs-oracle parity tests.

Fitness tolerance (reading of "fp32 fitness within 1e-5 relative"):
    |F_gpu - F_ref| <= 1e-5 * max(|F_ref|, S(x))
with S the magnitude of the terms the function sums, so that exact
cancellation at an optimum does not demand unbounded relative accuracy:
    Sphere, Rosenbrock, Rastrigin  S = |F|   (non-negative terms: Rastrigin as
                                              sum x^2 + 20 sin^2(pi x))
    Ackley              S = 20 + e
    Griewank            S = 2 + sum x^2 / 4000
    Schwefel            S = 418.9829 D + sum |x|
"""
import math

import numpy as np

REL = 1e-5
SPHERE, ACKLEY, RASTRIGIN, GRIEWANK, ROSENBROCK, SCHWEFEL = range(6)


def scale(fn, X, f_ref):
    X = np.asarray(X, dtype=np.float64)
    D = X.shape[1]
    f = np.abs(np.asarray(f_ref, dtype=np.float64))
    if fn in (SPHERE, ROSENBROCK, RASTRIGIN):
        return f
    if fn == ACKLEY:
        return np.maximum(f, 20.0 + math.e)
    if fn == GRIEWANK:
        return np.maximum(f, 2.0 + (X * X).sum(1) / 4000.0)
    if fn == SCHWEFEL:
        return np.maximum(f, 418.9829 * D + np.abs(X).sum(1))
    raise ValueError(fn)


def tol(fn, X, f_ref):
    return REL * scale(fn, X, f_ref)


def fitness_ok(fn, X, f_gpu, f_ref):
    """Boolean mask of rows whose GPU fitness is within tolerance."""
    f_gpu = np.asarray(f_gpu, dtype=np.float64)
    f_ref = np.asarray(f_ref, dtype=np.float64)
    both_inf = np.isinf(f_gpu) & np.isinf(f_ref) & (np.sign(f_gpu) == np.sign(f_ref))
    both_nan = np.isnan(f_gpu) & np.isnan(f_ref)
    with np.errstate(invalid="ignore"):
        close = np.abs(f_gpu - f_ref) <= tol(fn, X, f_ref)
    return close | both_inf | both_nan


def assert_fitness(fn, X, f_gpu, f_ref, what=""):
    ok = fitness_ok(fn, X, f_gpu, f_ref)
    if not ok.all():
        bad = np.nonzero(~ok)[0][:5]
        rows = [(int(i), float(f_gpu[i]), float(f_ref[i])) for i in bad]
        raise AssertionError(f"{what}: {int((~ok).sum())} rows out of tolerance, e.g. {rows}")


def index_ok(fn, X_rows, f_ref_all, i_gpu, i_ref):
    """Selected index: equal, or a tolerance tie (the two candidates' oracle
    values are within the fitness tolerance of each other)."""
    if i_gpu == i_ref:
        return True
    a, b = float(f_ref_all[i_gpu]), float(f_ref_all[i_ref])
    t = REL * max(abs(a), abs(b), float(scale(fn, X_rows, [b]).max()))
    return abs(a - b) <= t


def ulp_diff(a, b):
    """Distance in units in the last place between float32 arrays."""
    ai = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    bi = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    ai = np.where(ai < 0, -(ai & 0x7FFFFFFF), ai)
    bi = np.where(bi < 0, -(bi & 0x7FFFFFFF), bi)
    return np.abs(ai - bi)


def normal_tol(x_ref, mu, sigma):
    """Tolerance of the device normal deviates (Box-Muller in fp32 against
    the fp64 oracle): the hardware log2 and square root, each within one
    ulp, and the rounded 2 ln 2 put the radius r within 2^-23 relative (1.75
    ulp), the hardware cosine / sine of the exactly
    reduced angle is within 1.25e-7 absolute, so |z_gpu - z| <= 1.25e-7 r +
    1.8e-7 |z| <= 1e-6 max(1, |z|) for r <= sqrt(2 ln 2^24) = 5.77; the final
    fma adds at most one rounding of x."""
    x_ref = np.asarray(x_ref, dtype=np.float64)
    z = np.abs(x_ref - mu) / sigma if sigma else np.zeros_like(x_ref)
    ulp = np.spacing(np.abs(x_ref).astype(np.float32)).astype(np.float64)
    return abs(sigma) * 1e-6 * np.maximum(1.0, z) + ulp


def cso_lockstep(ref, g, r, what):
    """One CSO generation on both sides from the same swarm mean.

    The GPU sums the mean in fp64 in another order than the oracle; both
    round once to fp32, so the two agree within 1 ulp (checked here) and
    almost always exactly.  So that every generation compares the loser
    update bit for bit, the oracle's mean is then written into the GPU
    state's xbar, which the generation kernel reads."""
    import torch
    D = r.P.D
    xbar = ref.colmean(r.x)
    own = g.xbar[:D].cpu().numpy()
    assert ulp_diff(own, xbar).max() <= 1, f"{what}: the GPU's swarm mean is more than 1 ulp off"
    g.xbar[:D] = torch.from_numpy(xbar).to(g.xbar.device)
    g.step(1)
    r.step(1)
