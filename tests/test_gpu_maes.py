"""GPU parity of the MA-ES generation against the oracle, in lockstep.

Each generation starts both sides from the oracle's state (y, sigma, M, s;
inputs flow from the oracle to the GPU only) and compares the outcome with
bounds derived from the arithmetic of the two sides:
  - deviates: Box-Muller in fp32 with the device log and cosine against fp64,
    |dz| <= 2e-6 max(1, |z|) (the bound of the normal population);
  - steps d = M z: fp32 matrix-core sums of D products against fp64 sums
    rounded once, |dd_ki| <= (gamma_D + 2e-6) sum_j |M_ij| max(1, |z_kj|)
    + ulp(d_ki), gamma_D = D u / (1 - D u), u = 2^-24;
  - fitness: |dF| <= sum_i |dF/dx_i| |dx_i| (first order, per-function
    bounds on the partial derivatives) plus the evaluation tolerance;
  - parents: the GPU's order equals the oracle's, or differs only between
    samples whose oracle fitness lie within their bounds (then that
    generation's update is not compared; every case compares at least one);
  - y, s, sigma: the weighted sums of the step and deviate differences plus
    the final roundings;
  - M: the rank-mu form (1 - (c_1+c_w)/2) M + c_1/2 (M s) s^T + c_w/2 sum
    w_i d_i z_i^T with each factor's difference propagated, plus gamma_{mu+2}
    of the sum of the magnitudes of its terms, plus the final rounding.
"""
import math

import numpy as np
import pytest
import torch

from parity import tol

pytestmark = pytest.mark.gpu

U = 2.0 ** -24
SPHERE, ACKLEY, RASTRIGIN, GRIEWANK, ROSENBROCK, SCHWEFEL = range(6)


def gamma(n):
    return n * U / (1 - n * U)


def ulp(v):
    return np.spacing(np.abs(np.asarray(v, np.float64)).astype(np.float32)).astype(np.float64)


def grad_bound(fn, X):
    """Per-element bounds on |dF/dx_i| at the rows of X (fp64 [N, D])."""
    A = np.abs(X)
    D = X.shape[1]
    if fn == SPHERE:
        return 2 * A
    if fn == RASTRIGIN:
        return 2 * A + 20 * math.pi
    if fn == ACKLEY:
        return np.full_like(A, 4.0 / math.sqrt(D) + 2 * math.pi * math.e / D)
    if fn == GRIEWANK:
        return A / 2000 + 1.0
    if fn == SCHWEFEL:
        return 1.0 + np.sqrt(A) / 2
    if fn == ROSENBROCK:
        g = 2 * (1 + A)
        g[:, :-1] += 400 * A[:, :-1] * (A[:, 1:] + A[:, :-1] ** 2)
        g[:, 1:] += 200 * (A[:, 1:] + A[:, :-1] ** 2)
        return g
    raise ValueError(fn)


def pair(evox, ref, fn, N, D, seed, lb, ub, sigma):
    g = evox.Swarm(evox.make_params(evox.MAES, fn, N, D, lb, ub, seed=seed, es_sigma=sigma))
    r = ref.MAES(ref.make_params(fn, N, D, lb, ub, seed=seed, es_sigma=sigma))
    return g, r


def push(g, r):
    D = r.P.D
    g.x[:D] = torch.from_numpy(r.y).cuda()
    g.v[:D] = torch.from_numpy(r.s).cuda()
    g.mat[:, :D] = torch.from_numpy(r.M).cuda()
    g.sigma[:] = torch.from_numpy(r.sigma).cuda()


def lockstep(evox, ref, g, r, fn, what):
    N, D, seed, t = r.P.N, r.P.D, r.P.seed, r.t
    mu, w, c = ref.maes_consts(N, D)
    push(g, r)
    y0, s0, sig0 = r.y.astype(np.float64), r.s.astype(np.float64), float(r.sigma[0])
    M0 = r.M.astype(np.float64)
    g.step(1)
    r.step(1, keep_d=True)
    z = ref.maes_deviates(seed, t, N, D).astype(np.float64)
    d = r.d.astype(np.float64)
    Mabs = np.abs(M0)
    dz = 2e-6 * np.maximum(1.0, np.abs(z))
    dd = (gamma(D) + 2e-6) * (np.maximum(1.0, np.abs(z)) @ Mabs.T) + ulp(d)
    # fitness
    X = y0 + sig0 * d
    dx = sig0 * dd + ulp(X)
    fb = (grad_bound(fn, np.abs(X) + dx) * dx).sum(1)
    f_gpu, f_ref = g.fit.cpu().numpy().astype(np.float64), r.fit.astype(np.float64)
    ftol = 2 * (fb + tol(fn, np.abs(X) + dx, f_ref))
    bad = np.nonzero(np.abs(f_gpu - f_ref) > ftol)[0]
    assert bad.size == 0, f"{what}: sample fitness off at {bad[:5]}: {f_gpu[bad[:3]]} vs {f_ref[bad[:3]]}"
    # parents: the GPU's order (fitness, then index) must be the oracle's, or
    # differ only where the two samples' oracle fitness lie within the sum of
    # their bounds; in that case the update is not comparable this generation
    order = np.argsort(r.rank)
    gorder = np.lexsort((np.arange(N), f_gpu))
    bf, bi = g.best()
    assert bi == gorder[0], f"{what}: best index is not the GPU's own argmin"
    if not np.array_equal(gorder[:mu], order[:mu]):
        for p in np.nonzero(gorder[:mu] != order[:mu])[0]:
            a, b = gorder[p], order[p]
            assert abs(f_ref[a] - f_ref[b]) <= ftol[a] + ftol[b], f"{what}: parent {p} is {a}, oracle {b}"
        return False
    assert bf == pytest.approx(f_ref[order[0]], abs=ftol[order[0]]), f"{what}: best fitness"
    par = order[:mu]
    zp, dp, ddp, dzp = z[par], d[par], dd[par], dz[par]
    # center, path, step size
    y_gpu = g.x[:D].cpu().numpy().astype(np.float64)
    yb = sig0 * (w @ ddp) + 2 * ulp(r.y) + sig0 * gamma(mu) * (w @ np.abs(dp))
    bad = np.nonzero(np.abs(y_gpu - r.y) > yb)[0]
    assert bad.size == 0, f"{what}: center off at {bad[:5]}"
    cz = math.sqrt(c["mu_eff"] * c["c_s"] * (2 - c["c_s"]))
    s_gpu = g.v[:D].cpu().numpy().astype(np.float64)
    sb = cz * (w @ dzp) + 2 * ulp(r.s) + cz * gamma(mu) * (w @ np.abs(zp))
    bad = np.nonzero(np.abs(s_gpu - r.s) > sb)[0]
    assert bad.size == 0, f"{what}: path off at {bad[:5]}"
    s1 = r.s.astype(np.float64)
    nrm = np.linalg.norm(s1)
    dn = np.linalg.norm(sb) + gamma(D) * nrm
    sig_ref = float(r.sigma[0])
    sgb = sig_ref * (c["c_s"] / c["d_s"] / c["chi"] * dn + 8 * U)
    assert abs(float(g.sigma.cpu()[0]) - sig_ref) <= sgb, f"{what}: sigma"
    # the matrix, through the rank-mu form
    hc1, hcw = c["c_1"] / 2, c["c_w"] / 2
    beta = 1 - hc1 - hcw
    ms = M0 @ s1
    dms = (1 - c["c_s"]) * gamma(D) * (Mabs @ np.abs(s0)) + cz * (w @ ddp) + Mabs @ (sb + ulp(s1)) \
        + ulp(ms)
    W = hcw * w[:, None]
    err = (W * ddp).T @ np.abs(zp) + (W * np.abs(dp)).T @ dzp + hc1 * (np.outer(dms, np.abs(s1))
                                                                       + np.outer(np.abs(ms), sb))
    mag = (W * np.abs(dp)).T @ np.abs(zp) + hc1 * np.outer(np.abs(ms), np.abs(s1)) + beta * Mabs
    Mb = err + gamma(mu + 2) * mag + 2 * U * mag + 2 * ulp(r.M)
    M_gpu = g.mat[:, :D].cpu().numpy().astype(np.float64)
    bad = np.argwhere(np.abs(M_gpu - r.M) > Mb)
    assert bad.size == 0, f"{what}: matrix off at {bad[:5].tolist()}"
    return True


CASES = [
    dict(fn=SPHERE, N=12, D=8, seed=1, lb=-5.0, ub=5.0, sigma=0.5, gens=6),
    dict(fn=RASTRIGIN, N=100, D=300, seed=2, lb=-5.12, ub=5.12, sigma=1.0, gens=3),
    dict(fn=SPHERE, N=100, D=1000, seed=3, lb=-5.0, ub=5.0, sigma=0.3, gens=3),
    dict(fn=ROSENBROCK, N=20, D=130, seed=4, lb=-2.0, ub=2.0, sigma=0.1, gens=3),
    dict(fn=ACKLEY, N=300, D=257, seed=5, lb=-32.768, ub=32.768, sigma=2.0, gens=2),
    dict(fn=GRIEWANK, N=64, D=64, seed=6, lb=-600.0, ub=600.0, sigma=50.0, gens=3),
    dict(fn=SCHWEFEL, N=40, D=33, seed=7, lb=-500.0, ub=500.0, sigma=30.0, gens=3),
    dict(fn=SPHERE, N=2, D=1, seed=8, lb=-5.0, ub=5.0, sigma=0.5, gens=4),
    dict(fn=SPHERE, N=1000, D=600, seed=9, lb=-5.0, ub=5.0, sigma=0.5, gens=2),
]


@pytest.mark.parametrize("case", CASES, ids=[f"fn{c['fn']}-{c['N']}x{c['D']}" for c in CASES])
def test_lockstep_generations(evox_gpu, ref, case):
    c = dict(case)
    gens = c.pop("gens")
    print(f"maes {c} gens={gens}", flush=True)
    g, r = pair(evox_gpu, ref, **c)
    compared = sum(lockstep(evox_gpu, ref, g, r, c["fn"], f"gen {k}") for k in range(gens))
    print(f"  generations with the same parents: {compared} of {gens}", flush=True)
    assert compared >= 1


def test_initial_state(evox_gpu, ref):
    g, r = pair(evox_gpu, ref, SPHERE, 10, 37, 5, -5.0, 5.0, 0.7)
    D = 37
    assert np.array_equal(g.x[:D].cpu().numpy(), r.y)
    assert np.array_equal(g.mat[:, :D].cpu().numpy(), r.M) and not g.mat[:, D:].cpu().numpy().any()
    assert not g.v.cpu().numpy().any() and float(g.sigma.cpu()[0]) == r.sigma[0]


def test_free_run_converges_and_resumes(evox_gpu):
    import paper_2301_12457_amd as ev
    P = ev.make_params(ev.MAES, SPHERE, 16, 40, -5.0, 5.0, seed=11, es_sigma=1.0)
    a, b = ev.Swarm(P), ev.Swarm(P)
    f0 = float((a.x[:40].double() ** 2).sum())
    a.step(300)
    for n in (1, 99, 200):
        b.step(n)
    torch.cuda.synchronize()
    assert torch.equal(a.x, b.x) and torch.equal(a.mat, b.mat) and torch.equal(a.sigma, b.sigma)
    assert float((a.x[:40].double() ** 2).sum()) < 1e-6 * f0
    assert a.t == 300


def test_rejects_bad_sizes(evox_gpu):
    import paper_2301_12457_amd as ev
    for N, D in ((1, 10), (16385, 10), (10, 0)):
        with pytest.raises(ev.EvoxError):
            ev.Swarm(ev.make_params(ev.MAES, SPHERE, N, D, -1.0, 1.0))


def test_full_size_first_generation(evox_gpu, ref):
    """The benchmark's size, N = 100, D = 16384, one generation from the
    initial state.  With M = I the steps are the deviates exactly (every
    product but one is zero), so each sample's fitness is checked against
    F(fma(sigma, z_k, y)) from the oracle's deviates and evaluation; the
    parents against the oracle order of those values; and the new M, which
    is I T with T symmetric, for symmetry on sampled rows."""
    N, D, seed, sigma = 100, 16384, 10, 1.0
    g = evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.MAES, SPHERE, N, D, -5.0, 5.0, seed=seed, es_sigma=sigma))
    y0 = ref.init_uniform(seed, 0, 1, D, -5.0, 5.0)[0].astype(np.float64)
    g.step(1)
    z = ref.maes_deviates(seed, 0, N, D).astype(np.float64)
    X = (np.float64(np.float32(sigma)) * z + y0).astype(np.float32)
    f_ref = ref.evaluate(SPHERE, X).astype(np.float64)
    f_gpu = g.fit.cpu().numpy().astype(np.float64)
    ftol = 2 * (tol(SPHERE, X, f_ref) + (2 * np.abs(X.astype(np.float64)) * 2e-6 * np.maximum(1, np.abs(z))).sum(1))
    bad = np.nonzero(np.abs(f_gpu - f_ref) > ftol)[0]
    assert bad.size == 0, f"sample fitness off at {bad[:5]}"
    order = np.lexsort((np.arange(N), f_ref))
    gorder = np.lexsort((np.arange(N), f_gpu))
    for p in np.nonzero(gorder != order)[0]:
        a, b = gorder[p], order[p]
        assert abs(f_ref[a] - f_ref[b]) <= ftol[a] + ftol[b], f"rank {p}: {a} vs {b}"
    rows = np.random.default_rng(1).choice(D, 48, replace=False)
    Mr = g.mat[torch.from_numpy(rows).cuda()][:, :D].cpu().numpy().astype(np.float64)
    Mc = g.mat[:, torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64).T
    assert np.all(np.isfinite(Mr))
    assert np.allclose(Mr, Mc, rtol=1e-5, atol=1e-7), np.abs(Mr - Mc).max()
    sig = float(g.sigma.cpu()[0])
    assert np.isfinite(sig) and 0 < sig


def test_full_size_dense_matrix(evox_gpu, ref):
    """N = 100, D = 16384 (the benchmark shape) from a seeded dense,
    non-identity M pushed to the GPU at generation 7.  A plain oracle
    generation costs ~10^10 operations at this D, so the reference is
    composed from the oracle's own pieces -- its deviates, its evaluation and
    its constants -- and fp64 matrix products (BLAS) that follow the
    generation's definition: d_k = M z_k, samples fma(sigma, d_k, y), parents
    in the argmin order, y' = y + sigma sum w d, s' = (1 - c_s) s + sqrt(mu_eff
    c_s (2 - c_s)) sum w z, sigma' by path length, and on 48 sampled rows
    M' = M T in the rank-(mu + 1) form (equal to M T, an oracle pin).  The GPU
    must match within the bounds of the lockstep test: every sample's
    fitness, the parents, y', s', sigma' and the sampled rows of M' (so both
    the split-K sampling product and the rank pass are compared element by
    element at the benchmark shape).  At this D the default learning rates
    are ~1e-7 (c_1, c_w ~ 2 / D^2), so one generation moves M by about one
    fp32 ulp: the rows are checked to their bound, the steps (through every
    sample's fitness, the center and the path) carry the product's test."""
    from paper_2301_12457_amd.workloads import normal_matrix_np
    N, D, seed, t, fn = 100, 16384, 10, 7, SPHERE
    M = normal_matrix_np(D, D, 0.0, 0.5 / math.sqrt(D), 77)
    M[np.arange(D), np.arange(D)] += np.float32(1.0)
    y = normal_matrix_np(1, D, 0.0, 2.0, 78)[0]
    s0 = normal_matrix_np(1, D, 0.0, 0.3, 79)[0]
    sig0 = np.float32(0.7)
    g = evox_gpu.Swarm(evox_gpu.make_params(evox_gpu.MAES, fn, N, D, -5.0, 5.0, seed=seed, es_sigma=1.0))
    g.mat[:, :D] = torch.from_numpy(M).cuda()
    g.x[:D] = torch.from_numpy(y).cuda()
    g.v[:D] = torch.from_numpy(s0).cuda()
    g.sigma[:] = float(sig0)
    g.set_generation(t)
    g.step(1)
    torch.cuda.synchronize()
    mu, w, c = ref.maes_consts(N, D)
    z = ref.maes_deviates(seed, t, N, D).astype(np.float64)
    M64 = M.astype(np.float64)
    d = (z @ M64.T).astype(np.float32).astype(np.float64)          # d_k = M z_k, rounded once
    X = (np.float64(sig0) * d + y.astype(np.float64)).astype(np.float32)
    f_ref = ref.evaluate(fn, X).astype(np.float64)
    # bounds (as in the lockstep test): deviates within 2e-6 max(1, |z|), the
    # steps within (gamma_D + 2e-6) |M| max(1, |z|) + ulp
    Mabs = np.abs(M64)
    dz = 2e-6 * np.maximum(1.0, np.abs(z))
    dd = (gamma(D) + 2e-6) * (np.maximum(1.0, np.abs(z)) @ Mabs.T) + ulp(d)
    del Mabs
    dx = float(sig0) * dd + ulp(X)
    fb = (grad_bound(fn, np.abs(X.astype(np.float64)) + dx) * dx).sum(1)
    ftol = 2 * (fb + tol(fn, np.abs(X.astype(np.float64)) + dx, f_ref))
    f_gpu = g.fit.cpu().numpy().astype(np.float64)
    bad = np.nonzero(np.abs(f_gpu - f_ref) > ftol)[0]
    assert bad.size == 0, f"sample fitness off at {bad[:5]}"
    order = np.lexsort((np.arange(N), f_ref))
    gorder = np.lexsort((np.arange(N), f_gpu))
    assert np.array_equal(gorder[:mu], order[:mu]), "parents differ (not expected at this state)"
    par = order[:mu]
    zp, dp, ddp, dzp = z[par], d[par], dd[par], dz[par]
    zw, dw = w @ zp, w @ dp
    y1 = (y.astype(np.float64) + float(sig0) * dw).astype(np.float32)
    cz = math.sqrt(c["mu_eff"] * c["c_s"] * (2 - c["c_s"]))
    s1 = ((1 - c["c_s"]) * s0.astype(np.float64) + cz * zw).astype(np.float32)
    nrm = float(np.linalg.norm(s1.astype(np.float64)))
    sig1 = float(sig0) * math.exp(c["c_s"] / c["d_s"] * (nrm / c["chi"] - 1.0))
    y_gpu = g.x[:D].cpu().numpy().astype(np.float64)
    yb = float(sig0) * (w @ ddp) + 2 * ulp(y1) + float(sig0) * gamma(mu) * (w @ np.abs(dp))
    assert np.all(np.abs(y_gpu - y1) <= yb), "center"
    s_gpu = g.v[:D].cpu().numpy().astype(np.float64)
    sb = cz * (w @ dzp) + 2 * ulp(s1) + cz * gamma(mu) * (w @ np.abs(zp))
    assert np.all(np.abs(s_gpu - s1) <= sb), "path"
    dn = np.linalg.norm(sb) + gamma(D) * nrm
    assert abs(float(g.sigma.cpu()[0]) - sig1) <= sig1 * (c["c_s"] / c["d_s"] / c["chi"] * dn + 8 * U), "sigma"
    # M' on sampled rows, rank-(mu + 1) form: beta M + c_1/2 (M s') s'^T + c_w/2 sum w (M z) z^T
    rows = np.sort(np.random.default_rng(5).choice(D, 48, replace=False))
    hc1, hcw = c["c_1"] / 2, c["c_w"] / 2
    beta = 1 - hc1 - hcw
    s1d = s1.astype(np.float64)
    Mr = M64[rows]
    ms = Mr @ s1d
    Mz = dp[:, rows]                                                  # (M z_r)_i = d_r,i
    M1 = beta * Mr + hc1 * np.outer(ms, s1d) + hcw * (w[:, None] * Mz).T @ zp
    # bound: the terms' errors (steps, path) plus gamma_{mu+2} of their magnitudes
    W = hcw * w[:, None]
    Mrabs = np.abs(Mr)
    dms = (1 - c["c_s"]) * gamma(D) * (Mrabs @ np.abs(s0.astype(np.float64))) + cz * (w @ ddp[:, rows]) \
        + Mrabs @ (sb + ulp(s1d)) + ulp(ms)
    err = (W * ddp[:, rows]).T @ np.abs(zp) + (W * np.abs(dp[:, rows])).T @ dzp \
        + hc1 * (np.outer(dms, np.abs(s1d)) + np.outer(np.abs(ms), sb))
    mag = (W * np.abs(dp[:, rows])).T @ np.abs(zp) + hc1 * np.outer(np.abs(ms), np.abs(s1d)) + beta * Mrabs
    Mb = err + gamma(mu + 2) * mag + 2 * U * mag + 2 * ulp(M1)
    M_gpu = g.mat[torch.from_numpy(rows).cuda()][:, :D].cpu().numpy().astype(np.float64)
    bad = np.argwhere(np.abs(M_gpu - M1) > Mb)
    assert bad.size == 0, f"matrix off at {bad[:5].tolist()}"
