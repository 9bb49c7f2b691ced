"""ctypes wrapper of the CPU oracle (oracle/evox_ref.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py, never by the product package.  All arrays are
numpy, C-contiguous, row-major [N, D] (row pitch D).
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libevox_ref.so")

SPHERE, ACKLEY, RASTRIGIN, GRIEWANK, ROSENBROCK, SCHWEFEL = range(6)
FN_NAMES = ("sphere", "ackley", "rastrigin", "griewank", "rosenbrock", "schwefel")


class RefParams(ctypes.Structure):
    _fields_ = [
        ("fn", ctypes.c_int32), ("clamp_x", ctypes.c_int32),
        ("N", ctypes.c_int64), ("D", ctypes.c_int64),
        ("lb", ctypes.c_float), ("ub", ctypes.c_float),
        ("v_lo", ctypes.c_float), ("v_hi", ctypes.c_float),
        ("w", ctypes.c_float), ("c1", ctypes.c_float), ("c2", ctypes.c_float),
        ("phi", ctypes.c_float), ("vmax", ctypes.c_float),
        ("x_init", ctypes.c_int32), ("x_mu", ctypes.c_float), ("x_sigma", ctypes.c_float),
        ("de_f", ctypes.c_float), ("de_cr", ctypes.c_float),
        ("es_sigma", ctypes.c_float), ("es_lr", ctypes.c_float),
        ("pgpe_sigma_lr", ctypes.c_float), ("pgpe_max_change", ctypes.c_float),
        ("seed", ctypes.c_uint64),
        ("cso_local", ctypes.c_int32),
    ]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _b
            _b.build()
        L = ctypes.CDLL(LIB_PATH)
        u32, i64, u64, f32 = ctypes.c_uint32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_float
        P = ctypes.c_void_p
        L.evox_ref_philox4x32_10.argtypes = [P, P, P]
        L.evox_ref_philox_word.argtypes = [u64, u32, u32, u32, u32, ctypes.c_int]
        L.evox_ref_philox_word.restype = u32
        L.evox_ref_u01.argtypes = [u32]
        L.evox_ref_u01.restype = f32
        L.evox_ref_u01_array.argtypes = [P, i64, P]
        L.evox_ref_eval_row_f64.argtypes = [ctypes.c_int, P, i64]
        L.evox_ref_eval_row_f64.restype = ctypes.c_double
        L.evox_ref_eval.argtypes = [ctypes.c_int, P, i64, i64, i64, P]
        L.evox_ref_argmin.argtypes = [P, i64]
        L.evox_ref_argmin.restype = i64
        L.evox_ref_init_uniform.argtypes = [u64, ctypes.c_int, i64, i64, f32, f32, P]
        L.evox_ref_normal01.argtypes = [u64, i64, i64]
        L.evox_ref_normal01.restype = ctypes.c_double
        L.evox_ref_init_normal.argtypes = [u64, i64, i64, f32, f32, P]
        L.evox_ref_pso_init.argtypes = [P, P, P, P, P, P, P, P]
        L.evox_ref_pso_step.argtypes = [P, i64, i64, P, P, P, P, P, P, P]
        L.evox_ref_colmean.argtypes = [P, i64, i64, P]
        L.evox_ref_ring_mean.argtypes = [P, i64, i64, P]
        L.evox_ref_perm.argtypes = [u64, i64, i64, P]
        L.evox_ref_argsort_u32.argtypes = [P, i64, P]
        L.evox_ref_de_choices.argtypes = [u64, i64, i64, i64, i64, P]
        L.evox_ref_es_eps.argtypes = [u64, i64, i64, i64]
        L.evox_ref_es_eps.restype = ctypes.c_double
        L.evox_ref_es_init.argtypes = [P, P]
        L.evox_ref_es_step.argtypes = [P, i64, i64, P, P, P, P, P]
        L.evox_ref_gemm.argtypes = [ctypes.c_int, ctypes.c_int, i64, i64, i64, f32, P, i64, P, i64, f32, P, i64]
        L.evox_ref_pgpe_z.argtypes = [u64, i64, i64, i64]
        L.evox_ref_pgpe_z.restype = ctypes.c_double
        L.evox_ref_pgpe_init.argtypes = [P, P, P]
        L.evox_ref_pgpe_step.argtypes = [P, i64, i64, P, P, P, P, P, P]
        L.evox_ref_maes_z.argtypes = [u64, i64, i64, i64]
        L.evox_ref_maes_z.restype = ctypes.c_double
        L.evox_ref_maes_deviates.argtypes = [u64, i64, i64, i64, P]
        L.evox_ref_maes_consts.argtypes = [i64, i64, P, P]
        L.evox_ref_maes_consts.restype = i64
        L.evox_ref_maes_init.argtypes = [P, P, P, P, P]
        L.evox_ref_maes_step.argtypes = [P, i64, i64, P, P, P, P, P, P, P, P, i64, P, P]
        L.evox_ref_dtlz1.argtypes = [P, i64, ctypes.c_int32, P]
        L.evox_ref_dtlz1_rows.argtypes = [P, i64, i64, ctypes.c_int32, P]
        L.evox_ref_dominates.argtypes = [P, P, ctypes.c_int32]
        L.evox_ref_dominates.restype = ctypes.c_int
        L.evox_ref_nds.argtypes = [P, i64, ctypes.c_int32, P]
        L.evox_ref_nds.restype = ctypes.c_int32
        L.evox_ref_crowding.argtypes = [P, i64, ctypes.c_int32, P, P]
        L.evox_ref_nsga2_parents.argtypes = [u64, i64, i64, i64, P, P, P, P]
        L.evox_ref_poly_mutate.argtypes = [ctypes.c_double, ctypes.c_double, ctypes.c_double]
        L.evox_ref_poly_mutate.restype = ctypes.c_double
        L.evox_ref_nsga2_offspring.argtypes = [P, i64, i64, P, P, P, P]
        L.evox_ref_nsga2_init.argtypes = [P, P, P, P, P]
        L.evox_ref_nsga2_step.argtypes = [P, i64, i64, P, P, P, P]
        L.evox_ref_de_init.argtypes = [P, P, P]
        L.evox_ref_de_step.argtypes = [P, i64, i64, P, P, P, P, P]
        L.evox_ref_cso_init.argtypes = [P, P, P, P]
        L.evox_ref_cso_step.argtypes = [P, i64, i64, P, P, P, P, P, P]
        _lib = L
    return _lib


_mt = None
MT_LIB_PATH = os.path.join(HERE, "libevox_ref_mt.so")


def mt_lib():
    """The all-core CPU baseline (oracle/evox_ref_mt.c): the oracle's steps
    with their row loops split over threads, bit-identical results."""
    global _mt
    if _mt is None:
        if not os.path.exists(MT_LIB_PATH):
            from . import build as _b
            _b.build()
        L = ctypes.CDLL(MT_LIB_PATH)
        i64, P, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
        L.evox_mt_eval.argtypes = [ci, P, i64, i64, i64, P, ci]
        L.evox_mt_pso_step.argtypes = [P, i64, i64, P, P, P, P, P, P, P, ci]
        L.evox_mt_cso_step.argtypes = [P, i64, i64, P, P, P, P, P, ci]
        _mt = L
    return _mt


def mt_evaluate(fn, X, threads):
    X = _f32(X)
    N, D = X.shape
    out = np.zeros(N, dtype=np.float32)
    if mt_lib().evox_mt_eval(fn, _ptr(X), N, D, D, _ptr(out), threads) != 0:
        raise ValueError("evox_mt_eval failed")
    return out


def mt_step(state, n_gens, threads):
    """n_gens generations of an oracle PSO or CSO state on `threads` threads."""
    if isinstance(state, PSO):
        rc = mt_lib().evox_mt_pso_step(ctypes.byref(state.P), state.t, n_gens, _ptr(state.x), _ptr(state.v),
                                       _ptr(state.p), _ptr(state.pf), _ptr(state.g), ctypes.byref(state._gf),
                                       ctypes.byref(state._gi), threads)
    elif isinstance(state, CSO):
        bf, bi = ctypes.c_float(0.0), ctypes.c_int64(0)
        rc = mt_lib().evox_mt_cso_step(ctypes.byref(state.P), state.t, n_gens, _ptr(state.x), _ptr(state.v),
                                       _ptr(state.fit), ctypes.byref(bf), ctypes.byref(bi), threads)
        state.best_fit, state.best_idx = bf.value, bi.value
    else:
        raise TypeError(type(state))
    if rc != 0:
        raise ValueError(f"all-core step rc={rc}")
    state.t += n_gens


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f32(a):
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a


def philox4x32_10(ctr, key):
    """Four output words of Philox4x32-10 for counter ctr[4], key key[2]."""
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().evox_ref_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def philox_word(seed, c0, c1, c2, c3, word):
    return int(lib().evox_ref_philox_word(seed, c0, c1, c2, c3, word))


def u01(w):
    return float(lib().evox_ref_u01(int(w)))


def u01_array(words):
    w = np.ascontiguousarray(words, dtype=np.uint32)
    out = np.zeros(w.shape, dtype=np.float32)
    lib().evox_ref_u01_array(_ptr(w), w.size, _ptr(out))
    return out


def eval_row_f64(fn, x):
    x = _f32(x)
    return float(lib().evox_ref_eval_row_f64(fn, _ptr(x), x.shape[-1]))


def evaluate(fn, X):
    """fp32 fitness of every row of X [N, D] (fp64 inside, rounded once)."""
    X = _f32(X)
    N, D = X.shape
    out = np.zeros(N, dtype=np.float32)
    rc = lib().evox_ref_eval(fn, _ptr(X), N, D, D, _ptr(out))
    if rc != 0:
        raise ValueError(f"evox_ref_eval rc={rc}")
    return out


def argmin(f):
    f = _f32(f)
    return int(lib().evox_ref_argmin(_ptr(f), f.shape[0]))


def init_uniform(seed, stream, N, D, lo, hi):
    out = np.zeros((N, D), dtype=np.float32)
    lib().evox_ref_init_uniform(seed, stream, N, D, lo, hi, _ptr(out))
    return out


def normal01(seed, i, j):
    """The fp64 standard normal deviate of element (i, j) (stream 5)."""
    return lib().evox_ref_normal01(seed, i, j)


def init_normal(seed, N, D, mu, sigma):
    out = np.zeros((N, D), dtype=np.float32)
    lib().evox_ref_init_normal(seed, N, D, mu, sigma, _ptr(out))
    return out


def make_params(fn, N, D, lb, ub, v_lo=0.0, v_hi=0.0, w=0.6, c1=1.5, c2=1.5, phi=0.1,
                vmax=0.0, clamp_x=0, seed=0, x_init=0, x_mu=0.0, x_sigma=1.0, de_f=0.5, de_cr=0.9,
                es_sigma=0.1, es_lr=0.01, pgpe_sigma_lr=0.01, pgpe_max_change=0.2, cso_local=0):
    return RefParams(fn=fn, clamp_x=clamp_x, N=N, D=D, lb=lb, ub=ub, v_lo=v_lo, v_hi=v_hi,
                     w=w, c1=c1, c2=c2, phi=phi, vmax=vmax, x_init=x_init, x_mu=x_mu,
                     x_sigma=x_sigma, de_f=de_f, de_cr=de_cr, es_sigma=es_sigma, es_lr=es_lr,
                     pgpe_sigma_lr=pgpe_sigma_lr, pgpe_max_change=pgpe_max_change, seed=seed,
                     cso_local=cso_local)


class PSO:
    """Oracle PSO state: x, v, p, pf, g, gf, gi and the generation counter t."""

    def __init__(self, params: RefParams):
        self.P = params
        N, D = params.N, params.D
        self.x = np.zeros((N, D), np.float32)
        self.v = np.zeros((N, D), np.float32)
        self.p = np.zeros((N, D), np.float32)
        self.pf = np.zeros(N, np.float32)
        self.g = np.zeros(D, np.float32)
        self._gf = ctypes.c_float(0.0)
        self._gi = ctypes.c_int64(0)
        self.t = 0
        rc = lib().evox_ref_pso_init(ctypes.byref(self.P), _ptr(self.x), _ptr(self.v),
                                     _ptr(self.p), _ptr(self.pf), _ptr(self.g),
                                     ctypes.byref(self._gf), ctypes.byref(self._gi))
        if rc != 0:
            raise ValueError(f"evox_ref_pso_init rc={rc}")

    @property
    def gf(self):
        return self._gf.value

    @property
    def gi(self):
        return self._gi.value

    def step(self, n_gens):
        for a in (self.x, self.v, self.p, self.pf, self.g):
            assert a.flags.c_contiguous and a.dtype == np.float32
        rc = lib().evox_ref_pso_step(ctypes.byref(self.P), self.t, n_gens, _ptr(self.x),
                                     _ptr(self.v), _ptr(self.p), _ptr(self.pf), _ptr(self.g),
                                     ctypes.byref(self._gf), ctypes.byref(self._gi))
        if rc != 0:
            raise ValueError(f"evox_ref_pso_step rc={rc}")
        self.t += n_gens


def colmean(X):
    X = _f32(X)
    N, D = X.shape
    out = np.zeros(D, np.float32)
    lib().evox_ref_colmean(_ptr(X), N, D, _ptr(out))
    return out


def argsort_u32(keys):
    keys = np.ascontiguousarray(keys, dtype=np.uint32)
    out = np.zeros(keys.size, np.int64)
    lib().evox_ref_argsort_u32(_ptr(keys), keys.size, _ptr(out))
    return out


def perm(seed, t, N):
    out = np.zeros(N, np.int64)
    lib().evox_ref_perm(seed, t, N, _ptr(out))
    return out


class CSO:
    """Oracle CSO state: x, v, fit and the generation counter t."""

    def __init__(self, params: RefParams):
        self.P = params
        N, D = params.N, params.D
        self.x = np.zeros((N, D), np.float32)
        self.v = np.zeros((N, D), np.float32)
        self.fit = np.zeros(N, np.float32)
        self.loser = np.zeros(N, np.uint8)
        self.best_fit = float("nan")
        self.best_idx = -1
        self.t = 0
        rc = lib().evox_ref_cso_init(ctypes.byref(self.P), _ptr(self.x), _ptr(self.v),
                                     _ptr(self.fit))
        if rc != 0:
            raise ValueError(f"evox_ref_cso_init rc={rc}")

    def step(self, n_gens):
        bf = ctypes.c_float(0.0)
        bi = ctypes.c_int64(0)
        rc = lib().evox_ref_cso_step(ctypes.byref(self.P), self.t, n_gens, _ptr(self.x),
                                     _ptr(self.v), _ptr(self.fit), ctypes.byref(bf),
                                     ctypes.byref(bi), _ptr(self.loser))
        if rc != 0:
            raise ValueError(f"evox_ref_cso_step rc={rc}")
        self.best_fit, self.best_idx = bf.value, bi.value
        self.t += n_gens


def de_choices(seed, t, i, N, D):
    """(r1, r2, r3, j_rand) of target i at generation t."""
    out = np.zeros(4, np.int64)
    lib().evox_ref_de_choices(seed, t, i, N, D, _ptr(out))
    return tuple(int(v) for v in out)


class DE:
    """Oracle DE/rand/1/bin state: x, fit and the generation counter t."""

    def __init__(self, params: RefParams):
        self.P = params
        N, D = params.N, params.D
        self.x = np.zeros((N, D), np.float32)
        self.fit = np.zeros(N, np.float32)
        self.accepted = np.zeros(N, np.uint8)
        self.best_fit = float("nan")
        self.best_idx = -1
        self.t = 0
        rc = lib().evox_ref_de_init(ctypes.byref(self.P), _ptr(self.x), _ptr(self.fit))
        if rc != 0:
            raise ValueError(f"evox_ref_de_init rc={rc}")
        self.best_idx = argmin(self.fit)
        self.best_fit = float(self.fit[self.best_idx])

    def step(self, n_gens):
        for a in (self.x, self.fit):
            assert a.flags.c_contiguous and a.dtype == np.float32
        bf = ctypes.c_float(0.0)
        bi = ctypes.c_int64(0)
        rc = lib().evox_ref_de_step(ctypes.byref(self.P), self.t, n_gens, _ptr(self.x), _ptr(self.fit),
                                    ctypes.byref(bf), ctypes.byref(bi), _ptr(self.accepted))
        if rc != 0:
            raise ValueError(f"evox_ref_de_step rc={rc}")
        self.best_fit, self.best_idx = bf.value, bi.value
        self.t += n_gens


def es_eps(seed, t, k, j):
    """The fp64 perturbation eps_kj of antithetic pair k at generation t."""
    return lib().evox_ref_es_eps(seed, t, k, j)


class ES:
    """Oracle OpenES state: the center theta and the generation counter t."""

    def __init__(self, params: RefParams):
        self.P = params
        self.theta = np.zeros(params.D, np.float32)
        self.fit = np.zeros(params.N, np.float32)
        self.rank = np.zeros(params.N, np.int64)
        self.best_fit = float("nan")
        self.best_idx = -1
        self.t = 0
        if lib().evox_ref_es_init(ctypes.byref(self.P), _ptr(self.theta)) != 0:
            raise ValueError("evox_ref_es_init failed")

    def step(self, n_gens):
        assert self.theta.flags.c_contiguous and self.theta.dtype == np.float32
        bf = ctypes.c_float(0.0)
        bi = ctypes.c_int64(0)
        rc = lib().evox_ref_es_step(ctypes.byref(self.P), self.t, n_gens, _ptr(self.theta),
                                    _ptr(self.fit), _ptr(self.rank), ctypes.byref(bf), ctypes.byref(bi))
        if rc != 0:
            raise ValueError(f"evox_ref_es_step rc={rc}")
        if n_gens > 0:
            self.best_fit, self.best_idx = bf.value, bi.value
        self.t += n_gens


def pgpe_z(seed, t, k, j):
    """The fp64 standard deviate z_kj of PGPE pair k at generation t."""
    return lib().evox_ref_pgpe_z(seed, t, k, j)


class PGPE:
    """Oracle PGPE state: center mu, standard deviations sigma, generation t."""

    def __init__(self, params: RefParams):
        self.P = params
        self.mu = np.zeros(params.D, np.float32)
        self.sigma = np.zeros(params.D, np.float32)
        self.fit = np.zeros(params.N, np.float32)
        self.rank = np.zeros(params.N, np.int64)
        self.best_fit = float("nan")
        self.best_idx = -1
        self.t = 0
        if lib().evox_ref_pgpe_init(ctypes.byref(self.P), _ptr(self.mu), _ptr(self.sigma)) != 0:
            raise ValueError("evox_ref_pgpe_init failed")

    def step(self, n_gens):
        for a in (self.mu, self.sigma):
            assert a.flags.c_contiguous and a.dtype == np.float32
        bf = ctypes.c_float(0.0)
        bi = ctypes.c_int64(0)
        rc = lib().evox_ref_pgpe_step(ctypes.byref(self.P), self.t, n_gens, _ptr(self.mu), _ptr(self.sigma),
                                      _ptr(self.fit), _ptr(self.rank), ctypes.byref(bf), ctypes.byref(bi))
        if rc != 0:
            raise ValueError(f"evox_ref_pgpe_step rc={rc}")
        if n_gens > 0:
            self.best_fit, self.best_idx = bf.value, bi.value
        self.t += n_gens


def maes_z(seed, t, k, j):
    """The MA-ES deviate z_kj of sample k at generation t (fp64)."""
    return lib().evox_ref_maes_z(seed, t, k, j)


def maes_deviates(seed, t, N, D):
    """The generation's deviates z [N, D], rounded to fp32 as the step uses them."""
    z = np.zeros((N, D), np.float32)
    lib().evox_ref_maes_deviates(seed, t, N, D, _ptr(z))
    return z


def maes_consts(N, D):
    """(mu, weights[mu], dict of mu_eff, c_s, d_s, c_1, c_w, chi_D)."""
    w = np.zeros(max(N // 2, 1), np.float64)
    c = np.zeros(6, np.float64)
    mu = lib().evox_ref_maes_consts(N, D, _ptr(w), _ptr(c))
    if mu < 0:
        raise ValueError("invalid MA-ES sizes")
    return mu, w[:mu], dict(zip(("mu_eff", "c_s", "d_s", "c_1", "c_w", "chi"), c.tolist()))


class MAES:
    """Oracle MA-ES state: center y, step size sigma, transformation M [D, D],
    evolution path s, generation t."""

    def __init__(self, params: RefParams):
        D = params.D
        self.P = params
        self.y = np.zeros(D, np.float32)
        self.sigma = np.zeros(1, np.float32)
        self.M = np.zeros((D, D), np.float32)
        self.s = np.zeros(D, np.float32)
        self.fit = np.zeros(params.N, np.float32)
        self.rank = np.zeros(params.N, np.int64)
        self.d = None
        self.best_fit = float("nan")
        self.best_idx = -1
        self.t = 0
        if lib().evox_ref_maes_init(ctypes.byref(self.P), _ptr(self.y), _ptr(self.sigma), _ptr(self.M),
                                    _ptr(self.s)) != 0:
            raise ValueError("evox_ref_maes_init failed")

    def step(self, n_gens, rows=None, keep_d=False):
        """n_gens generations; rows (one generation only) limits the update
        of M to those rows; keep_d stores the last generation's d_k in .d."""
        for a in (self.y, self.sigma, self.M, self.s):
            assert a.flags.c_contiguous and a.dtype == np.float32
        bf = ctypes.c_float(0.0)
        bi = ctypes.c_int64(0)
        r = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
        self.d = np.zeros((self.P.N, self.P.D), np.float32) if keep_d else None
        rc = lib().evox_ref_maes_step(ctypes.byref(self.P), self.t, n_gens, _ptr(self.y), _ptr(self.sigma),
                                      _ptr(self.M), _ptr(self.s), _ptr(self.fit), _ptr(self.rank),
                                      ctypes.byref(bf), ctypes.byref(bi), 0 if r is None else r.size,
                                      _ptr(r), _ptr(self.d))
        if rc != 0:
            raise ValueError(f"evox_ref_maes_step rc={rc}")
        if n_gens > 0:
            self.best_fit, self.best_idx = bf.value, bi.value
        self.t += n_gens


class NSGA2Params(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int64), ("D", ctypes.c_int64), ("M", ctypes.c_int32),
                ("eta_c", ctypes.c_float), ("eta_m", ctypes.c_float), ("seed", ctypes.c_uint64)]


def dtlz1(X, M):
    """fp32 objectives [n, M] of the rows of X (fp64 inside, rounded once)."""
    X = _f32(np.atleast_2d(X))
    F = np.zeros((X.shape[0], M), np.float32)
    lib().evox_ref_dtlz1_rows(_ptr(X), X.shape[0], X.shape[1], M, _ptr(F))
    return F


def dtlz1_f64(x, M):
    x = _f32(np.asarray(x).reshape(1, -1))[0]
    f = np.zeros(M, np.float64)
    lib().evox_ref_dtlz1(_ptr(x), x.size, M, _ptr(f))
    return f


def dominates(a, b):
    a, b = _f32(np.asarray(a).reshape(1, -1))[0], _f32(np.asarray(b).reshape(1, -1))[0]
    return bool(lib().evox_ref_dominates(_ptr(a), _ptr(b), a.size))


def nds(F):
    """0-based front index of every row of F [n, M]."""
    F = _f32(np.atleast_2d(F))
    front = np.zeros(F.shape[0], np.int32)
    lib().evox_ref_nds(_ptr(F), F.shape[0], F.shape[1], _ptr(front))
    return front


def crowding(F, front):
    F = _f32(np.atleast_2d(F))
    front = np.ascontiguousarray(front, dtype=np.int32)
    crowd = np.zeros(F.shape[0], np.float64)
    lib().evox_ref_crowding(_ptr(F), F.shape[0], F.shape[1], _ptr(front), _ptr(crowd))
    return crowd


def nsga2_params(N, D, M=3, eta_c=20.0, eta_m=20.0, seed=0):
    return NSGA2Params(N=N, D=D, M=M, eta_c=eta_c, eta_m=eta_m, seed=seed)


def poly_mutate(x, u, eta):
    return lib().evox_ref_poly_mutate(x, u, eta)


def nsga2_parents(seed, t, p, N, front, crowd):
    front = np.ascontiguousarray(front, dtype=np.int32)
    crowd = np.ascontiguousarray(crowd, dtype=np.float64)
    a, b = ctypes.c_int64(0), ctypes.c_int64(0)
    lib().evox_ref_nsga2_parents(seed, t, p, N, _ptr(front), _ptr(crowd), ctypes.byref(a), ctypes.byref(b))
    return a.value, b.value


def nsga2_offspring(P, t, p, a, b):
    a, b = _f32(np.asarray(a).reshape(1, -1))[0], _f32(np.asarray(b).reshape(1, -1))[0]
    c0, c1 = np.zeros(P.D, np.float32), np.zeros(P.D, np.float32)
    lib().evox_ref_nsga2_offspring(ctypes.byref(P), t, p, _ptr(a), _ptr(b), _ptr(c0), _ptr(c1))
    return c0, c1


class NSGA2:
    """Oracle NSGA-II state on DTLZ1: population X [N, D], objectives F [N, M],
    fronts and crowding distances, generation t."""

    def __init__(self, params: NSGA2Params):
        self.P = params
        N, D, M = params.N, params.D, params.M
        self.X = np.zeros((N, D), np.float32)
        self.F = np.zeros((N, M), np.float32)
        self.front = np.zeros(N, np.int32)
        self.crowd = np.zeros(N, np.float64)
        self.t = 0
        if lib().evox_ref_nsga2_init(ctypes.byref(self.P), _ptr(self.X), _ptr(self.F), _ptr(self.front),
                                     _ptr(self.crowd)) != 0:
            raise ValueError("evox_ref_nsga2_init failed")

    def step(self, n_gens):
        for a in (self.X, self.F, self.front, self.crowd):
            assert a.flags.c_contiguous
        rc = lib().evox_ref_nsga2_step(ctypes.byref(self.P), self.t, n_gens, _ptr(self.X), _ptr(self.F),
                                       _ptr(self.front), _ptr(self.crowd))
        if rc != 0:
            raise ValueError(f"evox_ref_nsga2_step rc={rc}")
        self.t += n_gens


def ring_mean(X):
    """Each row's ring-neighbourhood mean (rows i - 1, i, i + 1 modulo N)."""
    X = _f32(np.atleast_2d(X))
    out = np.zeros_like(X)
    lib().evox_ref_ring_mean(_ptr(X), X.shape[0], X.shape[1], _ptr(out))
    return out


def gemm(A, B, ta=False, tb=False, alpha=1.0, beta=0.0, C=None):
    """alpha op(A) op(B) + beta C in fp64 per output, rounded to fp32."""
    A = np.ascontiguousarray(A, dtype=np.float32)
    B = np.ascontiguousarray(B, dtype=np.float32)
    M = A.shape[1] if ta else A.shape[0]
    K = A.shape[0] if ta else A.shape[1]
    N = B.shape[0] if tb else B.shape[1]
    out = np.zeros((M, N), np.float32) if C is None else np.ascontiguousarray(C, dtype=np.float32).copy()
    lib().evox_ref_gemm(int(ta), int(tb), M, N, K, alpha, _ptr(A), A.shape[1], _ptr(B), B.shape[1], beta,
                        _ptr(out), N)
    return out
