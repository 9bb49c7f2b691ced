"""Python binding of the gfx950 EvoX hot path (libevox.so, C ABI in include/evox.h).

Argument marshalling only: torch supplies device memory and the HIP stream,
every step of the path runs in the library's kernels.  Importing this module
does not touch the GPU; the first call that needs the library loads it and
raises if it has not been built (python paper_2301_12457_amd/build.py).
"""
import ctypes
import math
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libevox.so")

SPHERE, ACKLEY, RASTRIGIN, GRIEWANK, ROSENBROCK, SCHWEFEL = range(6)
FN_IDS = {"sphere": SPHERE, "ackley": ACKLEY, "rastrigin": RASTRIGIN, "griewank": GRIEWANK,
          "rosenbrock": ROSENBROCK, "schwefel": SCHWEFEL}
PSO, CSO, DE, ES, PGPE, MAES, NSGA2 = 0, 1, 2, 3, 4, 5, 6
OK, EINVAL, EHIP, ENOSPC, EALIGN = 0, -1, -2, -3, -4
MAX_D = 32768

# every symbol include/evox.h declares
EXPORTS = (
    "evox_scratch_bytes", "evox_state_create", "evox_state_destroy", "evox_eval", "evox_eval_ld",
    "evox_eval_argmin_scratch_bytes", "evox_eval_argmin", "evox_eval_argmin_noalloc", "evox_pso_step",
    "evox_cso_step",
    "evox_de_step", "evox_es_step", "evox_pgpe_step", "evox_maes_step", "evox_nsga2_step",
    "evox_nsga2_sort_scratch_bytes", "evox_nsga2_sort",
    "evox_cso_refresh", "evox_best", "evox_generation", "evox_set_generation", "evox_row_layout",
    "evox_default_ldx",
    "evox_fill_normal", "evox_sgemm", "evox_copy", "evox_pso_stream", "evox_pair_move", "evox_philox_fill",
    "evox_permutation_scratch_bytes",
    "evox_permutation", "evox_argsort_u32",
    "evox_profile", "evox_profile_read", "evox_strerror", "evox_last_error",
)


class EvoxError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"evox error {code}: {msg}")
        self.code = code


class Params(ctypes.Structure):
    _fields_ = [
        ("algo", ctypes.c_int32), ("fn_id", ctypes.c_int32),
        ("N", ctypes.c_int64), ("D", ctypes.c_int64), ("ldx", ctypes.c_int64),
        ("lb", ctypes.c_float), ("ub", ctypes.c_float),
        ("v_lo", ctypes.c_float), ("v_hi", ctypes.c_float),
        ("w", ctypes.c_float), ("c1", ctypes.c_float), ("c2", ctypes.c_float),
        ("phi", ctypes.c_float), ("vmax", ctypes.c_float),
        ("clamp_x", ctypes.c_int32),
        ("x_init", ctypes.c_int32), ("x_mu", ctypes.c_float), ("x_sigma", ctypes.c_float),
        ("de_f", ctypes.c_float), ("de_cr", ctypes.c_float),
        ("es_sigma", ctypes.c_float), ("es_lr", ctypes.c_float),
        ("pgpe_sigma_lr", ctypes.c_float), ("pgpe_max_change", ctypes.c_float),
        ("seed", ctypes.c_uint64),
        ("n_obj", ctypes.c_int32), ("sbx_eta", ctypes.c_float), ("pm_eta", ctypes.c_float),
        ("cso_local", ctypes.c_int32),
    ]


class Buffers(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("x", "v", "pbest", "pfit", "fit", "gbest", "xbar", "mat",
                                                "sigma", "obj", "front", "crowd")] + [
        ("scratch", ctypes.c_void_p), ("scratch_bytes", ctypes.c_size_t)]


_lib = None


def lib():
    """The loaded libevox.so (raises if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python paper_2301_12457_amd/build.py` (no fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, u32, u64, sz = (ctypes.c_void_p, ctypes.c_int, ctypes.c_int64,
                                     ctypes.c_uint32, ctypes.c_uint64, ctypes.c_size_t)
        sig = {
            "evox_scratch_bytes": ([P], sz),
            "evox_state_create": ([P, P, P, P], i32),
            "evox_state_destroy": ([P], i32),
            "evox_eval": ([i32, P, i64, i64, P, P], i32),
            "evox_eval_ld": ([i32, P, i64, i64, i64, P, P], i32),
            "evox_eval_argmin_scratch_bytes": ([i64], sz),
            "evox_eval_argmin": ([i32, P, i64, i64, i64, P, P, P, P, sz, P], i32),
            "evox_eval_argmin_noalloc": ([i32, P, i64, i64, i64, P, P, P, P], i32),
            "evox_pso_step": ([P, i64], i32),
            "evox_cso_step": ([P, i64], i32),
            "evox_de_step": ([P, i64], i32),
            "evox_es_step": ([P, i64], i32),
            "evox_pgpe_step": ([P, i64], i32),
            "evox_maes_step": ([P, i64], i32),
            "evox_nsga2_step": ([P, i64], i32),
            "evox_nsga2_sort_scratch_bytes": ([i64, i32], ctypes.c_size_t),
            "evox_nsga2_sort": ([P, i64, i32, P, P, P, ctypes.c_size_t, P], i32),
            "evox_cso_refresh": ([P, i32], i32),
            "evox_best": ([P, P, P, P], i32),
            "evox_generation": ([P], i64),
            "evox_set_generation": ([P, i64], i32),
            "evox_row_layout": ([i32, i64, P, P], i32),
            "evox_default_ldx": ([i32, i64], i64),
            "evox_fill_normal": ([u64, i64, i64, i64, ctypes.c_float, ctypes.c_float, P, P], i32),
            "evox_copy": ([P, P, i64, P], i32),
            "evox_pair_move": ([P, P, i64, i64, i64, P, P], i32),
            "evox_pso_stream": ([P, P, P, i64, P], i32),
            "evox_sgemm": ([i32, i32, i64, i64, i64, ctypes.c_float, P, i64, P, i64, ctypes.c_float, P, i64, P],
                           i32),
            "evox_permutation_scratch_bytes": ([i64, i64], sz),
            "evox_permutation": ([u64, i64, i64, i64, P, P, sz, P], i32),
            "evox_argsort_u32": ([P, i64, P, P, sz, P], i32),
            "evox_philox_fill": ([u64, u32, u32, u32, i64, P, P], i32),
            "evox_profile": ([P, i32], i32),
            "evox_profile_read": ([P, P, P, P], i32),
            "evox_strerror": ([i32], ctypes.c_char_p),
            "evox_last_error": ([], ctypes.c_char_p),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def _check(rc):
    if rc != OK:
        raise EvoxError(rc, lib().evox_last_error().decode())
    return rc


def _stream(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


LAYOUT_PSO, LAYOUT_CSO, LAYOUT_EVAL = 0, 1, 2


def row_layout(D, kernels=LAYOUT_PSO):
    """(threads per row, float4 chunks per thread) of a kernel family at dimension D."""
    g, n = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(lib().evox_row_layout(kernels, D, ctypes.byref(g), ctypes.byref(n)))
    return g.value, n.value


def evox_eval(fn_id, X, out, stream=None):
    """out[i] = F(X[i]) on the GPU (X: contiguous [N, D] float32 device tensor)."""
    assert X.dim() == 2 and X.is_contiguous()
    _check(lib().evox_eval(fn_id, _ptr(X), X.shape[0], X.shape[1], _ptr(out), _stream(stream)))
    return out


def evox_eval_ld(fn_id, X, N, D, ldx, out, stream=None):
    _check(lib().evox_eval_ld(fn_id, _ptr(X), N, D, ldx, _ptr(out), _stream(stream)))
    return out


def evox_eval_argmin(fn_id, X, N, D, ldx, out, best_fit, best_idx, scratch, stream=None):
    """Fitness of every row plus (best_fit[0], best_idx[0]) = argmin, on the GPU."""
    _check(lib().evox_eval_argmin(fn_id, _ptr(X), N, D, ldx, _ptr(out), _ptr(best_fit),
                                  _ptr(best_idx), _ptr(scratch), scratch.numel() * scratch.element_size(),
                                  _stream(stream)))
    return out


def evox_eval_argmin_noalloc(fn_id, X, N, D, ldx, out, best_fit, best_idx, stream=None):
    """evox_eval_argmin with the library's static per-device scratch (no allocation)."""
    _check(lib().evox_eval_argmin_noalloc(fn_id, _ptr(X), N, D, ldx, _ptr(out), _ptr(best_fit),
                                          _ptr(best_idx), _stream(stream)))
    return out


def evox_eval_argmin_scratch_bytes(N):
    return int(lib().evox_eval_argmin_scratch_bytes(N))


def evox_philox_fill(seed, c1, c2, c3, n_ctr, out, stream=None):
    _check(lib().evox_philox_fill(seed, c1, c2, c3, n_ctr, _ptr(out), _stream(stream)))
    return out


def evox_fill_normal(seed, N, D, ldx, mu, sigma, X, stream=None):
    """X[:N, :D] = mu + sigma z (Philox stream 5, Box-Muller); padding set to 0."""
    _check(lib().evox_fill_normal(seed, N, D, ldx, mu, sigma, _ptr(X), _stream(stream)))
    return X


def evox_sgemm(A, B, C, trans_a=False, trans_b=False, alpha=1.0, beta=0.0, stream=None):
    """C = alpha op(A) op(B) + beta C on the matrix cores (2-D fp32 tensors,
    row strides multiples of 4)."""
    M = A.shape[1] if trans_a else A.shape[0]
    K = A.shape[0] if trans_a else A.shape[1]
    N = B.shape[0] if trans_b else B.shape[1]
    _check(lib().evox_sgemm(int(trans_a), int(trans_b), M, N, K, alpha, _ptr(A), A.stride(0), _ptr(B),
                            B.stride(0), beta, _ptr(C), C.stride(0), _stream(stream)))
    return C


def evox_nsga2_sort(F, front, crowd, scratch=None, stream=None):
    """Fronts (int32) and crowding distances (float64) of the rows of F
    [n, M] (fp32 device tensor), through the library's sort."""
    import torch
    n, M = F.shape
    nbytes = int(lib().evox_nsga2_sort_scratch_bytes(n, M))
    if nbytes == 0:
        _check(EINVAL)
    if scratch is None:
        scratch = torch.empty((nbytes + 255) // 256 * 64, dtype=torch.int32, device=F.device)
    _check(lib().evox_nsga2_sort(_ptr(F), n, M, _ptr(front), _ptr(crowd), _ptr(scratch), scratch.numel() * 4,
                                 _stream(stream)))
    return front, crowd


def evox_copy(src, dst, n, stream=None):
    """dst[:n] = src[:n] by the library's streaming copy (bandwidth reference)."""
    _check(lib().evox_copy(_ptr(src), _ptr(dst), n, _stream(stream)))
    return dst


def evox_pso_stream(x, v, p, n, stream=None):
    """v[:n] += p[:n] - x[:n]; x[:n] += v[:n]: the 20 B per element stream of
    a PSO generation (diagnostic)."""
    _check(lib().evox_pso_stream(_ptr(x), _ptr(v), _ptr(p), n, _stream(stream)))


def evox_pair_move(x, v, N, D, ldx, winner_of, stream=None):
    """The data movement of one swarm-mean CSO generation (diagnostic)."""
    _check(lib().evox_pair_move(_ptr(x), _ptr(v), N, D, ldx, _ptr(winner_of), _stream(stream)))


def evox_permutation(seed, t0, n_gens, N, perm_out, scratch, stream=None):
    """perm_out[g] = the CSO pairing permutation of generation t0 + g."""
    _check(lib().evox_permutation(seed, t0, n_gens, N, _ptr(perm_out), _ptr(scratch),
                                  scratch.numel() * scratch.element_size(), _stream(stream)))
    return perm_out


def evox_argsort_u32(keys, N, perm_out, scratch, stream=None):
    """perm_out[:N] = stable argsort of the uint32 keys[:N] (as int32 tensors)."""
    _check(lib().evox_argsort_u32(_ptr(keys), N, _ptr(perm_out), _ptr(scratch),
                                  scratch.numel() * scratch.element_size(), _stream(stream)))
    return perm_out


def pitch(D, algo=PSO):
    """Recommended row pitch in floats for an algo's state (evox_default_ldx:
    128-byte-aligned rows where that pays, else 16-byte)."""
    ldx = lib().evox_default_ldx(algo, D)
    if ldx <= 0:
        raise EvoxError(EINVAL, f"no row pitch for algo {algo}, D = {D}")
    return ldx


def make_params(algo, fn_id, N, D, lb, ub, v_lo=0.0, v_hi=0.0, w=0.6, c1=1.5, c2=1.5, phi=0.1,
                vmax=0.0, clamp_x=0, seed=0, ldx=None, x_init=0, x_mu=0.0, x_sigma=1.0, de_f=0.5,
                de_cr=0.9, es_sigma=0.1, es_lr=0.01, pgpe_sigma_lr=0.01, pgpe_max_change=0.2, n_obj=3,
                sbx_eta=20.0, pm_eta=20.0, cso_local=0):
    return Params(algo=algo, fn_id=fn_id, N=N, D=D, ldx=pitch(D, algo) if ldx is None else ldx,
                  lb=lb, ub=ub, v_lo=v_lo, v_hi=v_hi, w=w, c1=c1, c2=c2, phi=phi, vmax=vmax,
                  clamp_x=clamp_x, x_init=x_init, x_mu=x_mu, x_sigma=x_sigma, de_f=de_f,
                  de_cr=de_cr, es_sigma=es_sigma, es_lr=es_lr, pgpe_sigma_lr=pgpe_sigma_lr,
                  pgpe_max_change=pgpe_max_change, seed=seed, n_obj=n_obj, sbx_eta=sbx_eta, pm_eta=pm_eta,
                  cso_local=cso_local)


def evox_scratch_bytes(params):
    return int(lib().evox_scratch_bytes(ctypes.byref(params)))


class Swarm:
    """A PSO, CSO, DE, OpenES, PGPE, MA-ES or NSGA-II state over torch-allocated device buffers.

    x, v (and pbest) are [N, ldx] float32 tensors whose first D columns are the
    population; pfit / fit are [N]; gbest / xbar are [ldx].  DE has x and fit
    only (its second population buffer lives in the scratch); ES has x = the
    center theta [ldx] and fit = the last generation's sample fitness [N];
    PGPE also v = the per-dimension deviations [ldx].  MA-ES has x = the center
    y [ldx], v = the path s [ldx], mat = M [D, ldx], sigma [1] and fit [N].
    NSGA-II has x [N, ldx], obj [N, n_obj] (DTLZ1), front [N] (int32) and
    crowd [N] (float64).
    """

    def __init__(self, params: Params, device="cuda", stream=None):
        import torch
        self.P = params
        self.stream = stream if stream is not None else torch.cuda.current_stream(device)
        N, ldx = params.N, params.ldx
        f32 = dict(dtype=torch.float32, device=device)
        # ES / PGPE: x is the center (one row); PGPE: v the deviations (one row)
        one_row = params.algo in (ES, PGPE, MAES)
        self.x = torch.empty((ldx,) if one_row else (N, ldx), **f32)
        self.v = (torch.empty((N, ldx), **f32) if params.algo in (PSO, CSO)
                  else torch.empty((ldx,), **f32) if params.algo in (PGPE, MAES) else None)
        self.mat = torch.empty((params.D, ldx), **f32) if params.algo == MAES else None
        self.sigma = torch.empty((1,), **f32) if params.algo == MAES else None
        nsga = params.algo == NSGA2
        self.obj = torch.empty((N, params.n_obj), **f32) if nsga else None
        self.front = torch.empty((N,), dtype=torch.int32, device=device) if nsga else None
        self.crowd = torch.empty((N,), dtype=torch.float64, device=device) if nsga else None
        if nsga:
            self.pbest = self.pfit = self.gbest = self.xbar = self.fit = None
        elif params.algo in (DE, ES, PGPE, MAES):
            self.pbest = self.pfit = self.gbest = self.xbar = None
            self.fit = torch.empty((N,), **f32)
        elif params.algo == PSO:
            self.pbest = torch.empty((N, ldx), **f32)
            self.pfit = torch.empty((N,), **f32)
            self.gbest = torch.empty((ldx,), **f32)
            self.fit = torch.empty((N,), **f32)
            self.xbar = None
        else:
            self.pbest = self.pfit = self.gbest = None
            self.fit = torch.empty((N,), **f32)
            self.xbar = torch.empty((ldx,), **f32)
        nbytes = evox_scratch_bytes(params)
        if nbytes == 0:
            _check(EINVAL)
        self.scratch = torch.empty((nbytes + 255) // 256 * 256 // 4, dtype=torch.int32, device=device)
        self.buffers = Buffers(x=_ptr(self.x), v=_ptr(self.v), pbest=_ptr(self.pbest),
                               pfit=_ptr(self.pfit), fit=_ptr(self.fit), gbest=_ptr(self.gbest),
                               xbar=_ptr(self.xbar), mat=_ptr(self.mat), sigma=_ptr(self.sigma),
                               obj=_ptr(self.obj), front=_ptr(self.front), crowd=_ptr(self.crowd),
                               scratch=_ptr(self.scratch),
                               scratch_bytes=self.scratch.numel() * 4)
        self.handle = ctypes.c_void_p()
        _check(lib().evox_state_create(ctypes.byref(self.P), ctypes.byref(self.buffers),
                                       _stream(self.stream), ctypes.byref(self.handle)))

    def __del__(self):
        h = getattr(self, "handle", None)
        if h and _lib is not None:
            _lib.evox_state_destroy(h)
            self.handle = None

    @property
    def D(self):
        return self.P.D

    @property
    def t(self):
        return int(lib().evox_generation(self.handle))

    def set_generation(self, t):
        _check(lib().evox_set_generation(self.handle, t))

    def step(self, n_gens=1):
        if self.P.algo == PSO:
            _check(lib().evox_pso_step(self.handle, n_gens))
        elif self.P.algo == CSO:
            _check(lib().evox_cso_step(self.handle, n_gens))
        elif self.P.algo == DE:
            _check(lib().evox_de_step(self.handle, n_gens))
        elif self.P.algo == ES:
            _check(lib().evox_es_step(self.handle, n_gens))
        elif self.P.algo == PGPE:
            _check(lib().evox_pgpe_step(self.handle, n_gens))
        elif self.P.algo == MAES:
            _check(lib().evox_maes_step(self.handle, n_gens))
        else:
            _check(lib().evox_nsga2_step(self.handle, n_gens))

    def refresh(self, refit=True):
        _check(lib().evox_cso_refresh(self.handle, 1 if refit else 0))

    def best(self, with_x=False):
        import numpy as np
        f = ctypes.c_float(0.0)
        i = ctypes.c_int64(0)
        xb = np.zeros(self.P.D, np.float32) if with_x else None
        _check(lib().evox_best(self.handle, ctypes.byref(f), ctypes.byref(i),
                               xb.ctypes.data_as(ctypes.c_void_p) if with_x else None))
        return (f.value, i.value, xb) if with_x else (f.value, i.value)

    def profile(self, enable):
        _check(lib().evox_profile(self.handle, 1 if enable else 0))

    def profile_read(self):
        ms, n, imp = ctypes.c_double(0), ctypes.c_int64(0), ctypes.c_int64(0)
        _check(lib().evox_profile_read(self.handle, ctypes.byref(ms), ctypes.byref(n),
                                       ctypes.byref(imp)))
        return ms.value, n.value, imp.value

    def view(self, name):
        """The [N, D] (or [D]) part of a buffer, without the padding columns."""
        t = getattr(self, name)
        return t[..., :self.P.D]
