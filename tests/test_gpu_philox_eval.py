"""GPU parity: the device Philox stream (bit-exact) and Problem.evaluate
(fitness within tolerance, argmin index exact) against the oracle."""
import numpy as np
import pytest
import torch

from parity import assert_fitness, index_ok

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seed,c1,c2,c3,n", [(0, 0, 0, 0, 1000), (2**64 - 1, 7, 123456, 3, 4097),
                                             (42, 2**32 - 1, 2**32 - 1, 4, 513)])
def test_philox_stream_bit_exact(evox_gpu, ref, seed, c1, c2, c3, n):
    out = torch.zeros(4 * n, dtype=torch.int32, device="cuda")
    evox_gpu.evox_philox_fill(seed, c1, c2, c3, n, out)
    got = out.cpu().numpy().view(np.uint32).reshape(n, 4)
    rows = list(range(0, n, max(1, n // 97))) + [n - 1]
    for k in rows:
        want = ref.philox4x32_10([k, c1, c2, c3], [seed & 0xFFFFFFFF, seed >> 32])
        assert np.array_equal(got[k], want), k


SHAPES = [(1, 1), (7, 3), (33, 10), (100, 10), (257, 100), (64, 257), (40, 1000), (9, 1001),
          (5, 4100), (3, 16385), (2, 32768)]


@pytest.mark.parametrize("fn", range(6))
@pytest.mark.parametrize("N,D", SHAPES)
def test_eval_matches_oracle(evox_gpu, ref, fn, N, D):
    print(f"eval fn={fn} N={N} D={D}", flush=True)
    rng = np.random.default_rng(1000 * fn + D)
    span = {0: 5.0, 1: 32.768, 2: 5.12, 3: 600.0, 4: 2.0, 5: 500.0}[fn]
    X = rng.uniform(-span, span, size=(N, D)).astype(np.float32)
    if N > 2:
        X[1] = 0.0            # optimum of most functions
        X[2] = 1.0            # Rosenbrock optimum
    Xd = torch.from_numpy(X).cuda()
    out = torch.empty(N, dtype=torch.float32, device="cuda")
    evox_gpu.evox_eval(fn, Xd, out)
    f_gpu = out.cpu().numpy()
    f_ref = ref.evaluate(fn, X)
    assert_fitness(fn, X, f_gpu, f_ref, f"fn {fn} N {N} D {D}")


@pytest.mark.parametrize("fn", range(6))
@pytest.mark.parametrize("N,D,ldx", [(50, 10, 12), (300, 100, 104), (33, 1000, 1024)])
def test_eval_argmin_pitched(evox_gpu, ref, fn, N, D, ldx):
    rng = np.random.default_rng(7 + fn)
    X = rng.uniform(-3, 3, size=(N, ldx)).astype(np.float32)
    X[:, D:] = np.nan          # padding must never be read into the fitness
    Xd = torch.from_numpy(X).cuda()
    out = torch.empty(N, dtype=torch.float32, device="cuda")
    bf = torch.empty(1, dtype=torch.float32, device="cuda")
    bi = torch.empty(1, dtype=torch.int64, device="cuda")
    scratch = torch.empty(evox_gpu.evox_eval_argmin_scratch_bytes(N) // 4 + 64, dtype=torch.int32,
                          device="cuda")
    evox_gpu.evox_eval_argmin(fn, Xd, N, D, ldx, out, bf, bi, scratch)
    f_gpu = out.cpu().numpy()
    f_ref = ref.evaluate(fn, X[:, :D])
    assert_fitness(fn, X[:, :D], f_gpu, f_ref, f"fn {fn}")
    i_gpu = int(bi.item())
    assert i_gpu == ref.argmin(f_gpu)                       # exact on the GPU's own values
    assert index_ok(fn, X[:, :D], f_ref, i_gpu, ref.argmin(f_ref))
    assert float(bf.item()) == f_gpu[i_gpu]


def test_eval_unaligned_input(evox_gpu, ref):
    N, D = 41, 13
    rng = np.random.default_rng(3)
    X = rng.uniform(-2, 2, size=(N, D)).astype(np.float32)
    buf = torch.zeros(N * D + 1, dtype=torch.float32, device="cuda")
    buf[1:] = torch.from_numpy(X.ravel()).cuda()
    out = torch.empty(N, dtype=torch.float32, device="cuda")
    Xv = buf[1:].view(N, D)          # 4-byte aligned only
    evox_gpu.evox_eval(4, Xv, out)
    assert_fitness(4, X, out.cpu().numpy(), ref.evaluate(4, X), "unaligned")


def test_argmin_ties_nan_and_signed_zero(evox_gpu, ref):
    # Sphere of rows with known values: ties at the minimum go to the lowest index
    N, D = 3000, 4
    X = np.full((N, D), 2.0, np.float32)
    X[[17, 1500, 2999]] = 0.0
    X[5] = np.nan
    Xd = torch.from_numpy(X).cuda()
    out = torch.empty(N, dtype=torch.float32, device="cuda")
    bf = torch.empty(1, dtype=torch.float32, device="cuda")
    bi = torch.empty(1, dtype=torch.int64, device="cuda")
    scratch = torch.empty(evox_gpu.evox_eval_argmin_scratch_bytes(N) // 4 + 64, dtype=torch.int32,
                          device="cuda")
    evox_gpu.evox_eval_argmin(0, Xd, N, D, D, out, bf, bi, scratch)
    assert int(bi.item()) == 17 and float(bf.item()) == 0.0
    X[:] = np.nan
    evox_gpu.evox_eval_argmin(0, torch.from_numpy(X).cuda(), N, D, D, out, bf, bi, scratch)
    assert int(bi.item()) == 0 and np.isnan(bf.item())


def test_eval_empty_population(evox_gpu):
    out = torch.empty(1, dtype=torch.float32, device="cuda")
    X = torch.empty((0, 5), dtype=torch.float32, device="cuda")
    evox_gpu.evox_eval(0, X, out)
    torch.cuda.synchronize()


@pytest.mark.parametrize("n", [4, 1028, 4096 * 1024 + 8])
def test_pso_stream(evox_gpu, n):
    """The PSO data-movement floor computes v + (p - x), then x + v, in fp32
    (one rounding per operation, as numpy does), and touches nothing past n."""
    g = torch.Generator().manual_seed(n)
    x, v, p = (torch.randn(n + 8, generator=g) for _ in range(3))
    xd, vd, pd = x.cuda(), v.cuda(), p.cuda()
    evox_gpu.evox_pso_stream(xd, vd, pd, n)
    xn, vn, pn = x.numpy(), v.numpy(), p.numpy()
    v_ref = vn[:n] + (pn[:n] - xn[:n])
    x_ref = xn[:n] + v_ref
    assert np.array_equal(vd.cpu().numpy()[:n], v_ref) and np.array_equal(xd.cpu().numpy()[:n], x_ref)
    assert torch.equal(vd[n:].cpu(), v[n:]) and torch.equal(xd[n:].cpu(), x[n:]) and torch.equal(pd.cpu(), p)


@pytest.mark.parametrize("n", [1, 3, 4, 1027, 4096 * 1024 + 5])
def test_stream_copy(evox_gpu, n):
    src = torch.randn(n + 8, device="cuda")
    dst = torch.zeros(n + 8, device="cuda")
    evox_gpu.evox_copy(src, dst, n)
    assert torch.equal(dst[:n], src[:n]) and torch.all(dst[n:] == 0)
