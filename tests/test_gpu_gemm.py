"""GPU parity of the matrix-core product against the oracle's fp64 product.

Bound per output: |C_gpu - C_ref| <= |alpha| gamma_K sum_k |a_ik b_kj|
+ |beta c_ij| u + ulp(C_ref), with u = 2^-24 and gamma_K = K u / (1 - K u),
the textbook bound of any order of an fp32 sum of K products (the kernel's
order is fixed but not the oracle's), the rounding of beta c, and the final
rounding of the oracle's fp64 result."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


def to_dev(X):
    """X in a zero-padded device buffer whose row stride is a multiple of 4."""
    rows, cols = X.shape
    buf = torch.zeros((max(rows, 1), max((cols + 3) // 4 * 4, 4)), dtype=torch.float32)
    buf[:rows, :cols] = torch.from_numpy(X)
    return buf.cuda()[:rows, :cols]


def limit(A, B, ta, tb, alpha, beta, C0, want):
    K = A.shape[0] if ta else A.shape[1]
    a = np.abs(A.astype(np.float64).T if ta else A.astype(np.float64))
    b = np.abs(B.astype(np.float64).T if tb else B.astype(np.float64))
    g = K * U / (1 - K * U)
    return abs(alpha) * g * (a @ b) + abs(beta) * np.abs(C0.astype(np.float64)) * U + \
        np.spacing(np.abs(want))


# (65..112 rows take the 16 x 16-tile kernel: a full 112-row block, a ragged
# one with ragged columns and K, and the 101 rows of the MA-ES sampling
# product)
SHAPES = [(1, 1, 1), (5, 7, 3), (128, 128, 16), (129, 130, 17), (300, 77, 1000), (64, 512, 2048),
          (1000, 1000, 1000), (33, 100, 0), (112, 64, 64), (65, 33, 129), (101, 300, 777)]


@pytest.mark.parametrize("ta", [False, True])
@pytest.mark.parametrize("tb", [False, True])
@pytest.mark.parametrize("M,N,K", SHAPES)
def test_gemm_matches_oracle(evox_gpu, ref, ta, tb, M, N, K):
    print(f"gemm ta={ta} tb={tb} {M}x{N}x{K}", flush=True)
    rng = np.random.default_rng([M, N, K, int(ta), int(tb)])
    A = rng.standard_normal((K, M) if ta else (M, K)).astype(np.float32)
    B = rng.standard_normal((N, K) if tb else (K, N)).astype(np.float32)
    C0 = rng.standard_normal((M, N)).astype(np.float32)
    for alpha, beta in ((1.0, 0.0), (0.5, -2.0)):
        Cd = to_dev(C0)
        evox_gpu.evox_sgemm(to_dev(A), to_dev(B), Cd, ta, tb, alpha, beta)
        got = Cd.cpu().numpy()
        want = ref.gemm(A, B, ta, tb, alpha, beta, C0)
        err = np.abs(got.astype(np.float64) - want.astype(np.float64))
        bad = np.argwhere(err > limit(A, B, ta, tb, alpha, beta, C0, want))
        assert bad.size == 0, f"alpha={alpha} beta={beta}: {len(bad)} entries off, e.g. {bad[:3].tolist()}"


def test_gemm_is_reproducible(evox_gpu):
    rng = np.random.default_rng(4)
    A, B = (to_dev(rng.standard_normal((300, 700)).astype(np.float32)),
            to_dev(rng.standard_normal((700, 260)).astype(np.float32)))
    C1, C2 = torch.empty(300, 260, device="cuda"), torch.empty(300, 260, device="cuda")
    evox_gpu.evox_sgemm(A, B, C1)
    evox_gpu.evox_sgemm(A, B, C2)
    assert torch.equal(C1, C2)


def test_gemm_rejects_bad_args(evox_gpu):
    L = evox_gpu.lib()
    x = torch.zeros(64, device="cuda")
    p = x.data_ptr()
    assert L.evox_sgemm(0, 0, 4, 4, 4, 1.0, p, 2, p, 4, 0.0, p, 4, None) == evox_gpu.EINVAL    # lda < K
    assert L.evox_sgemm(0, 0, 4, 4, 4, 1.0, p, 6, p, 4, 0.0, p, 4, None) == evox_gpu.EALIGN
    assert L.evox_sgemm(0, 0, 4, 4, 4, 1.0, p + 4, 4, p, 4, 0.0, p, 4, None) == evox_gpu.EALIGN
    assert L.evox_sgemm(0, 0, -1, 4, 4, 1.0, p, 4, p, 4, 0.0, p, 4, None) == evox_gpu.EINVAL
    assert L.evox_sgemm(0, 0, 0, 4, 4, 1.0, None, 4, None, 4, 0.0, None, 4, None) == evox_gpu.OK
