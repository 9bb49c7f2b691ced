"""GPU parity of the CSO pairing sort (integer work: bit-exact).

evox_permutation gives the pairing permutations the CSO generations use;
they are compared with the oracle's sort of the same Philox keys, across
launch batches, at the generation-counter edge and at the largest swarm
(2^24).  evox_argsort_u32 runs the same passes on caller keys, which is how
the path for a superbucket too large for the LDS sort (more than 4096 keys
sharing their top bits) is reached: all-equal keys, keys confined to the low
bits, heavy ties.
"""
import zlib

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def scratch_for(evox, N, batch):
    n = evox.lib().evox_permutation_scratch_bytes(N, batch)
    assert n > 0
    return torch.empty((n + 255) // 4 + 64, dtype=torch.int32, device="cuda")


def gpu_perms(evox, seed, t0, n_gens, N, batch=8):
    out = torch.full((n_gens, N), -1, dtype=torch.int32, device="cuda")
    evox.evox_permutation(seed, t0, n_gens, N, out, scratch_for(evox, N, batch))
    return out.cpu().numpy().astype(np.int64)


@pytest.mark.parametrize("N", [1, 2, 3, 4, 5, 1023, 4096, 4097, 100_003])
def test_permutations_match_oracle(evox_gpu, ref, N):
    seed, t0, n_gens = 1234567, 5, 11      # 11 generations: batches of 8 + 3
    print(f"perm N={N}", flush=True)
    got = gpu_perms(evox_gpu, seed, t0, n_gens, N)
    for g in range(n_gens):
        assert np.array_equal(got[g], ref.perm(seed, t0 + g, N)), g


def test_permutation_batch_size_does_not_matter(evox_gpu):
    a = gpu_perms(evox_gpu, 9, 0, 5, 50_000, batch=1)
    b = gpu_perms(evox_gpu, 9, 0, 5, 50_000, batch=8)
    assert np.array_equal(a, b)


def test_permutation_at_generation_counter_edge(evox_gpu, ref):
    t0 = 2**32 - 3
    got = gpu_perms(evox_gpu, 2**64 - 1, t0, 3, 777)
    for g in range(3):
        assert np.array_equal(got[g], ref.perm(2**64 - 1, t0 + g, 777))


def test_permutation_largest_swarm(evox_gpu, ref):
    N = 2**24
    got = gpu_perms(evox_gpu, 3, 17, 1, N, batch=1)[0]
    assert np.array_equal(got, ref.perm(3, 17, N))


def test_permutation_rejects_bad_args(evox_gpu):
    L = evox_gpu.lib()
    s = scratch_for(evox_gpu, 100, 1)
    out = torch.empty(200, dtype=torch.int32, device="cuda")
    assert L.evox_permutation(0, 0, 1, 0, out.data_ptr(), s.data_ptr(), 1 << 20, None) == evox_gpu.EINVAL
    assert L.evox_permutation(0, 0, 1, 2**24 + 1, out.data_ptr(), s.data_ptr(), 1 << 20, None) == evox_gpu.EINVAL
    assert L.evox_permutation(0, 2**32 - 1, 2, 100, out.data_ptr(), s.data_ptr(), 1 << 20, None) == evox_gpu.EINVAL
    assert L.evox_permutation(0, 0, 1, 100, out.data_ptr(), s.data_ptr(), 16, None) == evox_gpu.ENOSPC
    assert L.evox_permutation(0, 0, 0, 100, None, None, 0, None) == evox_gpu.OK


def gpu_argsort(evox, keys):
    N = keys.size
    k = torch.from_numpy(keys.astype(np.uint32).view(np.int32)).cuda()
    out = torch.full((max(N, 1),), -1, dtype=torch.int32, device="cuda")
    evox.evox_argsort_u32(k, N, out, scratch_for(evox, max(N, 1), 1))
    return out.cpu().numpy()[:N].astype(np.int64)


@pytest.mark.parametrize("case", ["random", "ties", "all_equal_lds", "all_equal_big", "low_bits",
                                  "top_heavy", "max_n", "tiny"])
def test_argsort_matches_oracle(evox_gpu, ref, case):
    rng = np.random.default_rng(zlib.crc32(case.encode()))
    keys = {
        "random": lambda: rng.integers(0, 2**32, size=30_000, dtype=np.uint64),
        "ties": lambda: rng.integers(0, 8, size=30_000),
        "all_equal_lds": lambda: np.full(4096, 123456),          # one bucket, at the LDS capacity
        "all_equal_big": lambda: np.full(20_000, 2**31 + 5),     # one bucket beyond it
        "low_bits": lambda: rng.integers(0, 2**16, size=20_000),  # top bits all zero
        "top_heavy": lambda: np.concatenate([rng.integers(0, 2**32, size=10_000, dtype=np.uint64),
                                             np.full(6_000, 2**32 - 1)]),
        "max_n": lambda: rng.integers(0, 2**32, size=65_536, dtype=np.uint64),
        "tiny": lambda: np.array([5, 5, 1]),
    }[case]().astype(np.uint32)
    print(f"argsort {case} N={keys.size}", flush=True)
    assert np.array_equal(gpu_argsort(evox_gpu, keys), ref.argsort_u32(keys))


def test_argsort_bounds(evox_gpu):
    L = evox_gpu.lib()
    assert L.evox_argsort_u32(None, 0, None, None, 0, None) == evox_gpu.OK
    assert L.evox_argsort_u32(None, 65_537, None, None, 0, None) == evox_gpu.EINVAL
