"""Pins of the oracle's random-number layer.

Philox4x32-10 (Salmon et al., SC'11) is checked against rocRAND's own
implementation, called through its host-callable engine.  The u32 -> U[0,1)
map is checked exhaustively over every 24-bit pattern.
"""
import numpy as np

from conftest import u01_exact


def test_philox_matches_rocrand_random_counters(ref, rocrand_philox):
    rng = np.random.default_rng(2301)
    seeds = rng.integers(0, 2**64, size=3000, dtype=np.uint64)
    ctrs = rng.integers(0, 2**32, size=(3000, 4), dtype=np.uint64)
    rows = np.concatenate([seeds[:, None], ctrs], axis=1)
    got = np.array([[ref.philox_word(int(r[0]), *[int(c) for c in r[1:]], k) for k in range(4)]
                    for r in rows], dtype=np.uint32)
    want = rocrand_philox(rows)
    assert np.array_equal(got, want)


def test_philox_matches_rocrand_edge_counters(ref, rocrand_philox):
    M = 0xFFFFFFFF
    rows = [(0, 0, 0, 0, 0), (2**64 - 1, M, M, M, M), (1, 1, 0, 0, 0), (1, 0, 1, 0, 0),
            (1, 0, 0, 1, 0), (1, 0, 0, 0, 1), (2**32, 0, 0, 0, 0), (7, M, 0, 0, 0),
            (3, 12345, 678, 9, 4)]
    got = np.array([[ref.philox_word(r[0], *r[1:], k) for k in range(4)] for r in rows],
                   dtype=np.uint32)
    assert np.array_equal(got, rocrand_philox(rows))


def test_philox_key_words_are_seed_low_high(ref):
    ctr = [5, 6, 7, 8]
    seed = (0x01234567 << 32) | 0x89ABCDEF
    w = ref.philox4x32_10(ctr, [0x89ABCDEF, 0x01234567])
    assert [ref.philox_word(seed, *ctr, k) for k in range(4)] == [int(v) for v in w]


def test_u01_exhaustive_over_24_bit_patterns(ref):
    top = np.arange(1 << 24, dtype=np.uint64)
    # low byte set to a mix of values: it must be ignored
    words = ((top << np.uint64(8)) | (top & np.uint64(0xFF))).astype(np.uint32)
    u = ref.u01_array(words)
    assert np.array_equal(u, u01_exact(words))
    assert u.min() == 0.0 and u.max() == np.float32(1.0 - 2.0**-24)
    assert np.all(np.diff(u) > 0)


def test_init_uniform_uses_stream_words(ref, rocrand_philox):
    seed, N, D, lo, hi = 11, 3, 9, -5.12, 5.12
    X = ref.init_uniform(seed, 0, N, D, lo, hi)
    rows = [(seed, j // 4, i, 0, 0) for i in range(N) for j in range(D)]
    words = rocrand_philox(rows)
    u = u01_exact([words[k, (k % D) % 4] for k in range(N * D)]).reshape(N, D)
    lo32, rng32 = np.float32(lo), np.float32(hi) - np.float32(lo)
    want = (u.astype(np.float64) * rng32 + lo32).astype(np.float32)  # single rounding = fma
    assert np.array_equal(X, want)
    assert X.min() >= lo32 and X.max() < np.float32(hi)
