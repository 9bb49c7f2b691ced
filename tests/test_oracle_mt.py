"""The all-core CPU baseline (oracle/evox_ref_mt.c: the oracle compiled with
its row loops split over threads) computes exactly what the oracle computes:
states bit for bit after several generations, at several thread counts."""
import numpy as np
import pytest


@pytest.mark.parametrize("threads", [1, 3, 8])
@pytest.mark.parametrize("fn,N,D,kw", [(2, 64, 37, dict(vmax=2.048)), (1, 33, 129, dict(v_lo=-1.0, v_hi=1.0)),
                                        (4, 17, 1001, {})])
def test_pso_all_core_equals_oracle(ref, threads, fn, N, D, kw):
    a = ref.PSO(ref.make_params(fn, N, D, -5.0, 5.0, seed=N + D, **kw))
    b = ref.PSO(ref.make_params(fn, N, D, -5.0, 5.0, seed=N + D, **kw))
    a.step(7)
    ref.mt_step(b, 7, threads)
    for name in ("x", "v", "p", "pf", "g"):
        assert np.array_equal(getattr(a, name), getattr(b, name)), name
    assert (a.gf, a.gi, a.t) == (b.gf, b.gi, b.t)


@pytest.mark.parametrize("threads", [1, 4, 7])
@pytest.mark.parametrize("fn,N,D,local", [(3, 301, 29, 0), (0, 1001, 5, 0), (2, 64, 37, 1), (5, 7, 3, 1)])
def test_cso_all_core_equals_oracle(ref, threads, fn, N, D, local):
    a = ref.CSO(ref.make_params(fn, N, D, -50.0, 50.0, seed=N, cso_local=local))
    b = ref.CSO(ref.make_params(fn, N, D, -50.0, 50.0, seed=N, cso_local=local))
    a.step(6)
    ref.mt_step(b, 6, threads)
    for name in ("x", "v", "fit"):
        assert np.array_equal(getattr(a, name), getattr(b, name)), name
    assert (a.best_idx, a.t) == (b.best_idx, b.t)


@pytest.mark.parametrize("fn", range(6))
def test_eval_all_core_equals_oracle(ref, fn):
    rng = np.random.default_rng(fn)
    X = rng.normal(0.5, 2.0, size=(513, 70)).astype(np.float32)
    assert np.array_equal(ref.mt_evaluate(fn, X, 5), ref.evaluate(fn, X))
