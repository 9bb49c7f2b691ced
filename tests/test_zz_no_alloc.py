"""evox_eval_argmin_noalloc, the evaluation + selection entry point that
allocates nothing (its selection slots are the library's static per-device
array), against evox_eval_argmin with a caller scratch: fitness bit for bit,
the same best value and index, on two calls in a row (the second smaller, so
a stale slot left by the first would show)."""
import pytest
import torch

from paper_2301_12457_amd.workloads import normal_matrix_torch

pytestmark = pytest.mark.gpu

# (function, N, D, ldx, seed): Rosenbrock on the evaluation workload's row
# shape, then a smaller ragged Ackley population
CALLS = [(4, 200_003, 1000, 1000, 41), (1, 4_097, 77, 80, 42)]


def test_noalloc_matches_scratch_entry_point(evox_gpu):
    ev = evox_gpu
    for fn, N, D, ldx, seed in CALLS:
        print(f"noalloc fn={fn} N={N} D={D} ldx={ldx}", flush=True)
        X = normal_matrix_torch(N, D, 1.0, 0.5, seed, ldx=ldx)
        out_a = torch.empty(N, dtype=torch.float32, device="cuda")
        out_b = torch.full((N,), float("nan"), dtype=torch.float32, device="cuda")
        bf_a = torch.empty(1, dtype=torch.float32, device="cuda")
        bi_a = torch.empty(1, dtype=torch.int64, device="cuda")
        bf_b = torch.full((1,), float("nan"), dtype=torch.float32, device="cuda")
        bi_b = torch.full((1,), -1, dtype=torch.int64, device="cuda")
        scratch = torch.empty(ev.evox_eval_argmin_scratch_bytes(N) // 4 + 64, dtype=torch.int32,
                              device="cuda")
        ev.evox_eval_argmin(fn, X, N, D, ldx, out_a, bf_a, bi_a, scratch)
        ev.evox_eval_argmin_noalloc(fn, X, N, D, ldx, out_b, bf_b, bi_b)
        torch.cuda.synchronize()
        assert torch.equal(out_a, out_b)
        assert int(bi_b.item()) == int(bi_a.item())
        assert torch.equal(bf_a, bf_b)
        i = int(bi_a.item())
        assert 0 <= i < N and float(bf_a.item()) == float(out_a[i].item())
        assert float(out_a.min().item()) == float(bf_a.item())
