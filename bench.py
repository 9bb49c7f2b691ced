"""Benchmark of the MI355X PSO / CSO generation hot path.

One step = one Workflow.step call of the workload's full generation count
(evox_pso_step / evox_cso_step(state, gens)), or one evaluation pass for the
evaluation-only workload, on inputs resident in HBM.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""
import argparse
import hashlib
import json
import os
import re
import sys
import statistics
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2301_12457_amd.workloads import WORKLOADS  # noqa: E402

METRIC = "individual·dim updates/sec per fused generation; % of HBM peak GB/s"
UNIT = "individual·dim updates/s"
HBM_PEAK_GBS = 8000.0
DEFAULT_WORKLOAD = "pso_rastrigin_1e5x1e3"
# the benchmark set: PSO Sphere 100 x 10, PSO Ackley 1e4 x 1e3, PSO Rastrigin
# 1e5 x 1e3 (the headline), CSO Griewank 1e6 x 100, evaluation + argmin of
# Rosenbrock 1,048,576 x 1000; every bench.py run times all of them
CONFIG_WORKLOADS = ("pso_sphere_100x10", "pso_ackley_1e4x1e3", "pso_rastrigin_1e5x1e3", "cso_griewank_1e6x100",
                    "eval_rosenbrock_1m_x1e3")
KERNEL_SOURCES = ("paper_2301_12457_amd/csrc/evox_device.hpp",
                  "paper_2301_12457_amd/csrc/evox_kernels.hpp")


def kernel_hash():
    """Hash of the kernel sources' code: comments and white space removed,
    so that a change of wording leaves the committed counters valid."""
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            src = f.read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        src = re.sub(r"//[^\n]*", "", src)
        h.update(re.sub(r"\s+", "", src).encode())
    return h.hexdigest()[:16]


def traffic_from_profile(name):
    """HBM bytes per launch of the dominant kernel from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE summary (KiB per dispatch, each scaled
    by what the counter reads for a device copy of known size), if it was
    taken on the current kernel sources; None otherwise."""
    path = os.path.join(ROOT, "profiles", f"{name}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_sha") != kernel_hash():
        return None
    return 1024.0 * (t["fetch_kib_per_dispatch"] * t["fetch_scale"] +
                     t["write_kib_per_dispatch"] * t["write_scale"])


def pso_bytes_per_generation(w, evaluations, improved_rows):
    # read x, v, pbest and write x, v (20 B per element); read pfit (4 B per
    # row); write pbest row and pfit of each improved row (the kernels' count
    # over `evaluations` generations)
    imp = improved_rows / max(evaluations, 1)
    return 20.0 * w.N * w.D + 4.0 * w.N + (4.0 * w.D + 4.0) * imp


def de_bytes_per_launch(w):
    # per target element: read the target, gather three partners, write the
    # next population (20 B); per target: read and write its fitness
    return 20.0 * w.N * w.D + 8.0 * w.N


# OpenES is bound by vector-ALU work (the perturbations are regenerated, not
# stored): lane-ops per perturbation element and generation, counted from
# the computation as written -- Philox4x32-10 is 10 rounds of two 32x32->64
# products (4 ops) and two three-input xors (one instruction each on gfx950)
# per 4 elements (15), Box-Muller 16 ops per 2 elements (8), the two samples
# and their Sphere terms (4); the gradient pass regenerates the perturbation
# (23) and adds its weighted value (1).
ES_OPS_PER_ELEMENT = 15 + 8 + 4 + 23 + 1
# PGPE: the same, with two weighted sums in the gradient pass (z and z^2 - 1)
PGPE_OPS_PER_ELEMENT = 15 + 8 + 4 + 23 + 3
ALU_PEAK_TOPS = 256 * 64 * 2.4e9 / 1e12   # 256 CUs x 64 lanes x 2.4 GHz, 32-bit lane-ops
MFMA_F32_PEAK_TFLOPS = 157.3              # dense fp32 matrix-core peak
# NSGA-II's dominance pass: per ordered pair of the merged population, two
# comparisons per objective, one combination of the two outcomes and one add
def nsga2_count_ops(w):
    return (2.0 * w.N) ** 2 * (2 * w.n_obj + 2)


def gemm_nt_label(rows):
    """The A B^T kernel the library picks for `rows` rows of A."""
    if 64 < rows <= 112:
        return "k_gemm_nt16<7>"          # 16 x 16 tiles, 112 rows
    return "k_gemm_nt<%d,%d>" % (64 if rows <= 64 else 128, 64 if rows <= 128 else 128)


def maes_flops(w):
    """Algorithmic flops of the MA-ES generation's two products: the steps
    and M s, 2 (N + 1) D^2, and the rank-mu update, 2 (mu + 1) D^2."""
    mu = w.N // 2
    return 2.0 * (w.N + 1) * w.D ** 2, 2.0 * (mu + 1) * w.D ** 2


def cso_bytes_per_launch(w):
    # per pair: read winner row, loser x and v, write loser x and v
    # (20 B per pair element = 10 B per individual element); fitness of both
    # and the permutation entries (4 B each), write loser fitness.  The
    # neighbourhood version writes the next positions to the other buffer:
    # it also writes the winner's row (4 B per pair element); every old row
    # is counted once, so the loser's neighbours (rows of other pairs) add
    # nothing
    pairs = w.N // 2
    return (24.0 if w.cso_local else 20.0) * pairs * w.D + pairs * (4 * 2 + 4 * 2 + 4)


def host_cpu():
    """Model name of the host CPU and the number of cores this process may use."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, len(os.sched_getaffinity(0))


def cpu_baseline(w, budget_s=12.0):
    """The oracle, single-threaded and pinned to one core, on a bounded sample
    of the workload; and, for PSO, CSO and evaluation, the all-core leg: the
    oracle's steps with their row loops split over every core this process
    may use (oracle/evox_ref_mt.c, bit-identical results), the comparison the
    paper's CPU runs make (all host threads)."""
    allowed = os.sched_getaffinity(0)
    os.sched_setaffinity(0, {min(allowed)})
    try:
        out = _cpu_baseline(w, budget_s)
    finally:
        os.sched_setaffinity(0, allowed)
    out["host_cpu"], out["host_cores_available"] = host_cpu()
    if w.algo in ("pso", "cso", "eval"):
        # every core of this process's share: the affinity set, bounded by the
        # OpenMP thread budget where the host sets one
        threads = len(allowed)
        if os.environ.get("OMP_NUM_THREADS", "").isdigit():
            threads = max(1, min(threads, int(os.environ["OMP_NUM_THREADS"])))
        out["all_cores"] = _cpu_all_cores(w, threads, budget_s)
    return out


def _cpu_all_cores(w, threads, budget_s):
    import oracle
    fn = oracle.FN_NAMES.index(w.fn)
    if w.algo == "eval":
        from paper_2301_12457_amd.workloads import normal_matrix_np
        rows = min(w.N, 10_000 * threads)
        X = normal_matrix_np(rows, w.D, w.x_mu, w.x_sigma, w.seed)
        t0 = time.perf_counter()
        n = 0
        while time.perf_counter() - t0 < budget_s:
            oracle.mt_evaluate(fn, X, threads)
            n += 1
        dt = time.perf_counter() - t0
        return {"value": rows * w.D * n / dt, "unit": UNIT, "cores": threads,
                "kind": "oracle, rows split over all cores",
                "sample": f"{rows} of {w.N} rows x D={w.D}, {n} evaluation passes, {dt:.1f} s"}
    rows = min(w.N, (20_000 if w.algo == "cso" else 2000) * threads)
    P = oracle.make_params(fn, rows, w.D, w.lb, w.ub, v_lo=w.v_lo, v_hi=w.v_hi, w=w.w, c1=w.c1, c2=w.c2,
                           phi=w.phi, vmax=w.vmax, seed=w.seed, cso_local=w.cso_local)
    s = (oracle.PSO if w.algo == "pso" else oracle.CSO)(P)
    oracle.mt_step(s, 1, threads)
    t0 = time.perf_counter()
    gens = 0
    while time.perf_counter() - t0 < budget_s and gens < w.gens:
        oracle.mt_step(s, 1, threads)
        gens += 1
    dt = time.perf_counter() - t0
    return {"value": rows * w.D * gens / dt, "unit": UNIT, "cores": threads,
            "kind": "oracle, rows split over all cores",
            "sample": f"{rows} of {w.N} individuals x D={w.D}, {gens} generations, {dt:.1f} s"}


def _cpu_baseline(w, budget_s):
    import oracle
    if w.algo == "nsga2":
        # the oracle's sorting is quadratic per front: a population of 1000
        rows = min(w.N, 1000)
        s = oracle.NSGA2(oracle.nsga2_params(rows, w.D, w.n_obj, seed=w.seed))
        t0 = time.perf_counter()
        gens = 0
        while time.perf_counter() - t0 < budget_s and gens < w.gens:
            s.step(1)
            gens += 1
        dt = time.perf_counter() - t0
        return {"value": rows * w.D * gens / dt, "unit": UNIT, "cores": 1, "kind": "oracle",
                "sample": f"{rows} of {w.N} individuals x D={w.D}, {gens} generations, {dt:.1f} s"}
    fn = {"sphere": 0, "ackley": 1, "rastrigin": 2, "griewank": 3, "rosenbrock": 4,
          "schwefel": 5}[w.fn]
    if w.algo == "eval":
        rows = 20_000
        X = oracle.init_normal(w.seed, rows, w.D, w.x_mu, w.x_sigma)
        t0 = time.perf_counter()
        n = 0
        while time.perf_counter() - t0 < budget_s:
            oracle.evaluate(fn, X)
            n += 1
        dt = time.perf_counter() - t0
        return {"value": rows * w.D * n / dt, "unit": UNIT, "cores": 1, "kind": "oracle",
                "sample": f"{rows} of {w.N} rows x D={w.D}, {n} evaluation passes, {dt:.1f} s"}
    rows = min(w.N, 20_000 if w.algo == "cso" else 200 if w.algo in ("es", "pgpe") else 2000)
    # MA-ES: the oracle's matrix product costs D^3 per generation, so the
    # sample keeps the population and shrinks the dimension
    D = min(w.D, 1024) if w.algo == "maes" else w.D
    P = oracle.make_params(fn, rows, D, w.lb, w.ub, cso_local=w.cso_local, v_lo=w.v_lo, v_hi=w.v_hi, w=w.w, c1=w.c1,
                           c2=w.c2, phi=w.phi, vmax=w.vmax, seed=w.seed, de_f=w.de_f,
                           de_cr=w.de_cr, es_sigma=w.es_sigma, es_lr=w.es_lr,
                           pgpe_sigma_lr=w.pgpe_sigma_lr, pgpe_max_change=w.pgpe_max_change)
    s = {"pso": oracle.PSO, "cso": oracle.CSO, "de": oracle.DE, "es": oracle.ES,
         "pgpe": oracle.PGPE, "maes": oracle.MAES}[w.algo](P)
    s.step(1)
    t0 = time.perf_counter()
    gens = 0
    while time.perf_counter() - t0 < budget_s and gens < w.gens:
        s.step(1)
        gens += 1
    dt = time.perf_counter() - t0
    return {"value": rows * D * gens / dt, "unit": UNIT, "cores": 1, "kind": "oracle",
            "sample": f"{rows} of {w.N} individuals x D={D} of {w.D}, {gens} generations, {dt:.1f} s"}


def copy_bandwidth(torch, evox, mib=1024, reps=5):
    """GB/s (read + write bytes) of the library's streaming 1 GiB device copy
    on this GPU, measured in the same run as a reference for the achieved
    bandwidth."""
    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    evox.evox_copy(a, b, n)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        evox.evox_copy(a, b, n)
    e1.record()
    torch.cuda.synchronize()
    sec = e0.elapsed_time(e1) / 1e3 / reps
    del a, b
    return 2.0 * n * 4 / sec / 1e9


def cso_data_floor(torch, evox, w, ldx, reps=5):
    """The data-movement floor of the CSO generation on this GPU: the row
    traffic of one swarm-mean generation alone (evox_pair_move: the winner
    gathers and the losers' x and v, read and written, in the generation
    kernel's traversal, with the pairs of generation 0 of the workload's
    pairing), timed like the generation kernel.  Returns its average launch
    duration and the algorithmic bytes per launch."""
    N, D = w.N, w.D
    perm = torch.empty(N, dtype=torch.int32, device="cuda")
    scratch = torch.empty(evox.lib().evox_permutation_scratch_bytes(N, 1) // 4 + 64, dtype=torch.int32, device="cuda")
    evox.evox_permutation(w.seed, 0, 1, N, perm, scratch)
    p = perm.long()
    pairs = N // 2
    winner_of = torch.full((N,), -1, dtype=torch.int32, device="cuda")
    winner_of[p[1::2][:pairs]] = p[0::2][:pairs].int()
    x = torch.zeros((N, ldx), dtype=torch.float32, device="cuda")
    v = torch.zeros_like(x)
    evox.evox_pair_move(x, v, N, D, ldx, winner_of)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        evox.evox_pair_move(x, v, N, D, ldx, winner_of)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / reps * 1e3
    del x, v, winner_of, perm, scratch
    torch.cuda.empty_cache()
    # rows: gather x_w, read x_l and v_l, write x_l and v_l; winner_of: 4 B per individual
    return us, 20.0 * pairs * D + 4.0 * N


def pso_data_floor(torch, evox, w, ldx, reps=5):
    """The data-movement floor of the PSO generation on this GPU: its 20 B per
    element (read x, v, pbest; write x, v) streamed alone by evox_pso_stream
    over arrays of the swarm's N x ldx floats, timed like the generation
    kernel.  Returns its average launch duration and the algorithmic bytes
    per launch (20 B per element of the N x D swarm)."""
    n = w.N * ldx
    x = torch.zeros(n, dtype=torch.float32, device="cuda")
    v = torch.zeros_like(x)
    p = torch.zeros_like(x)
    evox.evox_pso_stream(x, v, p, n)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        evox.evox_pso_stream(x, v, p, n)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / reps * 1e3
    del x, v, p
    torch.cuda.empty_cache()
    return us, 20.0 * w.N * w.D


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="time only the chosen workload, not the rest of the benchmark set")
    ap.add_argument("--ldx", type=int, default=0,
                    help="row pitch in floats (default: D rounded up to a multiple of 4)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run a plain device copy of this size (HBM-counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}): this implementation has no "
              "multi-GPU path", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2301_12457_amd as evox

    torch.cuda.set_device(0)
    w = WORKLOADS[args.workload]
    head = measure(torch, evox, w, args.steps, args.warmup, args.ldx or None)
    ms, roofline = head["ms_per_step"], head["roofline"]

    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b
    copy = copy_bandwidth(torch, evox)
    if roofline is not None and roofline["bound"] == "hbm":
        roofline["copy_gbs"] = round(copy, 1)
        roofline["frac_of_copy"] = round(roofline["achieved"] / copy, 4)

    # the other workloads of the benchmark set, timed in the same run
    configs = []
    if not args.no_configs:
        for name in CONFIG_WORKLOADS:
            if name == w.name:
                continue
            wc = WORKLOADS[name]
            r = measure(torch, evox, wc, 5, 1, None)
            if r["roofline"] is not None and r["roofline"]["bound"] == "hbm":
                r["roofline"]["frac_of_copy"] = round(r["roofline"]["achieved"] / copy, 4)
            configs.append(r)
            print(f"[bench] {name}: {r['ms_per_step']:.3f} ms/step", file=sys.stderr, flush=True)

    base = None
    if not args.no_cpu_baseline:
        base = cpu_baseline(w)
        print(f"[bench] cpu baseline: {base}", file=sys.stderr, flush=True)

    line = {
        "metric": METRIC, "value": head["value"], "unit": UNIT, "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "ms_per_step_median": head["ms_per_step_median"],
        "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": head["config"], "roofline": roofline, "cpu_baseline": base, "configs": configs,
    }
    print(json.dumps(line), flush=True)


def measure(torch, evox, w, steps, warmup, ldx):
    """Time `steps` steps of workload w after `warmup` untimed ones; the
    dominant kernel's roofline from HIP events around its launches."""
    stream = torch.cuda.current_stream()
    fn = evox.FN_IDS[w.fn] if w.algo != "nsga2" else 0   # NSGA-II: DTLZ1

    if w.algo == "eval":
        X = torch.empty((w.N, w.D), dtype=torch.float32, device="cuda")
        evox.evox_fill_normal(w.seed, w.N, w.D, w.D, w.x_mu, w.x_sigma, X)
        out = torch.empty(w.N, dtype=torch.float32, device="cuda")
        bf = torch.empty(1, dtype=torch.float32, device="cuda")
        bi = torch.empty(1, dtype=torch.int64, device="cuda")
        scratch = torch.empty(evox.evox_eval_argmin_scratch_bytes(w.N) // 4 + 64,
                              dtype=torch.int32, device="cuda")

        def step():
            evox.evox_eval_argmin(fn, X, w.N, w.D, w.D, out, bf, bi, scratch)
        swarm = None
    else:
        algo = {"pso": evox.PSO, "cso": evox.CSO, "de": evox.DE, "es": evox.ES,
                "pgpe": evox.PGPE, "maes": evox.MAES, "nsga2": evox.NSGA2}[w.algo]
        P = evox.make_params(algo, fn, w.N, w.D, w.lb, w.ub, v_lo=w.v_lo, v_hi=w.v_hi, w=w.w,
                             c1=w.c1, c2=w.c2, phi=w.phi, vmax=w.vmax, seed=w.seed,
                             ldx=ldx, de_f=w.de_f, de_cr=w.de_cr,
                             es_sigma=w.es_sigma, es_lr=w.es_lr, pgpe_sigma_lr=w.pgpe_sigma_lr,
                             pgpe_max_change=w.pgpe_max_change, n_obj=w.n_obj, cso_local=w.cso_local)
        swarm = evox.Swarm(P)

        def step():
            swarm.step(w.gens)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] {w.name}: warmup done", file=sys.stderr, flush=True)

    if swarm is not None:
        swarm.profile(True)
    # one event per step boundary: the total over the K steps is the
    # measurement, the per-step times give its median
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev0, ev1 = evs[0], evs[-1]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for k in range(steps):
        step()
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = ev0.elapsed_time(ev1) / steps
    ms_median = statistics.median(evs[k].elapsed_time(evs[k + 1]) for k in range(steps))
    print(f"[bench] {w.name}: timed {steps} steps: {ms:.3f} ms/step (wall {wall:.3f} s)",
          file=sys.stderr, flush=True)

    gens = w.gens if w.algo != "eval" else 1
    value = w.N * w.D * gens / (ms / 1e3)
    roofline = None
    if swarm is not None:
        fused_ms, launches, improved = swarm.profile_read()
        swarm.profile(False)
        if launches > 0 and w.algo == "nsga2":
            # the vector-ALU roofline of the all-pairs dominance count
            avg_ms = fused_ms / launches
            ops = nsga2_count_ops(w)
            achieved = ops / (avg_ms / 1e3) / 1e12
            roofline = {"bound": "alu", "achieved": round(achieved, 2), "peak": ALU_PEAK_TOPS,
                        "unit": "Tops/s", "frac": round(achieved / ALU_PEAK_TOPS, 4), "traffic": None,
                        "kernel": "k_nsga_count (dominators of 2N points)",
                        "avg_launch_us": round(avg_ms * 1e3, 2), "launches": launches,
                        "algorithmic_ops_per_launch": ops,
                        "generation_us": round(ms / 1e3 / w.gens * 1e6, 2)}
        elif launches > 0 and w.algo == "maes":
            # the matrix-core roofline of the sampling product (the timed
            # launch: k_gemm_nt and its split-K reduction)
            avg_ms = fused_ms / launches
            f_sample, f_update = maes_flops(w)
            achieved = f_sample / (avg_ms / 1e3) / 1e12
            gen_s = ms / 1e3 / w.gens
            roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": MFMA_F32_PEAK_TFLOPS,
                        "unit": "TFLOP/s", "frac": round(achieved / MFMA_F32_PEAK_TFLOPS, 4),
                        "traffic": None, "kernel": gemm_nt_label(w.N + 1) + " + k_splitk_reduce (Z M^T)",
                        "avg_launch_us": round(avg_ms * 1e3, 2), "launches": launches,
                        "algorithmic_flops_per_launch": f_sample,
                        "generation_us": round(gen_s * 1e6, 2),
                        "generation_tflops": round((f_sample + f_update) / gen_s / 1e12, 2)}
        elif launches > 0 and w.algo in ("es", "pgpe"):
            # the ALU roofline of the whole generation (samples, ranks,
            # gradient, step), timed over the step
            gen_s = ms / 1e3 / w.gens
            ops = (ES_OPS_PER_ELEMENT if w.algo == "es" else PGPE_OPS_PER_ELEMENT) * (w.N // 2) * w.D
            achieved = ops / gen_s / 1e12
            roofline = {"bound": "alu", "achieved": round(achieved, 2), "peak": ALU_PEAK_TOPS,
                        "unit": "Tops/s", "frac": round(achieved / ALU_PEAK_TOPS, 4),
                        "traffic": None, "kernel": "k_es_eval_s + k_es_rank + k_es_grad + k_es_update",
                        "sample_kernel_avg_us": round(fused_ms / launches * 1e3, 2),
                        "generation_us": round(gen_s * 1e6, 2), "launches": launches,
                        "algorithmic_ops_per_generation": ops}
        elif launches > 0:
            # per generation of the timed launches (a fused launch is one
            # generation; a small swarm's one-block launch is a whole step)
            avg_ms = fused_ms / launches
            bytes_per = {"pso": lambda: pso_bytes_per_generation(w, steps * w.gens, improved),
                         "cso": lambda: cso_bytes_per_launch(w),
                         "de": lambda: de_bytes_per_launch(w)}[w.algo]()
            achieved = bytes_per / (avg_ms / 1e3) / 1e9
            kname = {"pso": "k_pso_fused", "cso": "k_cso", "de": "k_de"}[w.algo]
            traffic = traffic_from_profile(w.name)
            roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                        "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                        "traffic": traffic, "kernel": kname,
                        "avg_launch_us": round(avg_ms * 1e3, 2), "launches": launches,
                        "algorithmic_bytes_per_launch": bytes_per}
            if w.algo == "pso":
                # the 20 B per element floor alone (read x, v, pbest; write
                # x, v), without the rows whose personal best improved
                floor_bytes = 20.0 * w.N * w.D
                roofline["frac_floor_20B"] = round(floor_bytes / (avg_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4)
                roofline["improved_rows_per_generation"] = round(improved / (steps * w.gens), 1)
                if launches == steps * w.gens:
                    # the one-block kernel: one launch per step, the figures
                    # above are per generation
                    roofline["kernel"] = "k_pso_small (one block, a whole step per launch)"
                    roofline["avg_launch_us"] = round(fused_ms / steps * 1e3, 2)
                    roofline["launches"] = steps
                    roofline["generation_us"] = round(avg_ms * 1e3, 3)
    else:
        bytes_per = 4.0 * w.N * w.D + 4.0 * w.N
        achieved = bytes_per / (ms / 1e3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "traffic": traffic_from_profile(w.name), "kernel": "k_eval",
                    "avg_launch_us": round(ms * 1e3, 2), "launches": steps,
                    "algorithmic_bytes_per_launch": bytes_per}
    if roofline is not None and w.algo == "pso" and roofline["kernel"] == "k_pso_fused":
        f_us, f_bytes = pso_data_floor(torch, evox, w, swarm.P.ldx)
        floor_gbs = f_bytes / (f_us / 1e6) / 1e9
        roofline["data_floor"] = {"kernel": "k_pso_stream (evox_pso_stream)", "avg_launch_us": round(f_us, 2),
                                  "algorithmic_bytes_per_launch": f_bytes,
                                  "frac": round(floor_gbs / HBM_PEAK_GBS, 4),
                                  "achieved_over_floor": round(roofline["achieved"] / floor_gbs, 4)}
    if roofline is not None and w.algo == "cso" and not w.cso_local:
        f_us, f_bytes = cso_data_floor(torch, evox, w, swarm.P.ldx)
        roofline["data_floor"] = {"kernel": "k_pair_move (evox_pair_move)", "avg_launch_us": round(f_us, 2),
                                  "algorithmic_bytes_per_launch": f_bytes,
                                  "frac": round(f_bytes / (f_us / 1e6) / 1e9 / HBM_PEAK_GBS, 4),
                                  "kernel_over_floor": round(roofline["avg_launch_us"] / f_us, 4)}
    config = {"workload": w.name, "algo": w.algo, "fn": w.fn, "N": w.N, "D": w.D,
              "ldx": (swarm.P.ldx if swarm is not None else w.D), "generations_per_step": gens, "seed": w.seed}
    result = {"workload": w.name, "value": value, "unit": UNIT, "ms_per_step": ms, "ms_per_step_median": ms_median,
              "steps": steps,
              "warmup": warmup, "ms_per_generation": ms / gens, "config": config, "roofline": roofline}
    del swarm
    torch.cuda.empty_cache()
    return result


if __name__ == "__main__":
    main()
