/*
 * evox.h -- C ABI of the MI355X (gfx950) population-optimizer hot path.
 *
 * EvoX (arXiv 2301.12457) states an evolutionary algorithm as a stream of
 * state transitions (Sec. IV-B, Eq. (1)-(3)):
 *     T_pop, S = ask(S);   T_fit, S = evaluate(S, T_pop);   S = tell(S, T_fit)
 * with the stateful signature (state, ...) -> (result, state) and the
 * Algorithm / Problem / Workflow modules of Table I (setup, ask, tell,
 * evaluate, init, step).  This library implements that loop over an fp32
 * population matrix X[N, D] for:
 *   - PSO (global-best, inertia weight; the PSO of the single-objective
 *     experiment, Sec. VII-A-1),
 *   - CSO, the competitive swarm optimizer listed in Table II (with the
 *     swarm mean, or the ring-neighbourhood mean),
 *   - DE/rand/1/bin, OpenES, PGPE, CMA-ES in its matrix-adaptation form
 *     (MA-ES) and NSGA-II on DTLZ1 (Table II; Sec. VII-A and VII-B),
 * on six benchmark functions (Sphere, the function of Sec. VII-A-1, and the
 * textbook Ackley, Rastrigin, Griewank, Rosenbrock and Schwefel).
 *
 * Everything runs in hand-written HIP kernels; every call enqueues work on the
 * caller's HIP stream and returns without waiting, except evox_best and
 * evox_profile_read, which synchronize that stream.
 *
 * Ownership: every device buffer is allocated by the caller and only borrowed
 * by the library.  The library allocates no device memory (its one device
 * array, the 32 KiB slots of evox_eval_argmin_noalloc, is static);
 * evox_state_create allocates one host-side handle, freed by
 * evox_state_destroy.
 *
 * Errors: every int-returning call returns EVOX_OK (0) or a negative
 * evox_status.  A call that fails validation enqueues nothing and leaves the
 * state unchanged.  evox_last_error() gives a message for the calling thread's
 * last failure.  Kernel faults are asynchronous and surface at the next
 * synchronizing call as EVOX_EHIP.
 *
 * Random numbers: Philox4x32-10 (Salmon et al., SC'11) keyed by the 64-bit
 * seed (key = (low word, high word)).  Draw k of K for element (i, j) at
 * generation t in stream s is word (j mod 4) of
 *     Philox(seed, counter = (K * floor(j / 4) + k, i, t, s)),
 * mapped to [0, 1) as (word >> 8) * 2^-24.  Streams: 0 initial positions,
 * 1 initial velocities, 2 PSO (K = 2: r1, r2), 3 CSO (K = 3: R1, R2, R3, row i
 * = the loser), 4 CSO pairing keys (key of individual i = word (i mod 4) of
 * Philox(seed, (floor(i / 4), 0, t, 4))).
 */
#ifndef EVOX_H
#define EVOX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Benchmark functions (Problem.evaluate).  F(x) for x in R^D:
 *   SPHERE      sum x_i^2
 *   ACKLEY      -20 exp(-0.2 sqrt(mean x_i^2)) - exp(mean cos(2 pi x_i)) + 20 + e
 *   RASTRIGIN   10 D + sum (x_i^2 - 10 cos(2 pi x_i)) = sum (x_i^2 + 20 sin^2(pi x_i)), evaluated
 *               in the second form (non-negative terms: relative accuracy at every x)
 *   GRIEWANK    1 + sum x_i^2 / 4000 - prod cos(x_i / sqrt(i)),  i = 1..D
 *   ROSENBROCK  sum_{i<D} 100 (x_{i+1} - x_i^2)^2 + (1 - x_i)^2
 *   SCHWEFEL    418.9829 D - sum x_i sin(sqrt(|x_i|))                        */
enum evox_fn {
    EVOX_SPHERE = 0,
    EVOX_ACKLEY = 1,
    EVOX_RASTRIGIN = 2,
    EVOX_GRIEWANK = 3,
    EVOX_ROSENBROCK = 4,
    EVOX_SCHWEFEL = 5
};

enum evox_algo { EVOX_PSO = 0, EVOX_CSO = 1, EVOX_DE = 2, EVOX_ES = 3, EVOX_PGPE = 4, EVOX_MAES = 5,
                 EVOX_NSGA2 = 6 };

enum evox_status {
    EVOX_OK = 0,
    EVOX_EINVAL = -1, /* bad argument: size, null pointer, unknown id, wrong algorithm */
    EVOX_EHIP = -2,   /* HIP runtime or launch error */
    EVOX_ENOSPC = -3, /* scratch buffer smaller than evox_scratch_bytes() */
    EVOX_EALIGN = -4  /* a device pointer or row pitch is not 16-byte aligned */
};

/* Largest dimension D supported by the generation kernels. */
#define EVOX_MAX_D 32768

/* Immutable hyperparameters (theta of Sec. IV-B), fixed at creation. */
typedef struct evox_params {
    int32_t algo;     /* EVOX_PSO, EVOX_CSO, EVOX_DE, EVOX_ES (OpenES), EVOX_PGPE, EVOX_MAES
                         (CMA-ES as matrix adaptation) or EVOX_NSGA2 (on DTLZ1) */
    int32_t fn_id;    /* enum evox_fn (NSGA2: ignored, the problem is DTLZ1) */
    int64_t N;        /* population size: PSO 1 .. 2^31 - 1, CSO 2 .. 2^24, DE 4 .. 2^31 - 1,
                         ES / PGPE even, 2 .. 16384 (N / 2 antithetic pairs), MAES 2 .. 16384,
                         NSGA2 even, 4 .. 32768 */
    int64_t D;        /* dimension, 1 .. EVOX_MAX_D */
    int64_t ldx;      /* row pitch of x, v, pbest in floats: ldx >= D, ldx % 4 == 0 */
    float lb, ub;     /* x_init 0: initial positions ~ U[lb, ub): x = fma(u, ub - lb, lb);
                         also the clamp box of clamp_x */
    float v_lo, v_hi; /* initial velocities ~ U[v_lo, v_hi); both 0 gives v = 0 */
    float w, c1, c2;  /* PSO inertia and acceleration coefficients */
    float phi;        /* CSO social factor */
    float vmax;       /* PSO velocity clamp to [-vmax, vmax]; <= 0: none */
    int32_t clamp_x;  /* nonzero: positions clamped to [lb, ub] after each move */
    int32_t x_init;   /* 0: uniform in [lb, ub); 1: normal, as evox_fill_normal(seed, x_mu,
                         x_sigma) */
    float x_mu, x_sigma;
    float de_f;       /* DE differential weight F */
    float de_cr;      /* DE crossover rate CR */
    float es_sigma;   /* ES perturbation scale sigma; PGPE initial deviation (every dimension);
                         MAES initial step size */
    float es_lr;      /* ES / PGPE center learning rate */
    float pgpe_sigma_lr;    /* PGPE deviation learning rate */
    float pgpe_max_change;  /* PGPE bound on a deviation's relative change per generation */
    uint64_t seed;    /* Philox key */
    int32_t n_obj;    /* NSGA2: objectives of DTLZ1, 2 .. 8 (D >= n_obj) */
    float sbx_eta;    /* NSGA2: distribution index of the simulated binary crossover */
    float pm_eta;     /* NSGA2: distribution index of the polynomial mutation */
    int32_t cso_local; /* CSO: 0 = losers learn from the swarm mean; 1 = from the mean of their
                          ring neighbourhood (rows i-1, i, i+1 modulo N, taken before the
                          generation moves anyone) */
} evox_params;

/* Caller-owned device buffers, borrowed by the state (row-major, pitch ldx;
 * the padding columns D..ldx-1 are kept at zero by the library).
 *   PSO: x, v, pbest [N][ldx]; pfit [N]; gbest [ldx]; fit [N] optional (the
 *        fitness of the last evaluated positions); xbar unused.
 *   CSO: x, v [N][ldx]; fit [N]; xbar [ldx] (swarm mean of x); pbest, pfit,
 *        gbest unused.  The neighbourhood version (cso_local = 1) keeps a
 *        second population buffer in the scratch and alternates between it
 *        and x inside a call; x holds the positions whenever a call returns.
 *   DE:  x [N][ldx]; fit [N] (the fitness of x); v, pbest, pfit, gbest, xbar
 *        unused (the second population buffer is part of the scratch).
 *   ES:  x [ldx] = the center theta (one row; x_init / lb / ub / seed give
 *        its first value, row 0 of the initial population); fit [N] = the
 *        fitness of the last generation's samples; the rest unused.
 *   PGPE: as ES, and v [ldx] = the per-dimension deviations sigma (es_sigma
 *        at creation, padding 0).
 *   NSGA2: x [N][ldx] = the population in [0, 1]^D (uniform at creation,
 *        lb and ub ignored), obj [N][n_obj] = its DTLZ1 objectives, front [N]
 *        = each individual's 0-based front and crowd [N] = its crowding
 *        distance within that front (of the merged population it survived);
 *        the rest unused.
 *   MAES: x [ldx] = the center y (as ES), v [ldx] = the evolution path s
 *        (zero at creation), mat [D][ldx] = the transformation matrix M
 *        (identity at creation; M M^T plays the covariance matrix), sigma [1]
 *        = the step size (es_sigma at creation), fit [N] = the last
 *        generation's sample fitness; the rest unused.
 * Every array pointer must be 16-byte aligned.  scratch must hold
 * evox_scratch_bytes(params) bytes, 256-byte aligned, and must not be used by
 * anything else while the state exists. */
typedef struct evox_buffers {
    float *x, *v, *pbest, *pfit, *fit, *gbest, *xbar;
    float *mat, *sigma;  /* MAES only */
    float *obj;          /* NSGA2 only: objectives */
    int32_t *front;      /* NSGA2 only */
    double *crowd;       /* NSGA2 only */
    void *scratch;
    size_t scratch_bytes;
} evox_buffers;

typedef struct evox_state evox_state; /* opaque host-side handle */

/* Bytes of device scratch the state needs for these parameters (0 if the
 * parameters are invalid). */
size_t evox_scratch_bytes(const evox_params *params);

/* Algorithm.setup + Workflow.init (Sec. IV-A, Table I): validates, fills the
 * buffers with the generation-0 state on `hip_stream` and returns the handle.
 *   PSO: x, v drawn as above, pbest = x, pfit = +inf, best = (+inf, 0),
 *        gbest = row 0 of pbest.
 *   CSO: x, v drawn as above, fit = F(x), xbar = column mean of x (fp64 sum,
 *        one rounding), best = argmin of fit.
 * The generation counter starts at 0. */
int evox_state_create(const evox_params *params, const evox_buffers *buffers, void *hip_stream,
                      evox_state **out);

/* Frees the host handle only; the caller's buffers are untouched. */
int evox_state_destroy(evox_state *state);

/* Problem.evaluate (Sec. IV-A): out[i] = F(X_i) for i < N over a dense
 * row-major X [N][D] (device pointer), fp32 out [N] (device pointer).  The
 * result is within 1e-5 relative of the fp64 value (relative to the
 * function's scale: see the tests).  Any alignment of X is accepted. */
int evox_eval(int fn_id, const float *X, int64_t N, int64_t D, float *out, void *hip_stream);

/* evox_eval with an explicit row pitch ldx >= D (floats). */
int evox_eval_ld(int fn_id, const float *X, int64_t N, int64_t D, int64_t ldx, float *out,
                 void *hip_stream);

/* Scratch bytes evox_eval_argmin needs for N rows. */
size_t evox_eval_argmin_scratch_bytes(int64_t N);

/* Evaluation plus selection of the best candidate: out as evox_eval_ld, and
 * (best_fit_dev[0], best_idx_dev[0]) = the lexicographic minimum of
 * (out[i], i): smaller value first, lower index on ties, -0 == +0, NaN after
 * every number (all NaN gives index 0).  best_fit_dev / best_idx_dev are
 * device pointers (float, int64); scratch is caller device memory of
 * evox_eval_argmin_scratch_bytes(N) bytes, 256-byte aligned. */
int evox_eval_argmin(int fn_id, const float *X, int64_t N, int64_t D, int64_t ldx, float *out,
                     float *best_fit_dev, int64_t *best_idx_dev, void *scratch,
                     size_t scratch_bytes, void *hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): evox_eval_argmin
 * without a scratch argument.  Its selection slots live in a device array of
 * the library (EVOX_NOALLOC_SCRATCH_BYTES, 32 KiB, one copy per device, held
 * until the process ends); the call allocates nothing (no hipMalloc, hipFree
 * or allocating library routine) and resets the slots it uses with a kernel
 * before the evaluation.  Every call on a device shares that device's array:
 * calls that overlap on one device (concurrent streams or threads) race and
 * give wrong results.  The caller's current device must be the device of
 * hip_stream (EVOX_EINVAL otherwise); N, D, ldx as evox_eval_argmin, which
 * also gives the same results bit for bit. */
#define EVOX_NOALLOC_SCRATCH_BYTES 32768
int evox_eval_argmin_noalloc(int fn_id, const float *X, int64_t N, int64_t D, int64_t ldx, float *out,
                             float *best_fit_dev, int64_t *best_idx_dev, void *hip_stream);

/* Workflow.step x n_gens for PSO (Sec. IV-A, Table I; Eq. (1)-(3)).  One
 * generation t: evaluate x (fitness f); where f_i < pfit_i strictly, pbest_i =
 * x_i and pfit_i = f_i; the global best is the minimum of pfit in the argmin
 * order above and gbest is a copy of that pbest row; then every element moves
 *     a = c1 r1;  b = c2 r2;  vn = fma(b, g - x, fma(a, p - x, w v))
 *     vn = clamp(vn, -vmax, vmax) if vmax > 0;  x = x + vn (clamped if clamp_x)
 * with r1, r2 from stream 2 at generation t.  After the call x holds the
 * moved, not yet evaluated positions, and the generation counter has grown by
 * n_gens.  step(a) then step(b) equals step(a + b) bit for bit. */
int evox_pso_step(evox_state *state, int64_t n_gens);

/* Workflow.step x n_gens (Sec. IV-A, Table I; Eq. (1)-(3)) for CSO, the
 * competitive swarm optimizer of Table II (after Cheng and Jin, whose update
 * rule the paper does not print).  One generation t: xbar is the mean of the
 * current positions; individuals are paired by a random permutation (sort by
 * (stream-4 key, index)): pairs (perm[2k], perm[2k+1]), k < floor(N/2); the
 * second wins when its fitness is strictly lower (or the first's is NaN and
 * its own is not); each loser l moves toward its winner w and the mean
 *     t0 = R1 v;  t1 = fma(R2, x_w - x_l, t0);  vn = fma(phi R3, xbar - x_l, t1)
 *     x_l = x_l + vn (clamped if clamp_x)
 * with R1..R3 from stream 3 at generation t, and only the losers are
 * re-evaluated.  Winners and an unpaired individual are untouched.  xbar is
 * then refreshed from the new positions.  With cso_local = 1 the mean of a
 * loser l is that of rows l - 1, l, l + 1 (modulo N) of the positions before
 * the generation, in fp64 rounded once. */
int evox_cso_step(evox_state *state, int64_t n_gens);

/* n_gens generations of DE/rand/1/bin (Storn & Price, J. Global Optim. 11,
 * 1997; the vanilla DE of Sec. VII-A-1) on a DE state.  Generation t, for
 * every target i, on the population of generation t:
 *   - partners r1, r2, r3, mutually distinct and distinct from i, and a
 *     crossover position j_rand, from words 0..3 of Philox(seed, (0, i, t,
 *     6)): a_k = floor(w_k (N - 1 - k) / 2^32) for k = 0, 1, 2, and r_k is
 *     the a_k-th (from 0) index not yet taken (i, r1, ...); j_rand =
 *     floor(w_3 D / 2^32);
 *   - mutant v = fma(de_f, x_r2 - x_r3, x_r1) (fp32);
 *   - binomial crossover u_j = v_j if u01(word j mod 4 of Philox(seed,
 *     (1 + floor(j/4), i, t, 6))) <= de_cr or j = j_rand, else x_ij;
 *   - the trial replaces the target when F(u) < fit_i (strictly: ties and
 *     NaN keep the target).
 * All targets of a generation see the same population (the next one is
 * written to the other buffer); when the call returns, x and fit hold the
 * population and fitness after n_gens generations, and evox_best reports the
 * best of them. */
int evox_de_step(evox_state *state, int64_t n_gens);

/* n_gens OpenES generations (Salimans et al., arXiv 1703.03864, 2017; an ES
 * of Table II) on an ES state.  Generation t:
 *   - perturbations eps_kj, pair k < N/2, element j: the Box-Muller deviates
 *     of Philox(seed, (floor(j/4), k, t, 7)) with the word layout of
 *     evox_fill_normal;
 *   - samples x_{2k} = fma(sigma, eps_k, theta), x_{2k+1} = fma(-sigma,
 *     eps_k, theta), fit_i = F(x_i) (the samples exist only in registers);
 *   - centered ranks u_i = rank_i / (N - 1) - 1/2, rank_i the position of
 *     sample i in the order of (fit_i, i) (NaN last);
 *   - g_j = sum_k (u_{2k} - u_{2k+1}) eps_kj / (N sigma) (fp64), the
 *     perturbations regenerated from Philox;
 *   - theta_j <- fma(-lr, g_j, theta_j), g_j rounded to fp32.
 * evox_best reports the best sample of the last generation (fitness, index)
 * and, as the solution, the current center theta. */
int evox_es_step(evox_state *state, int64_t n_gens);

/* n_gens PGPE generations with symmetric sampling (Sehnke et al., Neural
 * Networks 23, 2010; the ES of the paper's neuroevolution experiment,
 * Sec. VII-B) on a PGPE state.  Generation t, with H = N/2 pairs:
 *   - deviates z_kj from Philox(seed, (floor(j/4), k, t, 8)) with the
 *     Box-Muller layout of evox_fill_normal; samples x_{2k} = fma(sigma_j,
 *     z_kj, mu_j), x_{2k+1} = fma(-sigma_j, z_kj, mu_j); fit = F(x);
 *   - centered ranks u_i = rank_i / (N - 1) - 1/2 (the argmin order);
 *   - g_mu_j = sigma_j sum_k (u_{2k} - u_{2k+1}) z_kj / (2H),
 *     g_sigma_j = sigma_j sum_k (u_{2k} + u_{2k+1}) (z_kj^2 - 1) / (2H)
 *     (fp64; the baseline, the mean utility, is zero);
 *   - mu_j <- fma(-es_lr, g_mu_j, mu_j); sigma_j <- sigma_j + d_j with
 *     d_j = -pgpe_sigma_lr g_sigma_j clamped to +-pgpe_max_change sigma_j
 *     (gradients rounded to fp32 once).
 * evox_best reports the best sample of the last generation and the center
 * mu as the solution. */
int evox_pgpe_step(evox_state *state, int64_t n_gens);

/* n_gens generations of CMA-ES (Table II; Sec. VII-A-1 runs it on Sphere up to
 * D = 16384) in the matrix-adaptation form of Beyer and Sendhoff (IEEE TEVC
 * 21(5), 2017), with Hansen's default constants: mu = floor(N/2) parents,
 * weights w_i ~ ln(mu + 1/2) - ln i summing to one, mu_eff = 1 / sum w_i^2,
 * c_s = (mu_eff + 2) / (D + mu_eff + 5), d_s = 1 + c_s + 2 max(0,
 * sqrt((mu_eff - 1) / (D + 1)) - 1), c_1 = 2 / ((D + 1.3)^2 + mu_eff), c_w =
 * min(1 - c_1, 2 (mu_eff - 2 + 1/mu_eff) / ((D + 2)^2 + mu_eff)), chi_D =
 * sqrt(D) (1 - 1/(4D) + 1/(21 D^2)).  Generation t:
 *   - deviates z_kj from Philox(seed, (floor(j/4), k, t, 9)) (the Box-Muller
 *     layout of evox_fill_normal), steps d_k = M z_k (fp32 matrix-core
 *     product), samples fma(sigma, d_kj, y_j), fit = F(samples);
 *   - parents: the mu best in the argmin order;
 *   - y <- y + sigma sum w_i d_i, s <- (1 - c_s) s + sqrt(mu_eff c_s (2 - c_s))
 *     sum w_i z_i (fp64 sums, one rounding);
 *   - M <- M [I + c_1/2 (s s^T - I) + c_w/2 (sum w_i z_i z_i^T - I)],
 *     computed as (1 - (c_1 + c_w)/2) M + c_1/2 (M s) s^T + c_w/2 sum w_i d_i
 *     z_i^T (the mu + 1 terms summed in fp32 on the matrix cores, then one
 *     fused multiply-add with the rounded (1 - (c_1 + c_w)/2) M);
 *   - sigma <- sigma exp(c_s/d_s (|s| / chi_D - 1)).
 * evox_best reports the best sample of the last generation and the center y
 * as the solution. */
int evox_maes_step(evox_state *state, int64_t n_gens);

/* n_gens generations of NSGA-II (Table II; Sec. VII-A-2 runs it on DTLZ1) after
 * Deb, Pratap, Agarwal and Meyarivan (IEEE TEVC 6(2), 2002).  Generation t:
 *   - offspring pair p < N/2 from two crowded binary tournaments (candidates
 *     floor(w_q N / 2^32) for the words w_0..w_3 of Philox(seed, (0, p, t,
 *     10)); the lower front wins, then the larger crowding distance, then
 *     the lower index);
 *   - per variable j, words w of Philox(seed, (j, p, t, 11)) and v of
 *     (j, p, t, 12), u(w) = top 24 bits x 2^-24: simulated binary crossover
 *     with spread (2u)^(1/(sbx_eta+1)) for u = u(w_0) <= 1/2, else
 *     (2 - 2u)^(-1/(sbx_eta+1)), negated when w_1 is odd, 1 (no crossing)
 *     when u(w_1) >= 1/2; children (a + b)/2 +- beta (a - b)/2 clipped to
 *     [0, 1]; polynomial mutation (index pm_eta) of child q when u(w_{2+q})
 *     < 1/D with draw u(v_q); fp64, each child rounded to fp32 once;
 *   - DTLZ1 objectives of the offspring (fp64, rounded once);
 *   - non-dominated fronts and crowding distances of parents and offspring
 *     together (parents first), then the survivors: whole fronts while
 *     they fit, and from the next front its members of largest crowding
 *     distance (lower index on ties), kept in their merged order.
 * Synchronizes the stream once per front sorted.  evox_best returns
 * EVOX_EINVAL for this algorithm (there is no single best). */
int evox_nsga2_step(evox_state *state, int64_t n_gens);

/* Non-dominated sorting and crowding distances (the sorting step of
 * NSGA-II) of n points with M objectives (minimised): F (device, fp32,
 * [n][M], no NaN), front (device, int32 [n]) receives every point's 0-based
 * front, crowd (device, fp64 [n]) its crowding distance within the front
 * (per objective in order 0..M-1: +inf at either end of the front's order
 * of (value, index), else + (next - previous) / (last - first) when that
 * range is not zero).  1 <= n <= 65536, 2 <= M <= 8; scratch (device,
 * 256-byte aligned) of evox_nsga2_sort_scratch_bytes(n, M) bytes.  Returns
 * when the result is in place (the stream is synchronized once per front). */
size_t evox_nsga2_sort_scratch_bytes(int64_t n, int32_t M);
int evox_nsga2_sort(const float *F, int64_t n, int32_t M, int32_t *front, double *crowd, void *scratch,
                    size_t scratch_bytes, void *hip_stream);

/* If the caller has changed x (or fit) of a CSO state, recompute xbar from x
 * and, when refit is nonzero, fit = F(x). */
int evox_cso_refresh(evox_state *state, int refit);

/* Best solution so far (what a Monitor would record, Sec. IV-B).  Waits for
 * the state's stream.  PSO: (gf, gi) of the last evaluated generation and,
 * if best_x_host is non-null, the gbest row (D floats) copied to host memory.
 * CSO: argmin of the current fitness and that individual's row.  Before any
 * PSO generation: (+inf, 0) and row 0 of pbest. */
int evox_best(evox_state *state, float *best_fit, int64_t *best_idx, float *best_x_host);

/* Generations completed so far. */
int64_t evox_generation(const evox_state *state);

/* Resume at generation t (0 <= t < 2^32): the next step performs generation
 * t, drawing the random numbers of generation t (t is the generation index
 * in every Philox counter).  Together with buffers the caller has written
 * this restores a state saved at generation t (the state as a function of t
 * and its buffers, Sec. IV-B): for PSO, x, v, pbest and pfit (the next step
 * re-evaluates x and re-selects the global best from pfit); for CSO, x, v and
 * fit followed by evox_cso_refresh (swarm mean and best).  Enqueues nothing;
 * EVOX_EINVAL for a null state or t out of range. */
int evox_set_generation(evox_state *state, int64_t t);

/* Kernel families for evox_row_layout. */
enum evox_layout { EVOX_LAYOUT_PSO = 0, EVOX_LAYOUT_CSO = 1, EVOX_LAYOUT_EVAL = 2 };

/* Row layout the kernels of a family use for dimension D: threads per row
 * and float4 chunks per thread (for tests and reports).  The threads per row
 * are the fewest (a power of two, 4..1024) that hold the row in at most 2
 * (PSO), 1 (CSO) or 4 (evox_eval) chunks per thread, and 8 at 1024 threads. */
int evox_row_layout(int32_t kernels, int64_t D, int32_t *threads_per_row, int32_t *chunks_per_thread);

/* Normal synthetic population: X[i][j] = mu + sigma z_ij for i < N, j < D
 * (device X, [N][ldx] floats, 16-byte aligned, ldx % 4 == 0, ldx >= D;
 * columns D..ldx-1 set to 0).  z_ij is a standard normal deviate by the
 * Box-Muller transform (Box & Muller, 1958) of Philox stream 5: one call
 * Philox(seed, (floor(j/4), i, 0, 5)) per four elements; of its word pairs
 * (0, 1) and (2, 3), a pair (a, b) gives u1 = ((a >> 8) + 1) 2^-24 in (0, 1],
 * u2 = (b >> 8) 2^-24, r = sqrt(-2 ln u1), and elements r cos(2 pi u2) (even
 * j) and r sin(2 pi u2) (odd j).  Computed in fp32 with the hardware log2
 * (times -2 ln 2), square root, and cosine / sine of the exactly reduced
 * angle, so within sigma 1e-6 max(1, |z|) + 1 ulp of the exact value.
 * The initial population of an x_init = 1 state is the same matrix.  N = 0
 * does nothing. */
int evox_fill_normal(uint64_t seed, int64_t N, int64_t D, int64_t ldx, float mu, float sigma,
                     float *X, void *hip_stream);

/* The pairing permutations of CSO generations t0 .. t0 + n_gens - 1 for a
 * swarm of N individuals (1 <= N <= 2^24): perm_out[g][k] (device, uint32,
 * [n_gens][N]) is the k-th individual in the order of (key_i, i), key_i =
 * word (i mod 4) of Philox(seed, (floor(i/4), 0, t0 + g, 4)).  This is the
 * permutation an evox_cso_step of that generation pairs by ((perm[2k],
 * perm[2k+1]), Table II).  scratch (device, 256-byte aligned) holds at least
 * evox_permutation_scratch_bytes(N, 1) bytes; with room for a batch of up to
 * 8 generations, that many are sorted per launch.  Returns EVOX_ENOSPC if the
 * scratch is too small. */
size_t evox_permutation_scratch_bytes(int64_t N, int64_t batch);
int evox_permutation(uint64_t seed, int64_t t0, int64_t n_gens, int64_t N, uint32_t *perm_out,
                     void *scratch, size_t scratch_bytes, void *hip_stream);

/* The same sort on caller keys (device, uint32, N <= EVOX_ARGSORT_MAX_N):
 * perm_out[k] = the k-th index in the order of (keys[i], i), a stable
 * argsort.  Keys that share their top bits in groups of more than 4096 are
 * ranked by a quadratic pass, which is why N is bounded here.  scratch as for
 * evox_permutation(N, 1 generation). */
#define EVOX_ARGSORT_MAX_N 65536
int evox_argsort_u32(const uint32_t *keys, int64_t N, uint32_t *perm_out, void *scratch,
                     size_t scratch_bytes, void *hip_stream);

/* Recommended row pitch (ldx, in floats) of an algo's state of dimension D:
 * a multiple of 32 floats (rows start on 128-byte cache lines) where that
 * pays, else a multiple of 4.  PSO (rows streamed in order; its kernels also
 * write the padding so that row ends are whole lines): 32-multiples for
 * D >= 512, where the padding is at most ~6 %; DE, whose target rows are
 * streamed the same way, and ES / PGPE likewise.  CSO: D rounded up to a
 * multiple of 4 (dense rows: the generation writes a random half of the rows
 * in index order, and on the MI355X dense rows move faster than rows padded
 * to whole lines: 1e6 x 100 generation kernel 242 against 252 us).
 * Returns the pitch, or 0 for an unknown algo or D outside [1, EVOX_MAX_D]. */
int64_t evox_default_ldx(int32_t algo, int64_t D);

/* Dense fp32 product on the matrix cores, the contraction of the matrix-
 * adaptation ES (evox_mae_step): C = alpha op(A) op(B) + beta C with op(A)
 * M x K and op(B) K x N, row-major device matrices (op(X) = X^T when trans_x:
 * A is then stored K x M, B N x K), leading dimensions multiples of 4 and at
 * least the stored row lengths, 16-byte aligned pointers.  Accumulation in
 * fp32 (v_mfma_f32_32x32x2f32) in a fixed order, so results are reproducible;
 * beta = 0 ignores C's old contents.  M or N = 0 does nothing. */
int evox_sgemm(int32_t trans_a, int32_t trans_b, int64_t M, int64_t N, int64_t K, float alpha,
               const float *A, int64_t lda, const float *B, int64_t ldb, float beta, float *C,
               int64_t ldc, void *hip_stream);

/* Diagnostic, the bandwidth reference of the benchmark: dst[i] = src[i] for
 * i < n (device pointers, 16-byte aligned, not overlapping), streamed with
 * nontemporal 16-byte loads and stores.  n = 0 does nothing. */
int evox_copy(const float *src, float *dst, int64_t n, void *hip_stream);

/* Diagnostic, the data-movement floor of the CSO generation: the row traffic
 * of one swarm-mean generation (Table II's CSO as evox_cso_step runs it) and
 * nothing else.  For every i < N with winner_of[i] >= 0 (a loser; winner_of
 * device int32 [N], each winner index < N, every index the winner of at most
 * one loser and no loser a winner), in the generation kernel's traversal (row
 * groups of the CSO layout of D, losers in index order): the winner's row is
 * gathered, the loser's x and v are read, and v_i = v_i + (x_w - x_i), x_i =
 * x_i + v_i are written (device x, v [N][ldx], 16-byte aligned, ldx % 4 == 0,
 * padding columns zero).  No random numbers, fitness or swarm mean.  With the
 * pairs of a real generation it times the accesses the generation kernel
 * cannot avoid. */
int evox_pair_move(float *x, float *v, int64_t N, int64_t D, int64_t ldx, const int32_t *winner_of,
                   void *hip_stream);

/* Diagnostic, the data-movement floor of the PSO generation: its 20 bytes
 * per element (read x, v, pbest; write x, v; Sec. IV-B, Eq. (1)-(3) as
 * evox_pso_step runs them) streamed with nothing else: for every q < n,
 * v[q] = v[q] + (p[q] - x[q]), then x[q] = x[q] + v[q] (device x, v, p of n
 * floats each, 16-byte aligned, n a multiple of 4; pass N * ldx for a swarm).
 * One 16-byte element per thread with nontemporal loads and stores, the shape
 * that streams fastest on gfx950.  No random numbers, fitness or selection.
 * n = 0 does nothing. */
int evox_pso_stream(float *x, float *v, const float *p, int64_t n, void *hip_stream);

/* Diagnostic: out[4 k + m] = word m of Philox(seed, (k, c1, c2, c3)) for
 * k < n_ctr, computed by the device Philox the kernels use (device out). */
int evox_philox_fill(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t n_ctr,
                     uint32_t *out_dev, void *hip_stream);

/* Timing of the generation kernels with HIP events on the state's stream.
 * evox_profile(state, 1) starts recording (clears the totals), 0 stops.
 * evox_profile_read waits for the stream and returns the summed duration of
 * the timed generation-kernel launches, the number of generations those
 * launches performed (one per fused launch; a small PSO swarm, N D <= 16384,
 * runs a whole call in one launch), and the number of rows whose personal
 * best improved in every evaluation since profiling started (PSO). */
int evox_profile(evox_state *state, int enable);
int evox_profile_read(evox_state *state, double *fused_ms, int64_t *fused_launches,
                      int64_t *improved_rows);

const char *evox_strerror(int code);
const char *evox_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* EVOX_H */
