/*
 * evox_ref_mt.c -- the all-core CPU baseline: the oracle's PSO, CSO and
 * evaluation steps with their per-row work split over POSIX threads.
 *
 * BENCHMARK AND TEST INFRASTRUCTURE ONLY, like the oracle it is built from:
 * only tests/ and the cpu_baseline leg of bench.py load it.  The paper's CPU
 * runs used every thread of the host (Sec. VII-A-1); this is that
 * comparison for the oracle's arithmetic.
 *
 * It compiles the oracle itself (evox_ref.c is included, not copied) and
 * calls its own per-row and per-element routines, so every value is
 * computed exactly as the single-threaded oracle computes it; only the
 * loops over rows (and over the columns of the swarm mean, each summed in
 * the oracle's row order) run in parallel.  The results are bit-identical
 * to the oracle's (tests/test_oracle_mt.py).  Serial parts: the argmin, the
 * pairing permutation (the oracle's sort) and the gbest row copy.
 */
#include <pthread.h>

#include "evox_ref.c"

typedef void (*range_fn)(void *ctx, int64_t lo, int64_t hi);

typedef struct {
    range_fn fn;
    void *ctx;
    int64_t lo, hi;
} mt_job;

static void *mt_run(void *arg)
{
    mt_job *j = (mt_job *)arg;
    j->fn(j->ctx, j->lo, j->hi);
    return NULL;
}

/* fn over [0, n) in `threads` contiguous ranges, the last on the caller. */
static int parallel_for(int64_t n, int threads, range_fn fn, void *ctx)
{
    if (threads < 1) threads = 1;
    if (threads > 1024) threads = 1024;
    if ((int64_t)threads > n) threads = n > 0 ? (int)n : 1;
    mt_job jobs[1024];
    pthread_t tid[1024];
    for (int k = 0; k < threads; ++k) {
        jobs[k].fn = fn;
        jobs[k].ctx = ctx;
        jobs[k].lo = n * k / threads;
        jobs[k].hi = n * (k + 1) / threads;
    }
    int started = 0;
    for (int k = 0; k + 1 < threads; ++k) {
        if (pthread_create(&tid[k], NULL, mt_run, &jobs[k]) != 0) break;
        ++started;
    }
    for (int k = started; k < threads; ++k) mt_run(&jobs[k]);  /* what did not start runs here */
    for (int k = 0; k < started; ++k) pthread_join(tid[k], NULL);
    return 0;
}

/* ---- evaluation ---------------------------------------------------------- */

typedef struct {
    int fn;
    const float *X;
    int64_t D, ldx;
    float *out;
} eval_ctx;

static void eval_rows(void *c, int64_t lo, int64_t hi)
{
    eval_ctx *e = (eval_ctx *)c;
    for (int64_t i = lo; i < hi; ++i) e->out[i] = (float)evox_ref_eval_row_f64(e->fn, e->X + i * e->ldx, e->D);
}

int evox_mt_eval(int fn, const float *X, int64_t N, int64_t D, int64_t ldx, float *out, int threads)
{
    if (fn < 0 || fn >= FN_COUNT || N < 0 || D < 1 || ldx < D) return -1;
    eval_ctx e = {fn, X, D, ldx, out};
    return parallel_for(N, threads, eval_rows, &e);
}

/* ---- PSO ------------------------------------------------------------------ */

typedef struct {
    const evox_ref_params *P;
    int64_t t;
    float *x, *v, *p, *pf;
    const float *g;
} pso_ctx;

static void pso_eval_rows(void *c, int64_t lo, int64_t hi)
{
    pso_ctx *s = (pso_ctx *)c;
    const int64_t D = s->P->D;
    for (int64_t i = lo; i < hi; ++i) {
        float f = (float)evox_ref_eval_row_f64(s->P->fn, s->x + i * D, D);
        if (f < s->pf[i]) {
            s->pf[i] = f;
            memcpy(s->p + i * D, s->x + i * D, sizeof(float) * (size_t)D);
        }
    }
}

static void pso_move_rows(void *c, int64_t lo, int64_t hi)
{
    pso_ctx *s = (pso_ctx *)c;
    const evox_ref_params *P = s->P;
    const int64_t D = P->D;
    for (int64_t i = lo; i < hi; ++i)
        for (int64_t j = 0; j < D; ++j) {
            float r1 = draw(P->seed, i, j, 2, 0, s->t, STREAM_PSO);
            float r2 = draw(P->seed, i, j, 2, 1, s->t, STREAM_PSO);
            int64_t e = i * D + j;
            pso_move_element(P, r1, r2, s->x[e], s->v[e], s->p[e], s->g[j], &s->x[e], &s->v[e]);
        }
}

/* evox_ref_pso_step with the evaluation / personal-best pass and the move
 * split over rows. */
int evox_mt_pso_step(const evox_ref_params *P, int64_t t0, int64_t n_gens, float *x, float *v, float *p,
                     float *pf, float *g, float *gf, int64_t *gi, int threads)
{
    const int64_t N = P->N, D = P->D;
    if (N < 1 || D < 1 || n_gens < 0 || P->fn < 0 || P->fn >= FN_COUNT) return -1;
    pso_ctx s = {P, 0, x, v, p, pf, g};
    for (int64_t t = t0; t < t0 + n_gens; ++t) {
        s.t = t;
        parallel_for(N, threads, pso_eval_rows, &s);
        *gi = evox_ref_argmin(pf, N);
        *gf = pf[*gi];
        memcpy(g, p + *gi * D, sizeof(float) * (size_t)D);
        parallel_for(N, threads, pso_move_rows, &s);
    }
    return 0;
}

/* ---- CSO ------------------------------------------------------------------ */

typedef struct {
    const evox_ref_params *P;
    int64_t t;
    float *x, *v, *fit, *xbar;
    const int64_t *perm;
    uint8_t *is_loser;
} cso_ctx;

/* The swarm mean, columns split over threads; each column summed in row
 * order exactly as evox_ref_colmean does. */
static void cso_mean_cols(void *c, int64_t lo, int64_t hi)
{
    cso_ctx *s = (cso_ctx *)c;
    const int64_t N = s->P->N, D = s->P->D;
    for (int64_t j = lo; j < hi; ++j) {
        double sum = 0.0;
        for (int64_t i = 0; i < N; ++i) sum += (double)s->x[i * D + j];
        s->xbar[j] = (float)(sum / (double)N);
    }
}

static void cso_ring_rows(void *c, int64_t lo, int64_t hi)
{
    cso_ctx *s = (cso_ctx *)c;
    const int64_t N = s->P->N, D = s->P->D;
    for (int64_t i = lo; i < hi; ++i) {
        const int64_t a = (i + N - 1) % N, b = (i + 1) % N;
        for (int64_t j = 0; j < D; ++j)
            s->xbar[i * D + j] =
                (float)((((double)s->x[a * D + j] + (double)s->x[i * D + j]) + (double)s->x[b * D + j]) / 3.0);
    }
}

static void cso_pairs(void *c, int64_t lo, int64_t hi)
{
    cso_ctx *s = (cso_ctx *)c;
    const evox_ref_params *P = s->P;
    for (int64_t k = lo; k < hi; ++k) {
        int64_t a = s->perm[2 * k], b = s->perm[2 * k + 1];
        int64_t w = a, l = b;
        if (second_wins(s->fit[a], s->fit[b])) {
            w = b;
            l = a;
        }
        s->is_loser[l] = 1;
        cso_move_loser(P, s->t, l, w, s->x, s->v, s->xbar + (P->cso_local ? l * P->D : 0));
    }
}

static void cso_refit_rows(void *c, int64_t lo, int64_t hi)
{
    cso_ctx *s = (cso_ctx *)c;
    const int64_t D = s->P->D;
    for (int64_t i = lo; i < hi; ++i)
        if (s->is_loser[i]) s->fit[i] = (float)evox_ref_eval_row_f64(s->P->fn, s->x + i * D, D);
}

/* evox_ref_cso_step with the mean, the pairs' moves and the losers'
 * re-evaluation split over threads (pairs touch distinct rows, winners are
 * only read). */
int evox_mt_cso_step(const evox_ref_params *P, int64_t t0, int64_t n_gens, float *x, float *v, float *fit,
                     float *best_fit, int64_t *best_idx, int threads)
{
    const int64_t N = P->N, D = P->D;
    if (N < 1 || D < 1 || n_gens < 0 || P->fn < 0 || P->fn >= FN_COUNT) return -1;
    float *xbar = (float *)malloc(sizeof(float) * (size_t)(P->cso_local ? N * D : D));
    int64_t *perm = (int64_t *)malloc(sizeof(int64_t) * (size_t)N);
    uint8_t *is_loser = (uint8_t *)calloc((size_t)N, 1);
    cso_ctx s = {P, 0, x, v, fit, xbar, perm, is_loser};
    for (int64_t t = t0; t < t0 + n_gens; ++t) {
        s.t = t;
        if (P->cso_local)
            parallel_for(N, threads, cso_ring_rows, &s);
        else
            parallel_for(D, threads, cso_mean_cols, &s);
        evox_ref_perm(P->seed, t, N, perm);
        memset(is_loser, 0, (size_t)N);
        parallel_for(N / 2, threads, cso_pairs, &s);
        parallel_for(N, threads, cso_refit_rows, &s);
    }
    int64_t bi = evox_ref_argmin(fit, N);
    *best_idx = bi;
    *best_fit = fit[bi];
    free(xbar);
    free(perm);
    free(is_loser);
    return 0;
}
