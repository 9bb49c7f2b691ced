/*
 * evox_ref.c -- the CPU oracle for one generation of PSO / CSO over a
 * population matrix X[N,D] (EvoX, arXiv 2301.12457).
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
 * cpu_baseline leg of bench.py may load this library.  The product path
 * (the HIP library) never calls it and shares no code, header, table or
 * constant generator with it.
 *
 * Plain, slow, single-threaded C.  Everything follows the algorithm step by
 * step in the order of the ask-evaluate-tell loop (Sec. IV-B, Eq. (1)-(3)):
 * ask = produce the population to evaluate, evaluate = fitness per candidate,
 * tell = selection / state update.  The paper prints no update rules and no
 * benchmark formulas; the readings used here are:
 *
 *   - PSO: global-best PSO with inertia weight (the PSO of Sec. VII-A-1,
 *     Kennedy & Eberhart as cited there).  Per element
 *         v <- w v + c1 r1 (p - x) + c2 r2 (g - x),   x <- x + v
 *     with r1, r2 ~ U[0,1) drawn per element.  The population state is fp32;
 *     the element update is done in fp32 with fused multiply-adds placed
 *     exactly as in pso_move_element() below.
 *   - CSO: the competitive swarm optimizer listed in Table II (Cheng & Jin):
 *     random pairs, the loser learns from the winner and the swarm mean.
 *   - Benchmark functions: textbook definitions, evaluated in fp64 from the
 *     fp32 inputs, sequential sum in index order, rounded once to fp32.
 *   - Random numbers: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel
 *     random numbers: as easy as 1, 2, 3", SC'11), written from its
 *     published definition.  The paper itself names only JAX's rbg
 *     generator (Sec. VII); the counter layout below is chosen here (the paper fixes none).
 *
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared (no fast-math): every float
 * operation is one IEEE rounding, fma only where fmaf() is written.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (SC'11 paper, Sec. "Philox").                               */
/* ------------------------------------------------------------------------ */

/* Round multipliers and Weyl key increments, as published. */
#define PHILOX_M4x32_0 0xD2511F53u
#define PHILOX_M4x32_1 0xCD9E8D57u
#define PHILOX_W32_0 0x9E3779B9u
#define PHILOX_W32_1 0xBB67AE85u

void evox_ref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += PHILOX_W32_0;
            k1 += PHILOX_W32_1;
        }
        uint64_t p0 = (uint64_t)PHILOX_M4x32_0 * (uint64_t)x0;
        uint64_t p1 = (uint64_t)PHILOX_M4x32_1 * (uint64_t)x2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t y0 = hi1 ^ x1 ^ k0;
        uint32_t y1 = lo1;
        uint32_t y2 = hi0 ^ x3 ^ k1;
        uint32_t y3 = lo0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* One 32-bit word of Philox(key = seed, counter = (c0, c1, c2, c3)). */
uint32_t evox_ref_philox_word(uint64_t seed, uint32_t c0, uint32_t c1, uint32_t c2,
                              uint32_t c3, int word)
{
    uint32_t ctr[4] = {c0, c1, c2, c3};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t out[4];
    evox_ref_philox4x32_10(ctr, key, out);
    return out[word & 3];
}

/* u32 -> U[0,1): the top 24 bits, times 2^-24.  Exact in fp32. */
float evox_ref_u01(uint32_t w)
{
    return (float)(w >> 8) * 0x1p-24f;
}

/* Elementwise u01 over an array of words. */
void evox_ref_u01_array(const uint32_t *w, int64_t n, float *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = evox_ref_u01(w[i]);
}

/* Random-stream identifiers (the counter's fourth word). */
enum { STREAM_INIT_X = 0, STREAM_INIT_V = 1, STREAM_PSO = 2, STREAM_CSO = 3,
       STREAM_PERM = 4, STREAM_INIT_NORMAL = 5, STREAM_DE = 6, STREAM_ES = 7, STREAM_PGPE = 8,
       STREAM_MAES = 9, STREAM_NSGA_SEL = 10, STREAM_NSGA_VAR = 11, STREAM_NSGA_MUT = 12 };

/* Draw k of K for element (i, j) at generation t in stream s:
 * word (j mod 4) of Philox(seed, (K*floor(j/4) + k, i, t, s)). */
static float draw(uint64_t seed, int64_t i, int64_t j, int K, int k, int64_t t, int s)
{
    uint32_t c0 = (uint32_t)(K * (j / 4) + k);
    return evox_ref_u01(evox_ref_philox_word(seed, c0, (uint32_t)i, (uint32_t)t,
                                             (uint32_t)s, (int)(j % 4)));
}

/* ------------------------------------------------------------------------ */
/* Benchmark functions (Problem.evaluate, Sec. IV-A, Table I).  Sphere is   */
/* the function of Sec. VII-A-1; the others are the usual textbook ones.    */
/* fp64 throughout, sum in index order.                                      */
/* ------------------------------------------------------------------------ */

enum { FN_SPHERE = 0, FN_ACKLEY, FN_RASTRIGIN, FN_GRIEWANK, FN_ROSENBROCK, FN_SCHWEFEL,
       FN_COUNT };

static const double kPi = 3.14159265358979323846;

/* sum_i x_i^2 */
static double sphere(const float *x, int64_t D)
{
    double s = 0.0;
    for (int64_t i = 0; i < D; ++i) {
        double xi = x[i];
        s += xi * xi;
    }
    return s;
}

/* -a exp(-b sqrt(mean x^2)) - exp(mean cos(c x)) + a + e, a=20, b=0.2, c=2 pi */
static double ackley(const float *x, int64_t D)
{
    const double a = 20.0, b = 0.2, c = 2.0 * kPi;
    double s1 = 0.0, s2 = 0.0;
    for (int64_t i = 0; i < D; ++i) {
        double xi = x[i];
        s1 += xi * xi;
        s2 += cos(c * xi);
    }
    double n = (double)D;
    return -a * exp(-b * sqrt(s1 / n)) - exp(s2 / n) + a + exp(1.0);
}

/* A D + sum_i (x_i^2 - A cos(2 pi x_i)), A = 10, written term by term as
 * sum_i (x_i^2 + 2 A sin^2(pi x_i)) (1 - cos 2u = 2 sin^2 u): every term is
 * non-negative, so the sum has no cancellation.  sin(pi x_i) is taken of the
 * exactly reduced x_i - rint(x_i) (same square for any integer shift). */
static double rastrigin(const float *x, int64_t D)
{
    const double A = 10.0;
    double s = 0.0;
    for (int64_t i = 0; i < D; ++i) {
        double xi = x[i];
        double si = sin(kPi * (xi - rint(xi)));
        s += xi * xi + 2.0 * A * si * si;
    }
    return s;
}

/* 1 + sum_i x_i^2 / 4000 - prod_i cos(x_i / sqrt(i)), i = 1..D */
static double griewank(const float *x, int64_t D)
{
    double s = 0.0, p = 1.0;
    for (int64_t i = 0; i < D; ++i) {
        double xi = x[i];
        s += xi * xi / 4000.0;
        p *= cos(xi / sqrt((double)(i + 1)));
    }
    return 1.0 + s - p;
}

/* sum_{i=1}^{D-1} 100 (x_{i+1} - x_i^2)^2 + (1 - x_i)^2 */
static double rosenbrock(const float *x, int64_t D)
{
    double s = 0.0;
    for (int64_t i = 0; i + 1 < D; ++i) {
        double xi = x[i], xn = x[i + 1];
        double t1 = xn - xi * xi;
        double t2 = 1.0 - xi;
        s += 100.0 * t1 * t1 + t2 * t2;
    }
    return s;
}

/* 418.9829 D - sum_i x_i sin(sqrt(|x_i|)) */
static double schwefel(const float *x, int64_t D)
{
    double s = 0.0;
    for (int64_t i = 0; i < D; ++i) {
        double xi = x[i];
        s += xi * sin(sqrt(fabs(xi)));
    }
    return 418.9829 * (double)D - s;
}

/* Unrounded fp64 fitness of one row. */
double evox_ref_eval_row_f64(int fn, const float *x, int64_t D)
{
    switch (fn) {
    case FN_SPHERE: return sphere(x, D);
    case FN_ACKLEY: return ackley(x, D);
    case FN_RASTRIGIN: return rastrigin(x, D);
    case FN_GRIEWANK: return griewank(x, D);
    case FN_ROSENBROCK: return rosenbrock(x, D);
    case FN_SCHWEFEL: return schwefel(x, D);
    default: return NAN;
    }
}

/* Fitness of N rows of X (row pitch ldx >= D), rounded once to fp32. */
int evox_ref_eval(int fn, const float *X, int64_t N, int64_t D, int64_t ldx, float *out)
{
    if (fn < 0 || fn >= FN_COUNT || N < 0 || D < 1 || ldx < D) return -1;
    for (int64_t i = 0; i < N; ++i) out[i] = (float)evox_ref_eval_row_f64(fn, X + i * ldx, D);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Selection: index of the best fitness.                                     */
/* Order: smaller value first, lower index on ties, -0 == +0, NaN after      */
/* everything (an all-NaN array gives index 0).                              */
/* ------------------------------------------------------------------------ */

static int better(float a, int64_t ia, float b, int64_t ib)
{
    if (isnan(a)) return isnan(b) && ia < ib;
    if (isnan(b)) return 1;
    if (a < b) return 1;
    if (b < a) return 0;
    return ia < ib;
}

int64_t evox_ref_argmin(const float *f, int64_t N)
{
    int64_t best = 0;
    for (int64_t i = 1; i < N; ++i)
        if (better(f[i], i, f[best], best)) best = i;
    return best;
}

/* ------------------------------------------------------------------------ */
/* Parameters (the immutable hyperparameters theta of Sec. IV-B).            */
/* ------------------------------------------------------------------------ */

typedef struct {
    int32_t fn;         /* benchmark function id */
    int32_t clamp_x;    /* nonzero: clamp positions to [lb, ub] after a move */
    int64_t N, D;       /* population size, dimension */
    float lb, ub;       /* initial box (and the clamp box) */
    float v_lo, v_hi;   /* initial velocity box; both 0 means v = 0 */
    float w, c1, c2;    /* PSO inertia and acceleration coefficients */
    float phi;          /* CSO social factor */
    float vmax;         /* PSO velocity clamp; <= 0 means none */
    int32_t x_init;     /* 0: x ~ U[lb, ub); 1: x ~ N(x_mu, x_sigma^2) */
    float x_mu, x_sigma;
    float de_f, de_cr;  /* DE differential weight F and crossover rate CR */
    float es_sigma;     /* OpenES perturbation scale; PGPE initial standard deviation */
    float es_lr;        /* OpenES / PGPE center learning rate */
    float pgpe_sigma_lr;     /* PGPE standard-deviation learning rate */
    float pgpe_max_change;   /* PGPE bound on the relative change of a standard deviation */
    uint64_t seed;      /* Philox key */
    int32_t cso_local;  /* CSO: 0 = the swarm mean, 1 = the mean of the ring neighbourhood */
} evox_ref_params;

/* Algorithm.setup (Sec. IV-A): uniform initial population and velocity.
 * x_ij = lb + u (ub - lb), u from stream 0; v_ij likewise from stream 1. */
static float uniform_in(float u, float lo, float hi)
{
    return fmaf(u, hi - lo, lo);
}

void evox_ref_init_uniform(uint64_t seed, int stream, int64_t N, int64_t D, float lo, float hi,
                           float *out)
{
    for (int64_t i = 0; i < N; ++i)
        for (int64_t j = 0; j < D; ++j)
            out[i * D + j] = uniform_in(draw(seed, i, j, 1, 0, 0, stream), lo, hi);
}

/* Standard normal deviate for element (i, j) of the normal initial
 * population (stream 5, generation 0; box_muller also serves other streams
 * with the generation in the counter's third word), by the Box-Muller transform (Box & Muller, Ann. Math. Statist.
 * 29, 1958): one Philox call per four elements, Philox(seed, (floor(j/4), i,
 * 0, 5)); elements 4c, 4c+1 use words (0, 1) and elements 4c+2, 4c+3 words
 * (2, 3).  Of a word pair (a, b), u1 = ((a >> 8) + 1) 2^-24 lies in (0, 1]
 * (never 0, so the logarithm is finite) and u2 = (b >> 8) 2^-24 in [0, 1);
 * with radius r = sqrt(-2 ln u1) and angle 2 pi u2, the even element of the
 * pair is r cos(angle) and the odd one r sin(angle).  fp64 throughout. */
static double box_muller(uint64_t seed, int64_t i, int64_t j, int64_t t, int stream)
{
    const uint32_t c0 = (uint32_t)(j / 4);
    const int q = (int)(j % 4) / 2;
    const uint32_t a = evox_ref_philox_word(seed, c0, (uint32_t)i, (uint32_t)t, (uint32_t)stream, 2 * q);
    const uint32_t b = evox_ref_philox_word(seed, c0, (uint32_t)i, (uint32_t)t, (uint32_t)stream, 2 * q + 1);
    const double u1 = ((double)(a >> 8) + 1.0) * 0x1p-24;
    const double u2 = (double)(b >> 8) * 0x1p-24;
    const double r = sqrt(-2.0 * log(u1));
    const double angle = 2.0 * kPi * u2;
    return (j % 2 == 0) ? r * cos(angle) : r * sin(angle);
}

double evox_ref_normal01(uint64_t seed, int64_t i, int64_t j)
{
    return box_muller(seed, i, j, 0, STREAM_INIT_NORMAL);
}

/* x_ij = mu + sigma z_ij with z from evox_ref_normal01, rounded once. */
void evox_ref_init_normal(uint64_t seed, int64_t N, int64_t D, float mu, float sigma, float *out)
{
    for (int64_t i = 0; i < N; ++i)
        for (int64_t j = 0; j < D; ++j)
            out[i * D + j] = (float)((double)mu + (double)sigma * evox_ref_normal01(seed, i, j));
}

static void init_xv(const evox_ref_params *P, float *x, float *v)
{
    if (P->x_init == 1)
        evox_ref_init_normal(P->seed, P->N, P->D, P->x_mu, P->x_sigma, x);
    else
        evox_ref_init_uniform(P->seed, STREAM_INIT_X, P->N, P->D, P->lb, P->ub, x);
    if (P->v_lo == 0.0f && P->v_hi == 0.0f)
        memset(v, 0, sizeof(float) * (size_t)(P->N * P->D));
    else
        evox_ref_init_uniform(P->seed, STREAM_INIT_V, P->N, P->D, P->v_lo, P->v_hi, v);
}

/* ------------------------------------------------------------------------ */
/* PSO                                                                       */
/* State: x, v (current), p, pf (personal bests), g, gf, gi (global best).   */
/* ------------------------------------------------------------------------ */

int evox_ref_pso_init(const evox_ref_params *P, float *x, float *v, float *p, float *pf,
                      float *g, float *gf, int64_t *gi)
{
    if (P->N < 1 || P->D < 1) return -1;
    init_xv(P, x, v);
    memcpy(p, x, sizeof(float) * (size_t)(P->N * P->D));
    for (int64_t i = 0; i < P->N; ++i) pf[i] = INFINITY;
    *gf = INFINITY;
    *gi = 0;
    memcpy(g, p, sizeof(float) * (size_t)P->D);
    return 0;
}

/* One velocity/position update of one element. */
static void pso_move_element(const evox_ref_params *P, float r1, float r2, float xv, float vv,
                             float pv, float gv, float *xn_out, float *vn_out)
{
    float a = P->c1 * r1;
    float b = P->c2 * r2;
    float d1 = pv - xv;
    float d2 = gv - xv;
    float vn = fmaf(b, d2, fmaf(a, d1, P->w * vv));
    if (P->vmax > 0.0f) vn = fminf(fmaxf(vn, -P->vmax), P->vmax);
    float xn = xv + vn;
    if (P->clamp_x) xn = fminf(fmaxf(xn, P->lb), P->ub);
    *xn_out = xn;
    *vn_out = vn;
}

/* n_gens ask-evaluate-tell iterations starting at generation t0.
 * Each one: evaluate x (Problem.evaluate); personal bests take strictly
 * better values (tell); the global best is the best personal best; then
 * every particle moves (the next ask). */
int evox_ref_pso_step(const evox_ref_params *P, int64_t t0, int64_t n_gens, float *x, float *v,
                      float *p, float *pf, float *g, float *gf, int64_t *gi)
{
    const int64_t N = P->N, D = P->D;
    if (N < 1 || D < 1 || n_gens < 0 || P->fn < 0 || P->fn >= FN_COUNT) return -1;
    for (int64_t t = t0; t < t0 + n_gens; ++t) {
        for (int64_t i = 0; i < N; ++i) {
            float f = (float)evox_ref_eval_row_f64(P->fn, x + i * D, D);
            if (f < pf[i]) {
                pf[i] = f;
                memcpy(p + i * D, x + i * D, sizeof(float) * (size_t)D);
            }
        }
        *gi = evox_ref_argmin(pf, N);
        *gf = pf[*gi];
        memcpy(g, p + *gi * D, sizeof(float) * (size_t)D);
        for (int64_t i = 0; i < N; ++i) {
            for (int64_t j = 0; j < D; ++j) {
                float r1 = draw(P->seed, i, j, 2, 0, t, STREAM_PSO);
                float r2 = draw(P->seed, i, j, 2, 1, t, STREAM_PSO);
                int64_t e = i * D + j;
                pso_move_element(P, r1, r2, x[e], v[e], p[e], g[j], &x[e], &v[e]);
            }
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* CSO                                                                       */
/* State: x, v, fit (fitness of the current x).                              */
/* ------------------------------------------------------------------------ */

/* Column mean: fp64 sum in row order, fp64 divide, one rounding to fp32. */
void evox_ref_colmean(const float *X, int64_t N, int64_t D, float *xbar)
{
    for (int64_t j = 0; j < D; ++j) {
        double s = 0.0;
        for (int64_t i = 0; i < N; ++i) s += (double)X[i * D + j];
        xbar[j] = (float)(s / (double)N);
    }
}

typedef struct {
    uint32_t key;
    int64_t idx;
} keyed;

static int keyed_cmp(const void *pa, const void *pb)
{
    const keyed *a = (const keyed *)pa, *b = (const keyed *)pb;
    if (a->key != b->key) return a->key < b->key ? -1 : 1;
    return (a->idx > b->idx) - (a->idx < b->idx);
}

/* The indices 0..N-1 in the order of (keys[i], i): a stable argsort. */
void evox_ref_argsort_u32(const uint32_t *keys, int64_t N, int64_t *perm)
{
    keyed *kv = (keyed *)malloc(sizeof(keyed) * (size_t)(N > 0 ? N : 1));
    for (int64_t i = 0; i < N; ++i) {
        kv[i].key = keys[i];
        kv[i].idx = i;
    }
    qsort(kv, (size_t)N, sizeof(keyed), keyed_cmp);
    for (int64_t i = 0; i < N; ++i) perm[i] = kv[i].idx;
    free(kv);
}

/* Random permutation of 0..N-1 at generation t: sort the individuals by the
 * key (Philox word from stream 4), lower index first among equal keys. */
void evox_ref_perm(uint64_t seed, int64_t t, int64_t N, int64_t *perm)
{
    uint32_t *keys = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)(N > 0 ? N : 1));
    for (int64_t i = 0; i < N; ++i)
        keys[i] = evox_ref_philox_word(seed, (uint32_t)(i / 4), 0u, (uint32_t)t, STREAM_PERM,
                                       (int)(i % 4));
    evox_ref_argsort_u32(keys, N, perm);
    free(keys);
}

/* Pair (a, b): b wins when its fitness is strictly lower, or when a's is
 * NaN and b's is not; otherwise a wins (ties go to a). */
static int second_wins(float fa, float fb)
{
    return fb < fa || (isnan(fa) && !isnan(fb));
}

int evox_ref_cso_init(const evox_ref_params *P, float *x, float *v, float *fit)
{
    if (P->N < 1 || P->D < 1 || P->fn < 0 || P->fn >= FN_COUNT) return -1;
    init_xv(P, x, v);
    return evox_ref_eval(P->fn, x, P->N, P->D, P->D, fit);
}

/* The ring-neighbourhood means of CSO's local version (Cheng and Jin, 2015,
 * whose x-bar may be the mean of a predefined neighbourhood): individual i's
 * neighbourhood is i - 1, i, i + 1 (indices modulo N), and its mean
 * ((x_{i-1} + x_i) + x_{i+1}) / 3 is taken in fp64 and rounded once. */
void evox_ref_ring_mean(const float *X, int64_t N, int64_t D, float *out)
{
    for (int64_t i = 0; i < N; ++i) {
        const int64_t a = (i + N - 1) % N, b = (i + 1) % N;
        for (int64_t j = 0; j < D; ++j)
            out[i * D + j] = (float)((((double)X[a * D + j] + (double)X[i * D + j]) + (double)X[b * D + j]) / 3.0);
    }
}

/* Loser l of generation t moves toward its winner w and the mean xb (D
 * floats: the swarm mean, or l's ring-neighbourhood mean). */
static void cso_move_loser(const evox_ref_params *P, int64_t t, int64_t l, int64_t w, float *x, float *v,
                           const float *xb)
{
    const int64_t D = P->D;
    for (int64_t j = 0; j < D; ++j) {
        float R1 = draw(P->seed, l, j, 3, 0, t, STREAM_CSO);
        float R2 = draw(P->seed, l, j, 3, 1, t, STREAM_CSO);
        float R3 = draw(P->seed, l, j, 3, 2, t, STREAM_CSO);
        float xl = x[l * D + j], xw = x[w * D + j], vl = v[l * D + j];
        float t0v = R1 * vl;
        float t1v = fmaf(R2, xw - xl, t0v);
        float c = P->phi * R3;
        float vn = fmaf(c, xb[j] - xl, t1v);
        float xn = xl + vn;
        if (P->clamp_x) xn = fminf(fmaxf(xn, P->lb), P->ub);
        v[l * D + j] = vn;
        x[l * D + j] = xn;
    }
}

/* n_gens CSO iterations from generation t0.  Each: the mean xbar of the
 * current positions -- the swarm's, or with cso_local each loser's ring
 * neighbourhood mean, all taken before any loser moves; random pairing; each
 * loser l moves toward its winner w and the mean,
 *     v_l <- R1 v_l + R2 (x_w - x_l) + phi R3 (xbar - x_l),  x_l <- x_l + v_l,
 * and only the losers are re-evaluated.  Afterwards (best_fit, best_idx) is
 * the best of the current swarm.  loser_flag (nullable, N bytes) receives 1
 * for the rows updated by the last generation. */
int evox_ref_cso_step(const evox_ref_params *P, int64_t t0, int64_t n_gens, float *x, float *v,
                      float *fit, float *best_fit, int64_t *best_idx, uint8_t *loser_flag)
{
    const int64_t N = P->N, D = P->D;
    if (N < 1 || D < 1 || n_gens < 0 || P->fn < 0 || P->fn >= FN_COUNT) return -1;
    float *xbar = (float *)malloc(sizeof(float) * (size_t)(P->cso_local ? N * D : D));
    int64_t *perm = (int64_t *)malloc(sizeof(int64_t) * (size_t)N);
    uint8_t *is_loser = (uint8_t *)calloc((size_t)N, 1);
    for (int64_t t = t0; t < t0 + n_gens; ++t) {
        if (P->cso_local)
            evox_ref_ring_mean(x, N, D, xbar);
        else
            evox_ref_colmean(x, N, D, xbar);
        evox_ref_perm(P->seed, t, N, perm);
        memset(is_loser, 0, (size_t)N);
        for (int64_t k = 0; k < N / 2; ++k) {
            int64_t a = perm[2 * k], b = perm[2 * k + 1];
            int64_t w = a, l = b;
            if (second_wins(fit[a], fit[b])) { w = b; l = a; }
            is_loser[l] = 1;
            cso_move_loser(P, t, l, w, x, v, xbar + (P->cso_local ? l * D : 0));
        }
        for (int64_t i = 0; i < N; ++i)
            if (is_loser[i]) fit[i] = (float)evox_ref_eval_row_f64(P->fn, x + i * D, D);
    }
    int64_t bi = evox_ref_argmin(fit, N);
    *best_idx = bi;
    *best_fit = fit[bi];
    if (loser_flag) memcpy(loser_flag, is_loser, (size_t)N);
    free(xbar);
    free(perm);
    free(is_loser);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* DE: DE/rand/1/bin (Storn & Price, J. Global Optim. 11, 1997), the vanilla */
/* DE of the single-objective experiment (Sec. VII-A-1).                     */
/* State: x, fit (fitness of x).                                             */
/* ------------------------------------------------------------------------ */

/* floor(w m / 2^32): a 32-bit word mapped to [0, m). */
static int64_t below(uint32_t w, int64_t m)
{
    return (int64_t)(((uint64_t)w * (uint64_t)m) >> 32);
}

/* The random choices of target i at generation t: three partners r1, r2,
 * r3, mutually distinct and distinct from i, and the crossover position
 * j_rand in [0, D).  Words 0..3 of Philox(seed, (0, i, t, 6)) give a_k in
 * [0, N - 1 - k) for k = 0, 1, 2 and j_rand in [0, D); r_k is the a_k-th
 * (from 0) of the indices 0..N-1 not yet taken (i, r_1, ..., r_{k-1}),
 * found by stepping a_k past the taken ones in increasing order.  Needs
 * N >= 4.  out = (r1, r2, r3, j_rand). */
void evox_ref_de_choices(uint64_t seed, int64_t t, int64_t i, int64_t N, int64_t D, int64_t out[4])
{
    uint32_t w[4];
    for (int k = 0; k < 4; ++k)
        w[k] = evox_ref_philox_word(seed, 0u, (uint32_t)i, (uint32_t)t, STREAM_DE, k);
    int64_t taken[4] = {i, 0, 0, 0};
    int n_taken = 1;
    for (int k = 0; k < 3; ++k) {
        int64_t r = below(w[k], N - 1 - k);
        for (int e = 0; e < n_taken; ++e)  /* taken[] is in increasing order */
            if (r >= taken[e]) ++r;
        out[k] = r;
        int pos = n_taken;  /* insert r, keeping taken[] sorted */
        while (pos > 0 && taken[pos - 1] > r) {
            taken[pos] = taken[pos - 1];
            --pos;
        }
        taken[pos] = r;
        ++n_taken;
    }
    out[3] = below(w[3], D);
}

int evox_ref_de_init(const evox_ref_params *P, float *x, float *fit)
{
    if (P->N < 4 || P->D < 1 || P->fn < 0 || P->fn >= FN_COUNT) return -1;
    if (P->x_init == 1)
        evox_ref_init_normal(P->seed, P->N, P->D, P->x_mu, P->x_sigma, x);
    else
        evox_ref_init_uniform(P->seed, STREAM_INIT_X, P->N, P->D, P->lb, P->ub, x);
    return evox_ref_eval(P->fn, x, P->N, P->D, P->D, fit);
}

/* n_gens DE generations from generation t0.  For every target i, on the
 * population of the previous generation: mutant v = x_r1 + F (x_r2 - x_r3)
 * (fp32: fma(F, x_r2 - x_r3, x_r1)); binomial crossover u_j = v_j when the
 * crossover draw of element j is <= CR or j = j_rand, else x_ij (the draw of
 * element j is word j mod 4 of Philox(seed, (1 + floor(j/4), i, t, 6)));
 * the trial replaces the target when its fitness is strictly lower (so NaN
 * never replaces).  Afterwards (best_fit, best_idx) is the best of the
 * population.  accepted (nullable, N bytes) receives 1 for the targets the
 * last generation replaced. */
int evox_ref_de_step(const evox_ref_params *P, int64_t t0, int64_t n_gens, float *x, float *fit,
                     float *best_fit, int64_t *best_idx, uint8_t *accepted)
{
    const int64_t N = P->N, D = P->D;
    if (N < 4 || D < 1 || n_gens < 0 || P->fn < 0 || P->fn >= FN_COUNT) return -1;
    float *xn = (float *)malloc(sizeof(float) * (size_t)(N * D));
    float *fn = (float *)malloc(sizeof(float) * (size_t)N);
    float *u = (float *)malloc(sizeof(float) * (size_t)D);
    if (!xn || !fn || !u) {
        free(xn);
        free(fn);
        free(u);
        return -1;
    }
    for (int64_t t = t0; t < t0 + n_gens; ++t) {
        for (int64_t i = 0; i < N; ++i) {
            int64_t c[4];
            evox_ref_de_choices(P->seed, t, i, N, D, c);
            const float *xi = x + i * D, *x1 = x + c[0] * D, *x2 = x + c[1] * D, *x3 = x + c[2] * D;
            for (int64_t j = 0; j < D; ++j) {
                const float mutant = fmaf(P->de_f, x2[j] - x3[j], x1[j]);
                const float cr = draw(P->seed, i, j, 1, 1, t, STREAM_DE);
                u[j] = (cr <= P->de_cr || j == c[3]) ? mutant : xi[j];
            }
            const float fu = (float)evox_ref_eval_row_f64(P->fn, u, D);
            const int take = fu < fit[i];
            memcpy(xn + i * D, take ? u : xi, sizeof(float) * (size_t)D);
            fn[i] = take ? fu : fit[i];
            if (accepted && t == t0 + n_gens - 1) accepted[i] = (uint8_t)take;
        }
        memcpy(x, xn, sizeof(float) * (size_t)(N * D));
        memcpy(fit, fn, sizeof(float) * (size_t)N);
    }
    free(xn);
    free(fn);
    free(u);
    *best_idx = evox_ref_argmin(fit, N);
    *best_fit = fit[*best_idx];
    return 0;
}

/* ------------------------------------------------------------------------ */
/* OpenES (Salimans, Ho, Chen, Sidor, Sutskever, arXiv 1703.03864, 2017; one */
/* of the ES of Table II): antithetic Gaussian perturbations of a center,   */
/* centered-rank fitness shaping, one gradient step.                         */
/* State: theta (the center, fp32 [D]).                                      */
/* ------------------------------------------------------------------------ */

/* The perturbation eps_kj of antithetic pair k at generation t: the
 * Box-Muller deviate of Philox(seed, (floor(j/4), k, t, 7)), the word layout
 * of the normal initial population. */
double evox_ref_es_eps(uint64_t seed, int64_t t, int64_t k, int64_t j)
{
    return box_muller(seed, k, j, t, STREAM_ES);
}

/* Initial center: theta_j = lb + u (ub - lb), u from row 0 of stream 0. */
int evox_ref_es_init(const evox_ref_params *P, float *theta)
{
    if (P->N < 2 || (P->N & 1) || P->D < 1 || P->fn < 0 || P->fn >= FN_COUNT) return -1;
    evox_ref_init_uniform(P->seed, STREAM_INIT_X, 1, P->D, P->lb, P->ub, theta);
    return 0;
}

/* n_gens OpenES generations from generation t0.  Each: samples x_{2k} =
 * theta + sigma eps_k and x_{2k+1} = theta - sigma eps_k (fp32:
 * fma(+-sigma, eps, theta) with eps rounded to fp32), fitness f = F(x);
 * centered ranks u_i = rank_i / (N - 1) - 1/2, rank_i the position of i in
 * the order of (f_i, i) (NaN last, the argmin order); the gradient estimate
 * g_j = sum_k (u_{2k} - u_{2k+1}) eps_kj / (N sigma) in fp64 (a descent
 * direction for minimization: u grows with f); theta_j <- fma(-lr, g_j,
 * theta_j) with g_j rounded to fp32.  fit (nullable, N floats) receives the
 * last generation's fitness, rank (nullable) its ranks; (best_fit,
 * best_idx) is the best sample of the last generation. */
int evox_ref_es_step(const evox_ref_params *P, int64_t t0, int64_t n_gens, float *theta,
                     float *fit_out, int64_t *rank_out, float *best_fit, int64_t *best_idx)
{
    const int64_t N = P->N, D = P->D, H = N / 2;
    if (N < 2 || (N & 1) || D < 1 || n_gens < 0 || P->fn < 0 || P->fn >= FN_COUNT) return -1;
    float *x = (float *)malloc(sizeof(float) * (size_t)D);
    float *f = (float *)malloc(sizeof(float) * (size_t)N);
    int64_t *order = (int64_t *)malloc(sizeof(int64_t) * (size_t)N);
    int64_t *rank = (int64_t *)malloc(sizeof(int64_t) * (size_t)N);
    double *g = (double *)malloc(sizeof(double) * (size_t)D);
    if (!x || !f || !order || !rank || !g) {
        free(x); free(f); free(order); free(rank); free(g);
        return -1;
    }
    for (int64_t t = t0; t < t0 + n_gens; ++t) {
        for (int64_t i = 0; i < N; ++i) {
            const int64_t k = i / 2;
            const float s = (i & 1) ? -P->es_sigma : P->es_sigma;
            for (int64_t j = 0; j < D; ++j)
                x[j] = fmaf(s, (float)evox_ref_es_eps(P->seed, t, k, j), theta[j]);
            f[i] = (float)evox_ref_eval_row_f64(P->fn, x, D);
        }
        /* ranks: sort the indices in the argmin order, by insertion */
        for (int64_t i = 0; i < N; ++i) {
            int64_t p = i;
            while (p > 0 && better(f[i], i, f[order[p - 1]], order[p - 1])) {
                order[p] = order[p - 1];
                --p;
            }
            order[p] = i;
        }
        for (int64_t p = 0; p < N; ++p) rank[order[p]] = p;
        for (int64_t j = 0; j < D; ++j) g[j] = 0.0;
        for (int64_t k = 0; k < H; ++k) {
            const double u0 = (double)rank[2 * k] / (double)(N - 1) - 0.5;
            const double u1 = (double)rank[2 * k + 1] / (double)(N - 1) - 0.5;
            for (int64_t j = 0; j < D; ++j) g[j] += (u0 - u1) * evox_ref_es_eps(P->seed, t, k, j);
        }
        for (int64_t j = 0; j < D; ++j) {
            const float gj = (float)(g[j] / ((double)N * (double)P->es_sigma));
            theta[j] = fmaf(-P->es_lr, gj, theta[j]);
        }
        if (t == t0 + n_gens - 1) {
            if (fit_out) memcpy(fit_out, f, sizeof(float) * (size_t)N);
            if (rank_out) memcpy(rank_out, rank, sizeof(int64_t) * (size_t)N);
            *best_idx = order[0];
            *best_fit = f[order[0]];
        }
    }
    free(x); free(f); free(order); free(rank); free(g);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* PGPE with symmetric sampling (Sehnke, Osendorfer, Rueckstiess, Graves,    */
/* Peters, Schmidhuber, Neural Networks 23, 2010; the ES the paper runs in   */
/* its neuroevolution and EvoTorch comparisons).                             */
/* State: mu (center) and sigma (per-dimension standard deviation), fp32.    */
/* ------------------------------------------------------------------------ */

/* z_kj of pair k at generation t: the Box-Muller deviate of Philox(seed,
 * (floor(j/4), k, t, 8)); the perturbation is sigma_j z_kj. */
double evox_ref_pgpe_z(uint64_t seed, int64_t t, int64_t k, int64_t j)
{
    return box_muller(seed, k, j, t, STREAM_PGPE);
}

/* First center: row 0 of the uniform population; sigma_j = es_sigma. */
int evox_ref_pgpe_init(const evox_ref_params *P, float *mu, float *sigma)
{
    if (P->N < 2 || (P->N & 1) || P->D < 1 || P->fn < 0 || P->fn >= FN_COUNT) return -1;
    evox_ref_init_uniform(P->seed, STREAM_INIT_X, 1, P->D, P->lb, P->ub, mu);
    for (int64_t j = 0; j < P->D; ++j) sigma[j] = P->es_sigma;
    return 0;
}

/* n_gens PGPE generations from generation t0.  Each: perturbations
 * eps_kj = sigma_j z_kj (fp32 product) for pairs k < N/2; samples
 * x_{2k} = mu + eps_k, x_{2k+1} = mu - eps_k (fp32: fma(+-sigma_j, z_kj,
 * mu_j)); fitness f = F(x); centered ranks u_i = rank_i / (N - 1) - 1/2 in
 * the argmin order (the utilities, higher is worse); with H = N/2, in fp64:
 *     g_mu_j    = (1/H) sum_k (u_{2k} - u_{2k+1}) / 2 * sigma_j z_kj
 *     g_sigma_j = (1/H) sum_k (u_{2k} + u_{2k+1}) / 2 * sigma_j (z_kj^2 - 1)
 * (the symmetric-sampling gradients of the expected utility, whose baseline
 * -- the mean utility -- is zero); descent steps in fp32:
 *     mu_j    <- fma(-lr, g_mu_j, mu_j)
 *     d_j      = -sigma_lr g_sigma_j, clamped to [-c sigma_j, c sigma_j]
 *                with c = pgpe_max_change (c sigma_j rounded once)
 *     sigma_j <- sigma_j + d_j
 * with the gradients rounded to fp32 once.  fit / rank (nullable) receive
 * the last generation's; (best_fit, best_idx) its best sample. */
int evox_ref_pgpe_step(const evox_ref_params *P, int64_t t0, int64_t n_gens, float *mu, float *sigma,
                       float *fit_out, int64_t *rank_out, float *best_fit, int64_t *best_idx)
{
    const int64_t N = P->N, D = P->D, H = N / 2;
    if (N < 2 || (N & 1) || D < 1 || n_gens < 0 || P->fn < 0 || P->fn >= FN_COUNT) return -1;
    float *x = (float *)malloc(sizeof(float) * (size_t)D);
    float *f = (float *)malloc(sizeof(float) * (size_t)N);
    int64_t *order = (int64_t *)malloc(sizeof(int64_t) * (size_t)N);
    int64_t *rank = (int64_t *)malloc(sizeof(int64_t) * (size_t)N);
    double *gm = (double *)malloc(sizeof(double) * (size_t)D);
    double *gs = (double *)malloc(sizeof(double) * (size_t)D);
    if (!x || !f || !order || !rank || !gm || !gs) {
        free(x); free(f); free(order); free(rank); free(gm); free(gs);
        return -1;
    }
    for (int64_t t = t0; t < t0 + n_gens; ++t) {
        for (int64_t i = 0; i < N; ++i) {
            const int64_t k = i / 2;
            for (int64_t j = 0; j < D; ++j) {
                const float s = (i & 1) ? -sigma[j] : sigma[j];
                x[j] = fmaf(s, (float)evox_ref_pgpe_z(P->seed, t, k, j), mu[j]);
            }
            f[i] = (float)evox_ref_eval_row_f64(P->fn, x, D);
        }
        for (int64_t i = 0; i < N; ++i) {
            int64_t p = i;
            while (p > 0 && better(f[i], i, f[order[p - 1]], order[p - 1])) {
                order[p] = order[p - 1];
                --p;
            }
            order[p] = i;
        }
        for (int64_t p = 0; p < N; ++p) rank[order[p]] = p;
        for (int64_t j = 0; j < D; ++j) gm[j] = gs[j] = 0.0;
        for (int64_t k = 0; k < H; ++k) {
            const double u0 = (double)rank[2 * k] / (double)(N - 1) - 0.5;
            const double u1 = (double)rank[2 * k + 1] / (double)(N - 1) - 0.5;
            for (int64_t j = 0; j < D; ++j) {
                const double z = (double)(float)evox_ref_pgpe_z(P->seed, t, k, j);
                gm[j] += 0.5 * (u0 - u1) * (double)sigma[j] * z;
                gs[j] += 0.5 * (u0 + u1) * (double)sigma[j] * (z * z - 1.0);
            }
        }
        for (int64_t j = 0; j < D; ++j) {
            const float gmj = (float)(gm[j] / (double)H), gsj = (float)(gs[j] / (double)H);
            mu[j] = fmaf(-P->es_lr, gmj, mu[j]);
            const float cap = P->pgpe_max_change * sigma[j];
            const float d = fminf(fmaxf(-P->pgpe_sigma_lr * gsj, -cap), cap);
            sigma[j] = sigma[j] + d;
        }
        if (t == t0 + n_gens - 1) {
            if (fit_out) memcpy(fit_out, f, sizeof(float) * (size_t)N);
            if (rank_out) memcpy(rank_out, rank, sizeof(int64_t) * (size_t)N);
            *best_idx = order[0];
            *best_fit = f[order[0]];
        }
    }
    free(x); free(f); free(order); free(rank); free(gm); free(gs);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Dense matrix product (the contractions of the matrix-adaptation ES):      */
/* C = alpha op(A) op(B) + beta C, op(A) [M x K], op(B) [K x N], row-major    */
/* with leading dimensions; op(A) = A^T when ta (A stored K x M), likewise    */
/* for B.  Each output in fp64 from the fp32 inputs, rounded once.            */
/* ------------------------------------------------------------------------ */
void evox_ref_gemm(int ta, int tb, int64_t M, int64_t N, int64_t K, float alpha, const float *A,
                   int64_t lda, const float *B, int64_t ldb, float beta, float *C, int64_t ldc)
{
    for (int64_t i = 0; i < M; ++i)
        for (int64_t j = 0; j < N; ++j) {
            double acc = 0.0;
            for (int64_t k = 0; k < K; ++k) {
                const double a = ta ? A[k * lda + i] : A[i * lda + k];
                const double b = tb ? B[j * ldb + k] : B[k * ldb + j];
                acc += a * b;
            }
            const double c = beta != 0.0f ? (double)beta * (double)C[i * ldc + j] : 0.0;
            C[i * ldc + j] = (float)((double)alpha * acc + c);
        }
}

/* ------------------------------------------------------------------------ */
/* CMA-ES (Table II; an ES of the scaling experiment of Sec. VII-A-1) in its */
/* matrix-adaptation form, MA-ES (Beyer and Sendhoff, IEEE TEVC 21(5),       */
/* 2017): the transformation M with M M^T in the role of the covariance      */
/* matrix is adapted directly, so sampling needs no eigendecomposition.      */
/* State: center y [D], step size sigma, M [D x D] (identity at start),      */
/* evolution path s [D] (zero at start), all fp32.                           */
/* ------------------------------------------------------------------------ */

/* z_kj of sample k at generation t: the Box-Muller deviate of
 * Philox(seed, (floor(j/4), k, t, 9)). */
double evox_ref_maes_z(uint64_t seed, int64_t t, int64_t k, int64_t j)
{
    return box_muller(seed, k, j, t, STREAM_MAES);
}

/* The deviates of one generation rounded to fp32, z[k * D + j] = z_kj. */
void evox_ref_maes_deviates(uint64_t seed, int64_t t, int64_t N, int64_t D, float *z)
{
    for (int64_t k = 0; k < N; ++k)
        for (int64_t j = 0; j < D; ++j) z[k * D + j] = (float)evox_ref_maes_z(seed, t, k, j);
}

/* The default strategy constants for N = lambda samples in D dimensions
 * (Hansen's CMA-ES defaults, which MA-ES keeps): mu = floor(lambda/2)
 * parents; weights w_i proportional to ln(mu + 1/2) - ln i (i = 1..mu),
 * summing to one; mu_eff = 1 / sum w_i^2;
 *   c_s     = (mu_eff + 2) / (D + mu_eff + 5)
 *   d_s     = 1 + c_s + 2 max(0, sqrt((mu_eff - 1) / (D + 1)) - 1)
 *   c_1     = 2 / ((D + 1.3)^2 + mu_eff)
 *   c_w     = min(1 - c_1, 2 (mu_eff - 2 + 1/mu_eff) / ((D + 2)^2 + mu_eff))
 *   chi_D   = sqrt(D) (1 - 1/(4D) + 1/(21 D^2)), the expected length of a
 *             standard normal vector in D dimensions.
 * w (nullable) receives the mu weights; c the six numbers mu_eff, c_s, d_s,
 * c_1, c_w, chi_D.  Returns mu, or -1 for N < 2 or D < 1. */
int64_t evox_ref_maes_consts(int64_t N, int64_t D, double *w, double *c)
{
    if (N < 2 || D < 1) return -1;
    const int64_t mu = N / 2;
    double sw = 0.0, sw2 = 0.0;
    for (int64_t i = 1; i <= mu; ++i) sw += log((double)mu + 0.5) - log((double)i);
    for (int64_t i = 1; i <= mu; ++i) {
        const double wi = (log((double)mu + 0.5) - log((double)i)) / sw;
        if (w) w[i - 1] = wi;
        sw2 += wi * wi;
    }
    const double n = (double)D, me = 1.0 / sw2;
    const double cs = (me + 2.0) / (n + me + 5.0);
    const double ds = 1.0 + cs + 2.0 * fmax(0.0, sqrt((me - 1.0) / (n + 1.0)) - 1.0);
    const double c1 = 2.0 / ((n + 1.3) * (n + 1.3) + me);
    const double cw = fmin(1.0 - c1, 2.0 * (me - 2.0 + 1.0 / me) / ((n + 2.0) * (n + 2.0) + me));
    c[0] = me;
    c[1] = cs;
    c[2] = ds;
    c[3] = c1;
    c[4] = cw;
    c[5] = sqrt(n) * (1.0 - 1.0 / (4.0 * n) + 1.0 / (21.0 * n * n));
    return mu;
}

/* Initial state: y = row 0 of the uniform population (stream 0), sigma =
 * es_sigma, M = I, s = 0. */
int evox_ref_maes_init(const evox_ref_params *P, float *y, float *sigma, float *M, float *s)
{
    if (P->N < 2 || P->D < 1 || P->fn < 0 || P->fn >= FN_COUNT) return -1;
    const int64_t D = P->D;
    evox_ref_init_uniform(P->seed, STREAM_INIT_X, 1, D, P->lb, P->ub, y);
    *sigma = P->es_sigma;
    for (int64_t i = 0; i < D; ++i) {
        s[i] = 0.0f;
        for (int64_t j = 0; j < D; ++j) M[i * D + j] = i == j ? 1.0f : 0.0f;
    }
    return 0;
}

/* n_gens MA-ES generations from generation t0.  Each, with the constants of
 * evox_ref_maes_consts:
 *   z_k = (z_kj rounded to fp32), k < lambda
 *   d_k = M z_k                      (fp64 sums, rounded to fp32)
 *   x_k = y + sigma d_k              (fp32: fma(sigma, d_kj, y_j))
 *   f_k = F(x_k); order the samples by (f_k, k) (NaN last, the argmin order)
 *   <z>_w = sum_{i<mu} w_i z_{i:lambda},  <d>_w likewise   (fp64)
 *   y  <- y + sigma <d>_w
 *   s  <- (1 - c_s) s + sqrt(mu_eff c_s (2 - c_s)) <z>_w
 *   M  <- M [I + c_1/2 (s s^T - I) + c_w/2 (sum_{i<mu} w_i z_{i:lambda}
 *            z_{i:lambda}^T - I)]      (the new s; the bracket in fp64,
 *                                      the product in fp64 per element)
 *   sigma <- sigma exp(c_s/d_s (|s| / chi_D - 1))
 * each new fp32 value rounded once from fp64.  M is row-major D x D.
 * rows (nullable; n_gens must then be 1) restricts the update of M to the
 * n_rows listed rows, the others keeping their old values.  fit, rank
 * (nullable) receive the last generation's fitness and ranks, d_out
 * (nullable, N x D) its d_k; (best_fit, best_idx) is its best sample. */
int evox_ref_maes_step(const evox_ref_params *P, int64_t t0, int64_t n_gens, float *y, float *sigma,
                       float *M, float *s, float *fit_out, int64_t *rank_out, float *best_fit,
                       int64_t *best_idx, int64_t n_rows, const int64_t *rows, float *d_out)
{
    const int64_t N = P->N, D = P->D;
    if (N < 2 || D < 1 || n_gens < 0 || P->fn < 0 || P->fn >= FN_COUNT) return -1;
    if (rows && n_gens != 1) return -1;
    double c[6];
    double *w = (double *)malloc(sizeof(double) * (size_t)(N / 2));
    const int64_t mu = evox_ref_maes_consts(N, D, w, c);
    const double me = c[0], cs = c[1], ds = c[2], c1 = c[3], cw = c[4], chi = c[5];
    float *z = (float *)malloc(sizeof(float) * (size_t)(N * D));
    float *d = (float *)malloc(sizeof(float) * (size_t)(N * D));
    float *x = (float *)malloc(sizeof(float) * (size_t)D);
    float *f = (float *)malloc(sizeof(float) * (size_t)N);
    int64_t *order = (int64_t *)malloc(sizeof(int64_t) * (size_t)N);
    int64_t *rank = (int64_t *)malloc(sizeof(int64_t) * (size_t)N);
    double *zw = (double *)malloc(sizeof(double) * (size_t)D);
    double *dw = (double *)malloc(sizeof(double) * (size_t)D);
    double *T = (double *)malloc(sizeof(double) * (size_t)(D * D));
    double *row = (double *)malloc(sizeof(double) * (size_t)D);
    if (!w || !z || !d || !x || !f || !order || !rank || !zw || !dw || !T || !row) {
        free(w); free(z); free(d); free(x); free(f); free(order); free(rank); free(zw); free(dw);
        free(T); free(row);
        return -1;
    }
    for (int64_t t = t0; t < t0 + n_gens; ++t) {
        /* sampling and evaluation */
        evox_ref_maes_deviates(P->seed, t, N, D, z);
        for (int64_t k = 0; k < N; ++k) {
            for (int64_t i = 0; i < D; ++i) {
                double acc = 0.0;
                for (int64_t j = 0; j < D; ++j) acc += (double)M[i * D + j] * (double)z[k * D + j];
                d[k * D + i] = (float)acc;
            }
            for (int64_t i = 0; i < D; ++i) x[i] = fmaf(*sigma, d[k * D + i], y[i]);
            f[k] = (float)evox_ref_eval_row_f64(P->fn, x, D);
        }
        for (int64_t i = 0; i < N; ++i) {
            int64_t p = i;
            while (p > 0 && better(f[i], i, f[order[p - 1]], order[p - 1])) {
                order[p] = order[p - 1];
                --p;
            }
            order[p] = i;
        }
        for (int64_t p = 0; p < N; ++p) rank[order[p]] = p;
        /* recombination */
        for (int64_t j = 0; j < D; ++j) {
            zw[j] = dw[j] = 0.0;
            for (int64_t r = 0; r < mu; ++r) {
                zw[j] += w[r] * (double)z[order[r] * D + j];
                dw[j] += w[r] * (double)d[order[r] * D + j];
            }
        }
        const double sig = (double)*sigma;
        const double cz = sqrt(me * cs * (2.0 - cs));
        double s2 = 0.0;
        for (int64_t j = 0; j < D; ++j) {
            y[j] = (float)((double)y[j] + sig * dw[j]);
            s[j] = (float)((1.0 - cs) * (double)s[j] + cz * zw[j]);
            s2 += (double)s[j] * (double)s[j];
        }
        /* T = I + c_1/2 (s s^T - I) + c_w/2 (sum_r w_r z_r z_r^T - I) */
        for (int64_t a = 0; a < D; ++a)
            for (int64_t b = 0; b < D; ++b) {
                double zz = 0.0;
                for (int64_t r = 0; r < mu; ++r)
                    zz += w[r] * (double)z[order[r] * D + a] * (double)z[order[r] * D + b];
                const double id = a == b ? 1.0 : 0.0;
                T[a * D + b] = id + 0.5 * c1 * ((double)s[a] * (double)s[b] - id) + 0.5 * cw * (zz - id);
            }
        /* M <- M T, row by row */
        const int64_t nr = rows ? n_rows : D;
        for (int64_t q = 0; q < nr; ++q) {
            const int64_t i = rows ? rows[q] : q;
            if (i < 0 || i >= D) continue;
            for (int64_t b = 0; b < D; ++b) {
                double acc = 0.0;
                for (int64_t a = 0; a < D; ++a) acc += (double)M[i * D + a] * T[a * D + b];
                row[b] = acc;
            }
            for (int64_t b = 0; b < D; ++b) M[i * D + b] = (float)row[b];
        }
        *sigma = (float)(sig * exp(cs / ds * (sqrt(s2) / chi - 1.0)));
        if (t == t0 + n_gens - 1) {
            if (fit_out) memcpy(fit_out, f, sizeof(float) * (size_t)N);
            if (rank_out) memcpy(rank_out, rank, sizeof(int64_t) * (size_t)N);
            if (d_out) memcpy(d_out, d, sizeof(float) * (size_t)(N * D));
            *best_idx = order[0];
            *best_fit = f[order[0]];
        }
    }
    free(w); free(z); free(d); free(x); free(f); free(order); free(rank); free(zw); free(dw);
    free(T); free(row);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* NSGA-II (Table II; the multi-objective experiment of Sec. VII-A-2         */
/* runs it on DTLZ1) following Deb, Pratap, Agarwal and Meyarivan, IEEE TEVC */
/* 6(2), 2002: crowded binary tournaments, simulated binary crossover and    */
/* polynomial mutation, non-dominated sorting of parents and offspring       */
/* together, crowding distance, elitist truncation.                          */
/* ------------------------------------------------------------------------ */

typedef struct {
    int64_t N, D;       /* population (even), decision variables (>= M) */
    int32_t M;          /* objectives */
    float eta_c, eta_m; /* distribution indices of the crossover and the mutation */
    uint64_t seed;
} evox_ref_nsga2_params;

/* DTLZ1 (Deb, Thiele, Laumanns, Zitzler, 2002) on x in [0, 1]^D with M
 * objectives, k = D - M + 1 distance variables:
 *   g = 100 (k + sum_{i >= M-1} ((x_i - 1/2)^2 - cos(20 pi (x_i - 1/2))))
 *   f_0 = (1 + g)/2 x_0 x_1 ... x_{M-2}
 *   f_m = (1 + g)/2 x_0 ... x_{M-2-m} (1 - x_{M-1-m}),  m = 1 .. M-1
 * in fp64; the Pareto-optimal front is sum_m f_m = 1/2 at g = 0. */
void evox_ref_dtlz1(const float *x, int64_t D, int32_t M, double *f)
{
    const double pi = 3.14159265358979323846;
    double g = 0.0;
    for (int64_t i = M - 1; i < D; ++i) {
        const double d = (double)x[i] - 0.5;
        g += d * d - cos(20.0 * pi * d);
    }
    g = 100.0 * ((double)(D - M + 1) + g);
    for (int32_t m = 0; m < M; ++m) {
        double v = 0.5 * (1.0 + g);
        for (int32_t i = 0; i < M - 1 - m; ++i) v *= (double)x[i];
        if (m > 0) v *= 1.0 - (double)x[M - 1 - m];
        f[m] = v;
    }
}

/* Objectives of n rows (pitch D) rounded to fp32, F[i * M + m]. */
void evox_ref_dtlz1_rows(const float *X, int64_t n, int64_t D, int32_t M, float *F)
{
    double f[64];
    for (int64_t i = 0; i < n; ++i) {
        evox_ref_dtlz1(X + i * D, D, M, f);
        for (int32_t m = 0; m < M; ++m) F[i * M + m] = (float)f[m];
    }
}

/* a dominates b (minimisation): no objective worse, at least one better. */
int evox_ref_dominates(const float *a, const float *b, int32_t M)
{
    int strict = 0;
    for (int32_t m = 0; m < M; ++m) {
        if (a[m] > b[m]) return 0;
        if (a[m] < b[m]) strict = 1;
    }
    return strict;
}

/* Non-dominated sorting by its definition: front 0 holds the points no
 * point dominates; front k + 1 the points that only points of fronts <= k
 * dominate.  front[i] receives the 0-based front index.  Returns the number
 * of fronts. */
int32_t evox_ref_nds(const float *F, int64_t n, int32_t M, int32_t *front)
{
    for (int64_t i = 0; i < n; ++i) front[i] = -1;
    int64_t left = n;
    int32_t k = 0;
    while (left > 0) {
        /* members of front k: unassigned and dominated by no unassigned point */
        for (int64_t i = 0; i < n; ++i) {
            if (front[i] != -1) continue;
            int dominated = 0;
            for (int64_t j = 0; j < n && !dominated; ++j)  /* j still unassigned (-1, or -2 below) */
                if (front[j] < 0) dominated = evox_ref_dominates(F + j * M, F + i * M, M);
            if (!dominated) front[i] = -2; /* front k, marked once every point is checked */
        }
        for (int64_t i = 0; i < n; ++i)
            if (front[i] == -2) {
                front[i] = k;
                --left;
            }
        ++k;
    }
    return k;
}

/* Crowding distance within each front (Deb et al. 2002): per objective m
 * (in the order m = 0 .. M-1), the front's members in the order of (f_m,
 * index); the first and last get +inf, every other member adds
 * (f_m[next] - f_m[prev]) / (f_m,max - f_m,min) in fp64 when the range is
 * not zero.  A member of a front of one or two points gets +inf. */
void evox_ref_crowding(const float *F, int64_t n, int32_t M, const int32_t *front, double *crowd)
{
    int64_t *idx = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int32_t nf = 0;
    for (int64_t i = 0; i < n; ++i) {
        crowd[i] = 0.0;
        if (front[i] + 1 > nf) nf = front[i] + 1;
    }
    for (int32_t k = 0; k < nf; ++k) {
        int64_t c = 0;
        for (int64_t i = 0; i < n; ++i)
            if (front[i] == k) idx[c++] = i;
        for (int32_t m = 0; m < M; ++m) {
            /* insertion sort by (f_m, index) */
            for (int64_t a = 1; a < c; ++a) {
                const int64_t v = idx[a];
                int64_t b = a;
                while (b > 0 && (F[idx[b - 1] * M + m] > F[v * M + m] ||
                                 (F[idx[b - 1] * M + m] == F[v * M + m] && idx[b - 1] > v))) {
                    idx[b] = idx[b - 1];
                    --b;
                }
                idx[b] = v;
            }
            if (c == 0) continue;
            crowd[idx[0]] = INFINITY;
            crowd[idx[c - 1]] = INFINITY;
            const double lo = (double)F[idx[0] * M + m], hi = (double)F[idx[c - 1] * M + m];
            if (hi > lo)
                for (int64_t a = 1; a + 1 < c; ++a)
                    crowd[idx[a]] += ((double)F[idx[a + 1] * M + m] - (double)F[idx[a - 1] * M + m]) / (hi - lo);
        }
    }
    free(idx);
}

/* The crowded comparison of a binary tournament: the lower front wins, then
 * the larger crowding distance, then the lower index. */
static int64_t crowded_winner(int64_t a, int64_t b, const int32_t *front, const double *crowd)
{
    if (front[a] != front[b]) return front[a] < front[b] ? a : b;
    if (crowd[a] != crowd[b]) return crowd[a] > crowd[b] ? a : b;
    return a < b ? a : b;
}

/* The two parents of offspring pair p at generation t: tournaments between
 * the individuals floor(w_q N / 2^32) named by the four words w_0..w_3 of
 * Philox(seed, (0, p, t, 10)): (w_0, w_1) and (w_2, w_3). */
void evox_ref_nsga2_parents(uint64_t seed, int64_t t, int64_t p, int64_t N, const int32_t *front,
                            const double *crowd, int64_t *p1, int64_t *p2)
{
    int64_t c[4];
    for (int q = 0; q < 4; ++q)
        c[q] = (int64_t)(((uint64_t)evox_ref_philox_word(seed, 0, (uint32_t)p, (uint32_t)t, STREAM_NSGA_SEL, q) *
                          (uint64_t)N) >> 32);
    *p1 = crowded_winner(c[0], c[1], front, crowd);
    *p2 = crowded_winner(c[2], c[3], front, crowd);
}

/* Polynomial mutation of x in [0, 1] with distribution index eta and draw
 * u in [0, 1) (Deb and Goyal, 1996, in its bounded form): u < 1/2 moves
 * down by 1 - (2u + (1 - 2u)(1 - x)^(eta+1))^(1/(eta+1)), u >= 1/2 up by
 * 1 - (2(1 - u) + 2(u - 1/2) x^(eta+1))^(1/(eta+1)); clipped to [0, 1]. */
double evox_ref_poly_mutate(double x, double u, double eta)
{
    const double e1 = eta + 1.0, inv = 1.0 / e1;
    double y;
    if (u < 0.5)
        y = x + (pow(2.0 * u + (1.0 - 2.0 * u) * pow(1.0 - x, e1), inv) - 1.0);
    else
        y = x + (1.0 - pow(2.0 * (1.0 - u) + 2.0 * (u - 0.5) * pow(x, e1), inv));
    return y < 0.0 ? 0.0 : y > 1.0 ? 1.0 : y;
}

/* Offspring 2p and 2p + 1 from parents a and b (rows of D floats in [0,1]).
 * Per variable j, with the words w of Philox(seed, (j, p, t, 11)) and v of
 * Philox(seed, (j, p, t, 12)), u(w) = the top 24 bits times 2^-24:
 *   simulated binary crossover (Deb and Agrawal, 1995; crossover
 *   probability 1): spread beta = (2u)^(1/(eta_c+1)) for u = u(w_0) <= 1/2,
 *   else (2 - 2u)^(-1/(eta_c+1)); negated when w_1 is odd; 1 (the variable
 *   is not crossed) when u(w_1) >= 1/2; children (a + b)/2 +- beta (a - b)/2
 *   clipped to [0, 1] and rounded to fp32;
 *   polynomial mutation of child q (q = 0, 1) when u(w_{2+q}) < 1/D, with
 *   draw u(v_q), rounded to fp32.
 * Arithmetic in fp64. */
void evox_ref_nsga2_offspring(const evox_ref_nsga2_params *P, int64_t t, int64_t p, const float *a,
                              const float *b, float *c0, float *c1)
{
    const double ec = (double)P->eta_c, em = (double)P->eta_m, pm = 1.0 / (double)P->D;
    for (int64_t j = 0; j < P->D; ++j) {
        uint32_t w[4], v[2];
        for (int q = 0; q < 4; ++q)
            w[q] = evox_ref_philox_word(P->seed, (uint32_t)j, (uint32_t)p, (uint32_t)t, STREAM_NSGA_VAR, q);
        for (int q = 0; q < 2; ++q)
            v[q] = evox_ref_philox_word(P->seed, (uint32_t)j, (uint32_t)p, (uint32_t)t, STREAM_NSGA_MUT, q);
        const double u = (double)evox_ref_u01(w[0]);
        double beta = u <= 0.5 ? pow(2.0 * u, 1.0 / (ec + 1.0)) : pow(2.0 - 2.0 * u, -1.0 / (ec + 1.0));
        if (w[1] & 1u) beta = -beta;
        if ((double)evox_ref_u01(w[1]) >= 0.5) beta = 1.0;
        const double xa = (double)a[j], xb = (double)b[j];
        double y[2] = {0.5 * (xa + xb) + 0.5 * beta * (xa - xb), 0.5 * (xa + xb) - 0.5 * beta * (xa - xb)};
        float out[2];
        for (int q = 0; q < 2; ++q) {
            const double yc = y[q] < 0.0 ? 0.0 : y[q] > 1.0 ? 1.0 : y[q];
            out[q] = (float)yc;
            if ((double)evox_ref_u01(w[2 + q]) < pm)
                out[q] = (float)evox_ref_poly_mutate((double)out[q], (double)evox_ref_u01(v[q]), em);
        }
        c0[j] = out[0];
        c1[j] = out[1];
    }
}

/* Initial population: x ~ U[0, 1) from stream 0 (the uniform initial
 * population with lb = 0, ub = 1), its objectives, fronts and crowding. */
int evox_ref_nsga2_init(const evox_ref_nsga2_params *P, float *X, float *F, int32_t *front, double *crowd)
{
    if (P->N < 2 || (P->N & 1) || P->M < 2 || P->M > 64 || P->D < P->M) return -1;
    evox_ref_init_uniform(P->seed, STREAM_INIT_X, P->N, P->D, 0.0f, 1.0f, X);
    evox_ref_dtlz1_rows(X, P->N, P->D, P->M, F);
    evox_ref_nds(F, P->N, P->M, front);
    evox_ref_crowding(F, P->N, P->M, front, crowd);
    return 0;
}

/* n_gens generations from generation t0: offspring Q (pairs p < N/2 from
 * tournament parents), R = (P, Q) with P first, fronts and crowding of R,
 * then the survivors: whole fronts in order while they fit, and from the
 * first front that does not fit, its members of largest crowding distance
 * (ties: lower index in R) up to N; the survivors keep their order in R and
 * their fronts and crowding distances. */
int evox_ref_nsga2_step(const evox_ref_nsga2_params *P, int64_t t0, int64_t n_gens, float *X, float *F,
                        int32_t *front, double *crowd)
{
    const int64_t N = P->N, D = P->D, R = 2 * P->N;
    const int32_t M = P->M;
    if (N < 2 || (N & 1) || M < 2 || M > 64 || D < M || n_gens < 0) return -1;
    float *XR = (float *)malloc(sizeof(float) * (size_t)(R * D));
    float *FR = (float *)malloc(sizeof(float) * (size_t)(R * M));
    int32_t *fr = (int32_t *)malloc(sizeof(int32_t) * (size_t)R);
    double *cr = (double *)malloc(sizeof(double) * (size_t)R);
    char *keep = (char *)malloc((size_t)R);
    if (!XR || !FR || !fr || !cr || !keep) {
        free(XR); free(FR); free(fr); free(cr); free(keep);
        return -1;
    }
    for (int64_t t = t0; t < t0 + n_gens; ++t) {
        memcpy(XR, X, sizeof(float) * (size_t)(N * D));
        memcpy(FR, F, sizeof(float) * (size_t)(N * M));
        for (int64_t p = 0; p < N / 2; ++p) {
            int64_t a, b;
            evox_ref_nsga2_parents(P->seed, t, p, N, front, crowd, &a, &b);
            evox_ref_nsga2_offspring(P, t, p, X + a * D, X + b * D, XR + (N + 2 * p) * D, XR + (N + 2 * p + 1) * D);
        }
        evox_ref_dtlz1_rows(XR + N * D, N, D, M, FR + N * M);
        const int32_t nf = evox_ref_nds(FR, R, M, fr);
        evox_ref_crowding(FR, R, M, fr, cr);
        int64_t taken = 0;
        for (int64_t i = 0; i < R; ++i) keep[i] = 0;
        for (int32_t k = 0; k < nf && taken < N; ++k) {
            int64_t size = 0;
            for (int64_t i = 0; i < R; ++i) size += fr[i] == k;
            if (taken + size <= N) {
                for (int64_t i = 0; i < R; ++i)
                    if (fr[i] == k) keep[i] = 1;
                taken += size;
            } else {
                /* members of front k by (crowding descending, index) */
                while (taken < N) {
                    int64_t best = -1;
                    for (int64_t i = 0; i < R; ++i)
                        if (fr[i] == k && !keep[i] && (best < 0 || cr[i] > cr[best])) best = i;
                    keep[best] = 1;
                    ++taken;
                }
            }
        }
        int64_t q = 0;
        for (int64_t i = 0; i < R; ++i)
            if (keep[i]) {
                memcpy(X + q * D, XR + i * D, sizeof(float) * (size_t)D);
                memcpy(F + q * M, FR + i * M, sizeof(float) * (size_t)M);
                front[q] = fr[i];
                crowd[q] = cr[i];
                ++q;
            }
    }
    free(XR); free(FR); free(fr); free(cr); free(keep);
    return 0;
}
