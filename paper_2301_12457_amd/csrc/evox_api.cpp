// C ABI of the gfx950 population-optimizer hot path (include/evox.h):
// validation, scratch planning, and the launch sequences of one generation.
#include "evox.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <limits>
#include <mutex>
#include <utility>
#include <vector>

#include "evox_launch.hpp"

using namespace evox;

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int hip_fail(hipError_t e, const char *what)
{
    return fail(EVOX_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }
size_t round256(size_t n) { return (n + 255) & ~(size_t)255; }

// Superbuckets of the pairing sort: about 512-1024 individuals each.
int perm_bits(int64_t N)
{
    int bits = 0;
    while ((N >> bits) > 1024 && bits < kPermMaxBits) ++bits;
    return bits;
}

// Blocks of the CSO kernels (one fp64 column-sum row each): at most 16384
// and at most 2^24 doubles of partial sums.
int cso_grid_cap(int64_t ldx)
{
    int64_t cap = ((int64_t)1 << 24) / ldx;
    if (cap > 16384) cap = 16384;
    if (cap < 64) cap = 64;
    return (int)cap;
}

int grid_for(int64_t groups, int G, int64_t cap)
{
    const int64_t rpb = block_for(G) / G;
    int64_t g = (groups + rpb - 1) / rpb;
    if (g > cap) g = cap;
    if (g < 1) g = 1;
    return (int)g;
}

template <typename T>
T *at_off(void *base, size_t off)
{
    return reinterpret_cast<T *>(static_cast<char *>(base) + off);
}

struct Plan {
    Layout L{0, 0, 0};
    int grid = 0, cso_grid = 0, colsum_grid = 0, bits = 0;
    size_t best = 0, slots = 0;
    size_t hist = 0, offs = 0, cursor = 0, tkv = 0, perm = 0, xsum = 0, s1 = 0, ticket = 0;
    int64_t xsum_rows = 0;
    int perm_batch = 0;
    size_t x2 = 0, fit2 = 0;  // DE: the other population buffer and its fitness
    size_t xalt = 0;          // CSO neighbourhood version: the other population buffer
    size_t mate = 0, cfit2 = 0;  // CSO: mate arrays, the other fitness buffer
    size_t esrank = 0, espart = 0;  // ES: sample ranks, gradient partial sums
    // MA-ES: deviates, steps, split-K workspace, update factors, parents,
    // weights, path-norm partial sums
    size_t mae_z = 0, mae_d = 0, mae_work = 0, mae_at = 0, mae_bt = 0, mae_sel = 0, mae_w = 0, mae_part = 0;
    size_t mae_wpart = 0;
    int mae_splits = 1;
    int64_t mae_mu = 0, mae_kp = 0, mae_ldf = 0;
    // NSGA-II: offspring, survivors' rows, merged objectives / fronts /
    // crowding, the sorting scratch, survivor flags and their prefix sums
    size_t ns_q = 0, ns_x2 = 0, ns_fr = 0, ns_frontr = 0, ns_crowdr = 0, ns_keep = 0, ns_pre = 0, ns_sums = 0;
    size_t ns_cnt = 0, ns_list = 0, ns_foff = 0, ns_pos = 0, ns_sorted = 0, ns_len = 0;
    size_t total = 0;
};

// Scratch of the non-dominated sorting of n points with M objectives,
// placed from `off` on: counts, the front-ordered list, front offsets, the
// per-objective positions and orders, the list length.
struct NsgaSortScratch {
    size_t cnt, list, foff, pos, sorted, len, end;
};
NsgaSortScratch nsga_sort_layout(int64_t n, int32_t M, size_t off)
{
    NsgaSortScratch l{};
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off = round256(off + bytes);
        return at;
    };
    l.cnt = take(4 * (size_t)n);
    l.list = take(4 * (size_t)n);
    l.foff = take(4 * ((size_t)n + 1));
    l.pos = take(4 * (size_t)M * (size_t)n);
    l.sorted = take(4 * (size_t)M * (size_t)n);
    l.len = take(4 * (size_t)kNsgaPeelBatch);
    l.end = off;
    return l;
}

NsgaSortArgs nsga_sort_args(void *scratch, const NsgaSortScratch &l, const float *F, int64_t n, int32_t M,
                            int32_t *front, double *crowd)
{
    return NsgaSortArgs{F, n, M, front, crowd, at_off<uint32_t>(scratch, l.cnt), at_off<int32_t>(scratch, l.list),
                        at_off<int32_t>(scratch, l.foff), at_off<int32_t>(scratch, l.pos),
                        at_off<int32_t>(scratch, l.sorted), n, at_off<uint32_t>(scratch, l.len)};
}

// K-slices of the sampling product (N + 1) x D x D: a small population gives
// few output tiles, so the product is split along K until the blocks fill
// the chip -- a whole number of rounds of resident blocks when the occupancy
// is known (a partial last round idles most of the chip), else about 1024
// blocks -- with every slice at least 256 deep.
int mae_splits(int64_t N, int64_t D, int64_t resident)
{
    const int64_t rows = N + 1, bm = rows <= 64 ? 64 : rows <= 112 ? 112 : 128, bn = rows <= 128 ? 64 : 128;
    const int64_t tiles = ((D + bn - 1) / bn) * ((rows + bm - 1) / bm);
    int64_t sp = resident > 0 ? resident / tiles : (1024 + tiles - 1) / tiles;
    const int64_t deep = D / 256 > 1 ? D / 256 : 1;
    if (sp > deep) sp = deep;
    if (sp > 16) sp = 16;
    return (int)(sp < 1 ? 1 : sp);
}

// Blocks of the sampling product's thin tile shape resident on the device at
// once (0 if unknown).
int64_t resident_thin_blocks(int64_t M)
{
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    return (int64_t)cus * occupancy_gemm_nt_thin(M);
}

int make_plan(const evox_params *P, Plan *pl)
{
    if (!P) return fail(EVOX_EINVAL, "params is null");
    if (P->algo != EVOX_PSO && P->algo != EVOX_CSO && P->algo != EVOX_DE && P->algo != EVOX_ES &&
        P->algo != EVOX_PGPE && P->algo != EVOX_MAES && P->algo != EVOX_NSGA2)
        return fail(EVOX_EINVAL, "unknown algo %d", P->algo);
    const bool es_like = P->algo == EVOX_ES || P->algo == EVOX_PGPE;
    if (P->fn_id < 0 || P->fn_id >= FN_COUNT) return fail(EVOX_EINVAL, "unknown fn_id %d", P->fn_id);
    const int64_t nmin = P->algo == EVOX_CSO ? 2 : P->algo == EVOX_DE ? 4 : 1;
    if (P->N < nmin || P->N >= ((int64_t)1 << 31))
        return fail(EVOX_EINVAL, "N = %lld out of range [%lld, 2^31)", (long long)P->N, (long long)nmin);
    if (P->D < 1 || P->D > EVOX_MAX_D)
        return fail(EVOX_EINVAL, "D = %lld out of range [1, %d]", (long long)P->D, EVOX_MAX_D);
    if (P->algo == EVOX_CSO && P->N > kCsoMaxN)
        return fail(EVOX_EINVAL, "CSO N = %lld above %lld", (long long)P->N, (long long)kCsoMaxN);
    if (es_like && (P->N < 2 || (P->N & 1) || P->N > kEsMaxN))
        return fail(EVOX_EINVAL, "ES / PGPE N = %lld must be even, in [2, %d]", (long long)P->N, kEsMaxN);
    if (P->algo == EVOX_MAES && (P->N < 2 || P->N > kEsMaxN))
        return fail(EVOX_EINVAL, "MAES N = %lld out of range [2, %d]", (long long)P->N, kEsMaxN);
    if (P->algo == EVOX_NSGA2) {
        if (P->N < 4 || (P->N & 1) || P->N > kNsgaMaxN)
            return fail(EVOX_EINVAL, "NSGA2 N = %lld must be even, in [4, %lld]", (long long)P->N,
                        (long long)kNsgaMaxN);
        if (P->n_obj < 2 || P->n_obj > kNsgaMaxM || P->D < P->n_obj)
            return fail(EVOX_EINVAL, "NSGA2 n_obj = %d must be in [2, %d] and <= D", P->n_obj, kNsgaMaxM);
        if (!(P->sbx_eta >= 0.0f) || !(P->pm_eta >= 0.0f))
            return fail(EVOX_EINVAL, "NSGA2 distribution indices must be >= 0");
    }
    if (P->ldx < P->D || (P->ldx & 3))
        return fail(EVOX_EINVAL, "ldx = %lld must be >= D and a multiple of 4", (long long)P->ldx);
    if (P->x_init != 0 && P->x_init != 1) return fail(EVOX_EINVAL, "unknown x_init %d", P->x_init);
    if (P->cso_local != 0 && (P->cso_local != 1 || P->algo != EVOX_CSO))
        return fail(EVOX_EINVAL, "cso_local = %d: 0, or 1 for CSO", P->cso_local);
    Plan p;
    const int family = P->algo == EVOX_CSO ? LAYOUT_CSO : LAYOUT_PSO;
    if (!row_layout(P->D, family, &p.L)) return fail(EVOX_EINVAL, "no row layout for D = %lld", (long long)P->D);
    p.grid = grid_for(es_like ? P->N / 2 : P->N, p.L.G, kMaxGrid);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off = round256(off + bytes);
        return at;
    };
    p.best = take(sizeof(DevBest));
    p.slots = take(sizeof(SelSlots));
    if (P->algo == EVOX_CSO) {
        const int cap = cso_grid_cap(P->ldx);
        // both versions sweep ranges of individuals
        int64_t ranges = (P->N + kCsoSweep - 1) / kCsoSweep;
        p.cso_grid = (int)(ranges > cap ? cap : ranges);
        p.colsum_grid = grid_for(P->N, p.L.G, cap);
        p.bits = perm_bits(P->N);
        // permutations and their mate arrays sorted kPermBatch generations
        // at a time, within 256 MB
        const int64_t per = 16;
        int64_t batch = ((int64_t)256 << 20) / (per * P->N);
        p.perm_batch = (int)(batch < 1 ? 1 : batch > kPermBatch ? kPermBatch : batch);
        const size_t B = (size_t)p.perm_batch, nb = (size_t)1 << p.bits;
        p.hist = take(4 * nb * B);
        p.offs = take(4 * (nb + 1) * B);
        p.cursor = take(4 * nb * B);
        p.tkv = take(8 * (size_t)P->N * B);
        p.perm = take(4 * (size_t)P->N * B);
        p.mate = take(4 * (size_t)P->N * B);
        p.cfit2 = take(sizeof(float) * (size_t)P->N);
        p.xsum_rows = cap;
        p.xsum = take(sizeof(double) * (size_t)cap * (size_t)P->ldx);
        p.s1 = take(sizeof(double) * (size_t)kMeanStages * (size_t)P->ldx);
        p.ticket = take(sizeof(uint32_t) * (size_t)((P->ldx + 63) / 64));
        if (P->cso_local) p.xalt = take(sizeof(float) * (size_t)P->N * (size_t)P->ldx);
    }
    if (P->algo == EVOX_DE) {
        p.x2 = take(sizeof(float) * (size_t)P->N * (size_t)P->ldx);
        p.fit2 = take(sizeof(float) * (size_t)P->N);
    }
    if (es_like) {
        const size_t H = (size_t)P->N / 2, chunks = (H + kEsPairChunk - 1) / kEsPairChunk;
        const size_t sums = P->algo == EVOX_PGPE ? 2 : 1;  // PGPE: center and deviation gradients
        p.esrank = take(sizeof(uint32_t) * 2 * H);
        p.espart = take(sizeof(double) * sums * chunks * 4 * (size_t)((P->D + 3) / 4));
    }
    if (P->algo == EVOX_MAES) {
        const size_t rows = (size_t)P->N + 1, D = (size_t)P->D;
        p.mae_mu = P->N / 2;
        // factor terms: ceil((mu + 1) / 2) steps of two when an unrolled rank
        // kernel exists for that count, else a multiple of 32 terms
        const int64_t steps = (p.mae_mu + 2) / 2;
        p.mae_kp = steps <= kMaeRankUnrolled ? 2 * steps : (p.mae_mu + 1 + 31) / 32 * 32;
        p.mae_ldf = (P->D + 127) / 128 * 128;
        p.mae_splits = mae_splits(P->N, P->D, resident_thin_blocks(P->N + 1));
        p.mae_z = take(sizeof(float) * rows * (size_t)P->ldx);
        p.mae_d = take(sizeof(float) * rows * (size_t)P->ldx);
        p.mae_work = p.mae_splits > 1 ? take(sizeof(float) * (size_t)p.mae_splits * rows * D) : 0;
        p.mae_at = take(sizeof(float) * (size_t)p.mae_ldf * (size_t)p.mae_kp);
        p.mae_bt = take(sizeof(float) * (size_t)p.mae_ldf * (size_t)p.mae_kp);
        p.esrank = take(sizeof(uint32_t) * (size_t)P->N);
        p.mae_sel = take(sizeof(int32_t) * (size_t)p.mae_mu);
        p.mae_w = take(sizeof(double) * (size_t)p.mae_mu);
        p.mae_part = take(sizeof(double) * ((D + kMaeBlock - 1) / kMaeBlock));
        p.mae_wpart = take(sizeof(double) * 2 * D * (size_t)((p.mae_mu + kMaeChunk - 1) / kMaeChunk));
    }
    if (P->algo == EVOX_NSGA2) {
        const size_t N = (size_t)P->N, R = 2 * N, M = (size_t)P->n_obj;
        p.ns_q = take(sizeof(float) * N * (size_t)P->ldx);
        p.ns_x2 = take(sizeof(float) * N * (size_t)P->ldx);
        p.ns_fr = take(sizeof(float) * R * M);
        p.ns_frontr = take(sizeof(int32_t) * R);
        p.ns_crowdr = take(sizeof(double) * R);
        p.ns_keep = take(sizeof(int32_t) * R);
        p.ns_pre = take(sizeof(int32_t) * R);
        p.ns_sums = take(sizeof(int32_t) * ((R + 1023) / 1024));
        const NsgaSortScratch l = nsga_sort_layout((int64_t)R, P->n_obj, off);
        p.ns_cnt = l.cnt;
        p.ns_list = l.list;
        p.ns_foff = l.foff;
        p.ns_pos = l.pos;
        p.ns_sorted = l.sorted;
        p.ns_len = l.len;
        off = l.end;
    }
    p.total = off;
    *pl = p;
    return EVOX_OK;
}

}  // namespace

struct evox_state {
    evox_params P;
    evox_buffers B;
    hipStream_t stream;
    int64_t t;
    Plan pl;
    uint32_t k0, k1;
    DevBest *best;
    SelSlots *slots;
    uint32_t *hist, *offs, *cursor, *perm, *ticket;
    uint32_t *mate;    // CSO: mate arrays of the permutation batch
    float *cfit2;      // CSO: the other fitness buffer
    uint2 *tkv;
    int64_t perm_t0;  // first generation of the stored permutation batch (-1: none)
    double *xsum, *s1;
    float *x2, *fit2;  // DE: the other population buffer
    uint32_t *esrank;  // ES: sample ranks
    double *espart;    // ES: gradient partial sums
    MaeArgs mae;       // MA-ES: the generation's buffers and constants (t set per generation)
    float mae_beta;    // 1 - (c_1 + c_w) / 2
    float *mae_work;
    std::vector<double> mae_w;  // the weights, host copy of the device table
    NsgaSortArgs ns_sort;       // NSGA-II: sorting of the merged population
    NsgaSelArgs ns_sel;         // NSGA-II: survivor selection
    // profiling of the fused generation kernel
    bool prof;
    std::vector<std::pair<hipEvent_t, hipEvent_t>> ev;
    size_t ev_used;
    int64_t prof_gens;  // generations performed by the timed launches
    uint64_t improved_base;
};

namespace {

template <typename T>
T *at(void *base, size_t off)
{
    return reinterpret_cast<T *>(static_cast<char *>(base) + off);
}

// Enqueue `launch` bracketed by profiling events when enabled; the launch
// performs `gens` generations.
template <typename F>
hipError_t timed(evox_state *s, F &&launch, int64_t gens = 1)
{
    if (!s->prof) return launch();
    s->prof_gens += gens;
    if (s->ev_used == s->ev.size()) {
        hipEvent_t a, b;
        hipError_t e = hipEventCreate(&a);
        if (e != hipSuccess) return e;
        e = hipEventCreate(&b);
        if (e != hipSuccess) return e;
        s->ev.emplace_back(a, b);
    }
    auto &pr = s->ev[s->ev_used++];
    hipError_t e = hipEventRecord(pr.first, s->stream);
    if (e != hipSuccess) return e;
    e = launch();
    if (e != hipSuccess) return e;
    return hipEventRecord(pr.second, s->stream);
}

hipError_t best_init(evox_state *s, float f, int64_t i) { return launch_best_init(s->best, f, i, s->stream); }

PsoArgs pso_args(evox_state *s)
{
    const evox_params &P = s->P;
    PsoArgs a{};
    a.x = s->B.x;
    a.v = s->B.v;
    a.p = s->B.pbest;
    a.pf = s->B.pfit;
    a.fit = s->B.fit;
    a.gbest = s->B.gbest;
    a.N = P.N;
    a.D = P.D;
    a.ldx = P.ldx;
    a.w = P.w;
    a.c1 = P.c1;
    a.c2 = P.c2;
    a.vmax = P.vmax;
    a.lb = P.lb;
    a.ub = P.ub;
    a.vclamp = P.vmax > 0.0f;
    a.xclamp = P.clamp_x != 0;
    a.k0 = s->k0;
    a.k1 = s->k1;
    a.t = 0;
    a.slots = s->slots;
    a.nt = 20 * P.N * P.D > kStreamBytes;
    return a;
}

// Swarm mean from nparts partial rows; also the selection from the slots.
// First-stage blocks per column tile: a power of two near nparts / 32, so
// that a first-stage lane sums about 8 partial rows (one batch of loads) and
// the last block about as few stage sums (at most kMeanStages blocks).
MeanArgs mean_args(evox_state *s, int nparts)
{
    int stages = 4;
    while (stages < kMeanStages && 32 * (int64_t)stages < nparts) stages *= 2;
    return MeanArgs{s->xsum, nparts, s->P.N, s->P.D, s->P.ldx, s->B.xbar, s->s1, stages, s->ticket, s->slots,
                    s->best};
}

// CSO: fit (optional), swarm mean and best of the current positions.
int cso_refresh(evox_state *s, bool refit)
{
    const evox_params &P = s->P;
    const Plan &pl = s->pl;
    hipError_t e;
    if (refit) {
        EvalArgs ea{s->B.x, P.N, P.D, P.ldx, s->B.fit, nullptr, 4 * P.N * P.ldx > kStreamBytes};
        if ((e = launch_eval(P.fn_id, pl.L, true, ea, pl.grid, s->stream)) != hipSuccess)
            return hip_fail(e, "evaluate");
    }
    if ((e = launch_colsum(pl.L, s->B.x, P.N, P.D, P.ldx, s->xsum, pl.colsum_grid, s->stream)) != hipSuccess)
        return hip_fail(e, "column sums");
    if ((e = launch_argmin_slots(s->B.fit, P.N, s->slots, s->stream)) != hipSuccess)
        return hip_fail(e, "select");
    if ((e = launch_cso_mean(mean_args(s, pl.colsum_grid), s->stream)) != hipSuccess)
        return hip_fail(e, "swarm mean");
    return EVOX_OK;
}

}  // namespace

extern "C" {

size_t evox_scratch_bytes(const evox_params *params)
{
    Plan pl;
    if (make_plan(params, &pl) != EVOX_OK) return 0;
    return pl.total;
}

int evox_state_create(const evox_params *params, const evox_buffers *b, void *hip_stream,
                      evox_state **out)
{
    if (!out) return fail(EVOX_EINVAL, "out is null");
    *out = nullptr;
    Plan pl;
    int rc = make_plan(params, &pl);
    if (rc != EVOX_OK) return rc;
    const evox_params &P = *params;
    if (!b) return fail(EVOX_EINVAL, "buffers is null");
    if (!b->x || !b->scratch) return fail(EVOX_EINVAL, "x and scratch are required");
    if ((P.algo == EVOX_PSO || P.algo == EVOX_CSO) && !b->v) return fail(EVOX_EINVAL, "PSO and CSO need v");
    if ((P.algo == EVOX_DE || P.algo == EVOX_ES || P.algo == EVOX_PGPE || P.algo == EVOX_MAES) && !b->fit)
        return fail(EVOX_EINVAL, "DE, ES, PGPE and MAES need fit");
    if (P.algo == EVOX_MAES && (!b->v || !b->mat || !b->sigma))
        return fail(EVOX_EINVAL, "MAES needs v (the path), mat and sigma");
    if (P.algo == EVOX_NSGA2 && (!b->obj || !b->front || !b->crowd))
        return fail(EVOX_EINVAL, "NSGA2 needs obj, front and crowd");
    if (P.algo == EVOX_PGPE && !b->v) return fail(EVOX_EINVAL, "PGPE needs v (the deviations)");
    if (P.algo == EVOX_PSO && (!b->pbest || !b->pfit || !b->gbest))
        return fail(EVOX_EINVAL, "PSO needs pbest, pfit and gbest");
    if (P.algo == EVOX_CSO && (!b->fit || !b->xbar)) return fail(EVOX_EINVAL, "CSO needs fit and xbar");
    const void *ptrs[] = {b->x, b->v, b->pbest, b->pfit, b->fit, b->gbest, b->xbar, b->mat, b->sigma, b->obj,
                          b->front, b->crowd};
    for (const void *p : ptrs)
        if (p && !aligned16(p)) return fail(EVOX_EALIGN, "buffer %p is not 16-byte aligned", p);
    if (((uintptr_t)b->scratch & 255u) != 0) return fail(EVOX_EALIGN, "scratch is not 256-byte aligned");
    if (b->scratch_bytes < pl.total)
        return fail(EVOX_ENOSPC, "scratch has %zu bytes, needs %zu", b->scratch_bytes, pl.total);

    evox_state *s = new evox_state();
    s->P = P;
    s->B = *b;
    s->stream = (hipStream_t)hip_stream;
    s->t = 0;
    s->pl = pl;
    s->k0 = (uint32_t)P.seed;
    s->k1 = (uint32_t)(P.seed >> 32);
    s->best = at<DevBest>(b->scratch, pl.best);
    s->slots = at<SelSlots>(b->scratch, pl.slots);
    s->hist = s->offs = s->cursor = s->perm = s->mate = nullptr;
    s->cfit2 = nullptr;
    s->tkv = nullptr;
    s->xsum = s->s1 = nullptr;
    s->perm_t0 = -1;
    s->ticket = nullptr;
    s->x2 = s->fit2 = nullptr;
    s->esrank = nullptr;
    s->espart = nullptr;
    if (P.algo == EVOX_ES || P.algo == EVOX_PGPE) {
        s->esrank = at<uint32_t>(b->scratch, pl.esrank);
        s->espart = at<double>(b->scratch, pl.espart);
    }
    if (P.algo == EVOX_DE) {
        s->x2 = at<float>(b->scratch, pl.x2);
        s->fit2 = at<float>(b->scratch, pl.fit2);
    }
    s->mae = MaeArgs{};
    s->mae_beta = 1.0f;
    s->mae_work = nullptr;
    if (P.algo == EVOX_MAES) {
        // Hansen's default strategy constants for N samples in D dimensions
        const int64_t mu = pl.mae_mu;
        const double n = (double)P.D;
        double sw = 0.0, sw2 = 0.0;
        s->mae_w.resize((size_t)mu);
        for (int64_t i = 0; i < mu; ++i) sw += std::log((double)mu + 0.5) - std::log((double)(i + 1));
        for (int64_t i = 0; i < mu; ++i) {
            s->mae_w[(size_t)i] = (std::log((double)mu + 0.5) - std::log((double)(i + 1))) / sw;
            sw2 += s->mae_w[(size_t)i] * s->mae_w[(size_t)i];
        }
        const double me = 1.0 / sw2, cs = (me + 2.0) / (n + me + 5.0);
        const double ds = 1.0 + cs + 2.0 * std::fmax(0.0, std::sqrt((me - 1.0) / (n + 1.0)) - 1.0);
        const double c1 = 2.0 / ((n + 1.3) * (n + 1.3) + me);
        const double cw = std::fmin(1.0 - c1, 2.0 * (me - 2.0 + 1.0 / me) / ((n + 2.0) * (n + 2.0) + me));
        MaeArgs &m = s->mae;
        m.Z = at<float>(b->scratch, pl.mae_z);
        m.Dm = at<float>(b->scratch, pl.mae_d);
        m.N = P.N;
        m.D = P.D;
        m.ldx = P.ldx;
        m.mu = mu;
        m.kp = pl.mae_kp;
        m.ldf = pl.mae_ldf;
        s->esrank = at<uint32_t>(b->scratch, pl.esrank);
        m.rank = s->esrank;
        m.sel = at<int32_t>(b->scratch, pl.mae_sel);
        m.w = at<double>(b->scratch, pl.mae_w);
        m.y = b->x;
        m.s = b->v;
        m.sigma = b->sigma;
        m.At = at<float>(b->scratch, pl.mae_at);
        m.Bt = at<float>(b->scratch, pl.mae_bt);
        m.part = at<double>(b->scratch, pl.mae_part);
        m.wpart = at<double>(b->scratch, pl.mae_wpart);
        m.cs = cs;
        m.cz = std::sqrt(me * cs * (2.0 - cs));
        m.hc1 = 0.5 * c1;
        m.hcw = 0.5 * cw;
        m.damp = cs / ds;
        m.chi = std::sqrt(n) * (1.0 - 1.0 / (4.0 * n) + 1.0 / (21.0 * n * n));
        m.k0 = s->k0;
        m.k1 = s->k1;
        s->mae_beta = (float)(1.0 - 0.5 * (c1 + cw));
        if (pl.mae_splits > 1) s->mae_work = at<float>(b->scratch, pl.mae_work);
    }
    s->ns_sort = NsgaSortArgs{};
    s->ns_sel = NsgaSelArgs{};
    if (P.algo == EVOX_NSGA2) {
        const int64_t R = 2 * P.N;
        float *FR = at<float>(b->scratch, pl.ns_fr);
        int32_t *frontR = at<int32_t>(b->scratch, pl.ns_frontr);
        double *crowdR = at<double>(b->scratch, pl.ns_crowdr);
        s->ns_sort = NsgaSortArgs{FR, R, P.n_obj, frontR, crowdR, at<uint32_t>(b->scratch, pl.ns_cnt),
                                  at<int32_t>(b->scratch, pl.ns_list), at<int32_t>(b->scratch, pl.ns_foff),
                                  at<int32_t>(b->scratch, pl.ns_pos), at<int32_t>(b->scratch, pl.ns_sorted), R,
                                  at<uint32_t>(b->scratch, pl.ns_len)};
        s->ns_sel = NsgaSelArgs{b->x, at<float>(b->scratch, pl.ns_q), P.N, P.ldx, P.n_obj, FR, frontR, crowdR,
                                s->ns_sort.list, at<int32_t>(b->scratch, pl.ns_keep),
                                at<int32_t>(b->scratch, pl.ns_pre), s->ns_sort.pos,
                                at<int32_t>(b->scratch, pl.ns_sums), at<float>(b->scratch, pl.ns_x2), b->obj,
                                b->front, b->crowd};
    }
    if (P.algo == EVOX_CSO) {
        s->hist = at<uint32_t>(b->scratch, pl.hist);
        s->offs = at<uint32_t>(b->scratch, pl.offs);
        s->cursor = at<uint32_t>(b->scratch, pl.cursor);
        s->tkv = at<uint2>(b->scratch, pl.tkv);
        s->perm = at<uint32_t>(b->scratch, pl.perm);
        s->mate = at<uint32_t>(b->scratch, pl.mate);
        s->cfit2 = at<float>(b->scratch, pl.cfit2);
        s->xsum = at<double>(b->scratch, pl.xsum);
        s->s1 = at<double>(b->scratch, pl.s1);
        s->ticket = at<uint32_t>(b->scratch, pl.ticket);
    }
    s->prof = false;
    s->ev_used = 0;
    s->prof_gens = 0;
    s->improved_base = 0;
    if (P.algo == EVOX_CSO) {
        // persistent grid for the pair kernel: every block resident at once
        int dev = 0, cus = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess) {
            const int occ = occupancy_cso(P.fn_id, pl.L, P.cso_local != 0);
            const int64_t resident = (int64_t)cus * (occ > 0 ? occ : 1);
            if (resident < s->pl.cso_grid) s->pl.cso_grid = (int)resident;
        }
    }

    hipError_t e;
    // ES / PGPE: x is the center, one row
    const bool own_v = P.algo == EVOX_PSO || P.algo == EVOX_CSO;
    const bool es_like = P.algo == EVOX_ES || P.algo == EVOX_PGPE || P.algo == EVOX_MAES;
    const bool unit_box = P.algo == EVOX_NSGA2;  // DTLZ1's domain
    InitArgs ia{b->x, own_v ? b->v : nullptr, P.algo == EVOX_PSO ? b->pbest : nullptr,
                es_like ? 1 : P.N, P.D, P.ldx, unit_box ? 0.0f : P.lb, unit_box ? 1.0f : P.ub,
                P.v_lo, P.v_hi, P.v_lo == 0.0f && P.v_hi == 0.0f, P.x_init == 1, P.x_mu, P.x_sigma,
                s->k0, s->k1};
    if ((e = launch_init(ia, s->stream)) != hipSuccess) {
        delete s;
        return hip_fail(e, "init");
    }
    if ((e = launch_slots_init(s->slots, s->stream)) != hipSuccess) {
        delete s;
        return hip_fail(e, "init");
    }
    if (P.algo == EVOX_NSGA2) {
        // the offspring rows' padding stays zero; objectives, fronts and
        // crowding of the initial population
        NsgaSortArgs init = s->ns_sort;
        init.F = b->obj;
        init.n = P.N;
        init.front = b->front;
        init.crowd = b->crowd;
        NsgaSortResult r;
        if ((e = launch_fill(at<float>(b->scratch, pl.ns_q), P.N * P.ldx, 0.0f, s->stream)) != hipSuccess ||
            (e = launch_nsga_dtlz1(b->x, P.N, P.D, P.ldx, P.n_obj, b->obj, s->stream)) != hipSuccess ||
            (e = nsga_sort(init, P.N, &r, s->stream)) != hipSuccess) {
            delete s;
            return hip_fail(e, "init");
        }
    } else if (P.algo == EVOX_PSO) {
        if ((e = best_init(s, std::numeric_limits<float>::infinity(), 0)) != hipSuccess ||
            (e = launch_fill(b->pfit, P.N, std::numeric_limits<float>::infinity(), s->stream)) != hipSuccess ||
            (e = launch_copy_row(b->pbest, b->gbest, P.ldx, s->stream)) != hipSuccess) {
            delete s;
            return hip_fail(e, "init");
        }
    } else if (es_like) {
        // PGPE: v holds the deviations, es_sigma in every dimension (padding 0)
        if ((e = best_init(s, std::numeric_limits<float>::infinity(), 0)) != hipSuccess ||
            (P.algo == EVOX_PGPE && (e = launch_fill(b->v, P.ldx, 0.0f, s->stream)) != hipSuccess) ||
            (P.algo == EVOX_PGPE && (e = launch_fill(b->v, P.D, P.es_sigma, s->stream)) != hipSuccess)) {
            delete s;
            return hip_fail(e, "init");
        }
        // MA-ES: s = 0, M = I, sigma = es_sigma, the weight table
        if (P.algo == EVOX_MAES &&
            ((e = launch_fill(b->v, P.ldx, 0.0f, s->stream)) != hipSuccess ||
             (e = launch_mae_identity(b->mat, P.D, P.ldx, s->stream)) != hipSuccess ||
             (e = launch_fill(s->mae.At, s->mae.kp * s->mae.ldf, 0.0f, s->stream)) != hipSuccess ||
             (e = launch_fill(s->mae.Bt, s->mae.kp * s->mae.ldf, 0.0f, s->stream)) != hipSuccess ||
             (e = launch_fill(b->sigma, 1, P.es_sigma, s->stream)) != hipSuccess ||
             (e = hipMemcpyAsync((void *)s->mae.w, s->mae_w.data(), sizeof(double) * s->mae_w.size(),
                                 hipMemcpyHostToDevice, s->stream)) != hipSuccess ||
             (e = hipStreamSynchronize(s->stream)) != hipSuccess)) {
            delete s;
            return hip_fail(e, "init");
        }
    } else if (P.algo == EVOX_DE) {
        // the other buffer starts zero, so padding columns the kernels do
        // not reach stay zero in both; then fit = F(x) and the first best
        EvalArgs ea{b->x, P.N, P.D, P.ldx, b->fit, s->slots, 4 * P.N * P.ldx > kStreamBytes};
        if ((e = launch_fill(s->x2, P.N * P.ldx, 0.0f, s->stream)) != hipSuccess ||
            (e = best_init(s, std::numeric_limits<float>::infinity(), 0)) != hipSuccess ||
            (e = launch_eval(P.fn_id, pl.L, true, ea, pl.grid, s->stream)) != hipSuccess ||
            (e = launch_select(s->slots, nullptr, 0, nullptr, s->best, nullptr, nullptr, s->stream)) != hipSuccess) {
            delete s;
            return hip_fail(e, "init");
        }
    } else {
        const size_t nb = ((size_t)1 << pl.bits) * (size_t)pl.perm_batch;
        // the neighbourhood version's other population buffer starts zero,
        // so the padding columns the kernels never write stay zero in both
        if ((P.cso_local && (e = launch_fill(at<float>(b->scratch, pl.xalt), P.N * P.ldx, 0.0f, s->stream)) !=
                                hipSuccess) ||
            (e = launch_zero_u32(s->hist, (int64_t)nb, s->stream)) != hipSuccess ||
            (e = launch_zero_u32(s->cursor, (int64_t)nb, s->stream)) != hipSuccess ||
            (e = launch_zero_u32(s->ticket, (P.ldx + 63) / 64, s->stream)) != hipSuccess ||
            // every mate entry is an index below N or kUnpaired at all times
            (s->mate && (e = launch_fill_u32(s->mate, P.N * pl.perm_batch, kUnpaired, s->stream)) != hipSuccess) ||
            (e = best_init(s, std::numeric_limits<float>::infinity(), 0)) != hipSuccess) {
            delete s;
            return hip_fail(e, "init");
        }
        rc = cso_refresh(s, true);
        if (rc != EVOX_OK) {
            delete s;
            return rc;
        }
    }
    *out = s;
    return EVOX_OK;
}

int evox_state_destroy(evox_state *s)
{
    if (!s) return fail(EVOX_EINVAL, "state is null");
    for (auto &pr : s->ev) {
        (void)hipEventDestroy(pr.first);
        (void)hipEventDestroy(pr.second);
    }
    delete s;
    return EVOX_OK;
}

static int eval_common(int fn_id, const float *X, int64_t N, int64_t D, int64_t ldx, float *out,
                       SelSlots *slots, hipStream_t st)
{
    if (fn_id < 0 || fn_id >= FN_COUNT) return fail(EVOX_EINVAL, "unknown fn_id %d", fn_id);
    if (N < 0 || N >= ((int64_t)1 << 31)) return fail(EVOX_EINVAL, "N = %lld out of range", (long long)N);
    if (D < 1 || D > EVOX_MAX_D) return fail(EVOX_EINVAL, "D = %lld out of range [1, %d]", (long long)D, EVOX_MAX_D);
    if (ldx < D) return fail(EVOX_EINVAL, "ldx = %lld < D", (long long)ldx);
    if (N > 0 && (!X || !out)) return fail(EVOX_EINVAL, "X and out are required");
    Layout L;
    if (!row_layout(D, LAYOUT_EVAL, &L)) return fail(EVOX_EINVAL, "no row layout for D = %lld", (long long)D);
    const int grid = grid_for(N, L.G, kMaxGrid);
    if (N == 0) return EVOX_OK;
    const bool vec = (ldx & 3) == 0 && aligned16(X);
    EvalArgs a{X, N, D, ldx, out, slots, 4 * N * ldx > kStreamBytes};
    hipError_t e = launch_eval(fn_id, L, vec, a, grid, st);
    if (e != hipSuccess) return hip_fail(e, "evaluate");
    return EVOX_OK;
}

int evox_eval(int fn_id, const float *X, int64_t N, int64_t D, float *out, void *hip_stream)
{
    return eval_common(fn_id, X, N, D, D, out, nullptr, (hipStream_t)hip_stream);
}

int evox_eval_ld(int fn_id, const float *X, int64_t N, int64_t D, int64_t ldx, float *out,
                 void *hip_stream)
{
    return eval_common(fn_id, X, N, D, ldx, out, nullptr, (hipStream_t)hip_stream);
}

size_t evox_eval_argmin_scratch_bytes(int64_t)
{
    return round256(sizeof(SelSlots));
}

int evox_eval_argmin(int fn_id, const float *X, int64_t N, int64_t D, int64_t ldx, float *out,
                     float *best_fit_dev, int64_t *best_idx_dev, void *scratch, size_t scratch_bytes,
                     void *hip_stream)
{
    if (N < 1 || N >= ((int64_t)1 << 31))
        return fail(EVOX_EINVAL, "N = %lld out of range [1, 2^31) for a selection", (long long)N);
    if (!best_fit_dev || !best_idx_dev || !scratch) return fail(EVOX_EINVAL, "best outputs and scratch are required");
    if (((uintptr_t)scratch & 255u) != 0) return fail(EVOX_EALIGN, "scratch is not 256-byte aligned");
    if (scratch_bytes < evox_eval_argmin_scratch_bytes(N))
        return fail(EVOX_ENOSPC, "scratch has %zu bytes, needs %zu", scratch_bytes, evox_eval_argmin_scratch_bytes(N));
    SelSlots *slots = at<SelSlots>(scratch, 0);
    hipStream_t st = (hipStream_t)hip_stream;
    // validate before enqueueing anything
    int rc = eval_common(fn_id, nullptr, 0, D, ldx, nullptr, nullptr, st);
    if (rc != EVOX_OK) return rc;
    if (!X || !out) return fail(EVOX_EINVAL, "X and out are required");
    hipError_t e = launch_slots_init(slots, st);
    if (e != hipSuccess) return hip_fail(e, "select init");
    rc = eval_common(fn_id, X, N, D, ldx, out, slots, st);
    if (rc != EVOX_OK) return rc;
    e = launch_select(slots, nullptr, 0, nullptr, nullptr, best_fit_dev, best_idx_dev, st);
    if (e != hipSuccess) return hip_fail(e, "select");
    return EVOX_OK;
}

}  // extern "C"

namespace {

// Scratch of evox_eval_argmin_noalloc: the selection slots, one copy per
// device.  Host code never uses this name as an address: the device's own
// address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[EVOX_NOALLOC_SCRATCH_BYTES];
static_assert(sizeof(SelSlots) <= EVOX_NOALLOC_SCRATCH_BYTES, "selection slots fit the static scratch");

constexpr int kMaxDevices = 64;
std::mutex g_noalloc_mu;
void *g_noalloc_ptr[kMaxDevices] = {};

// The static scratch's address on device `dev` (the current device).
int noalloc_scratch(int dev, void **out)
{
    if (dev < 0 || dev >= kMaxDevices) return fail(EVOX_EINVAL, "device %d beyond the %d supported", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_noalloc_mu);
    if (!g_noalloc_ptr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "address of the static scratch");
        if (!p) return fail(EVOX_EHIP, "address of the static scratch is null");
        g_noalloc_ptr[dev] = p;
    }
    *out = g_noalloc_ptr[dev];
    return EVOX_OK;
}

}  // namespace

extern "C" {

int evox_eval_argmin_noalloc(int fn_id, const float *X, int64_t N, int64_t D, int64_t ldx, float *out,
                             float *best_fit_dev, int64_t *best_idx_dev, void *hip_stream)
{
    if (N < 1 || N >= ((int64_t)1 << 31))
        return fail(EVOX_EINVAL, "N = %lld out of range [1, 2^31) for a selection", (long long)N);
    if (!best_fit_dev || !best_idx_dev) return fail(EVOX_EINVAL, "best outputs are required");
    const size_t need = evox_eval_argmin_scratch_bytes(N);
    if (need > EVOX_NOALLOC_SCRATCH_BYTES)
        return fail(EVOX_ENOSPC, "N = %lld needs %zu scratch bytes, the static scratch holds %d", (long long)N, need,
                    EVOX_NOALLOC_SCRATCH_BYTES);
    hipStream_t st = (hipStream_t)hip_stream;
    // validate before enqueueing anything
    int rc = eval_common(fn_id, nullptr, 0, D, ldx, nullptr, nullptr, st);
    if (rc != EVOX_OK) return rc;
    if (!X || !out) return fail(EVOX_EINVAL, "X and out are required");
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "current device");
    if (st) {
        hipDevice_t sdev = -1;
        if ((e = hipStreamGetDevice(st, &sdev)) != hipSuccess) return hip_fail(e, "device of the stream");
        if ((int)sdev != dev)
            return fail(EVOX_EINVAL, "the stream belongs to device %d, the current device is %d", (int)sdev, dev);
    }
    void *ptr = nullptr;
    if ((rc = noalloc_scratch(dev, &ptr)) != EVOX_OK) return rc;
    SelSlots *slots = static_cast<SelSlots *>(ptr);
    if ((e = launch_slots_init(slots, st)) != hipSuccess) return hip_fail(e, "select init");
    rc = eval_common(fn_id, X, N, D, ldx, out, slots, st);
    if (rc != EVOX_OK) return rc;
    if ((e = launch_select(slots, nullptr, 0, nullptr, nullptr, best_fit_dev, best_idx_dev, st)) != hipSuccess)
        return hip_fail(e, "select");
    return EVOX_OK;
}

int evox_pso_step(evox_state *s, int64_t n_gens)
{
    if (!s) return fail(EVOX_EINVAL, "state is null");
    if (s->P.algo != EVOX_PSO) return fail(EVOX_EINVAL, "evox_pso_step on a CSO state");
    if (n_gens < 0) return fail(EVOX_EINVAL, "n_gens = %lld < 0", (long long)n_gens);
    if (s->t + n_gens >= ((int64_t)1 << 32)) return fail(EVOX_EINVAL, "generation counter would pass 2^32");
    if (n_gens == 0) return EVOX_OK;
    const Plan &pl = s->pl;
    const int fn = s->P.fn_id;
    PsoArgs a = pso_args(s);
    hipError_t e;
    if (pl.L.G <= 64 && s->P.N * s->P.D <= kPsoSmallElems && s->P.ldx <= kPsoSmallMaxLdx) {
        // a small swarm: the whole call in one block, one launch
        a.t = (uint32_t)s->t;
        e = timed(s, [&] { return launch_pso_small(fn, pl.L, a, n_gens, s->B.gbest, s->best, s->stream); }, n_gens);
        if (e != hipSuccess) return hip_fail(e, "pso generations");
        s->t += n_gens;
        return EVOX_OK;
    }
    // generation t: evaluate x_t, personal and global bests
    if ((e = launch_pso(fn, pl.L, PSO_EVAL, a, pl.grid, s->stream)) != hipSuccess) return hip_fail(e, "pso eval");
    if ((e = launch_select(s->slots, s->B.pbest, s->P.ldx, s->B.gbest, s->best, nullptr, nullptr,
                           s->stream)) != hipSuccess)
        return hip_fail(e, "select");
    for (int64_t k = 1; k < n_gens; ++k) {
        a.t = (uint32_t)(s->t + k - 1);  // move of generation t+k-1, evaluation of t+k
        e = timed(s, [&] { return launch_pso(fn, pl.L, PSO_FUSED, a, pl.grid, s->stream); });
        if (e != hipSuccess) return hip_fail(e, "pso generation");
        if ((e = launch_select(s->slots, s->B.pbest, s->P.ldx, s->B.gbest, s->best, nullptr, nullptr,
                               s->stream)) != hipSuccess)
            return hip_fail(e, "select");
    }
    a.t = (uint32_t)(s->t + n_gens - 1);
    if ((e = launch_pso(fn, pl.L, PSO_MOVE, a, pl.grid, s->stream)) != hipSuccess) return hip_fail(e, "pso move");
    s->t += n_gens;
    return EVOX_OK;
}

int evox_cso_step(evox_state *s, int64_t n_gens)
{
    if (!s) return fail(EVOX_EINVAL, "state is null");
    if (s->P.algo != EVOX_CSO) return fail(EVOX_EINVAL, "evox_cso_step on a PSO state");
    if (n_gens < 0) return fail(EVOX_EINVAL, "n_gens = %lld < 0", (long long)n_gens);
    if (s->t + n_gens >= ((int64_t)1 << 32)) return fail(EVOX_EINVAL, "generation counter would pass 2^32");
    const evox_params &P = s->P;
    const Plan &pl = s->pl;
    const bool local = P.cso_local != 0;
    hipError_t e;
    // both versions alternate the fitness between fit and a second buffer (a
    // generation reads every individual's fitness before it and writes every
    // one after it); the neighbourhood version also alternates the positions
    // between x and a second buffer (a loser's mean reads its neighbours'
    // rows as they were before the generation)
    float *cur = s->B.x, *alt = local ? at<float>(s->B.scratch, pl.xalt) : nullptr;
    float *fcur = s->B.fit;
    for (int64_t k = 0; k < n_gens; ++k) {
        const int64_t t = s->t + k;
        if (s->perm_t0 < 0 || t < s->perm_t0 || t >= s->perm_t0 + pl.perm_batch) {
            PermArgs pa{P.N, pl.bits, s->k0, s->k1, (uint32_t)t, (uint32_t)pl.perm_batch, s->hist, s->offs,
                        s->cursor, s->tkv, s->perm, nullptr, s->mate};
            if ((e = launch_perm(pa, s->stream)) != hipSuccess) return hip_fail(e, "pairing");
            s->perm_t0 = t;
        }
        const int64_t slice = (t - s->perm_t0) * P.N;
        float *dst = local ? (cur == s->B.x ? alt : s->B.x) : s->B.x;
        float *fnext = fcur == s->B.fit ? s->cfit2 : s->B.fit;
        CsoArgs ca{dst, s->B.v, fnext, fcur, s->B.xbar, s->perm + slice, s->mate + slice,
                   P.N, P.D, P.ldx, P.phi, P.lb, P.ub, P.clamp_x != 0, s->k0, s->k1, (uint32_t)t, s->slots,
                   s->xsum, cur};
        e = timed(s, [&] { return launch_cso(P.fn_id, pl.L, ca, pl.cso_grid, s->stream); });
        if (e != hipSuccess) return hip_fail(e, "cso generation");
        if ((e = launch_cso_mean(mean_args(s, pl.cso_grid), s->stream)) != hipSuccess)
            return hip_fail(e, "swarm mean");
        cur = dst;
        fcur = fnext;
    }
    // the caller's x and fit hold the state after the call
    if (cur != s->B.x && (e = launch_stream_copy(cur, s->B.x, P.N * P.ldx, s->stream)) != hipSuccess)
        return hip_fail(e, "positions");
    if (fcur != s->B.fit && (e = launch_stream_copy(fcur, s->B.fit, P.N, s->stream)) != hipSuccess)
        return hip_fail(e, "fitness");
    s->t += n_gens;
    return EVOX_OK;
}

int evox_de_step(evox_state *s, int64_t n_gens)
{
    if (!s) return fail(EVOX_EINVAL, "state is null");
    if (s->P.algo != EVOX_DE) return fail(EVOX_EINVAL, "evox_de_step on a PSO or CSO state");
    if (n_gens < 0) return fail(EVOX_EINVAL, "n_gens = %lld < 0", (long long)n_gens);
    if (s->t + n_gens >= ((int64_t)1 << 32)) return fail(EVOX_EINVAL, "generation counter would pass 2^32");
    if (n_gens == 0) return EVOX_OK;
    const evox_params &P = s->P;
    const Plan &pl = s->pl;
    hipError_t e;
    for (int64_t k = 0; k < n_gens; ++k) {
        // generation k reads one buffer and writes the other
        const bool even = (k & 1) == 0;
        DeArgs a{even ? s->B.x : s->x2, even ? s->B.fit : s->fit2, even ? s->x2 : s->B.x,
                 even ? s->fit2 : s->B.fit, P.N, P.D, P.ldx, P.de_f, P.de_cr, s->k0, s->k1,
                 (uint32_t)(s->t + k), k == n_gens - 1 ? s->slots : nullptr, 20 * P.N * P.D > kStreamBytes};
        e = timed(s, [&] { return launch_de(P.fn_id, pl.L, a, pl.grid, s->stream); });
        if (e != hipSuccess) return hip_fail(e, "de generation");
    }
    if ((e = launch_select(s->slots, nullptr, 0, nullptr, s->best, nullptr, nullptr, s->stream)) != hipSuccess)
        return hip_fail(e, "select");
    if (n_gens & 1) {  // the population ended in the other buffer: bring it home
        if ((e = launch_stream_copy(s->x2, s->B.x, P.N * P.ldx, s->stream)) != hipSuccess ||
            (e = launch_stream_copy(s->fit2, s->B.fit, P.N, s->stream)) != hipSuccess)
            return hip_fail(e, "de copy");
    }
    s->t += n_gens;
    return EVOX_OK;
}

}  // extern "C"

namespace {

// n_gens OpenES (pgpe false) or PGPE generations: samples and fitness,
// ranks, gradients and steps per generation; the selection after the last.
int es_generations(evox_state *s, int64_t n_gens, bool pgpe)
{
    if (n_gens < 0) return fail(EVOX_EINVAL, "n_gens = %lld < 0", (long long)n_gens);
    if (s->t + n_gens >= ((int64_t)1 << 32)) return fail(EVOX_EINVAL, "generation counter would pass 2^32");
    if (n_gens == 0) return EVOX_OK;
    const evox_params &P = s->P;
    const Plan &pl = s->pl;
    const uint32_t stream = pgpe ? STREAM_PGPE : STREAM_ES;
    float *sig = pgpe ? s->B.v : nullptr;
    hipError_t e;
    for (int64_t k = 0; k < n_gens; ++k) {
        const uint32_t t = (uint32_t)(s->t + k);
        EsArgs a{s->B.x, sig, s->B.fit, s->esrank, P.N, P.D, P.es_sigma, s->k0, s->k1, t, stream,
                 k == n_gens - 1 ? s->slots : nullptr};
        e = timed(s, [&] { return launch_es_eval(P.fn_id, pl.L, a, pl.grid, s->stream); });
        if (e != hipSuccess) return hip_fail(e, "samples");
        if ((e = launch_es_rank(s->B.fit, P.N, s->esrank, s->stream)) != hipSuccess) return hip_fail(e, "ranks");
        EsGradArgs ga{s->esrank, s->espart, s->B.x, sig, P.N / 2, P.D, P.es_sigma, P.es_lr,
                      P.pgpe_sigma_lr, P.pgpe_max_change, s->k0, s->k1, t, stream};
        if ((e = launch_es_grad(ga, s->stream)) != hipSuccess) return hip_fail(e, "gradient");
    }
    if ((e = launch_select(s->slots, nullptr, 0, nullptr, s->best, nullptr, nullptr, s->stream)) != hipSuccess)
        return hip_fail(e, "select");
    s->t += n_gens;
    return EVOX_OK;
}

int nsga_generations(evox_state *s, int64_t n_gens)
{
    if (n_gens < 0) return fail(EVOX_EINVAL, "n_gens = %lld < 0", (long long)n_gens);
    if (s->t + n_gens >= ((int64_t)1 << 32)) return fail(EVOX_EINVAL, "generation counter would pass 2^32");
    const evox_params &P = s->P;
    const int32_t M = P.n_obj;
    hipError_t e;
    for (int64_t k = 0; k < n_gens; ++k) {
        const uint32_t t = (uint32_t)(s->t + k);
        NsgaVarArgs va{s->B.x, P.N, P.D, P.ldx, s->B.front, s->B.crowd, at<float>(s->B.scratch, s->pl.ns_q),
                       (double)P.sbx_eta,
                       (double)P.pm_eta, s->k0, s->k1, t};
        NsgaSortResult r;
        if ((e = launch_nsga_var(va, s->stream)) != hipSuccess) return hip_fail(e, "variation");
        if ((e = launch_stream_copy(s->B.obj, (float *)s->ns_sort.F, P.N * M, s->stream)) != hipSuccess)
            return hip_fail(e, "merge");
        if ((e = launch_nsga_dtlz1(s->ns_sel.Q, P.N, P.D, P.ldx, M, (float *)s->ns_sort.F + P.N * M, s->stream)) !=
            hipSuccess)
            return hip_fail(e, "objectives");
        if ((e = timed(s, [&] { return nsga_count(s->ns_sort, s->stream); })) != hipSuccess ||
            (e = nsga_fronts(s->ns_sort, P.N, &r, s->stream)) != hipSuccess)
            return hip_fail(e, "non-dominated sorting");
        if ((e = launch_nsga_select(s->ns_sel, r, s->stream)) != hipSuccess) return hip_fail(e, "selection");
        if ((e = launch_stream_copy(s->ns_sel.X2, s->B.x, P.N * P.ldx, s->stream)) != hipSuccess)
            return hip_fail(e, "survivors");
    }
    s->t += n_gens;
    return EVOX_OK;
}

int mae_generations(evox_state *s, int64_t n_gens)
{
    if (n_gens < 0) return fail(EVOX_EINVAL, "n_gens = %lld < 0", (long long)n_gens);
    if (s->t + n_gens >= ((int64_t)1 << 32)) return fail(EVOX_EINVAL, "generation counter would pass 2^32");
    if (n_gens == 0) return EVOX_OK;
    const evox_params &P = s->P;
    const Plan &pl = s->pl;
    MaeArgs m = s->mae;
    // the sampling product Dm = Z M^T ((N + 1) x D over K = D); the update
    // M <- beta M + At^T Bt is the rank pass
    const GemmArgs sample{P.N + 1, P.D, P.D, 1.0f, m.Z, P.ldx, s->B.mat, P.ldx, 0.0f, m.Dm, P.ldx};
    hipError_t e;
    for (int64_t k = 0; k < n_gens; ++k) {
        m.t = (uint32_t)(s->t + k);
        MaeEvalArgs ea{s->B.x, m.Dm, P.ldx, s->B.sigma, s->B.fit, s->esrank, P.N, P.D,
                       k == n_gens - 1 ? s->slots : nullptr};
        if ((e = launch_mae_sample(m, s->stream)) != hipSuccess) return hip_fail(e, "deviates");
        if ((e = timed(s, [&] { return launch_gemm_nt(sample, pl.mae_splits, s->mae_work, s->stream); })) !=
            hipSuccess)
            return hip_fail(e, "sampling product");
        if ((e = launch_mae_eval(P.fn_id, pl.L, ea, pl.grid, s->stream)) != hipSuccess)
            return hip_fail(e, "samples");
        if ((e = launch_es_rank(s->B.fit, P.N, s->esrank, s->stream)) != hipSuccess) return hip_fail(e, "ranks");
        if ((e = launch_mae_select(m, s->stream)) != hipSuccess) return hip_fail(e, "parents");
        if ((e = launch_mae_recombine(m, s->stream)) != hipSuccess) return hip_fail(e, "recombination");
        if ((e = launch_mae_rank(m, s->B.mat, s->mae_beta, s->stream)) != hipSuccess)
            return hip_fail(e, "matrix update");
    }
    if ((e = launch_select(s->slots, nullptr, 0, nullptr, s->best, nullptr, nullptr, s->stream)) != hipSuccess)
        return hip_fail(e, "select");
    s->t += n_gens;
    return EVOX_OK;
}

}  // namespace

extern "C" {

int evox_es_step(evox_state *s, int64_t n_gens)
{
    if (!s) return fail(EVOX_EINVAL, "state is null");
    if (s->P.algo != EVOX_ES) return fail(EVOX_EINVAL, "evox_es_step on a state of another algorithm");
    return es_generations(s, n_gens, false);
}

int evox_pgpe_step(evox_state *s, int64_t n_gens)
{
    if (!s) return fail(EVOX_EINVAL, "state is null");
    if (s->P.algo != EVOX_PGPE) return fail(EVOX_EINVAL, "evox_pgpe_step on a state of another algorithm");
    return es_generations(s, n_gens, true);
}

int evox_nsga2_step(evox_state *s, int64_t n_gens)
{
    if (!s) return fail(EVOX_EINVAL, "state is null");
    if (s->P.algo != EVOX_NSGA2) return fail(EVOX_EINVAL, "evox_nsga2_step on a state of another algorithm");
    return nsga_generations(s, n_gens);
}

size_t evox_nsga2_sort_scratch_bytes(int64_t n, int32_t M)
{
    if (n < 1 || n > EVOX_ARGSORT_MAX_N || M < 2 || M > kNsgaMaxM) return 0;
    return nsga_sort_layout(n, M, 0).end;
}

int evox_nsga2_sort(const float *F, int64_t n, int32_t M, int32_t *front, double *crowd, void *scratch,
                    size_t scratch_bytes, void *hip_stream)
{
    if (n < 1 || n > EVOX_ARGSORT_MAX_N || M < 2 || M > kNsgaMaxM)
        return fail(EVOX_EINVAL, "n = %lld, M = %d: need 1 <= n <= %d, 2 <= M <= %d", (long long)n, M,
                    EVOX_ARGSORT_MAX_N, kNsgaMaxM);
    if (!F || !front || !crowd || !scratch) return fail(EVOX_EINVAL, "F, front, crowd and scratch are required");
    if (((uintptr_t)F & 3u) || ((uintptr_t)front & 3u) || ((uintptr_t)crowd & 7u))
        return fail(EVOX_EALIGN, "F, front or crowd is misaligned");
    if (((uintptr_t)scratch & 255u) != 0) return fail(EVOX_EALIGN, "scratch is not 256-byte aligned");
    const NsgaSortScratch l = nsga_sort_layout(n, M, 0);
    if (scratch_bytes < l.end) return fail(EVOX_ENOSPC, "scratch has %zu bytes, needs %zu", scratch_bytes, l.end);
    NsgaSortResult r;
    hipError_t e = nsga_sort(nsga_sort_args(scratch, l, F, n, M, front, crowd), n, &r, (hipStream_t)hip_stream);
    if (e != hipSuccess) return hip_fail(e, "non-dominated sorting");
    return EVOX_OK;
}

int evox_maes_step(evox_state *s, int64_t n_gens)
{
    if (!s) return fail(EVOX_EINVAL, "state is null");
    if (s->P.algo != EVOX_MAES) return fail(EVOX_EINVAL, "evox_maes_step on a state of another algorithm");
    return mae_generations(s, n_gens);
}

int evox_cso_refresh(evox_state *s, int refit)
{
    if (!s) return fail(EVOX_EINVAL, "state is null");
    if (s->P.algo != EVOX_CSO) return fail(EVOX_EINVAL, "evox_cso_refresh on a PSO state");
    return cso_refresh(s, refit != 0);
}

int evox_best(evox_state *s, float *best_fit, int64_t *best_idx, float *best_x_host)
{
    if (!s) return fail(EVOX_EINVAL, "state is null");
    if (s->P.algo == EVOX_NSGA2) return fail(EVOX_EINVAL, "NSGA-II has no single best (read front and obj)");
    DevBest h{};
    hipError_t e = hipMemcpyAsync(&h, s->best, sizeof h, hipMemcpyDeviceToHost, s->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
    if (e != hipSuccess) return hip_fail(e, "read best");
    if (best_fit) *best_fit = h.f;
    if (best_idx) *best_idx = h.i;
    if (best_x_host) {
        const bool center = s->P.algo == EVOX_ES || s->P.algo == EVOX_PGPE || s->P.algo == EVOX_MAES;
        const float *src = s->P.algo == EVOX_PSO ? s->B.gbest : center ? s->B.x : s->B.x + h.i * s->P.ldx;
        e = hipMemcpyAsync(best_x_host, src, sizeof(float) * (size_t)s->P.D, hipMemcpyDeviceToHost, s->stream);
        if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
        if (e != hipSuccess) return hip_fail(e, "read best row");
    }
    return EVOX_OK;
}

int64_t evox_generation(const evox_state *s) { return s ? s->t : -1; }

int evox_set_generation(evox_state *s, int64_t t)
{
    if (!s) return fail(EVOX_EINVAL, "state is null");
    if (t < 0 || t >= ((int64_t)1 << 32)) return fail(EVOX_EINVAL, "t = %lld out of range [0, 2^32)", (long long)t);
    s->t = t;
    return EVOX_OK;
}

int evox_row_layout(int32_t kernels, int64_t D, int32_t *threads_per_row, int32_t *chunks_per_thread)
{
    static const int family[3] = {LAYOUT_PSO, LAYOUT_CSO, LAYOUT_EVAL};
    if (kernels < EVOX_LAYOUT_PSO || kernels > EVOX_LAYOUT_EVAL)
        return fail(EVOX_EINVAL, "unknown kernel family %d", kernels);
    Layout L;
    if (D > EVOX_MAX_D || !row_layout(D, family[kernels], &L))
        return fail(EVOX_EINVAL, "no row layout for D = %lld", (long long)D);
    if (threads_per_row) *threads_per_row = L.G;
    if (chunks_per_thread) *chunks_per_thread = L.nit;
    return EVOX_OK;
}

int64_t evox_default_ldx(int32_t algo, int64_t D)
{
    if (D < 1 || D > EVOX_MAX_D) return 0;
    const int64_t line = (D + 31) / 32 * 32, quad = (D + 3) / 4 * 4;
    if (algo == EVOX_PSO || algo == EVOX_DE || algo == EVOX_ES || algo == EVOX_PGPE || algo == EVOX_MAES ||
        algo == EVOX_NSGA2)
        return D >= 512 ? line : quad;
    if (algo == EVOX_CSO) return quad;
    return 0;
}

namespace {

// Scratch of the pairing sort for `batch` generations of N individuals:
// counts, offsets and cursors per superbucket, (key, index) per entry.
size_t perm_scratch(int64_t N, int64_t batch, size_t *hist, size_t *offs, size_t *cursor, size_t *tkv)
{
    const size_t B = (size_t)batch, nb = (size_t)1 << perm_bits(N);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off = round256(off + bytes);
        return at;
    };
    *hist = take(4 * nb * B);
    *offs = take(4 * (nb + 1) * B);
    *cursor = take(4 * nb * B);
    *tkv = take(8 * (size_t)N * B);
    return off;
}

size_t perm_scratch_total(int64_t N, int64_t batch)
{
    size_t a, b, c, d;
    return perm_scratch(N, batch, &a, &b, &c, &d);
}

// n_gens sorts of N keys into perm_out[n_gens][N], as many per launch as the
// scratch holds (at most kPermBatch); keys (caller keys, n_gens 1) or null.
int sort_batches(uint64_t seed, int64_t t0, int64_t n_gens, int64_t N, const uint32_t *keys,
                 uint32_t *perm_out, void *scratch, size_t scratch_bytes, hipStream_t st)
{
    int64_t B = n_gens < kPermBatch ? n_gens : kPermBatch;
    while (B > 1 && perm_scratch_total(N, B) > scratch_bytes) --B;
    if (perm_scratch_total(N, B) > scratch_bytes)
        return fail(EVOX_ENOSPC, "scratch has %zu bytes, needs %zu", scratch_bytes, perm_scratch_total(N, 1));
    size_t oh, oo, oc, ok;
    perm_scratch(N, B, &oh, &oo, &oc, &ok);
    uint32_t *hist = at<uint32_t>(scratch, oh), *cursor = at<uint32_t>(scratch, oc);
    const int bits = perm_bits(N);
    hipError_t e;
    if ((e = launch_zero_u32(hist, ((int64_t)1 << bits) * B, st)) != hipSuccess ||
        (e = launch_zero_u32(cursor, ((int64_t)1 << bits) * B, st)) != hipSuccess)
        return hip_fail(e, "sort");
    for (int64_t g = 0; g < n_gens; g += B) {
        const int64_t b = n_gens - g < B ? n_gens - g : B;
        PermArgs pa{N, bits, (uint32_t)seed, (uint32_t)(seed >> 32), (uint32_t)(t0 + g), (uint32_t)b, hist,
                    at<uint32_t>(scratch, oo), cursor, at<uint2>(scratch, ok), perm_out + g * N, keys};
        if ((e = launch_perm(pa, st)) != hipSuccess) return hip_fail(e, "sort");
    }
    return EVOX_OK;
}

}  // namespace

size_t evox_permutation_scratch_bytes(int64_t N, int64_t batch)
{
    if (N < 1 || N > kCsoMaxN || batch < 1 || batch > kPermBatch) return 0;
    return perm_scratch_total(N, batch);
}

int evox_permutation(uint64_t seed, int64_t t0, int64_t n_gens, int64_t N, uint32_t *perm_out, void *scratch,
                     size_t scratch_bytes, void *hip_stream)
{
    if (N < 1 || N > kCsoMaxN) return fail(EVOX_EINVAL, "N = %lld out of range [1, 2^24]", (long long)N);
    if (t0 < 0 || n_gens < 0 || t0 + n_gens > ((int64_t)1 << 32))
        return fail(EVOX_EINVAL, "generations [%lld, %lld) outside [0, 2^32)", (long long)t0,
                    (long long)(t0 + n_gens));
    if (n_gens == 0) return EVOX_OK;
    if (!perm_out || !scratch) return fail(EVOX_EINVAL, "perm_out and scratch are required");
    if (((uintptr_t)perm_out & 3u) != 0) return fail(EVOX_EALIGN, "perm_out is not 4-byte aligned");
    if (((uintptr_t)scratch & 255u) != 0) return fail(EVOX_EALIGN, "scratch is not 256-byte aligned");
    return sort_batches(seed, t0, n_gens, N, nullptr, perm_out, scratch, scratch_bytes, (hipStream_t)hip_stream);
}

int evox_argsort_u32(const uint32_t *keys, int64_t N, uint32_t *perm_out, void *scratch, size_t scratch_bytes,
                     void *hip_stream)
{
    if (N < 0 || N > EVOX_ARGSORT_MAX_N)
        return fail(EVOX_EINVAL, "N = %lld out of range [0, %d]", (long long)N, EVOX_ARGSORT_MAX_N);
    if (N == 0) return EVOX_OK;
    if (!keys || !perm_out || !scratch) return fail(EVOX_EINVAL, "keys, perm_out and scratch are required");
    if (((uintptr_t)keys & 3u) != 0 || ((uintptr_t)perm_out & 3u) != 0)
        return fail(EVOX_EALIGN, "keys or perm_out is not 4-byte aligned");
    if (((uintptr_t)scratch & 255u) != 0) return fail(EVOX_EALIGN, "scratch is not 256-byte aligned");
    return sort_batches(0, 0, 1, N, keys, perm_out, scratch, scratch_bytes, (hipStream_t)hip_stream);
}

int evox_fill_normal(uint64_t seed, int64_t N, int64_t D, int64_t ldx, float mu, float sigma,
                     float *X, void *hip_stream)
{
    if (N < 0 || N >= ((int64_t)1 << 31)) return fail(EVOX_EINVAL, "N = %lld out of range [0, 2^31)", (long long)N);
    if (D < 1 || ldx < D || (ldx & 3) || ldx / 4 >= ((int64_t)1 << 32))
        return fail(EVOX_EINVAL, "D = %lld, ldx = %lld: need 1 <= D <= ldx, ldx %% 4 == 0", (long long)D,
                    (long long)ldx);
    if (N == 0) return EVOX_OK;
    if (!X) return fail(EVOX_EINVAL, "X is null");
    if (!aligned16(X)) return fail(EVOX_EALIGN, "X is not 16-byte aligned");
    InitArgs ia{X, nullptr, nullptr, N, D, ldx, 0.0f, 0.0f, 0.0f, 0.0f, 1, 1, mu, sigma,
                (uint32_t)seed, (uint32_t)(seed >> 32)};
    hipError_t e = launch_init(ia, (hipStream_t)hip_stream);
    if (e != hipSuccess) return hip_fail(e, "fill normal");
    return EVOX_OK;
}

int evox_sgemm(int32_t trans_a, int32_t trans_b, int64_t M, int64_t N, int64_t K, float alpha, const float *A,
               int64_t lda, const float *B, int64_t ldb, float beta, float *C, int64_t ldc, void *hip_stream)
{
    if (M < 0 || N < 0 || K < 0) return fail(EVOX_EINVAL, "negative size");
    if (M == 0 || N == 0) return EVOX_OK;
    const int64_t a_cols = trans_a ? M : K, b_cols = trans_b ? K : N;
    if (lda < a_cols || ldb < b_cols || ldc < N) return fail(EVOX_EINVAL, "leading dimension below the row length");
    if ((lda & 3) || (ldb & 3) || (ldc & 3)) return fail(EVOX_EALIGN, "leading dimensions must be multiples of 4");
    if (!C || (K > 0 && (!A || !B))) return fail(EVOX_EINVAL, "null matrix");
    if ((M + 127) / 128 > 65535 || (N + 127) / 128 > INT32_MAX) return fail(EVOX_EINVAL, "matrix too tall");
    if ((A && !aligned16(A)) || (B && !aligned16(B)) || !aligned16(C))
        return fail(EVOX_EALIGN, "matrices must be 16-byte aligned");
    GemmArgs g{M, N, K, alpha, A, lda, B, ldb, beta, C, ldc};
    hipError_t e = launch_gemm(trans_a != 0, trans_b != 0, g, (hipStream_t)hip_stream);
    if (e != hipSuccess) return hip_fail(e, "gemm");
    return EVOX_OK;
}

int evox_copy(const float *src, float *dst, int64_t n, void *hip_stream)
{
    if (n < 0) return fail(EVOX_EINVAL, "n = %lld < 0", (long long)n);
    if (n == 0) return EVOX_OK;
    if (!src || !dst) return fail(EVOX_EINVAL, "src and dst are required");
    if (!aligned16(src) || !aligned16(dst)) return fail(EVOX_EALIGN, "src or dst is not 16-byte aligned");
    hipError_t e = launch_stream_copy(src, dst, n, (hipStream_t)hip_stream);
    if (e != hipSuccess) return hip_fail(e, "copy");
    return EVOX_OK;
}

int evox_pso_stream(float *x, float *v, const float *p, int64_t n, void *hip_stream)
{
    if (n < 0 || (n & 3)) return fail(EVOX_EINVAL, "n = %lld must be >= 0 and a multiple of 4", (long long)n);
    if (n == 0) return EVOX_OK;
    if (!x || !v || !p) return fail(EVOX_EINVAL, "x, v and p are required");
    if (!aligned16(x) || !aligned16(v) || !aligned16(p)) return fail(EVOX_EALIGN, "x, v or p is not 16-byte aligned");
    hipError_t e = launch_pso_stream(x, v, p, n, (hipStream_t)hip_stream);
    if (e != hipSuccess) return hip_fail(e, "pso stream");
    return EVOX_OK;
}

int evox_pair_move(float *x, float *v, int64_t N, int64_t D, int64_t ldx, const int32_t *winner_of,
                   void *hip_stream)
{
    if (N < 2 || N > kCsoMaxN) return fail(EVOX_EINVAL, "N = %lld out of range [2, 2^24]", (long long)N);
    if (D < 1 || D > EVOX_MAX_D) return fail(EVOX_EINVAL, "D = %lld out of range [1, %d]", (long long)D, EVOX_MAX_D);
    if (ldx < D || (ldx & 3)) return fail(EVOX_EINVAL, "ldx = %lld must be >= D and a multiple of 4", (long long)ldx);
    if (!x || !v || !winner_of) return fail(EVOX_EINVAL, "x, v and winner_of are required");
    if (!aligned16(x) || !aligned16(v)) return fail(EVOX_EALIGN, "x or v is not 16-byte aligned");
    Layout L;
    if (!row_layout(D, LAYOUT_CSO, &L)) return fail(EVOX_EINVAL, "no row layout for D = %lld", (long long)D);
    hipError_t e = launch_pair_move(L.G, x, v, N, D, ldx, winner_of, (hipStream_t)hip_stream);
    if (e != hipSuccess) return hip_fail(e, "pair move");
    return EVOX_OK;
}

int evox_philox_fill(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t n_ctr,
                     uint32_t *out_dev, void *hip_stream)
{
    if (n_ctr < 0 || n_ctr > ((int64_t)1 << 32)) return fail(EVOX_EINVAL, "n_ctr out of range");
    if (n_ctr == 0) return EVOX_OK;
    if (!out_dev) return fail(EVOX_EINVAL, "out is null");
    if (!aligned16(out_dev)) return fail(EVOX_EALIGN, "out is not 16-byte aligned");
    hipError_t e = launch_philox_fill((uint32_t)seed, (uint32_t)(seed >> 32), c1, c2, c3, n_ctr, out_dev,
                                      (hipStream_t)hip_stream);
    if (e != hipSuccess) return hip_fail(e, "philox fill");
    return EVOX_OK;
}

int evox_profile(evox_state *s, int enable)
{
    if (!s) return fail(EVOX_EINVAL, "state is null");
    if (enable) {
        s->ev_used = 0;
        s->prof_gens = 0;
        DevBest h{};
        hipError_t e = hipMemcpyAsync(&h, s->best, sizeof h, hipMemcpyDeviceToHost, s->stream);
        if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
        if (e != hipSuccess) return hip_fail(e, "profile start");
        s->improved_base = h.improved;
    }
    s->prof = enable != 0;
    return EVOX_OK;
}

int evox_profile_read(evox_state *s, double *fused_ms, int64_t *fused_launches, int64_t *improved_rows)
{
    if (!s) return fail(EVOX_EINVAL, "state is null");
    hipError_t e = hipStreamSynchronize(s->stream);
    if (e != hipSuccess) return hip_fail(e, "profile read");
    double ms = 0.0;
    for (size_t k = 0; k < s->ev_used; ++k) {
        float m = 0.0f;
        e = hipEventElapsedTime(&m, s->ev[k].first, s->ev[k].second);
        if (e != hipSuccess) return hip_fail(e, "event time");
        ms += m;
    }
    DevBest h{};
    e = hipMemcpy(&h, s->best, sizeof h, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "profile read");
    if (fused_ms) *fused_ms = ms;
    if (fused_launches) *fused_launches = s->prof_gens;
    if (improved_rows) *improved_rows = (int64_t)(h.improved - s->improved_base);
    return EVOX_OK;
}

const char *evox_strerror(int code)
{
    switch (code) {
    case EVOX_OK: return "ok";
    case EVOX_EINVAL: return "invalid argument";
    case EVOX_EHIP: return "HIP runtime error";
    case EVOX_ENOSPC: return "scratch buffer too small";
    case EVOX_EALIGN: return "misaligned pointer or pitch";
    default: return "unknown error";
    }
}

const char *evox_last_error(void) { return g_err; }

}  // extern "C"
