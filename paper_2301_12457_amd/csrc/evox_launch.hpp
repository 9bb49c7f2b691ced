// Host-side launchers of the gfx950 kernels (one per kernel family).  Each
// dispatches on (function id, lanes per row) to a template instantiation.
// All return hipSuccess or the launch error.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "evox_device.hpp"

namespace evox {

enum PsoMode { PSO_EVAL = 0, PSO_FUSED = 1, PSO_MOVE = 2 };

struct PsoArgs {
    float *x, *v, *p, *pf, *fit;
    const float *gbest;
    int64_t N, D, ldx;
    float w, c1, c2, vmax, lb, ub;
    int32_t vclamp, xclamp;
    uint32_t k0, k1;
    uint32_t t;  // generation whose move this launch performs
    SelSlots *slots;
    bool nt;     // streaming hint on row accesses
};

struct DeArgs {
    const float *x, *fit;  // generation t population and fitness
    float *xn, *fitn;      // generation t + 1
    int64_t N, D, ldx;
    float F, CR;
    uint32_t k0, k1;
    uint32_t t;
    SelSlots *slots;       // nullable: no selection in this launch
    bool nt;               // streaming hint on the target rows
};

// OpenES and PGPE.  k_es_eval_s / k_es_eval: both samples center +-
// sigma z_k of each antithetic pair from registers (sigma a scalar, or per
// dimension for PGPE) and their fitness; k_es_rank: the ranks by counting (N <= kEsMaxN); k_es_grad /
// k_es_update: the gradient estimates with the deviates regenerated from
// Philox (never stored) and the steps.
constexpr int kEsMaxN = 16384;
constexpr int kEsPairChunk = 32;  // pairs per thread of the gradient pass
struct EsArgs {
    const float *theta;
    const float *sig;      // PGPE: per-dimension deviations; null: the scalar sigma
    float *fit;            // [N] sample fitness
    uint32_t *rank;        // [N] zeroed here for k_es_rank
    int64_t N, D;
    float sigma;
    uint32_t k0, k1, t, stream;
    SelSlots *slots;       // nullable
};
struct EsGradArgs {
    const uint32_t *rank;  // [N] sample ranks
    double *part;          // [1 or 2][ceil(H / kEsPairChunk)][4 * ceil(D / 4)] partial sums
    float *theta;
    float *sig;            // PGPE: per-dimension deviations (updated); null for OpenES
    int64_t H, D;
    float sigma, lr, sig_lr, max_change;
    uint32_t k0, k1, t, stream;
};

// Matrix-adaptation ES.  One generation: k_mae_sample writes the deviates Z
// [(N + 1) rows][ldx] (row N is the path s, so that the product also yields
// M s); the product Dm = Z M^T gives the steps d_k = M z_k and M s; k_mae_eval
// the fitness of y + sigma d_k; k_es_rank the ranks; k_mae_select the parents
// in rank order; k_mae_recombine the new center and path and the two
// K-contiguous factors of the matrix update; k_mae_sigma the step size; the
// rank-(mu + 1) pass M <- beta M + At^T Bt the new M.
constexpr int kMaeBlock = 256;  // threads (columns) per block of the recombination
constexpr int kMaeChunk = 64;   // parents per partial weighted sum
constexpr int kMaeRankUnrolled = 32;  // rank-pass step counts with an unrolled kernel of their own
struct MaeEvalArgs {
    const float *y, *d;   // center [ldx]; steps [N][ldd]
    int64_t ldd;
    const float *sigma;   // step size (device scalar)
    float *fit;           // [N]
    uint32_t *rank;       // [N] zeroed here for k_es_rank
    int64_t N, D;
    SelSlots *slots;      // nullable
};
struct MaeArgs {
    float *Z, *Dm;        // [(N + 1)][ldx]
    int64_t N, D, ldx, mu;
    int64_t kp, ldf;      // factor terms (mu + 1 padded with zero terms) and their pitch
    const uint32_t *rank; // [N]
    int32_t *sel;         // [mu] the parents' sample indices, best first
    const double *w;      // [mu] recombination weights
    float *y, *s, *sigma; // center [ldx], path [ldx], step size [1]
    float *At, *Bt;       // [kp][ldf], k-major, zero past term mu and column D
    double *part;         // [ceil(D / kMaeBlock)] partial sums of |s|^2
    double *wpart;        // [ceil(mu / kMaeChunk)][2][D] weighted parent sums per chunk
    double cs, cz, hc1, hcw, damp, chi;  // c_s, sqrt(mu_eff c_s (2 - c_s)), c_1 / 2, c_w / 2, c_s / d_s, chi_D
    uint32_t k0, k1, t;
};
hipError_t launch_mae_sample(const MaeArgs &a, hipStream_t s);
hipError_t launch_mae_select(const MaeArgs &a, hipStream_t s);
hipError_t launch_mae_recombine(const MaeArgs &a, hipStream_t s);  // and the step size
hipError_t launch_mae_rank(const MaeArgs &a, float *M, float beta, hipStream_t s);  // M <- beta M + At^T Bt
hipError_t launch_mae_identity(float *M, int64_t D, int64_t ldx, hipStream_t s);
int occupancy_gemm_nt_thin(int64_t M);  // resident blocks per CU of the tile shape for M rows (M <= 128)

// NSGA-II on DTLZ1.
constexpr int kNsgaMaxM = 8;          // objectives
constexpr int64_t kNsgaMaxN = 32768;  // population (the merged population is 2N)
constexpr int kNsgaPeelBatch = 8;     // fronts peeled per host round trip
struct NsgaVarArgs {
    const float *X;        // parents [N][ldx]
    int64_t N, D, ldx;
    const int32_t *front;  // [N]
    const double *crowd;   // [N]
    float *Q;              // offspring [N][ldx]
    double eta_c, eta_m;
    uint32_t k0, k1, t;
};
struct NsgaSortArgs {
    const float *F;        // [n][M]
    int64_t n;
    int32_t M;
    int32_t *front;        // [n] out: front index, -1 past the fronts needed
    double *crowd;         // [n] out: crowding distance within the front
    uint32_t *cnt;         // [n] dominator counts
    int32_t *list;         // [n] points front by front
    int32_t *foff;         // [n + 1] first list position of each front
    int32_t *pos, *sorted; // [M][cap] order within the front per objective
    int64_t cap;           // >= n
    uint32_t *len;         // [kNsgaPeelBatch] sizes of the fronts of a peeling batch
};
struct NsgaSortResult {
    int32_t fronts;        // fronts assigned
    int64_t assigned;      // points in them
    int64_t last;          // points in the last one
};
struct NsgaSelArgs {
    const float *X, *Q;    // parents, offspring [N][ldx]
    int64_t N, ldx;
    int32_t M;
    const float *FR;       // [2N][M]
    const int32_t *frontR; // [2N]
    const double *crowdR;  // [2N]
    const int32_t *list;   // [2N] from the sort
    int32_t *keep, *pre;   // [2N]
    int32_t *rank;         // [2N] last-front ranks (the sort's free per-objective positions)
    int32_t *sums;         // [ceil(2N / 1024)] block sums of the survivor prefix sums
    float *X2;             // [N][ldx] survivors' rows
    float *F;              // [N][M]
    int32_t *front;        // [N]
    double *crowd;         // [N]
};
hipError_t launch_nsga_var(const NsgaVarArgs &a, hipStream_t s);
hipError_t launch_nsga_dtlz1(const float *X, int64_t n, int64_t D, int64_t ldx, int32_t M, float *F, hipStream_t s);
// Fronts until at least `need` points are assigned, and the crowding
// distances within them; synchronizes the stream once per front.  The same
// in two parts: the dominator counts over all pairs, then the peeling and
// the crowding distances.
hipError_t nsga_sort(const NsgaSortArgs &a, int64_t need, NsgaSortResult *res, hipStream_t s);
hipError_t nsga_count(const NsgaSortArgs &a, hipStream_t s);
hipError_t nsga_fronts(const NsgaSortArgs &a, int64_t need, NsgaSortResult *res, hipStream_t s);
hipError_t launch_nsga_select(const NsgaSelArgs &a, const NsgaSortResult &r, hipStream_t s);

// C = alpha op(A) op(B) + beta C (row-major; op(A) is M x K, op(B) K x N;
// leading dimensions and pointers 16-byte multiples for the vector loads).
struct GemmArgs {
    int64_t M, N, K;
    float alpha;
    const float *A;
    int64_t lda;
    const float *B;
    int64_t ldb;
    float beta;
    float *C;
    int64_t ldc;
};
hipError_t launch_gemm(bool ta, bool tb, const GemmArgs &g, hipStream_t s);
// The A B^T product (A [M x K], B [N x K]) with `splits` K-slices; splits > 1
// needs a workspace of splits * M * N floats.  gemm_nt_chunk: the K extent of
// one slice.
hipError_t launch_gemm_nt(const GemmArgs &g, int splits, float *work, hipStream_t s);
int64_t gemm_nt_chunk(int64_t K, int splits);

struct EvalArgs {
    const float *X;
    int64_t N, D, ldx;
    float *out;
    SelSlots *slots;  // nullable: no selection
    bool nt;          // streaming hint on row accesses
};

struct InitArgs {
    float *x, *v, *p;  // v, p nullable
    int64_t N, D, ldx;
    float lb, ub, v_lo, v_hi;
    int32_t v_zero;
    int32_t x_normal;  // x = mu + sigma z (stream 5) instead of U[lb, ub)
    float mu, sigma;
    uint32_t k0, k1;
};

// CSO pairing in individual order (the swarm-mean generation): entry i of a
// generation's mate array is the index of i's partner, with kMateFirst set
// when i is the first of its pair (the one that wins ties); kUnpaired marks
// the individual left over when N is odd.
constexpr uint32_t kMateFirst = 0x80000000u;
constexpr uint32_t kUnpaired = 0xFFFFFFFFu;
constexpr int kCsoSweep = 128;  // individuals per range of the swarm-mean generation kernel

struct CsoArgs {
    float *x, *v;
    float *fit;            // fitness after the generation (every entry written)
    const float *fit_in;   // fitness before the generation (another buffer than fit)
    const float *xbar;
    const uint32_t *perm;  // this generation's permutation (not read by the generation kernels)
    const uint32_t *mate;  // this generation's mate array
    int64_t N, D, ldx;
    float phi, lb, ub;
    int32_t xclamp;
    uint32_t k0, k1, t;
    SelSlots *slots;
    double *xsum;  // [grid][ldx] column partial sums of the new positions
    // positions before the generation: x itself (swarm mean: the losers are
    // moved in place), or the other population buffer (neighbourhood
    // version: every row of x is written, the losers' new rows and copies of
    // the others, and loser l's mean is that of rows l - 1, l, l + 1 of xs)
    const float *xs;
};

hipError_t launch_pso(int fn, Layout L, int mode, const PsoArgs &a, int grid, hipStream_t s);
// A whole n-generation PSO call in one block of kPsoSmallBlock threads, for
// N D <= kPsoSmallElems, rows in at most 64 lanes and ldx <= kPsoSmallMaxLdx.
constexpr int kPsoSmallBlock = 1024;
constexpr int64_t kPsoSmallElems = 16384;
constexpr int64_t kPsoSmallMaxLdx = 1024;
hipError_t launch_pso_small(int fn, Layout L, const PsoArgs &a, int64_t n_gens, float *gbest_out, DevBest *best,
                            hipStream_t s);
template <int FN>
hipError_t launch_pso_small_t(Layout L, const PsoArgs &a, int64_t n_gens, float *gbest_out, DevBest *best,
                              hipStream_t s);
template <int FN>
hipError_t launch_pso_t(Layout L, int mode, const PsoArgs &a, int grid, hipStream_t s);
template <int FN>
hipError_t launch_eval_t(Layout L, bool vec, const EvalArgs &a, int grid, hipStream_t s);
template <int FN>
hipError_t launch_cso_t(Layout L, const CsoArgs &a, int grid, hipStream_t s);
template <int FN>
hipError_t launch_de_t(Layout L, const DeArgs &a, int grid, hipStream_t s);
template <int FN>
hipError_t launch_es_eval_t(Layout L, const EsArgs &a, int grid, hipStream_t s);
template <int FN>
hipError_t launch_mae_eval_t(Layout L, const MaeEvalArgs &a, int grid, hipStream_t s);
template <int FN>
int occupancy_cso_t(Layout L, bool local);  // resident blocks per CU of k_cso
hipError_t launch_eval(int fn, Layout L, bool vec, const EvalArgs &a, int grid, hipStream_t s);
// Second pass of the selection: reduce and reset the slots, store the result
// (best and/or the two outputs, each nullable) and copy the selected row of
// `rows` (ldx floats) to row_out (nullable).
hipError_t launch_select(SelSlots *slots, const float *rows, int64_t ldx, float *row_out,
                         DevBest *best, float *best_f_out, int64_t *best_i_out, hipStream_t s);
hipError_t launch_slots_init(SelSlots *slots, hipStream_t s);
hipError_t launch_init(const InitArgs &a, hipStream_t s);
hipError_t launch_philox_fill(uint32_t k0, uint32_t k1, uint32_t c1, uint32_t c2, uint32_t c3,
                              int64_t n, uint32_t *out, hipStream_t s);
hipError_t launch_stream_copy(const float *src, float *dst, int64_t n, hipStream_t s);
// The 20 B per element stream of a PSO generation (diagnostic): n floats,
// n % 4 == 0.
hipError_t launch_pso_stream(float *x, float *v, const float *p, int64_t n, hipStream_t s);
// The data movement of a swarm-mean CSO generation with G lanes per row
// (diagnostic): loser i = every index with winner_of[i] >= 0.
hipError_t launch_pair_move(int G, float *x, float *v, int64_t N, int64_t D, int64_t ldx, const int32_t *winner_of,
                            hipStream_t s);
// dst[0 .. ldx) = src[0 .. ldx).
hipError_t launch_copy_row(const float *src, float *dst, int64_t ldx, hipStream_t s);
hipError_t launch_fill(float *dst, int64_t n, float value, hipStream_t s);
hipError_t launch_best_init(DevBest *best, float f, int64_t i, hipStream_t s);
hipError_t launch_zero_u32(uint32_t *dst, int64_t n, hipStream_t s);
hipError_t launch_fill_u32(uint32_t *dst, int64_t n, uint32_t value, hipStream_t s);
// First pass of the selection over a stored fitness array.
hipError_t launch_argmin_slots(const float *f, int64_t N, SelSlots *slots, hipStream_t s);

// CSO pairing: superbucket sort of the stream-4 keys by (key, index).
constexpr int kPermChunk = 4096;        // individuals per block of the count / place passes
constexpr int kPermMaxBits = 13;        // superbuckets <= 8192
constexpr int kPermMaxBuckets = 1 << kPermMaxBits;
constexpr int kPermSortCap = 4096;      // LDS capacity of one superbucket sort (mean <= 2048)
constexpr int64_t kCsoMaxN = (int64_t)1 << 24;
constexpr int kPermBatch = 8;           // generations per permutation batch at most
struct PermArgs {
    int64_t N;
    int bits;           // superbuckets = 2^bits
    uint32_t k0, k1;
    uint32_t t0;        // first generation of the batch
    uint32_t batch;     // generations in the batch
    uint32_t *hist, *offs, *cursor;  // [batch][...] slices
    uint2 *tkv;                      // [batch][N] (key, index) placed by superbucket
    uint32_t *perm;                  // [batch][N]
    const uint32_t *keys;  // caller keys (batch 1), or null: Philox stream-4 keys
    uint32_t *mate;        // [batch][N] mate arrays of the permutations, or null: none
};
hipError_t launch_perm(const PermArgs &a, hipStream_t s);
hipError_t launch_cso(int fn, Layout L, const CsoArgs &a, int grid, hipStream_t s);
hipError_t launch_de(int fn, Layout L, const DeArgs &a, int grid, hipStream_t s);
hipError_t launch_es_eval(int fn, Layout L, const EsArgs &a, int grid, hipStream_t s);
hipError_t launch_es_rank(const float *fit, int64_t N, uint32_t *rank, hipStream_t s);
hipError_t launch_mae_eval(int fn, Layout L, const MaeEvalArgs &a, int grid, hipStream_t s);
hipError_t launch_es_grad(const EsGradArgs &a, hipStream_t s);
int occupancy_cso(int fn, Layout L, bool local);
hipError_t launch_colsum(Layout L, const float *x, int64_t N, int64_t D, int64_t ldx, double *xsum,
                         int grid, hipStream_t s);

// Swarm mean from per-block fp64 column sums.
constexpr int kMeanStages = 128;  // first-stage blocks per column tile at most
struct MeanArgs {
    const double *xsum;  // [nparts][ldx]
    int64_t nparts, N, D, ldx;
    float *xbar;         // [ldx]
    double *s1;          // [kMeanStages][ldx] stage sums
    int32_t stages;      // first-stage blocks per column tile, 1..kMeanStages
    uint32_t *ticket;    // [ceil(ldx / 64)], zero between launches
    SelSlots *slots;     // nullable: also reduce these selection slots into best
    DevBest *best;
};
hipError_t launch_cso_mean(const MeanArgs &m, hipStream_t s);

}  // namespace evox
