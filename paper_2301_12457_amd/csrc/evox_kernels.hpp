// Kernel templates over (benchmark function, lanes per row) of the gfx950
// generation path, and their per-function launchers.  evox_fn.hip
// instantiates them once per function so the six compile in parallel.
//
// PSO.  Generation t of the ask-evaluate-tell loop (Sec. IV-B, Eq. (1)-(3))
// needs a grid-wide reduction (the global best) between "evaluate + personal
// best" and "move".  The kernels cut the loop there:
//   k_pso<EVAL>   evaluate x_t, update personal bests, block argmin partials
//   k_select      grid argmin over the partials, copy the gbest row
//   k_pso<FUSED>  move(t) -> x_{t+1}, evaluate x_{t+1}, personal bests,
//                 block argmin partials, all from one read of x, v, pbest
//   k_pso<MOVE>   the final move of a call (nothing to evaluate after it)
// so an n-generation call is EVAL, select, (n-1) x (FUSED, select), MOVE:
// one HBM pass of 20 B per element per generation (read x, v, p; write x, v)
// plus 4 B per element of rows whose personal best improved.
//
// CSO (the competitive swarm optimizer of Table II).  k_cso / k_cso5 sweep
// the individuals in index order: each decides from its mate entry and the
// two fitness values whether it lost its pair; a loser reads its winner's
// row (a random gather), its own x and v (in address order), moves, writes x
// and v, is re-evaluated from registers, and both rows' new values are
// accumulated into per-block fp64 column sums for the next swarm mean: 20 B
// per pair element, i.e. 10 B per individual element.  The neighbourhood
// version sweeps the same way, reads the positions from the other
// population buffer (xs): the loser's neighbours l - 1 and l + 1 besides its
// own row (three consecutive rows), and writes every row of x (the others'
// as copies).
#pragma once

#include "evox_launch.hpp"

namespace evox {

// ---------------------------------------------------------------------------
// The PSO move of float4 chunk c of a row at generation a.t: r1, r2 from
// Philox stream 2 (counters 2c and 2c + 1), vn = fma(c2 r2, g - x, fma(c1 r1,
// p - x, w v)), optional clamps, x + vn; elements past D give zeros.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void pso_move4(const PsoArgs &a, int64_t row, int64_t c, float4 xv, float4 vv,
                                          float4 pv, float4 gv, float4 &xn, float4 &vn)
{
    const U4 r1 = philox((uint32_t)(2 * c), (uint32_t)row, a.t, STREAM_PSO, a.k0, a.k1);
    const U4 r2 = philox((uint32_t)(2 * c + 1), (uint32_t)row, a.t, STREAM_PSO, a.k0, a.k1);
    float xo[4], vo[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float xe = comp(xv, e);
        const float A = a.c1 * wcomp(r1, e);
        const float Bc = a.c2 * wcomp(r2, e);
        float nv = fmaf(Bc, comp(gv, e) - xe, fmaf(A, comp(pv, e) - xe, a.w * comp(vv, e)));
        if (a.vclamp) nv = fminf(fmaxf(nv, -a.vmax), a.vmax);
        float nx = xe + nv;
        if (a.xclamp) nx = fminf(fmaxf(nx, a.lb), a.ub);
        const bool in = 4 * c + e < a.D;
        xo[e] = in ? nx : 0.0f;
        vo[e] = in ? nv : 0.0f;
    }
    xn = make_float4(xo[0], xo[1], xo[2], xo[3]);
    vn = make_float4(vo[0], vo[1], vo[2], vo[3]);
}

// ---------------------------------------------------------------------------
// The PSO generation kernel (modes above).  One group of block_for(G) / G
// rows per block (grid-stride only beyond kMaxGrid blocks); the loop bound is
// uniform over the block, so the barriers inside row_fitness are reached by
// every thread.  Each block folds its best (pfit, row) into a selection slot.
// ---------------------------------------------------------------------------
template <int FN, int G, int MAXIT, int MODE>
__global__ __launch_bounds__(block_for(G)) void k_pso(PsoArgs a)
{
    constexpr int B = block_for(G), RPB = B / G;
    constexpr bool MOVE = MODE != PSO_EVAL, EVAL = MODE != PSO_MOVE;
    __shared__ float nbr[(FN == FN_ROSENBROCK && G > 64) ? B * MAXIT : 1];
    __shared__ float red[2 * (B / 64)];
    __shared__ uint64_t sk[B / 64];
    __shared__ uint32_t sc[B / 64];

    const int tid = threadIdx.x, g = tid % G, slot = tid / G;
    const int64_t C4 = (a.D + 3) >> 2;
    // chunks written per row: the padding up to the row pitch is rewritten
    // (with zeros) where the lanes cover it, so that rows of a 128-byte-
    // aligned pitch are written as whole cache lines
    const int64_t CW = a.ldx / 4 < (int64_t)G * MAXIT ? a.ldx / 4 : (int64_t)G * MAXIT;
    uint64_t best = kNoKey;
    uint32_t nimp = 0;

    for (int64_t rb = (int64_t)blockIdx.x * RPB; rb < a.N; rb += (int64_t)gridDim.x * RPB) {
        const int64_t row = rb + slot;
        const bool active = row < a.N;
        float4 xr[MAXIT];
#pragma unroll
        for (int it = 0; it < MAXIT; ++it) {
            const int64_t c = g + (int64_t)G * it;
            float4 xn = make_float4(0.f, 0.f, 0.f, 0.f);
            if (active && c < C4) {
                const int64_t off = row * a.ldx + 4 * c;
                const float4 xv = ld_row(a.x + off, a.nt);
                if constexpr (MOVE) {
                    const float4 vv = ld_row(a.v + off, a.nt);
                    const float4 pv = ld_row(a.p + off, a.nt);
                    const float4 gv = *reinterpret_cast<const float4 *>(a.gbest + 4 * c);
                    float4 vn;
                    pso_move4(a, row, c, xv, vv, pv, gv, xn, vn);
                    st_row(a.x + off, xn, a.nt);
                    st_row(a.v + off, vn, a.nt);
                } else {
                    xn = xv;
                }
            } else if (MOVE && active && c < CW) {
                const int64_t off = row * a.ldx + 4 * c;
                st_row(a.x + off, xn, a.nt);
                st_row(a.v + off, xn, a.nt);
            }
            xr[it] = xn;
        }
        if constexpr (EVAL) {
            // the personal-best fitness is read before the evaluation's
            // block barriers: when a row spans several waves, lane 0 of its
            // first wave rewrites it below, and a wave that read it after
            // that store would take the opposite decision for its chunks
            const float pold = active ? a.pf[row] : 0.0f;
            const float f = row_fitness<FN, G, MAXIT>(xr, g, a.D, nbr, red);
            if (active) {
                const bool imp = f < pold;
                if (imp) {
#pragma unroll
                    for (int it = 0; it < MAXIT; ++it) {
                        const int64_t c = g + (int64_t)G * it;
                        if (c < CW) st_row(a.p + row * a.ldx + 4 * c, xr[it], a.nt);
                    }
                }
                if (g == 0) {
                    if (imp) a.pf[row] = f;
                    if (a.fit) a.fit[row] = f;
                    const uint64_t k = sel_key(imp ? f : pold, row);
                    best = k < best ? k : best;
                    nimp += imp ? 1u : 0u;
                }
            }
        }
    }
    if constexpr (EVAL) {
        block_min_key(best, nimp, sk, sc);
        if (tid == 0) slot_commit(a.slots, best, nimp);
    }
}

// ---------------------------------------------------------------------------
// A whole n-generation PSO call in one block, for swarms that one CU
// evaluates and moves in a few microseconds (N D <= kPsoSmallElems, a row in
// at most one wave): the grid-wide step between evaluation and move (the
// global best) becomes a block barrier, so the call is one launch instead of
// 2 n + 1.  Per generation t: evaluation of x_t and personal bests with the
// row layout and reduction of k_pso (the same fitness bits, hence the same
// decisions), the lexicographic minimum of (pfit, row) over the block, the
// gbest row from pbest through LDS, then the move.  When every row fits in
// one pass of the block the swarm stays in registers for the whole call;
// otherwise the rows are walked in passes through global memory.
// ---------------------------------------------------------------------------
template <int FN, int G, int MAXIT>
__global__ __launch_bounds__(kPsoSmallBlock) void k_pso_small(PsoArgs a, int64_t n_gens, float *gbest_out,
                                                              DevBest *best)
{
    static_assert(G <= 64, "a row within one wave");
    constexpr int B = kPsoSmallBlock, RPB = B / G;
    __shared__ __align__(16) float gb[kPsoSmallMaxLdx];
    __shared__ uint64_t sk[B / 64];
    __shared__ uint32_t sc[B / 64];
    __shared__ int64_t sel;
    const int tid = threadIdx.x, g = tid % G, slot = tid / G;
    const int64_t C4 = (a.D + 3) >> 2;
    const int64_t CW = a.ldx / 4 < (int64_t)G * MAXIT ? a.ldx / 4 : (int64_t)G * MAXIT;
    const uint32_t t0 = a.t;
    for (int64_t j = tid; j < a.ldx; j += B) gb[j] = 0.0f;  // padding past the lanes' reach
    __syncthreads();
    if (a.N <= RPB) {
        // every row in one pass of the block: x, v, pbest and pfit stay in
        // registers for the whole call, only the gbest row goes through LDS
        const int64_t row = slot;
        const bool active = row < a.N;
        float4 xr[MAXIT], vr[MAXIT], pr[MAXIT];
#pragma unroll
        for (int it = 0; it < MAXIT; ++it) {
            const int64_t c = g + (int64_t)G * it, off = row * a.ldx + 4 * c;
            const bool in = active && c < C4;
            const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
            xr[it] = in ? *reinterpret_cast<const float4 *>(a.x + off) : z;
            vr[it] = in ? *reinterpret_cast<const float4 *>(a.v + off) : z;
            pr[it] = in ? *reinterpret_cast<const float4 *>(a.p + off) : z;
        }
        float pf = active ? a.pf[row] : 0.0f, f = 0.0f;
        uint64_t bk = kNoKey;
        uint32_t nimp = 0, total_imp = 0;
        for (int64_t k = 0; k < n_gens; ++k) {
            a.t = t0 + (uint32_t)k;
            f = row_fitness<FN, G, MAXIT>(xr, g, a.D, nullptr, nullptr);
            const bool imp = active && f < pf;
            if (imp) {
#pragma unroll
                for (int it = 0; it < MAXIT; ++it) pr[it] = xr[it];
                pf = f;
            }
            bk = active && g == 0 ? sel_key(pf, row) : kNoKey;
            nimp = imp && g == 0 ? 1u : 0u;
            block_min_key(bk, nimp, sk, sc);
            if (tid == 0) {
                sel = bk == kNoKey ? 0 : key_index(bk);
                total_imp += nimp;
            }
            __syncthreads();
            if (row == sel) {
#pragma unroll
                for (int it = 0; it < MAXIT; ++it) {
                    const int64_t c = g + (int64_t)G * it;
                    if (c < CW) *reinterpret_cast<float4 *>(gb + 4 * c) = pr[it];
                }
            }
            __syncthreads();
#pragma unroll
            for (int it = 0; it < MAXIT; ++it) {
                const int64_t c = g + (int64_t)G * it;
                if (active && c < C4) {
                    const float4 gv = *reinterpret_cast<const float4 *>(gb + 4 * c);
                    pso_move4(a, row, c, xr[it], vr[it], pr[it], gv, xr[it], vr[it]);
                }
            }
            // the next write of gb follows the barriers of the next block minimum
        }
        if (active) {
#pragma unroll
            for (int it = 0; it < MAXIT; ++it) {
                const int64_t c = g + (int64_t)G * it, off = row * a.ldx + 4 * c;
                if (c < CW) {
                    *reinterpret_cast<float4 *>(a.x + off) = xr[it];
                    *reinterpret_cast<float4 *>(a.v + off) = vr[it];
                    *reinterpret_cast<float4 *>(a.p + off) = pr[it];
                }
            }
            if (g == 0) {
                a.pf[row] = pf;
                if (a.fit) a.fit[row] = f;
            }
        }
        for (int64_t j = tid; j < a.ldx; j += B) gbest_out[j] = gb[j];
        if (tid == 0) {
            best->f = key_value(bk);
            best->i = sel;
            best->improved += total_imp;
        }
        return;
    }
    for (int64_t k = 0; k < n_gens; ++k) {
        a.t = t0 + (uint32_t)k;
        // evaluate x_t, personal bests
        uint64_t bk = kNoKey;
        uint32_t nimp = 0;
        for (int64_t rb = 0; rb < a.N; rb += RPB) {  // uniform trip count
            const int64_t row = rb + slot;
            const bool active = row < a.N;
            float4 xr[MAXIT];
#pragma unroll
            for (int it = 0; it < MAXIT; ++it) {
                const int64_t c = g + (int64_t)G * it;
                xr[it] = active && c < C4 ? *reinterpret_cast<const float4 *>(a.x + row * a.ldx + 4 * c)
                                          : make_float4(0.f, 0.f, 0.f, 0.f);
            }
            const float f = row_fitness<FN, G, MAXIT>(xr, g, a.D, nullptr, nullptr);
            if (active) {
                const float pold = a.pf[row];
                const bool imp = f < pold;
                if (imp) {
#pragma unroll
                    for (int it = 0; it < MAXIT; ++it) {
                        const int64_t c = g + (int64_t)G * it;
                        if (c < CW) *reinterpret_cast<float4 *>(a.p + row * a.ldx + 4 * c) = xr[it];
                    }
                }
                if (g == 0) {
                    if (imp) a.pf[row] = f;
                    if (a.fit) a.fit[row] = f;
                    const uint64_t key = sel_key(imp ? f : pold, row);
                    bk = key < bk ? key : bk;
                    nimp += imp ? 1u : 0u;
                }
            }
        }
        block_min_key(bk, nimp, sk, sc);
        if (tid == 0) {
            const int64_t i = bk == kNoKey ? 0 : key_index(bk);
            best->f = key_value(bk);
            best->i = i;
            best->improved += nimp;
            sel = i;
        }
        __syncthreads();
        for (int64_t j = tid; j < a.ldx; j += B) {
            const float v = a.p[sel * a.ldx + j];
            gb[j] = v;
            gbest_out[j] = v;
        }
        __syncthreads();
        // move of generation t
        for (int64_t rb = 0; rb < a.N; rb += RPB) {
            const int64_t row = rb + slot;
            if (row >= a.N) continue;
#pragma unroll
            for (int it = 0; it < MAXIT; ++it) {
                const int64_t c = g + (int64_t)G * it;
                const int64_t off = row * a.ldx + 4 * c;
                if (c < C4) {
                    const float4 xv = *reinterpret_cast<const float4 *>(a.x + off);
                    const float4 vv = *reinterpret_cast<const float4 *>(a.v + off);
                    const float4 pv = *reinterpret_cast<const float4 *>(a.p + off);
                    const float4 gv = *reinterpret_cast<const float4 *>(gb + 4 * c);
                    float4 xn, vn;
                    pso_move4(a, row, c, xv, vv, pv, gv, xn, vn);
                    *reinterpret_cast<float4 *>(a.x + off) = xn;
                    *reinterpret_cast<float4 *>(a.v + off) = vn;
                } else if (c < CW) {
                    *reinterpret_cast<float4 *>(a.x + off) = make_float4(0.f, 0.f, 0.f, 0.f);
                    *reinterpret_cast<float4 *>(a.v + off) = make_float4(0.f, 0.f, 0.f, 0.f);
                }
            }
        }
        __syncthreads();  // the next generation reads every moved row
    }
}

// ---------------------------------------------------------------------------
// Problem.evaluate over any row pitch / alignment; optionally folds each
// block's best (fitness, row) into a selection slot.  VEC: 16-byte aligned
// rows, float4 loads.
// ---------------------------------------------------------------------------
template <int FN, int G, int MAXIT, bool VEC>
__global__ __launch_bounds__(block_for(G)) void k_eval(EvalArgs a)
{
    constexpr int B = block_for(G), RPB = B / G;
    __shared__ float nbr[(FN == FN_ROSENBROCK && G > 64) ? B * MAXIT : 1];
    __shared__ float red[2 * (B / 64)];
    __shared__ uint64_t sk[B / 64];
    __shared__ uint32_t sc[B / 64];

    const int tid = threadIdx.x, g = tid % G, slot = tid / G;
    const int64_t C4 = (a.D + 3) >> 2;
    uint64_t best = kNoKey;
    uint32_t none = 0;

    for (int64_t rb = (int64_t)blockIdx.x * RPB; rb < a.N; rb += (int64_t)gridDim.x * RPB) {
        const int64_t row = rb + slot;
        const bool active = row < a.N;
        float4 xr[MAXIT];
#pragma unroll
        for (int it = 0; it < MAXIT; ++it) {
            const int64_t c = g + (int64_t)G * it;
            float4 xv = make_float4(0.f, 0.f, 0.f, 0.f);
            if (active && c < C4) {
                const float *src = a.X + row * a.ldx + 4 * c;
                if constexpr (VEC) {
                    xv = ld_row(src, a.nt);
                } else {
                    const int64_t left = a.D - 4 * c;
                    xv.x = src[0];
                    if (left > 1) xv.y = src[1];
                    if (left > 2) xv.z = src[2];
                    if (left > 3) xv.w = src[3];
                }
            }
            xr[it] = xv;
        }
        const float f = row_fitness<FN, G, MAXIT>(xr, g, a.D, nbr, red);
        if (active && g == 0) {
            a.out[row] = f;
            const uint64_t k = sel_key(f, row);
            best = k < best ? k : best;
        }
    }
    if (a.slots) {
        block_min_key(best, none, sk, sc);
        if (tid == 0) slot_commit(a.slots, best, 0);
    }
}

// ---------------------------------------------------------------------------
// Column sums of a block's rows for the swarm mean.  Each thread accumulates
// fp64 sums of its columns 4 (g + G it) + e over the rows it handles (in LDS
// when a block holds several row slots, in registers otherwise); at the end
// the slots are combined in slot order and written to xsum[blockIdx][*].
// The order of every addition is fixed, so the result is reproducible.
// ---------------------------------------------------------------------------
template <int G, int MAXIT>
struct ColAcc {
    static constexpr int B = block_for(G), RPB = B / G;
    static constexpr bool kLds = RPB > 1;
    double *lds;                            // [4 MAXIT][B] when kLds
    double reg[kLds ? 1 : MAXIT][4];

    __device__ explicit ColAcc(double *l) : lds(l)
    {
#pragma unroll
        for (int it = 0; it < MAXIT; ++it)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if constexpr (kLds)
                    lds[(it * 4 + e) * B + threadIdx.x] = 0.0;
                else
                    reg[it][e] = 0.0;
            }
    }
    __device__ void add(int it, int e, double v)
    {
        if constexpr (kLds)
            lds[(it * 4 + e) * B + threadIdx.x] += v;
        else
            reg[it][e] += v;
    }
    // Reached by every thread of the block.
    __device__ void write(int64_t D, int64_t ldx, double *xsum)
    {
        const int tid = threadIdx.x;
        double *dst = xsum + (int64_t)blockIdx.x * ldx;
        if constexpr (kLds) {
            __syncthreads();
            for (int q = tid; q < 4 * G * MAXIT; q += B) {
                const int it = q / (4 * G), r = q - it * 4 * G, g = r / 4, e = r % 4;
                const int64_t j = 4 * ((int64_t)g + (int64_t)G * it) + e;
                if (j < D) {
                    const double *col = lds + (it * 4 + e) * B + g;
                    double t = col[0];
                    for (int sl = 1; sl < RPB; ++sl) t += col[sl * G];
                    dst[j] = t;
                }
            }
        } else {
            const int g = tid;  // one row slot: lane g of the row
#pragma unroll
            for (int it = 0; it < MAXIT; ++it)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int64_t j = 4 * ((int64_t)g + (int64_t)G * it) + e;
                    if (j < D) dst[j] = reg[it][e];
                }
        }
    }
};

// ---------------------------------------------------------------------------
// The swarm-mean generation, swept in individual order.  A block takes
// ranges of kCsoSweep consecutive individuals: every individual of the range
// reads its mate entry and both fitness values (before the generation) and
// decides whether it lost its pair; winners (and the odd one out) copy their
// fitness to the output buffer, losers are listed in LDS in index order (a
// ballot per wave, waves in order, so the list and the order of the column
// sums are deterministic).  The row groups then move the listed losers:
// gather the winner's row, read the loser's x and v -- rows in increasing
// address order, so the loser traffic is a forward sweep over the
// population instead of random rows -- update, write x and v, re-evaluate
// from registers, and accumulate winner + new loser rows into the fp64
// column sums of the next swarm mean.  The odd individual's row is listed
// too, for its column sums only.
// ---------------------------------------------------------------------------
template <int FN, int G, int MAXIT>
__device__ __forceinline__ void cso_sweep_body(const CsoArgs &a)
{
    constexpr int B = block_for(G), RPB = B / G, NW = B / 64, R = kCsoSweep;
    static_assert(R <= B, "one individual per thread in the decision phase");
    __shared__ float nbr[(FN == FN_ROSENBROCK && G > 64) ? B * MAXIT : 1];
    __shared__ float red[2 * (B / 64)];
    __shared__ uint64_t sk[B / 64];
    __shared__ uint32_t sc[B / 64];
    __shared__ double acc_lds[RPB > 1 ? 4 * MAXIT * B : 1];
    __shared__ int32_t lst_l[R], lst_w[R];  // listed individual, its winner (-1: the odd one out)
    __shared__ int32_t wcnt[NW];

    const int tid = threadIdx.x, g = tid % G, slot = tid / G, lane = tid & 63, wave = tid >> 6;
    const int64_t C4 = (a.D + 3) >> 2;
    uint64_t best = kNoKey;
    uint32_t none = 0;
    ColAcc<G, MAXIT> acc(acc_lds);

    for (int64_t base = (int64_t)blockIdx.x * R; base < a.N; base += (int64_t)gridDim.x * R) {
        bool listed = false;
        int32_t me = 0, other = -1;
        if (tid < R && base + tid < a.N) {
            const int64_t i = base + tid;
            const uint32_t m = a.mate[i];
            const float fi = a.fit_in[i];
            bool loser = false;
            if (m != kUnpaired) {
                const int64_t j = m & ~kMateFirst;
                const float fj = a.fit_in[j];
                const bool first = (m & kMateFirst) != 0;
                const float f0 = first ? fi : fj, f1 = first ? fj : fi;
                const bool second_wins = f1 < f0 || (f0 != f0 && f1 == f1);
                loser = first ? second_wins : !second_wins;
                other = (int32_t)j;
            }
            if (!loser) {
                a.fit[i] = fi;
                const uint64_t k = sel_key(fi, i);
                best = k < best ? k : best;
            }
            listed = loser || m == kUnpaired;
            me = (int32_t)i;
        }
        const uint64_t bal = __ballot(listed);
        if (lane == 0) wcnt[wave] = __popcll(bal);
        __syncthreads();
        int off = 0, total = 0;
#pragma unroll
        for (int q = 0; q < NW; ++q) {
            off += q < wave ? wcnt[q] : 0;
            total += wcnt[q];
        }
        if (listed) {
            const int at = off + __popcll(bal & ((1ull << lane) - 1ull));
            lst_l[at] = me;
            lst_w[at] = other;
        }
        __syncthreads();
        const int rounds = (total + RPB - 1) / RPB;  // uniform: every thread reaches the barriers
        for (int r = 0; r < rounds; ++r) {
            const int q = r * RPB + slot;
            const bool active = q < total;
            const int64_t l = active ? lst_l[q] : 0;
            const int64_t w = active ? lst_w[q] : -1;
            const bool paired = w >= 0;
            float4 xr[MAXIT];
#pragma unroll
            for (int it = 0; it < MAXIT; ++it) {
                const int64_t c = g + (int64_t)G * it;
                float4 xn = make_float4(0.f, 0.f, 0.f, 0.f);
                if (active && c < C4) {
                    const int64_t off_l = l * a.ldx + 4 * c;
                    const float4 xl = ld_stream(a.x + off_l);
                    if (paired) {
                        const float4 xw = *reinterpret_cast<const float4 *>(a.x + w * a.ldx + 4 * c);
                        const float4 vl = ld_stream(a.v + off_l);
                        const float4 xb = *reinterpret_cast<const float4 *>(a.xbar + 4 * c);
                        const U4 R1 = philox((uint32_t)(3 * c), (uint32_t)l, a.t, STREAM_CSO, a.k0, a.k1);
                        const U4 R2 = philox((uint32_t)(3 * c + 1), (uint32_t)l, a.t, STREAM_CSO, a.k0, a.k1);
                        const U4 R3 = philox((uint32_t)(3 * c + 2), (uint32_t)l, a.t, STREAM_CSO, a.k0, a.k1);
                        float xo[4], vo[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float xle = comp(xl, e);
                            const float t0 = wcomp(R1, e) * comp(vl, e);
                            const float t1 = fmaf(wcomp(R2, e), comp(xw, e) - xle, t0);
                            const float cc = a.phi * wcomp(R3, e);
                            const float nv = fmaf(cc, comp(xb, e) - xle, t1);
                            float nx = xle + nv;
                            if (a.xclamp) nx = fminf(fmaxf(nx, a.lb), a.ub);
                            const bool in = 4 * c + e < a.D;
                            xo[e] = in ? nx : 0.0f;
                            vo[e] = in ? nv : 0.0f;
                        }
                        xn = make_float4(xo[0], xo[1], xo[2], xo[3]);
                        st_stream(a.x + off_l, xn);
                        st_stream(a.v + off_l, make_float4(vo[0], vo[1], vo[2], vo[3]));
#pragma unroll
                        for (int e = 0; e < 4; ++e) acc.add(it, e, (double)comp(xw, e) + (double)comp(xn, e));
                    } else {
                        xn = xl;  // the odd one out: unchanged, counted in the column sums
#pragma unroll
                        for (int e = 0; e < 4; ++e) acc.add(it, e, (double)comp(xl, e));
                    }
                }
                xr[it] = xn;
            }
            const float f = row_fitness<FN, G, MAXIT>(xr, g, a.D, nbr, red);
            if (active && paired && g == 0) {
                a.fit[l] = f;
                const uint64_t k = sel_key(f, l);
                best = k < best ? k : best;
            }
        }
        __syncthreads();  // the next range overwrites the list
    }
    block_min_key(best, none, sk, sc);
    if (tid == 0) slot_commit(a.slots, best, 0);
    acc.write(a.D, a.ldx, a.xsum);
}

// ---------------------------------------------------------------------------
// The neighbourhood version's generation, swept in individual order like
// the swarm version: the old positions are read from xs and every row of the
// next population buffer x is written.  Per range of kCsoSweep individuals
// each one decides from its mate entry and both fitness values (before the
// generation) whether it lost; the others (winners and the odd one out) are
// listed first and copied, x_i = xs_i, their fitness carried over; then the
// losers, listed in index order, learn from their winner's row and from the
// fp64 mean of the old rows l - 1, l, l + 1 (modulo N, neighbours that the
// sweep reads around the same time), are written and re-evaluated.  Both
// lists are in index order, so the column sums' order is deterministic.
// ---------------------------------------------------------------------------
template <int FN, int G, int MAXIT>
__device__ __forceinline__ void cso_local_body(const CsoArgs &a)
{
    constexpr int B = block_for(G), RPB = B / G, NW = B / 64, R = kCsoSweep;
    static_assert(R <= B, "one individual per thread in the decision phase");
    __shared__ float nbr[(FN == FN_ROSENBROCK && G > 64) ? B * MAXIT : 1];
    __shared__ float red[2 * (B / 64)];
    __shared__ uint64_t sk[B / 64];
    __shared__ uint32_t sc[B / 64];
    __shared__ double acc_lds[RPB > 1 ? 4 * MAXIT * B : 1];
    __shared__ int32_t lst_c[R];            // copied individuals (winners, the odd one out)
    __shared__ int32_t lst_l[R], lst_w[R];  // losers and their winners
    __shared__ int32_t ccnt[NW], lcnt[NW];

    const int tid = threadIdx.x, g = tid % G, slot = tid / G, lane = tid & 63, wave = tid >> 6;
    const int64_t C4 = (a.D + 3) >> 2;
    uint64_t best = kNoKey;
    uint32_t none = 0;
    ColAcc<G, MAXIT> acc(acc_lds);

    for (int64_t base = (int64_t)blockIdx.x * R; base < a.N; base += (int64_t)gridDim.x * R) {
        bool in = false, loser = false;
        int32_t me = 0, other = -1;
        if (tid < R && base + tid < a.N) {
            const int64_t i = base + tid;
            const uint32_t m = a.mate[i];
            const float fi = a.fit_in[i];
            if (m != kUnpaired) {
                const int64_t j = m & ~kMateFirst;
                const float fj = a.fit_in[j];
                const bool first = (m & kMateFirst) != 0;
                const float f0 = first ? fi : fj, f1 = first ? fj : fi;
                const bool second_wins = f1 < f0 || (f0 != f0 && f1 == f1);
                loser = first ? second_wins : !second_wins;
                other = (int32_t)j;
            }
            if (!loser) {
                a.fit[i] = fi;
                const uint64_t k = sel_key(fi, i);
                best = k < best ? k : best;
            }
            in = true;
            me = (int32_t)i;
        }
        const uint64_t bl = __ballot(loser), bc = __ballot(in && !loser);
        if (lane == 0) {
            lcnt[wave] = __popcll(bl);
            ccnt[wave] = __popcll(bc);
        }
        __syncthreads();
        int offl = 0, offc = 0, nl = 0, nc = 0;
#pragma unroll
        for (int q = 0; q < NW; ++q) {
            offl += q < wave ? lcnt[q] : 0;
            offc += q < wave ? ccnt[q] : 0;
            nl += lcnt[q];
            nc += ccnt[q];
        }
        const uint64_t below = (1ull << lane) - 1ull;
        if (loser) {
            const int at = offl + __popcll(bl & below);
            lst_l[at] = me;
            lst_w[at] = other;
        } else if (in) {
            lst_c[offc + __popcll(bc & below)] = me;
        }
        __syncthreads();
        // the copies: a whole row per row group, counted in the column sums
        for (int r = 0; r < (nc + RPB - 1) / RPB; ++r) {
            const int q = r * RPB + slot;
            if (q < nc) {
                const int64_t i = lst_c[q];
#pragma unroll
                for (int it = 0; it < MAXIT; ++it) {
                    const int64_t c = g + (int64_t)G * it;
                    if (c < C4) {
                        const float4 xi = *reinterpret_cast<const float4 *>(a.xs + i * a.ldx + 4 * c);
                        st_stream(a.x + i * a.ldx + 4 * c, xi);
#pragma unroll
                        for (int e = 0; e < 4; ++e) acc.add(it, e, (double)comp(xi, e));
                    }
                }
            }
        }
        // the losers (uniform trip count: every thread reaches the barriers)
        for (int r = 0; r < (nl + RPB - 1) / RPB; ++r) {
            const int q = r * RPB + slot;
            const bool active = q < nl;
            const int64_t l = active ? lst_l[q] : 0;
            const int64_t w = active ? lst_w[q] : 0;
            float4 xr[MAXIT];
#pragma unroll
            for (int it = 0; it < MAXIT; ++it) {
                const int64_t c = g + (int64_t)G * it;
                float4 xn = make_float4(0.f, 0.f, 0.f, 0.f);
                if (active && c < C4) {
                    const int64_t off = l * a.ldx + 4 * c;
                    const float4 xl = *reinterpret_cast<const float4 *>(a.xs + off);
                    const float4 vl = ld_stream(a.v + off);
                    const float4 xw = *reinterpret_cast<const float4 *>(a.xs + w * a.ldx + 4 * c);
                    // ring mean of the rows before the generation: ((x_{l-1} + x_l) + x_{l+1}) / 3
                    // in fp64, rounded once
                    const int64_t lm = l == 0 ? a.N - 1 : l - 1, lp = l == a.N - 1 ? 0 : l + 1;
                    const float4 xa = *reinterpret_cast<const float4 *>(a.xs + lm * a.ldx + 4 * c);
                    const float4 xc = *reinterpret_cast<const float4 *>(a.xs + lp * a.ldx + 4 * c);
                    float mo[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        mo[e] = (float)((((double)comp(xa, e) + (double)comp(xl, e)) + (double)comp(xc, e)) / 3.0);
                    const float4 xb = make_float4(mo[0], mo[1], mo[2], mo[3]);
                    const U4 R1 = philox((uint32_t)(3 * c), (uint32_t)l, a.t, STREAM_CSO, a.k0, a.k1);
                    const U4 R2 = philox((uint32_t)(3 * c + 1), (uint32_t)l, a.t, STREAM_CSO, a.k0, a.k1);
                    const U4 R3 = philox((uint32_t)(3 * c + 2), (uint32_t)l, a.t, STREAM_CSO, a.k0, a.k1);
                    float xo[4], vo[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float xle = comp(xl, e);
                        const float t0 = wcomp(R1, e) * comp(vl, e);
                        const float t1 = fmaf(wcomp(R2, e), comp(xw, e) - xle, t0);
                        const float cc = a.phi * wcomp(R3, e);
                        const float nv = fmaf(cc, comp(xb, e) - xle, t1);
                        float nx = xle + nv;
                        if (a.xclamp) nx = fminf(fmaxf(nx, a.lb), a.ub);
                        const bool inb = 4 * c + e < a.D;
                        xo[e] = inb ? nx : 0.0f;
                        vo[e] = inb ? nv : 0.0f;
                    }
                    xn = make_float4(xo[0], xo[1], xo[2], xo[3]);
                    st_stream(a.x + off, xn);
                    st_stream(a.v + off, make_float4(vo[0], vo[1], vo[2], vo[3]));
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc.add(it, e, (double)comp(xn, e));
                }
                xr[it] = xn;
            }
            const float f = row_fitness<FN, G, MAXIT>(xr, g, a.D, nbr, red);
            if (active && g == 0) {
                a.fit[l] = f;
                const uint64_t k = sel_key(f, l);
                best = k < best ? k : best;
            }
        }
        __syncthreads();  // the next range overwrites the lists
    }
    block_min_key(best, none, sk, sc);
    if (tid == 0) slot_commit(a.slots, best, 0);
    acc.write(a.D, a.ldx, a.xsum);
}

template <int FN, int G, int MAXIT, bool LOCAL>
__global__ __launch_bounds__(block_for(G)) void k_cso(CsoArgs a)
{
    if constexpr (LOCAL)
        cso_local_body<FN, G, MAXIT>(a);
    else
        cso_sweep_body<FN, G, MAXIT>(a);
}

// The swarm-mean generation with one chunk per lane and at most 32 lanes per
// row (D <= 128), compiled for 5 waves per SIMD (within 96 registers): the
// shape of the large-population, moderate-D workloads.
template <int FN, int G>
__global__ __launch_bounds__(block_for(G)) __attribute__((amdgpu_waves_per_eu(5))) void k_cso5(CsoArgs a)
{
    cso_sweep_body<FN, G, 1>(a);
}

// ---------------------------------------------------------------------------
// DE/rand/1/bin generation (Storn & Price, 1997), one target row per row
// group: the target's three partners and crossover position from one Philox
// call (stream 6, counter (0, i, t)); partners mutually distinct and distinct
// from the target by stepping a draw in [0, N - 1 - k) past the indices
// already taken, in increasing order (no rejection loop); per float4 chunk
// the target row (streamed) and the three partner rows (gathered), the
// crossover draws of Philox (1 + c, i, t, 6), mutant fma(F, x_r2 - x_r3,
// x_r1), the trial evaluated from registers and kept when strictly better.
// Philox in its two-input xor form here: the three-input form schedules the
// kernel past 96 registers (4 instead of 5 waves per SIMD, 5 % slower).
// Every target writes its next row (trial or copy) to the other buffer, so
// all targets of a generation see the same population.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int64_t below(uint32_t w, int64_t m)
{
    return (int64_t)(((uint64_t)w * (uint64_t)m) >> 32);
}

template <int FN, int G, int MAXIT>
__global__ __launch_bounds__(block_for(G)) void k_de(DeArgs a)
{
    constexpr int B = block_for(G), RPB = B / G;
    __shared__ float nbr[(FN == FN_ROSENBROCK && G > 64) ? B * MAXIT : 1];
    __shared__ float red[2 * (B / 64)];
    __shared__ uint64_t sk[B / 64];
    __shared__ uint32_t sc[B / 64];

    const int tid = threadIdx.x, g = tid % G, slot = tid / G;
    const int64_t C4 = (a.D + 3) >> 2;
    const int64_t CW = a.ldx / 4 < (int64_t)G * MAXIT ? a.ldx / 4 : (int64_t)G * MAXIT;
    uint64_t best = kNoKey;
    uint32_t nacc = 0;

    for (int64_t rb = (int64_t)blockIdx.x * RPB; rb < a.N; rb += (int64_t)gridDim.x * RPB) {
        const int64_t row = rb + slot;
        const bool active = row < a.N;
        int64_t r[3] = {0, 0, 0}, jr = 0;
        if (active) {
            const U4 w = philox<false>(0u, (uint32_t)row, a.t, STREAM_DE, a.k0, a.k1);
            const uint32_t wk[3] = {w.x, w.y, w.z};
            int64_t taken[3] = {row, 0, 0};
#pragma unroll
            for (int k = 0; k < 3; ++k) {
                int64_t v = below(wk[k], a.N - 1 - k);
#pragma unroll
                for (int e = 0; e <= k; ++e)  // taken[0..k] in increasing order
                    if (v >= taken[e]) ++v;
                r[k] = v;
                if (k < 2) {  // insert v into taken[0..k]
                    int pos = k + 1;
#pragma unroll
                    for (int e = k; e >= 0; --e)
                        if (taken[e] > v) {
                            taken[e + 1] = taken[e];
                            pos = e;
                        }
                    taken[pos] = v;
                }
            }
            jr = below(w.w, a.D);
        }
        float4 xi[MAXIT], ur[MAXIT];
#pragma unroll
        for (int it = 0; it < MAXIT; ++it) {
            const int64_t c = g + (int64_t)G * it;
            float4 xv = make_float4(0.f, 0.f, 0.f, 0.f), uv = xv;
            if (active && c < C4) {
                const int64_t off = 4 * c;
                xv = ld_row(a.x + row * a.ldx + off, a.nt);
                const float4 v1 = *reinterpret_cast<const float4 *>(a.x + r[0] * a.ldx + off);
                const float4 v2 = *reinterpret_cast<const float4 *>(a.x + r[1] * a.ldx + off);
                const float4 v3 = *reinterpret_cast<const float4 *>(a.x + r[2] * a.ldx + off);
                const U4 cw = philox<false>((uint32_t)(1 + c), (uint32_t)row, a.t, STREAM_DE, a.k0, a.k1);
                float uo[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int64_t j = 4 * c + e;
                    const float mutant = fmaf(a.F, comp(v2, e) - comp(v3, e), comp(v1, e));
                    const bool take = wcomp(cw, e) <= a.CR || j == jr;
                    uo[e] = j < a.D ? (take ? mutant : comp(xv, e)) : 0.0f;
                }
                uv = make_float4(uo[0], uo[1], uo[2], uo[3]);
            }
            xi[it] = xv;
            ur[it] = uv;
        }
        const float fu = row_fitness<FN, G, MAXIT>(ur, g, a.D, nbr, red);
        if (active) {
            const float fi = a.fit[row];
            const bool acc = fu < fi;
#pragma unroll
            for (int it = 0; it < MAXIT; ++it) {
                const int64_t c = g + (int64_t)G * it;
                if (c < CW) st_row(a.xn + row * a.ldx + 4 * c, acc ? ur[it] : xi[it], a.nt);
            }
            if (g == 0) {
                const float fn = acc ? fu : fi;
                a.fitn[row] = fn;
                const uint64_t k = sel_key(fn, row);
                best = k < best ? k : best;
                nacc += acc ? 1u : 0u;
            }
        }
    }
    if (a.slots) {
        block_min_key(best, nacc, sk, sc);
        if (tid == 0) slot_commit(a.slots, best, nacc);
    }
}

// ---------------------------------------------------------------------------
// OpenES / PGPE samples and fitness: one row group per antithetic pair k;
// the deviate chunk z_k (Philox stream 7 or 8, generation t, Box-Muller) and
// both samples fma(+-sigma, z, center) live in registers only, and both rows
// are reduced to their fitness.  The center (and PGPE's sigma) are read by
// every pair from the caches.
//
// k_es_eval_s (functions without neighbour coupling): each lane folds its
// chunks into the two fitness partials as it generates them, so a lane can
// take many chunks (kEsChunksPerLane) and the per-pair reductions and
// barriers are spread over more deviates; k_es_eval (Rosenbrock) holds the
// rows in registers for the neighbour term.
// ---------------------------------------------------------------------------
constexpr int kEsChunksPerLane = 16;

template <int FN, int G>
__global__ __launch_bounds__(block_for(G)) void k_es_eval_s(EsArgs a)
{
    using F = Fn<FN>;
    static_assert(!F::kNeighbour, "neighbour-coupled functions use k_es_eval");
    constexpr int B = block_for(G), RPB = B / G;
    __shared__ float red[2 * (B / 64)];
    __shared__ uint64_t sk[B / 64];
    __shared__ uint32_t sc[B / 64];

    const int tid = threadIdx.x, g = tid % G, slot = tid / G;
    const int64_t C4 = (a.D + 3) >> 2, H = a.N / 2;
    uint64_t best = kNoKey;
    for (int64_t kb = (int64_t)blockIdx.x * RPB; kb < H; kb += (int64_t)gridDim.x * RPB) {
        const int64_t k = kb + slot;
        const bool active = k < H;
        Acc sp = F::init(), sm = F::init();
        if (active) {
            for (int64_t c = g; c < C4; c += G) {
                const float4 th = *reinterpret_cast<const float4 *>(a.theta + 4 * c);
                const float4 sg = a.sig ? *reinterpret_cast<const float4 *>(a.sig + 4 * c)
                                        : make_float4(a.sigma, a.sigma, a.sigma, a.sigma);
                const float4 z = normal4((uint32_t)c, (uint32_t)k, a.t, a.stream, a.k0, a.k1);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int64_t j = 4 * c + e;
                    if (j < a.D) {
                        F::elem(sp, fmaf(comp(sg, e), comp(z, e), comp(th, e)), 0.0f, j);
                        F::elem(sm, fmaf(-comp(sg, e), comp(z, e), comp(th, e)), 0.0f, j);
                    }
                }
            }
        }
        const float fp = F::finish(group_reduce<FN, G>(sp, red), a.D);
        const float fm = F::finish(group_reduce<FN, G>(sm, red), a.D);
        if (active && g == 0) {
            a.fit[2 * k] = fp;
            a.fit[2 * k + 1] = fm;
            a.rank[2 * k] = 0u;
            a.rank[2 * k + 1] = 0u;
            const uint64_t kp = sel_key(fp, 2 * k), km = sel_key(fm, 2 * k + 1);
            best = kp < best ? kp : best;
            best = km < best ? km : best;
        }
    }
    if (a.slots) {
        uint32_t none = 0;
        block_min_key(best, none, sk, sc);
        if (tid == 0) slot_commit(a.slots, best, 0);
    }
}

template <int FN, int G, int MAXIT>
__global__ __launch_bounds__(block_for(G)) void k_es_eval(EsArgs a)
{
    constexpr int B = block_for(G), RPB = B / G;
    __shared__ float nbr[(FN == FN_ROSENBROCK && G > 64) ? B * MAXIT : 1];
    __shared__ float red[2 * (B / 64)];
    __shared__ uint64_t sk[B / 64];
    __shared__ uint32_t sc[B / 64];

    const int tid = threadIdx.x, g = tid % G, slot = tid / G;
    const int64_t C4 = (a.D + 3) >> 2, H = a.N / 2;
    uint64_t best = kNoKey;
    for (int64_t kb = (int64_t)blockIdx.x * RPB; kb < H; kb += (int64_t)gridDim.x * RPB) {
        const int64_t k = kb + slot;
        const bool active = k < H;
        float4 xp[MAXIT], xm[MAXIT];
#pragma unroll
        for (int it = 0; it < MAXIT; ++it) {
            const int64_t c = g + (int64_t)G * it;
            float po[4] = {0.f, 0.f, 0.f, 0.f}, mo[4] = {0.f, 0.f, 0.f, 0.f};
            if (active && c < C4) {
                const float4 th = *reinterpret_cast<const float4 *>(a.theta + 4 * c);
                const float4 sg = a.sig ? *reinterpret_cast<const float4 *>(a.sig + 4 * c)
                                        : make_float4(a.sigma, a.sigma, a.sigma, a.sigma);
                const float4 z = normal4((uint32_t)c, (uint32_t)k, a.t, a.stream, a.k0, a.k1);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (4 * c + e < a.D) {
                        po[e] = fmaf(comp(sg, e), comp(z, e), comp(th, e));
                        mo[e] = fmaf(-comp(sg, e), comp(z, e), comp(th, e));
                    }
            }
            xp[it] = make_float4(po[0], po[1], po[2], po[3]);
            xm[it] = make_float4(mo[0], mo[1], mo[2], mo[3]);
        }
        const float fp = row_fitness<FN, G, MAXIT>(xp, g, a.D, nbr, red);
        const float fm = row_fitness<FN, G, MAXIT>(xm, g, a.D, nbr, red);
        if (active && g == 0) {
            a.fit[2 * k] = fp;
            a.fit[2 * k + 1] = fm;
            a.rank[2 * k] = 0u;
            a.rank[2 * k + 1] = 0u;
            const uint64_t kp = sel_key(fp, 2 * k), km = sel_key(fm, 2 * k + 1);
            best = kp < best ? kp : best;
            best = km < best ? km : best;
        }
    }
    if (a.slots) {
        uint32_t none = 0;
        block_min_key(best, none, sk, sc);
        if (tid == 0) slot_commit(a.slots, best, 0);
    }
}

// ---------------------------------------------------------------------------
// MA-ES samples: row k < N of the steps d (pitch ldd, from the matrix product)
// becomes x_k = fma(sigma, d_k, y) in registers and is reduced to its fitness;
// the sample's rank counter is cleared for the counting pass, and the last
// generation feeds the best-sample selection.
// ---------------------------------------------------------------------------
template <int FN, int G, int MAXIT>
__global__ __launch_bounds__(block_for(G)) void k_mae_eval(MaeEvalArgs a)
{
    constexpr int B = block_for(G), RPB = B / G;
    __shared__ float nbr[(FN == FN_ROSENBROCK && G > 64) ? B * MAXIT : 1];
    __shared__ float red[2 * (B / 64)];
    __shared__ uint64_t sk[B / 64];
    __shared__ uint32_t sc[B / 64];

    const int tid = threadIdx.x, g = tid % G, slot = tid / G;
    const int64_t C4 = (a.D + 3) >> 2;
    const float sg = *a.sigma;
    uint64_t best = kNoKey;
    for (int64_t kb = (int64_t)blockIdx.x * RPB; kb < a.N; kb += (int64_t)gridDim.x * RPB) {
        const int64_t k = kb + slot;
        const bool active = k < a.N;
        float4 xr[MAXIT];
#pragma unroll
        for (int it = 0; it < MAXIT; ++it) {
            const int64_t c = g + (int64_t)G * it;
            float o[4] = {0.f, 0.f, 0.f, 0.f};
            if (active && c < C4) {
                const float4 y = *reinterpret_cast<const float4 *>(a.y + 4 * c);
                const float4 d = *reinterpret_cast<const float4 *>(a.d + k * a.ldd + 4 * c);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (4 * c + e < a.D) o[e] = fmaf(sg, comp(d, e), comp(y, e));
            }
            xr[it] = make_float4(o[0], o[1], o[2], o[3]);
        }
        const float f = row_fitness<FN, G, MAXIT>(xr, g, a.D, nbr, red);
        if (active && g == 0) {
            a.fit[k] = f;
            a.rank[k] = 0u;
            const uint64_t key = sel_key(f, k);
            best = key < best ? key : best;
        }
    }
    if (a.slots) {
        uint32_t none = 0;
        block_min_key(best, none, sk, sc);
        if (tid == 0) slot_commit(a.slots, best, 0);
    }
}

// Column sums of all rows of x (the swarm mean at creation / refresh).
template <int G, int MAXIT>
__global__ __launch_bounds__(block_for(G)) void k_colsum(const float *x, int64_t N, int64_t D,
                                                        int64_t ldx, double *xsum)
{
    constexpr int B = block_for(G), RPB = B / G;
    __shared__ double acc_lds[RPB > 1 ? 4 * MAXIT * B : 1];
    const int tid = threadIdx.x, g = tid % G, slot = tid / G;
    const int64_t C4 = (D + 3) >> 2;
    ColAcc<G, MAXIT> acc(acc_lds);
    for (int64_t rb = (int64_t)blockIdx.x * RPB; rb < N; rb += (int64_t)gridDim.x * RPB) {
        const int64_t row = rb + slot;
        if (row >= N) continue;
#pragma unroll
        for (int it = 0; it < MAXIT; ++it) {
            const int64_t c = g + (int64_t)G * it;
            if (c < C4) {
                const float4 xv = ld_stream(x + row * ldx + 4 * c);
#pragma unroll
                for (int e = 0; e < 4; ++e) acc.add(it, e, (double)comp(xv, e));
            }
        }
    }
    acc.write(D, ldx, xsum);
}

// Dispatch on the row layout (G, MAXIT) of a family.
#define EVOX_FAMILY_CASES(M, F, ...)                                                              \
    case 4 * 16 + F: M(4, F, __VA_ARGS__); break;                                                 \
    case 8 * 16 + F: M(8, F, __VA_ARGS__); break;                                                 \
    case 16 * 16 + F: M(16, F, __VA_ARGS__); break;                                               \
    case 32 * 16 + F: M(32, F, __VA_ARGS__); break;                                               \
    case 64 * 16 + F: M(64, F, __VA_ARGS__); break;                                               \
    case 128 * 16 + F: M(128, F, __VA_ARGS__); break;                                             \
    case 256 * 16 + F: M(256, F, __VA_ARGS__); break;                                             \
    case 512 * 16 + F: M(512, F, __VA_ARGS__); break;
// 1024 lanes per row: the family's own chunk count while it holds the row,
// else the smallest of 4 and 8 chunks that does (row_layout's maxit)
#define EVOX_BIG_4_8(M, ...)                                                                      \
    case 1024 * 16 + 4: M(1024, 4, __VA_ARGS__); break;                                           \
    case 1024 * 16 + 8: M(1024, 8, __VA_ARGS__); break;
#define EVOX_BIG_CASES(M, F, ...)                                                                 \
    case 1024 * 16 + F: M(1024, F, __VA_ARGS__); break;                                           \
    EVOX_BIG_4_8(M, __VA_ARGS__)

#define EVOX_LAUNCH_PSO(GG, MM, MODEE) \
    hipLaunchKernelGGL((k_pso<FN, GG, MM, MODEE>), dim3(grid), dim3(block_for(GG)), 0, s, a)
#define EVOX_LAUNCH_EVAL(GG, MM, VECC) \
    hipLaunchKernelGGL((k_eval<FN, GG, MM, VECC>), dim3(grid), dim3(block_for(GG)), 0, s, a)
#define EVOX_LAUNCH_CSO(GG, MM, LOC) \
    hipLaunchKernelGGL((k_cso<FN, GG, MM, LOC>), dim3(grid), dim3(block_for(GG)), 0, s, a)
#define EVOX_LAUNCH_DE(GG, MM, UNUSED) \
    hipLaunchKernelGGL((k_de<FN, GG, MM>), dim3(grid), dim3(block_for(GG)), 0, s, a)
#define EVOX_LAUNCH_ES(GG, MM, UNUSED) \
    hipLaunchKernelGGL((k_es_eval<FN, GG, MM>), dim3(grid), dim3(block_for(GG)), 0, s, a)
#define EVOX_LAUNCH_MAE(GG, MM, UNUSED) \
    hipLaunchKernelGGL((k_mae_eval<FN, GG, MM>), dim3(grid), dim3(block_for(GG)), 0, s, a)

template <int FN>
hipError_t launch_pso_t(Layout L, int mode, const PsoArgs &a, int grid, hipStream_t s)
{
    const int key = L.G * 16 + L.maxit;
    if (mode == PSO_EVAL) {
        switch (key) {
            EVOX_FAMILY_CASES(EVOX_LAUNCH_PSO, LAYOUT_PSO, PSO_EVAL)
            EVOX_BIG_CASES(EVOX_LAUNCH_PSO, LAYOUT_PSO, PSO_EVAL)
            default: return hipErrorInvalidValue;
        }
    } else if (mode == PSO_FUSED) {
        switch (key) {
            EVOX_FAMILY_CASES(EVOX_LAUNCH_PSO, LAYOUT_PSO, PSO_FUSED)
            EVOX_BIG_CASES(EVOX_LAUNCH_PSO, LAYOUT_PSO, PSO_FUSED)
            default: return hipErrorInvalidValue;
        }
    } else {
        if constexpr (FN != FN_SPHERE) {
            return hipErrorInvalidValue;  // the move does not evaluate: instantiated once
        } else {
            switch (key) {
                EVOX_FAMILY_CASES(EVOX_LAUNCH_PSO, LAYOUT_PSO, PSO_MOVE)
                EVOX_BIG_CASES(EVOX_LAUNCH_PSO, LAYOUT_PSO, PSO_MOVE)
                default: return hipErrorInvalidValue;
            }
        }
    }
    return hipGetLastError();
}

template <int FN>
hipError_t launch_pso_small_t(Layout L, const PsoArgs &a, int64_t n_gens, float *gbest_out, DevBest *best,
                              hipStream_t s)
{
    if (L.maxit != LAYOUT_PSO) return hipErrorInvalidValue;
    switch (L.G) {
#define EVOX_SMALL(GG)                                                                                        \
    case GG: hipLaunchKernelGGL((k_pso_small<FN, GG, LAYOUT_PSO>), dim3(1), dim3(kPsoSmallBlock), 0, s, a, \
                                n_gens, gbest_out, best); break;
        EVOX_SMALL(4)
        EVOX_SMALL(8)
        EVOX_SMALL(16)
        EVOX_SMALL(32)
        EVOX_SMALL(64)
#undef EVOX_SMALL
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int FN>
hipError_t launch_eval_t(Layout L, bool vec, const EvalArgs &a, int grid, hipStream_t s)
{
    const int key = L.G * 16 + L.maxit;
    if (vec) {
        switch (key) {
            EVOX_FAMILY_CASES(EVOX_LAUNCH_EVAL, LAYOUT_EVAL, true)
            EVOX_FAMILY_CASES(EVOX_LAUNCH_EVAL, LAYOUT_CSO, true)
            EVOX_FAMILY_CASES(EVOX_LAUNCH_EVAL, LAYOUT_PSO, true)
            case 1024 * 16 + 1: EVOX_LAUNCH_EVAL(1024, 1, true); break;
            case 1024 * 16 + 2: EVOX_LAUNCH_EVAL(1024, 2, true); break;
            EVOX_BIG_4_8(EVOX_LAUNCH_EVAL, true)
            default: return hipErrorInvalidValue;
        }
    } else {
        switch (key) {
            EVOX_FAMILY_CASES(EVOX_LAUNCH_EVAL, LAYOUT_EVAL, false)
            EVOX_FAMILY_CASES(EVOX_LAUNCH_EVAL, LAYOUT_CSO, false)
            case 1024 * 16 + 1: EVOX_LAUNCH_EVAL(1024, 1, false); break;
            case 1024 * 16 + 2: EVOX_LAUNCH_EVAL(1024, 2, false); break;
            EVOX_BIG_4_8(EVOX_LAUNCH_EVAL, false)
            default: return hipErrorInvalidValue;
        }
    }
    return hipGetLastError();
}

template <int FN>
hipError_t launch_cso_t(Layout L, const CsoArgs &a, int grid, hipStream_t s)
{
    if (a.xs == a.x && L.maxit == 1 && L.G <= 32) {  // swarm mean, one chunk per lane: 5 waves per SIMD
        switch (L.G) {
            case 4: hipLaunchKernelGGL((k_cso5<FN, 4>), dim3(grid), dim3(block_for(4)), 0, s, a); break;
            case 8: hipLaunchKernelGGL((k_cso5<FN, 8>), dim3(grid), dim3(block_for(8)), 0, s, a); break;
            case 16: hipLaunchKernelGGL((k_cso5<FN, 16>), dim3(grid), dim3(block_for(16)), 0, s, a); break;
            case 32: hipLaunchKernelGGL((k_cso5<FN, 32>), dim3(grid), dim3(block_for(32)), 0, s, a); break;
            default: return hipErrorInvalidValue;
        }
    } else if (a.xs != a.x) {  // the neighbourhood version
        switch (L.G * 16 + L.maxit) {
            EVOX_FAMILY_CASES(EVOX_LAUNCH_CSO, LAYOUT_CSO, true)
            EVOX_BIG_CASES(EVOX_LAUNCH_CSO, LAYOUT_CSO, true)
            default: return hipErrorInvalidValue;
        }
    } else {
        switch (L.G * 16 + L.maxit) {
            EVOX_FAMILY_CASES(EVOX_LAUNCH_CSO, LAYOUT_CSO, false)
            EVOX_BIG_CASES(EVOX_LAUNCH_CSO, LAYOUT_CSO, false)
            default: return hipErrorInvalidValue;
        }
    }
    return hipGetLastError();
}

template <int FN>
hipError_t launch_de_t(Layout L, const DeArgs &a, int grid, hipStream_t s)
{
    switch (L.G * 16 + L.maxit) {
        EVOX_FAMILY_CASES(EVOX_LAUNCH_DE, LAYOUT_PSO, 0)
        EVOX_BIG_CASES(EVOX_LAUNCH_DE, LAYOUT_PSO, 0)
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int FN>
hipError_t launch_es_eval_t(Layout L, const EsArgs &a, int grid, hipStream_t s)
{
    if constexpr (Fn<FN>::kNeighbour) {
        switch (L.G * 16 + L.maxit) {
            EVOX_FAMILY_CASES(EVOX_LAUNCH_ES, LAYOUT_PSO, 0)
            EVOX_BIG_CASES(EVOX_LAUNCH_ES, LAYOUT_PSO, 0)
            default: return hipErrorInvalidValue;
        }
    } else {
        // the fewest lanes (a power of two, 4..1024) that hold the row in at
        // most kEsChunksPerLane chunks per lane
        const int64_t c4 = (a.D + 3) / 4;
        int G = 4;
        while (G < kMaxG && (c4 + G - 1) / G > kEsChunksPerLane) G *= 2;
        const int64_t rpb = block_for(G) / G, H = a.N / 2;
        int64_t nb = (H + rpb - 1) / rpb;
        nb = nb < 1 ? 1 : nb > kMaxGrid ? kMaxGrid : nb;
        const dim3 gs((unsigned)nb), bs((unsigned)block_for(G));
        (void)grid;
        switch (G) {
            case 4: hipLaunchKernelGGL((k_es_eval_s<FN, 4>), gs, bs, 0, s, a); break;
            case 8: hipLaunchKernelGGL((k_es_eval_s<FN, 8>), gs, bs, 0, s, a); break;
            case 16: hipLaunchKernelGGL((k_es_eval_s<FN, 16>), gs, bs, 0, s, a); break;
            case 32: hipLaunchKernelGGL((k_es_eval_s<FN, 32>), gs, bs, 0, s, a); break;
            case 64: hipLaunchKernelGGL((k_es_eval_s<FN, 64>), gs, bs, 0, s, a); break;
            case 128: hipLaunchKernelGGL((k_es_eval_s<FN, 128>), gs, bs, 0, s, a); break;
            case 256: hipLaunchKernelGGL((k_es_eval_s<FN, 256>), gs, bs, 0, s, a); break;
            case 512: hipLaunchKernelGGL((k_es_eval_s<FN, 512>), gs, bs, 0, s, a); break;
            case 1024: hipLaunchKernelGGL((k_es_eval_s<FN, 1024>), gs, bs, 0, s, a); break;
            default: return hipErrorInvalidValue;
        }
    }
    return hipGetLastError();
}

template <int FN>
hipError_t launch_mae_eval_t(Layout L, const MaeEvalArgs &a, int grid, hipStream_t s)
{
    switch (L.G * 16 + L.maxit) {
        EVOX_FAMILY_CASES(EVOX_LAUNCH_MAE, LAYOUT_PSO, 0)
        EVOX_BIG_CASES(EVOX_LAUNCH_MAE, LAYOUT_PSO, 0)
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int FN>
int occupancy_cso_t(Layout L, bool local)
{
    int n = 0;
    if (!local && L.maxit == 1 && L.G <= 32) {
        switch (L.G) {
            case 4: (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_cso5<FN, 4>, block_for(4), 0); break;
            case 8: (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_cso5<FN, 8>, block_for(8), 0); break;
            case 16: (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_cso5<FN, 16>, block_for(16), 0); break;
            case 32: (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_cso5<FN, 32>, block_for(32), 0); break;
            default: return 0;
        }
        return n;
    }
#define EVOX_OCC_CSO(GG, MM, UNUSED)                                                                             \
    (void)(local ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_cso<FN, GG, MM, true>, block_for(GG), 0)  \
                 : hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_cso<FN, GG, MM, false>, block_for(GG), 0))
    switch (L.G * 16 + L.maxit) {
        EVOX_FAMILY_CASES(EVOX_OCC_CSO, LAYOUT_CSO, 0)
        EVOX_BIG_CASES(EVOX_OCC_CSO, LAYOUT_CSO, 0)
        default: return 0;
    }
#undef EVOX_OCC_CSO
    return n;
}

}  // namespace evox
