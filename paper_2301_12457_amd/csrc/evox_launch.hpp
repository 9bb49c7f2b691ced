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
    float *pval;
    int64_t *pidx;
    uint32_t *pcnt;
};

struct EvalArgs {
    const float *X;
    int64_t N, D, ldx;
    float *out;
    float *pval;  // nullable: no selection partials
    int64_t *pidx;
};

struct InitArgs {
    float *x, *v, *p;  // p nullable
    int64_t N, D, ldx;
    float lb, ub, v_lo, v_hi;
    int32_t v_zero;
    uint32_t k0, k1;
};

struct CsoArgs {
    float *x, *v, *fit;
    const float *xbar;
    const uint32_t *perm;
    int64_t N, D, ldx;
    float phi, lb, ub;
    int32_t xclamp;
    uint32_t k0, k1, t;
    float *pval;
    int64_t *pidx;
    double *xsum;  // [grid][ldx] column partial sums of the new positions
};

hipError_t launch_pso(int fn, int G, int mode, const PsoArgs &a, int grid, hipStream_t s);
template <int FN>
hipError_t launch_pso_t(int G, int mode, const PsoArgs &a, int grid, hipStream_t s);
template <int FN>
hipError_t launch_eval_t(int G, bool vec, const EvalArgs &a, int grid, hipStream_t s);
template <int FN>
hipError_t launch_cso_t(int G, const CsoArgs &a, int grid, hipStream_t s);
hipError_t launch_eval(int fn, int G, bool vec, const EvalArgs &a, int grid, hipStream_t s);
hipError_t launch_select(const float *pval, const int64_t *pidx, const uint32_t *pcnt, int nparts,
                         const float *rows, int64_t ldx, float *row_out, DevBest *best,
                         float *best_f_out, int64_t *best_i_out, hipStream_t s);
hipError_t launch_init(const InitArgs &a, hipStream_t s);
hipError_t launch_philox_fill(uint32_t k0, uint32_t k1, uint32_t c1, uint32_t c2, uint32_t c3,
                              int64_t n, uint32_t *out, hipStream_t s);
hipError_t launch_copy_row(const float *src, float *dst, int64_t ldx, hipStream_t s);
hipError_t launch_fill(float *dst, int64_t n, float value, hipStream_t s);
hipError_t launch_best_init(DevBest *best, float f, int64_t i, hipStream_t s);
hipError_t launch_zero_u32(uint32_t *dst, int64_t n, hipStream_t s);
// Selection partials over a fitness array (first pass of the argmin).
int argmin_partials_grid(int64_t N);
hipError_t launch_argmin_partials(const float *f, int64_t N, float *pval, int64_t *pidx, int grid,
                                  hipStream_t s);

// CSO pairing: bucket sort of the stream-4 keys by (key, index).
struct PermArgs {
    int64_t N;
    int bits;  // buckets = 2^bits
    uint32_t k0, k1, t;
    uint32_t *hist, *offs, *cursor, *tkey, *tidx, *perm;
};
hipError_t launch_perm(const PermArgs &a, hipStream_t s);
hipError_t launch_cso(int fn, int G, const CsoArgs &a, int grid, hipStream_t s);
hipError_t launch_colsum(int G, const float *x, int64_t N, int64_t D, int64_t ldx, double *xsum,
                         int grid, hipStream_t s);
// xbar = (sum of the partial rows, in order) / N, rounded once to fp32.
hipError_t launch_cso_mean(const double *xsum, int nparts, int64_t N, int64_t D, int64_t ldx,
                           float *xbar, hipStream_t s);

}  // namespace evox
