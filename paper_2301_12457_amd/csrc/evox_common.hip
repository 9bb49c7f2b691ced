// Function-independent kernels of the gfx950 path: initialisation, selection
// (second pass), fills, the CSO pairing sort and swarm mean, the Philox
// diagnostic, and the dispatch from a function id to its instantiation.
//
// Pairing (CSO).  The permutation is the order of the individuals by
// (key, index), key_i = Philox stream-4 word of individual i at generation t.
// Keys are uniform 32-bit numbers, so a bucket sort does it in four light
// passes:
//   k_perm_hist     count the keys per bucket (top `bits` key bits)
//   k_perm_scan     exclusive scan of the counts -> bucket offsets
//   k_perm_scatter  place (key, index) into its bucket
//   k_perm_rank     rank each entry inside its bucket by (key, index) and
//                   write the index to its final position
// Buckets hold 8-16 entries on average, so the in-bucket rank is a short scan.
#include "evox_kernels.hpp"

namespace evox {

// ---------------------------------------------------------------------------
// Initialisation (Algorithm.setup): x ~ U[lb, ub), v ~ U[v_lo, v_hi) or 0,
// p = x; padding columns zero.  One thread per float4 chunk.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_init(InitArgs a)
{
    const int64_t C4 = (a.D + 3) / 4, L4 = a.ldx / 4;
    const int64_t total = a.N * L4;
    const float xr = a.ub - a.lb, vr = a.v_hi - a.v_lo;
    for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < total;
         q += (int64_t)gridDim.x * 256) {
        const int64_t row = q / L4, c = q - row * L4;
        float xo[4] = {0.f, 0.f, 0.f, 0.f}, vo[4] = {0.f, 0.f, 0.f, 0.f};
        if (c < C4) {
            const U4 rx = philox((uint32_t)c, (uint32_t)row, 0u, STREAM_INIT_X, a.k0, a.k1);
            U4 rv{0, 0, 0, 0};
            if (!a.v_zero) rv = philox((uint32_t)c, (uint32_t)row, 0u, STREAM_INIT_V, a.k0, a.k1);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (4 * c + e < a.D) {
                    xo[e] = fmaf(wcomp(rx, e), xr, a.lb);
                    vo[e] = a.v_zero ? 0.0f : fmaf(wcomp(rv, e), vr, a.v_lo);
                }
            }
        }
        const float4 X = make_float4(xo[0], xo[1], xo[2], xo[3]);
        const float4 V = make_float4(vo[0], vo[1], vo[2], vo[3]);
        reinterpret_cast<float4 *>(a.x)[q] = X;
        reinterpret_cast<float4 *>(a.v)[q] = V;
        if (a.p) reinterpret_cast<float4 *>(a.p)[q] = X;
    }
}

hipError_t launch_init(const InitArgs &a, hipStream_t s)
{
    const int64_t total = a.N * (a.ldx / 4);
    int64_t grid = (total + 255) / 256;
    if (grid > 8 * kGridCap) grid = 8 * kGridCap;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(k_init, dim3((unsigned)grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Second pass of the selection: one block reduces the partials, stores the
// result, and copies the selected row (ldx floats) to row_out.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void k_select(const float *pval, const int64_t *pidx,
                                                 const uint32_t *pcnt, int n, const float *rows,
                                                 int64_t ldx, float *row_out, DevBest *best,
                                                 float *bf_out, int64_t *bi_out)
{
    __shared__ float sv[16];
    __shared__ int64_t si[16];
    __shared__ uint32_t sc[16];
    __shared__ int64_t sel;
    float v = __builtin_nanf("");
    int64_t i = INT64_MAX;
    uint32_t cnt = 0;
    for (int q = threadIdx.x; q < n; q += blockDim.x) {
        if (cand_better(pval[q], pidx[q], v, i)) {
            v = pval[q];
            i = pidx[q];
        }
        if (pcnt) cnt += pcnt[q];
    }
    block_argmin(v, i, cnt, sv, si, sc);
    if (threadIdx.x == 0) {
        if (i == INT64_MAX) i = 0;
        if (best) {
            best->f = v;
            best->i = i;
            best->improved += cnt;
        }
        if (bf_out) *bf_out = v;
        if (bi_out) *bi_out = i;
        sel = i;
    }
    __syncthreads();
    if (row_out) {
        const float *src = rows + sel * ldx;
        for (int64_t j = threadIdx.x; j < ldx; j += blockDim.x) row_out[j] = src[j];
    }
}

hipError_t launch_select(const float *pval, const int64_t *pidx, const uint32_t *pcnt, int nparts,
                         const float *rows, int64_t ldx, float *row_out, DevBest *best,
                         float *best_f_out, int64_t *best_i_out, hipStream_t s)
{
    hipLaunchKernelGGL(k_select, dim3(1), dim3(1024), 0, s, pval, pidx, pcnt, nparts, rows, ldx,
                       row_out, best, best_f_out, best_i_out);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void k_copy_row(const float *src, float *dst, int64_t n)
{
    for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < n; j += (int64_t)gridDim.x * 256)
        dst[j] = src[j];
}

hipError_t launch_copy_row(const float *src, float *dst, int64_t ldx, hipStream_t s)
{
    hipLaunchKernelGGL(k_copy_row, dim3(1), dim3(256), 0, s, src, dst, ldx);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void k_fill(float *dst, int64_t n, float value)
{
    for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < n; j += (int64_t)gridDim.x * 256)
        dst[j] = value;
}

__global__ void k_best_init(DevBest *best, float f, int64_t i)
{
    best->f = f;
    best->pad = 0;
    best->i = i;
    best->improved = 0;
}

hipError_t launch_best_init(DevBest *best, float f, int64_t i, hipStream_t s)
{
    hipLaunchKernelGGL(k_best_init, dim3(1), dim3(1), 0, s, best, f, i);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void k_zero_u32(uint32_t *dst, int64_t n)
{
    for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < n; j += (int64_t)gridDim.x * 256)
        dst[j] = 0u;
}

static unsigned flat_grid(int64_t n)
{
    int64_t g = (n + 255) / 256;
    if (g > kGridCap) g = kGridCap;
    if (g < 1) g = 1;
    return (unsigned)g;
}

hipError_t launch_fill(float *dst, int64_t n, float value, hipStream_t s)
{
    hipLaunchKernelGGL(k_fill, dim3(flat_grid(n)), dim3(256), 0, s, dst, n, value);
    return hipGetLastError();
}

hipError_t launch_zero_u32(uint32_t *dst, int64_t n, hipStream_t s)
{
    hipLaunchKernelGGL(k_zero_u32, dim3(flat_grid(n)), dim3(256), 0, s, dst, n);
    return hipGetLastError();
}

// First pass of the selection over a stored fitness array.
__global__ __launch_bounds__(256) void k_argmin_partials(const float *f, int64_t n, float *pval,
                                                         int64_t *pidx)
{
    __shared__ float sv[4];
    __shared__ int64_t si[4];
    __shared__ uint32_t sc[4];
    float v = __builtin_nanf("");
    int64_t i = INT64_MAX;
    uint32_t dummy = 0;
    for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < n; j += (int64_t)gridDim.x * 256)
        if (cand_better(f[j], j, v, i)) {
            v = f[j];
            i = j;
        }
    block_argmin(v, i, dummy, sv, si, sc);
    if (threadIdx.x == 0) {
        pval[blockIdx.x] = v;
        pidx[blockIdx.x] = i;
    }
}

int argmin_partials_grid(int64_t N) { return (int)flat_grid(N); }

hipError_t launch_argmin_partials(const float *f, int64_t N, float *pval, int64_t *pidx, int grid,
                                  hipStream_t s)
{
    hipLaunchKernelGGL(k_argmin_partials, dim3(grid), dim3(256), 0, s, f, N, pval, pidx);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Diagnostic: raw Philox words of the device generator.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_philox_fill(uint32_t k0, uint32_t k1, uint32_t c1,
                                                     uint32_t c2, uint32_t c3, int64_t n,
                                                     uint32_t *out)
{
    for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < n; k += (int64_t)gridDim.x * 256) {
        const U4 r = philox((uint32_t)k, c1, c2, c3, k0, k1);
        reinterpret_cast<uint4 *>(out)[k] = make_uint4(r.x, r.y, r.z, r.w);
    }
}

hipError_t launch_philox_fill(uint32_t k0, uint32_t k1, uint32_t c1, uint32_t c2, uint32_t c3,
                              int64_t n, uint32_t *out, hipStream_t s)
{
    int64_t grid = (n + 255) / 256;
    if (grid > kGridCap) grid = kGridCap;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(k_philox_fill, dim3((unsigned)grid), dim3(256), 0, s, k0, k1, c1, c2, c3, n,
                       out);
    return hipGetLastError();
}

__device__ __forceinline__ uint32_t bucket_of(uint32_t key, int bits)
{
    return bits ? key >> (32 - bits) : 0u;
}

__global__ __launch_bounds__(256) void k_perm_hist(PermArgs a)
{
    const int64_t nq = (a.N + 3) / 4;
    for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < nq; q += (int64_t)gridDim.x * 256) {
        const U4 r = philox((uint32_t)q, 0u, a.t, STREAM_PERM, a.k0, a.k1);
        const uint32_t k4[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (4 * q + e < a.N) atomicAdd(&a.hist[bucket_of(k4[e], a.bits)], 1u);
    }
}

// One block: offs[b] = sum of hist[0..b), offs[nb] = N, cursor = offs, and
// the counts are cleared for the next generation.
__global__ __launch_bounds__(1024) void k_perm_scan(PermArgs a)
{
    __shared__ uint32_t part[1024];
    const int64_t nb = (int64_t)1 << a.bits;
    const int64_t per = (nb + 1023) / 1024;
    const int64_t lo = threadIdx.x * per, hi = lo + per < nb ? lo + per : nb;
    uint32_t s = 0;
    for (int64_t b = lo; b < hi; ++b) s += a.hist[b];
    part[threadIdx.x] = s;
    __syncthreads();
    // Hillis-Steele inclusive scan over the 1024 thread sums
    for (int off = 1; off < 1024; off <<= 1) {
        const uint32_t v = threadIdx.x >= off ? part[threadIdx.x - off] : 0u;
        __syncthreads();
        part[threadIdx.x] += v;
        __syncthreads();
    }
    uint32_t run = threadIdx.x ? part[threadIdx.x - 1] : 0u;
    for (int64_t b = lo; b < hi; ++b) {
        const uint32_t c = a.hist[b];
        a.offs[b] = run;
        a.cursor[b] = run;
        a.hist[b] = 0u;
        run += c;
    }
    if (threadIdx.x == 0) a.offs[nb] = (uint32_t)a.N;
}

__global__ __launch_bounds__(256) void k_perm_scatter(PermArgs a)
{
    const int64_t nq = (a.N + 3) / 4;
    for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < nq; q += (int64_t)gridDim.x * 256) {
        const U4 r = philox((uint32_t)q, 0u, a.t, STREAM_PERM, a.k0, a.k1);
        const uint32_t k4[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int64_t i = 4 * q + e;
            if (i < a.N) {
                const uint32_t pos = atomicAdd(&a.cursor[bucket_of(k4[e], a.bits)], 1u);
                a.tkey[pos] = k4[e];
                a.tidx[pos] = (uint32_t)i;
            }
        }
    }
}

__global__ __launch_bounds__(256) void k_perm_rank(PermArgs a)
{
    for (int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x; p < a.N; p += (int64_t)gridDim.x * 256) {
        const uint32_t key = a.tkey[p], idx = a.tidx[p];
        const uint32_t b = bucket_of(key, a.bits);
        const uint32_t lo = a.offs[b], hi = a.offs[b + 1];
        uint32_t rank = 0;
        for (uint32_t q = lo; q < hi; ++q) {
            const uint32_t kq = a.tkey[q], iq = a.tidx[q];
            rank += (kq < key || (kq == key && iq < idx)) ? 1u : 0u;
        }
        a.perm[lo + rank] = idx;
    }
}

hipError_t launch_perm(const PermArgs &a, hipStream_t s)
{
    const int64_t nq = (a.N + 3) / 4;
    int64_t g1 = (nq + 255) / 256, g2 = (a.N + 255) / 256;
    if (g1 > kGridCap) g1 = kGridCap;
    if (g2 > kGridCap) g2 = kGridCap;
    hipLaunchKernelGGL(k_perm_hist, dim3((unsigned)g1), dim3(256), 0, s, a);
    hipLaunchKernelGGL(k_perm_scan, dim3(1), dim3(1024), 0, s, a);
    hipLaunchKernelGGL(k_perm_scatter, dim3((unsigned)g1), dim3(256), 0, s, a);
    hipLaunchKernelGGL(k_perm_rank, dim3((unsigned)g2), dim3(256), 0, s, a);
    return hipGetLastError();
}

// xbar_j = (sum over the partial rows, in order) / N, rounded once; zero in
// the padding columns.  Block: 64 columns x 4 partial-row lanes.
__global__ __launch_bounds__(256) void k_cso_mean(const double *xsum, int nparts, int64_t N,
                                                  int64_t D, int64_t ldx, float *xbar)
{
    __shared__ double part[4][64];
    const int col = threadIdx.x & 63, lane = threadIdx.x >> 6;
    const int64_t j = (int64_t)blockIdx.x * 64 + col;
    double s = 0.0;
    if (j < D)
        for (int q = lane; q < nparts; q += 4) s += xsum[(int64_t)q * ldx + j];
    part[lane][col] = s;
    __syncthreads();
    if (lane == 0 && j < ldx) {
        const double t = ((part[0][col] + part[1][col]) + part[2][col]) + part[3][col];
        xbar[j] = j < D ? (float)(t / (double)N) : 0.0f;
    }
}

hipError_t launch_cso_mean(const double *xsum, int nparts, int64_t N, int64_t D, int64_t ldx,
                           float *xbar, hipStream_t s)
{
    const int64_t grid = (ldx + 63) / 64;
    hipLaunchKernelGGL(k_cso_mean, dim3((unsigned)grid), dim3(256), 0, s, xsum, nparts, N, D, ldx,
                       xbar);
    return hipGetLastError();
}

#define EVOX_LAUNCH_COLSUM(GG, UNUSED) \
    hipLaunchKernelGGL((k_colsum<GG>), dim3(grid), dim3(block_for(GG)), 0, s, x, N, D, ldx, xsum)

hipError_t launch_colsum(int G, const float *x, int64_t N, int64_t D, int64_t ldx, double *xsum,
                         int grid, hipStream_t s)
{
    EVOX_G_CASES(EVOX_LAUNCH_COLSUM, 0)
    return hipGetLastError();
}

#define EVOX_FN_SWITCH(CALL)                                                                      \
    switch (fn) {                                                                                 \
    case FN_SPHERE: return CALL(FN_SPHERE);                                                       \
    case FN_ACKLEY: return CALL(FN_ACKLEY);                                                       \
    case FN_RASTRIGIN: return CALL(FN_RASTRIGIN);                                                 \
    case FN_GRIEWANK: return CALL(FN_GRIEWANK);                                                   \
    case FN_ROSENBROCK: return CALL(FN_ROSENBROCK);                                               \
    case FN_SCHWEFEL: return CALL(FN_SCHWEFEL);                                                   \
    default: return hipErrorInvalidValue;                                                         \
    }

hipError_t launch_pso(int fn, int G, int mode, const PsoArgs &a, int grid, hipStream_t s)
{
    if (mode == PSO_MOVE) fn = FN_SPHERE;  // the move does not evaluate
#define EVOX_CALL_PSO(F) launch_pso_t<F>(G, mode, a, grid, s)
    EVOX_FN_SWITCH(EVOX_CALL_PSO)
}

hipError_t launch_eval(int fn, int G, bool vec, const EvalArgs &a, int grid, hipStream_t s)
{
#define EVOX_CALL_EVAL(F) launch_eval_t<F>(G, vec, a, grid, s)
    EVOX_FN_SWITCH(EVOX_CALL_EVAL)
}

hipError_t launch_cso(int fn, int G, const CsoArgs &a, int grid, hipStream_t s)
{
#define EVOX_CALL_CSO(F) launch_cso_t<F>(G, a, grid, s)
    EVOX_FN_SWITCH(EVOX_CALL_CSO)
}

}  // namespace evox
