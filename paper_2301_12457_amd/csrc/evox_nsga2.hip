// NSGA-II on DTLZ1 (Table II; the multi-objective scaling experiment of
// Sec. VII-A-2, whose speed-up the paper attributes to computing the dominance
// relations in parallel).  Deb, Pratap, Agarwal, Meyarivan (2002):
//   variation   crowded binary tournaments, simulated binary crossover and
//               polynomial mutation (one thread per pair and variable, fp64);
//   objectives  DTLZ1 (one wave per row, fp64: its g is a difference of
//               numbers near 100 k that fp32 would not resolve near the front);
//   sorting     dominator counts over all pairs (tiled through LDS, exact
//               integer atomics), then fronts peeled one at a time: the
//               unassigned points with no unassigned dominator form the next
//               front, whose members are appended to a list (fronts stored
//               contiguously) and their dominance subtracted from the rest;
//   crowding    each front member's position in every objective's order of
//               (value, index) by counting within its front (tiles of the
//               front through LDS), then the distance summed objective by
//               objective in that order;
//   selection   whole fronts, then the last front's members of largest
//               crowding distance (lower index on ties) by counting, and a
//               compaction that keeps the merged order.
#include "evox_launch.hpp"

#include <cmath>

namespace evox {

namespace {

constexpr int kSpan = 512;  // points per LDS tile of the pair kernels
constexpr double kPi = 3.14159265358979323846;

__device__ __forceinline__ int64_t crowded_winner(int64_t a, int64_t b, const int32_t *front, const double *crowd)
{
    if (front[a] != front[b]) return front[a] < front[b] ? a : b;
    if (crowd[a] != crowd[b]) return crowd[a] > crowd[b] ? a : b;
    return a < b ? a : b;
}

// Polynomial mutation of x in [0, 1] with draw u and index eta (the bounded
// form of Deb and Goyal): u < 1/2 lowers x by 1 - (2u + (1 - 2u)(1 - x)^(eta+1))
// ^(1/(eta+1)), u >= 1/2 raises it by 1 - (2(1 - u) + 2(u - 1/2) x^(eta+1))
// ^(1/(eta+1)); clipped to [0, 1].
__device__ double poly_mutate(double x, double u, double eta)
{
    const double e1 = eta + 1.0, inv = 1.0 / e1;
    double y;
    if (u < 0.5)
        y = x + (pow(2.0 * u + (1.0 - 2.0 * u) * pow(1.0 - x, e1), inv) - 1.0);
    else
        y = x + (1.0 - pow(2.0 * (1.0 - u) + 2.0 * (u - 0.5) * pow(x, e1), inv));
    return y < 0.0 ? 0.0 : y > 1.0 ? 1.0 : y;
}

// Offspring rows 2p and 2p + 1, variable j (one thread each): parents from
// the tournaments (w of Philox(0, p, t, 10): candidates floor(w_q N / 2^32),
// (w_0, w_1) and (w_2, w_3)); crossover and mutation draws from Philox(j, p,
// t, 11) and (j, p, t, 12).
__global__ __launch_bounds__(256) void k_nsga_var(NsgaVarArgs a)
{
    const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x, H = a.N / 2;
    if (q >= H * a.D) return;
    const int64_t p = q / a.D, j = q % a.D;
    const U4 ws = philox(0u, (uint32_t)p, a.t, STREAM_NSGA_SEL, a.k0, a.k1);
    const uint64_t n = (uint64_t)a.N;
    const int64_t c0 = (int64_t)(((uint64_t)ws.x * n) >> 32), c1 = (int64_t)(((uint64_t)ws.y * n) >> 32);
    const int64_t c2 = (int64_t)(((uint64_t)ws.z * n) >> 32), c3 = (int64_t)(((uint64_t)ws.w * n) >> 32);
    const int64_t pa = crowded_winner(c0, c1, a.front, a.crowd), pb = crowded_winner(c2, c3, a.front, a.crowd);
    const U4 w = philox((uint32_t)j, (uint32_t)p, a.t, STREAM_NSGA_VAR, a.k0, a.k1);
    const U4 v = philox((uint32_t)j, (uint32_t)p, a.t, STREAM_NSGA_MUT, a.k0, a.k1);
    const double ec = a.eta_c, em = a.eta_m, pm = 1.0 / (double)a.D;
    const double u = (double)u01(w.x);
    double beta = u <= 0.5 ? pow(2.0 * u, 1.0 / (ec + 1.0)) : pow(2.0 - 2.0 * u, -1.0 / (ec + 1.0));
    if (w.y & 1u) beta = -beta;
    if ((double)u01(w.y) >= 0.5) beta = 1.0;
    const double xa = (double)a.X[pa * a.ldx + j], xb = (double)a.X[pb * a.ldx + j];
    const double y[2] = {0.5 * (xa + xb) + 0.5 * beta * (xa - xb), 0.5 * (xa + xb) - 0.5 * beta * (xa - xb)};
    const uint32_t coin[2] = {w.z, w.w}, mu[2] = {v.x, v.y};
    for (int c = 0; c < 2; ++c) {
        const double yc = y[c] < 0.0 ? 0.0 : y[c] > 1.0 ? 1.0 : y[c];
        float out = (float)yc;
        if ((double)u01(coin[c]) < pm) out = (float)poly_mutate((double)out, (double)u01(mu[c]), em);
        a.Q[(2 * p + c) * a.ldx + j] = out;
    }
}

// DTLZ1 of row r (one wave): g = 100 (k + sum_{i >= M-1} ((x_i - 1/2)^2 -
// cos(20 pi (x_i - 1/2)))), f_0 = (1 + g)/2 x_0 ... x_{M-2}, f_m = (1 + g)/2
// x_0 ... x_{M-2-m} (1 - x_{M-1-m}); fp64, each objective rounded once.
__global__ __launch_bounds__(256) void k_nsga_dtlz1(const float *X, int64_t n, int64_t D, int64_t ldx, int32_t M,
                                                    float *F)
{
    const int64_t r = (int64_t)blockIdx.x * 4 + threadIdx.x / 64;
    const int lane = threadIdx.x % 64;
    if (r >= n) return;
    const float *x = X + r * ldx;
    double acc = 0.0;
    for (int64_t i = M - 1 + lane; i < D; i += 64) {
        const double d = (double)x[i] - 0.5;
        acc += d * d - cos(20.0 * kPi * d);
    }
    for (int o = 32; o > 0; o /= 2) acc += __shfl_xor(acc, o);
    if (lane < M) {
        const int m = lane;
        const double g = 100.0 * ((double)(D - M + 1) + acc);
        double f = 0.5 * (1.0 + g);
        for (int i = 0; i < M - 1 - m; ++i) f *= (double)x[i];
        if (m > 0) f *= 1.0 - (double)x[M - 1 - m];
        F[r * M + m] = (float)f;
    }
}

// Objectives of a point padded to P = 4 or 8 floats in LDS (read back as
// float4 broadcasts: every lane of a wave reads the same point).
template <int P>
__device__ __forceinline__ void load_pad(float *dst, const float *F, int64_t row, int32_t M)
{
#pragma unroll
    for (int m = 0; m < P; ++m) dst[m] = m < M ? F[row * M + m] : 0.0f;
}

// Dominance of b by a for M objectives known at compile time (comparisons as
// written: NaN neither dominates nor is dominated differently than in the
// definition).
template <int M>
__device__ __forceinline__ bool dominates_t(const float *a, const float *b)
{
    bool worse = false, better = false;
#pragma unroll
    for (int m = 0; m < M; ++m) {
        worse |= a[m] > b[m];
        better |= a[m] < b[m];
    }
    return !worse && better;
}

// cnt[i] += #{j in this block's span : F_j dominates F_i}.
template <int M>
__global__ __launch_bounds__(256) void k_nsga_count(const float *F, int64_t n, uint32_t *cnt)
{
    constexpr int P = M <= 4 ? 4 : 8;
    __shared__ __align__(16) float fj[kSpan * P];
    const int64_t j0 = (int64_t)blockIdx.y * kSpan, nj = n - j0 < kSpan ? n - j0 : kSpan;
    for (int64_t q = threadIdx.x; q < nj; q += 256) load_pad<P>(fj + q * P, F, j0 + q, M);
    __syncthreads();
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    float fi[M];
#pragma unroll
    for (int m = 0; m < M; ++m) fi[m] = F[i * M + m];
    uint32_t c = 0;
#pragma unroll 4
    for (int64_t q = 0; q < nj; ++q) {
        float v[P];
#pragma unroll
        for (int h = 0; h < P / 4; ++h) {
            const float4 t = *reinterpret_cast<const float4 *>(fj + q * P + 4 * h);
            v[4 * h] = t.x, v[4 * h + 1] = t.y, v[4 * h + 2] = t.z, v[4 * h + 3] = t.w;
        }
        c += dominates_t<M>(v, fi);
    }
    if (c) atomicAdd(cnt + i, c);
}

// Front k: unassigned points with no unassigned dominator, appended to list.
// Fronts are peeled kNsgaPeelBatch at a time without a host round trip:
// lens[kb] counts front (k0 + kb) of the batch, the fronts before the batch
// hold `assigned0` points, and a front is only marked (peeled) while the
// points assigned before it (with it) are fewer than `need`.
__device__ __forceinline__ int64_t batch_base(const uint32_t *lens, int32_t kb, int64_t assigned0)
{
    int64_t base = assigned0;
    for (int32_t r = 0; r < kb; ++r) base += lens[r];
    return base;
}

__global__ __launch_bounds__(256) void k_nsga_mark(int32_t *front, const uint32_t *cnt, int64_t n, int32_t k,
                                                   int32_t kb, int64_t assigned0, int64_t need, int32_t *list,
                                                   uint32_t *lens)
{
    const int64_t base = batch_base(lens, kb, assigned0);
    if (base >= need) return;  // the fronts needed are complete
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n || front[i] != -1 || cnt[i] != 0) return;
    front[i] = k;
    list[base + atomicAdd(lens + kb, 1u)] = (int32_t)i;
}

// cnt[i] -= #{j in this block's span of the new front : F_j dominates F_i}
// for the points still unassigned.
template <int M>
__global__ __launch_bounds__(256) void k_nsga_peel(const float *F, int64_t n, const int32_t *list_all,
                                                   const uint32_t *lens, int32_t kb, int64_t assigned0,
                                                   int64_t need, const int32_t *front, uint32_t *cnt)
{
    constexpr int P = M <= 4 ? 4 : 8;
    __shared__ __align__(16) float fj[kSpan * P];
    const int64_t base = batch_base(lens, kb, assigned0), size = lens[kb];
    const int64_t q0 = (int64_t)blockIdx.y * kSpan;
    // the grid covers the largest possible front; spans past this one's
    // size, and every span once no later front is needed, exit at once
    // (uniform over the block, before the barrier)
    if (base + size >= need || q0 >= size) return;
    const int32_t *list = list_all + base;
    const int64_t nq = size - q0 < kSpan ? size - q0 : kSpan;
    for (int64_t q = threadIdx.x; q < nq; q += 256) load_pad<P>(fj + q * P, F, list[q0 + q], M);
    __syncthreads();
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n || front[i] != -1) return;
    float fi[M];
#pragma unroll
    for (int m = 0; m < M; ++m) fi[m] = F[i * M + m];
    uint32_t c = 0;
#pragma unroll 4
    for (int64_t q = 0; q < nq; ++q) {
        float v[P];
#pragma unroll
        for (int h = 0; h < P / 4; ++h) {
            const float4 t = *reinterpret_cast<const float4 *>(fj + q * P + 4 * h);
            v[4 * h] = t.x, v[4 * h + 1] = t.y, v[4 * h + 2] = t.z, v[4 * h + 3] = t.w;
        }
        c += dominates_t<M>(v, fi);
    }
    if (c) atomicSub(cnt + i, c);
}

// foff[k] = first list position of front k; foff[K] = total.
__global__ __launch_bounds__(256) void k_nsga_foff(const int32_t *list, int64_t total, const int32_t *front,
                                                   int32_t *foff)
{
    const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (q >= total) return;
    const int32_t k = front[list[q]];
    if (q == 0 || front[list[q - 1]] != k) foff[k] = (int32_t)q;
    if (q == total - 1) foff[k + 1] = (int32_t)total;
}

// Position of list entry q in each objective's order of (value, index)
// within its front: pos[m][q] += #{list entries r of the same front in this
// block's span : (F_r,m, r's point) < (F_q,m, q's point)}.  Fronts are
// contiguous in the list, so a block whose span lies outside its entries'
// fronts exits at once; the work is the sum of the squared front sizes.
template <int M>
__global__ __launch_bounds__(256) void k_nsga_order(NsgaSortArgs a, int64_t total)
{
    constexpr int P = M <= 4 ? 4 : 8;
    __shared__ __align__(16) float fj[kSpan * P];
    __shared__ int32_t ij[kSpan], kj[kSpan];
    const int64_t q0 = (int64_t)blockIdx.x * 256, r0 = (int64_t)blockIdx.y * kSpan;
    const int64_t qlast = q0 + 255 < total ? q0 + 255 : total - 1;
    const int32_t lo = a.foff[a.front[a.list[q0]]], hi = a.foff[a.front[a.list[qlast]] + 1];
    const int64_t nr = total - r0 < kSpan ? total - r0 : kSpan;
    if (r0 >= hi || r0 + nr <= lo) return;
    for (int64_t r = threadIdx.x; r < nr; r += 256) {
        const int32_t j = a.list[r0 + r];
        ij[r] = j;
        kj[r] = a.front[j];
        load_pad<P>(fj + r * P, a.F, j, M);
    }
    __syncthreads();
    const int64_t q = q0 + threadIdx.x;
    if (q >= total) return;
    const int32_t i = a.list[q], k = a.front[i];
    float fi[M];
    int32_t c[M];
#pragma unroll
    for (int m = 0; m < M; ++m) {
        fi[m] = a.F[(int64_t)i * M + m];
        c[m] = 0;
    }
    for (int64_t r = 0; r < nr; ++r) {
        if (kj[r] != k) continue;
        const int32_t j = ij[r];
        float v[P];
#pragma unroll
        for (int h = 0; h < P / 4; ++h) {
            const float4 t = *reinterpret_cast<const float4 *>(fj + r * P + 4 * h);
            v[4 * h] = t.x, v[4 * h + 1] = t.y, v[4 * h + 2] = t.z, v[4 * h + 3] = t.w;
        }
#pragma unroll
        for (int m = 0; m < M; ++m) c[m] += (v[m] < fi[m]) || (v[m] == fi[m] && j < i);
    }
#pragma unroll
    for (int m = 0; m < M; ++m)
        if (c[m]) atomicAdd(a.pos + m * a.cap + q, c[m]);
}

// sorted[m][foff[k] + pos[m][q]] = the point of list entry q.
__global__ __launch_bounds__(256) void k_nsga_scatter(NsgaSortArgs a, int64_t total)
{
    const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (q >= total) return;
    const int32_t i = a.list[q], b = a.foff[a.front[i]];
    for (int m = 0; m < a.M; ++m) a.sorted[m * a.cap + b + a.pos[m * a.cap + q]] = i;
}

// Crowding distance of list entry q: per objective in order, +inf at either
// end of the front's order, else + (next - previous) / (last - first) when
// the range is not zero (fp64).
__global__ __launch_bounds__(256) void k_nsga_crowd(NsgaSortArgs a, int64_t total)
{
    const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (q >= total) return;
    const int32_t i = a.list[q], k = a.front[i];
    const int32_t b = a.foff[k], e = a.foff[k + 1], size = e - b;
    double d = 0.0;
    for (int m = 0; m < a.M; ++m) {
        const int32_t p = a.pos[m * a.cap + q];
        const int32_t *srt = a.sorted + m * a.cap + b;
        if (p == 0 || p == size - 1) {
            d = INFINITY;
        } else {
            const double lo = (double)a.F[(int64_t)srt[0] * a.M + m];
            const double hi = (double)a.F[(int64_t)srt[size - 1] * a.M + m];
            if (hi > lo)
                d += ((double)a.F[(int64_t)srt[p + 1] * a.M + m] - (double)a.F[(int64_t)srt[p - 1] * a.M + m]) /
                     (hi - lo);
        }
    }
    a.crowd[i] = d;
}

// Rank of the last front's entry q (list positions [full, total)) in the
// order of (crowding descending, index): rank[q - full] += #{entries of this
// block's span ahead of it}.
__global__ __launch_bounds__(256) void k_nsga_trunc(const int32_t *list, int64_t full, int64_t total,
                                                    const double *crowd, int32_t *rank)
{
    __shared__ double cj[kSpan];
    __shared__ int32_t ij[kSpan];
    const int64_t size = total - full, r0 = (int64_t)blockIdx.y * kSpan;
    const int64_t nr = size - r0 < kSpan ? size - r0 : kSpan;
    for (int64_t r = threadIdx.x; r < nr; r += 256) {
        const int32_t j = list[full + r0 + r];
        ij[r] = j;
        cj[r] = crowd[j];
    }
    __syncthreads();
    const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (q >= size) return;
    const int32_t i = list[full + q];
    const double ci = crowd[i];
    int32_t c = 0;
    // bitwise, not short-circuit: no branch per entry, so the loop unrolls
#pragma unroll 8
    for (int64_t r = 0; r < nr; ++r) c += (int32_t)((cj[r] > ci) | ((cj[r] == ci) & (ij[r] < i)));
    if (c) atomicAdd(rank + q, c);
}

// keep[i] for the survivors: the members of the fronts before the last, and
// the last front's entries ranked below `need`.
__global__ __launch_bounds__(256) void k_nsga_keep(const int32_t *list, int64_t full, int64_t total, int64_t need,
                                                   const int32_t *rank, int32_t *keep)
{
    const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (q >= total) return;
    if (q < full || rank[q - full] < need) keep[list[q]] = 1;
}

// Exclusive prefix sums of keep[0 .. n) in three passes: each block of
// kScanChunk entries sums its entries; one block turns the block sums into
// exclusive offsets; each block scans its entries from its offset.
constexpr int kScanChunk = 1024;

__global__ __launch_bounds__(256) void k_nsga_scan_sums(const int32_t *keep, int64_t n, int32_t *sums)
{
    __shared__ int32_t part[256];
    const int64_t b = (int64_t)blockIdx.x * kScanChunk;
    int32_t v = 0;
    for (int64_t i = b + threadIdx.x; i < b + kScanChunk && i < n; i += 256) v += keep[i];
    part[threadIdx.x] = v;
    __syncthreads();
    for (int o = 128; o > 0; o /= 2) {
        if (threadIdx.x < (unsigned)o) part[threadIdx.x] += part[threadIdx.x + o];
        __syncthreads();
    }
    if (threadIdx.x == 0) sums[blockIdx.x] = part[0];
}

__global__ __launch_bounds__(256) void k_nsga_scan_offsets(int32_t *sums, int64_t nb)
{
    if (threadIdx.x != 0) return;
    int32_t run = 0;
    for (int64_t q = 0; q < nb; ++q) {
        const int32_t v = sums[q];
        sums[q] = run;
        run += v;
    }
}

__global__ __launch_bounds__(256) void k_nsga_scan_local(const int32_t *keep, int64_t n, const int32_t *sums,
                                                         int32_t *pre)
{
    __shared__ int32_t part[256];
    const int64_t b = (int64_t)blockIdx.x * kScanChunk + 4 * threadIdx.x;
    int32_t v[4], s = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        v[e] = b + e < n ? keep[b + e] : 0;
        s += v[e];
    }
    part[threadIdx.x] = s;
    __syncthreads();
    for (int o = 1; o < 256; o *= 2) {
        const int32_t t = threadIdx.x >= (unsigned)o ? part[threadIdx.x - o] : 0;
        __syncthreads();
        part[threadIdx.x] += t;
        __syncthreads();
    }
    int32_t run = sums[blockIdx.x] + (threadIdx.x ? part[threadIdx.x - 1] : 0);
#pragma unroll
    for (int e = 0; e < 4; ++e)
        if (b + e < n) {
            pre[b + e] = run;
            run += v[e];
        }
}

// Survivor i of the merged population (parents 0..N-1, offspring N..2N-1)
// to row pre[i]: its row (float4 chunk c per thread), objectives, front and
// crowding distance.
__global__ __launch_bounds__(256) void k_nsga_compact(NsgaSelArgs a)
{
    const int64_t c4 = a.ldx / 4, q = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (q >= 2 * a.N * c4) return;
    const int64_t i = q / c4, c = q % c4;
    if (!a.keep[i]) return;
    const int64_t r = a.pre[i];
    const float *src = i < a.N ? a.X + i * a.ldx : a.Q + (i - a.N) * a.ldx;
    *reinterpret_cast<float4 *>(a.X2 + r * a.ldx + 4 * c) = *reinterpret_cast<const float4 *>(src + 4 * c);
    if (c == 0) {
        for (int m = 0; m < a.M; ++m) a.F[r * a.M + m] = a.FR[i * a.M + m];
        a.front[r] = a.frontR[i];
        a.crowd[r] = a.crowdR[i];
    }
}

__global__ __launch_bounds__(256) void k_fill_i32(int32_t *p, int64_t n, int32_t v)
{
    for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < n; q += (int64_t)gridDim.x * 256) p[q] = v;
}

unsigned blocks(int64_t n, int64_t per) { return (unsigned)((n + per - 1) / per); }

#define EVOX_NSGA_M_SWITCH(M, CALL) \
    switch (M) {                   \
        case 2: CALL(2); break;    \
        case 3: CALL(3); break;    \
        case 4: CALL(4); break;    \
        case 5: CALL(5); break;    \
        case 6: CALL(6); break;    \
        case 7: CALL(7); break;    \
        case 8: CALL(8); break;    \
        default: return hipErrorInvalidValue; \
    }

}  // namespace

hipError_t launch_nsga_var(const NsgaVarArgs &a, hipStream_t s)
{
    const int64_t n = a.N / 2 * a.D;
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_nsga_var, dim3(blocks(n, 256)), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_nsga_dtlz1(const float *X, int64_t n, int64_t D, int64_t ldx, int32_t M, float *F, hipStream_t s)
{
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_nsga_dtlz1, dim3(blocks(n, 4)), dim3(256), 0, s, X, n, D, ldx, M, F);
    return hipGetLastError();
}

hipError_t nsga_count(const NsgaSortArgs &a, hipStream_t s)
{
    const int64_t n = a.n;
    if (n == 0) return hipSuccess;
    hipError_t e;
    hipLaunchKernelGGL(k_fill_i32, dim3(blocks(n, 256) < 4096 ? blocks(n, 256) : 4096), dim3(256), 0, s, a.front,
                       n, -1);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_zero_u32(a.cnt, n, s)) != hipSuccess) return e;
    const dim3 grid(blocks(n, 256), blocks(n, kSpan));
#define EVOX_COUNT(MM) hipLaunchKernelGGL((k_nsga_count<MM>), grid, dim3(256), 0, s, a.F, n, a.cnt)
    EVOX_NSGA_M_SWITCH(a.M, EVOX_COUNT)
#undef EVOX_COUNT
    return hipGetLastError();
}

hipError_t nsga_fronts(const NsgaSortArgs &a, int64_t need, NsgaSortResult *res, hipStream_t s)
{
    const int64_t n = a.n;
    *res = NsgaSortResult{0, 0, 0};
    if (n == 0) return hipSuccess;
    hipError_t e;
    // every slot of the per-objective orders holds a valid index even if the
    // order kernel were handed values without a total order
    hipLaunchKernelGGL(k_fill_i32, dim3(4096), dim3(256), 0, s, a.sorted, (int64_t)a.M * a.cap, 0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    int64_t assigned = 0, last = 0;
    int32_t k = 0;
    uint32_t lens[kNsgaPeelBatch];
    while (assigned < need) {
        if ((e = launch_zero_u32(a.len, kNsgaPeelBatch, s)) != hipSuccess) return e;
        const dim3 grid(blocks(n, 256), blocks(n - assigned, kSpan));
        for (int32_t kb = 0; kb < kNsgaPeelBatch; ++kb) {
            hipLaunchKernelGGL(k_nsga_mark, dim3(blocks(n, 256)), dim3(256), 0, s, a.front,
                               (const uint32_t *)a.cnt, n, k + kb, kb, assigned, need, a.list, a.len);
            if ((e = hipGetLastError()) != hipSuccess) return e;
#define EVOX_PEEL(MM)                                                                                      \
    hipLaunchKernelGGL((k_nsga_peel<MM>), grid, dim3(256), 0, s, a.F, n, (const int32_t *)a.list,          \
                       (const uint32_t *)a.len, kb, assigned, need, (const int32_t *)a.front, a.cnt)
            EVOX_NSGA_M_SWITCH(a.M, EVOX_PEEL)
#undef EVOX_PEEL
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        if ((e = hipMemcpyAsync(lens, a.len, sizeof lens, hipMemcpyDeviceToHost, s)) != hipSuccess ||
            (e = hipStreamSynchronize(s)) != hipSuccess)
            return e;
        for (int32_t kb = 0; kb < kNsgaPeelBatch && assigned < need; ++kb) {
            if (lens[kb] == 0) return hipErrorUnknown;  // cannot happen: a finite set has a non-dominated point
            last = lens[kb];
            assigned += last;
            ++k;
        }
    }
    hipLaunchKernelGGL(k_nsga_foff, dim3(blocks(assigned, 256)), dim3(256), 0, s, (const int32_t *)a.list, assigned,
                       (const int32_t *)a.front, a.foff);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_fill_i32, dim3(4096), dim3(256), 0, s, a.pos, (int64_t)a.M * a.cap, 0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const dim3 og(blocks(assigned, 256), blocks(assigned, kSpan));
#define EVOX_ORDER(MM) hipLaunchKernelGGL((k_nsga_order<MM>), og, dim3(256), 0, s, a, assigned)
    EVOX_NSGA_M_SWITCH(a.M, EVOX_ORDER)
#undef EVOX_ORDER
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_nsga_scatter, dim3(blocks(assigned, 256)), dim3(256), 0, s, a, assigned);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_nsga_crowd, dim3(blocks(assigned, 256)), dim3(256), 0, s, a, assigned);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    *res = NsgaSortResult{k, assigned, last};
    return hipSuccess;
}

hipError_t nsga_sort(const NsgaSortArgs &a, int64_t need, NsgaSortResult *res, hipStream_t s)
{
    hipError_t e = nsga_count(a, s);
    return e != hipSuccess ? e : nsga_fronts(a, need, res, s);
}

hipError_t launch_nsga_select(const NsgaSelArgs &a, const NsgaSortResult &r, hipStream_t s)
{
    const int64_t full = r.assigned - r.last, need = a.N - full;
    hipError_t e;
    hipLaunchKernelGGL(k_fill_i32, dim3(blocks(2 * a.N, 256) < 4096 ? blocks(2 * a.N, 256) : 4096), dim3(256), 0, s,
                       a.keep, 2 * a.N, 0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_zero_u32((uint32_t *)a.rank, r.last, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_nsga_trunc, dim3(blocks(r.last, 256), blocks(r.last, kSpan)), dim3(256), 0, s, a.list, full,
                       r.assigned, a.crowdR, a.rank);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_nsga_keep, dim3(blocks(r.assigned, 256)), dim3(256), 0, s, a.list, full, r.assigned, need,
                       (const int32_t *)a.rank, a.keep);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int64_t nb = (2 * a.N + kScanChunk - 1) / kScanChunk;
    hipLaunchKernelGGL(k_nsga_scan_sums, dim3((unsigned)nb), dim3(256), 0, s, (const int32_t *)a.keep, 2 * a.N,
                       a.sums);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_nsga_scan_offsets, dim3(1), dim3(256), 0, s, a.sums, nb);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_nsga_scan_local, dim3((unsigned)nb), dim3(256), 0, s, (const int32_t *)a.keep, 2 * a.N,
                       (const int32_t *)a.sums, a.pre);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_nsga_compact, dim3(blocks(2 * a.N * (a.ldx / 4), 256)), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace evox
