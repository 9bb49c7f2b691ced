// The matrix-adaptation ES generation (CMA-ES of Table II in the form of
// Beyer and Sendhoff, 2017) apart from its two matrix products and the
// fitness pass: deviates, parent selection, recombination of the center and
// the path together with the factors of the rank-mu update, and the step
// size.  With s' the new path and d_i = M z_i the steps of the parents,
//     M [I + c_1/2 (s' s'^T - I) + c_w/2 (sum_i w_i z_i z_i^T - I)]
//   = (1 - (c_1 + c_w)/2) M + (M s') (c_1/2 s')^T + sum_i d_i (c_w/2 w_i z_i)^T,
// and M s' = (1 - c_s) M s + sqrt(mu_eff c_s (2 - c_s)) sum_i w_i d_i, so the
// update is one rank-(mu + 1) product of two factors that this file writes
// k-major ([term][column], so that a wave's operand loads are coalesced) and
// then applies to M in one streaming pass, and M s comes from the sampling
// product (the path rides along as an extra deviate row).
#include "evox_launch.hpp"

namespace evox {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

// Deviates z_k (rows k < N, Philox stream 9 with the generation in the
// counter) and the path s (row N); columns D..ldx-1 zero.
__global__ __launch_bounds__(256) void k_mae_sample(MaeArgs a)
{
    const int64_t q4 = a.ldx / 4, total = (a.N + 1) * q4;
    for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < total; q += (int64_t)gridDim.x * 256) {
        const int64_t row = q / q4, c = q % q4;
        float4 v;
        if (row < a.N) {
            const float4 z = normal4((uint32_t)c, (uint32_t)row, a.t, STREAM_MAES, a.k0, a.k1);
            v.x = 4 * c + 0 < a.D ? z.x : 0.0f;
            v.y = 4 * c + 1 < a.D ? z.y : 0.0f;
            v.z = 4 * c + 2 < a.D ? z.z : 0.0f;
            v.w = 4 * c + 3 < a.D ? z.w : 0.0f;
        } else {
            v = *reinterpret_cast<const float4 *>(a.s + 4 * c);
        }
        *reinterpret_cast<float4 *>(a.Z + row * a.ldx + 4 * c) = v;
    }
}

// sel[r] = the sample of rank r, for the mu best.
__global__ __launch_bounds__(256) void k_mae_select(MaeArgs a)
{
    const int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (k >= a.N) return;
    const uint32_t r = a.rank[k];
    if (r < (uint32_t)a.mu) a.sel[r] = (int32_t)k;
}

// Factor terms r < mu, one thread per (column j, term r): At[r][j] = d_{r:N, j}
// and Bt[r][j] = c_w/2 w_r z_{r:N, j} (rounded once).
__global__ __launch_bounds__(256) void k_mae_gather(MaeArgs a)
{
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x, r = blockIdx.y;
    if (j >= a.D) return;
    const int64_t k = a.sel[r];
    a.At[r * a.ldf + j] = a.Dm[k * a.ldx + j];
    a.Bt[r * a.ldf + j] = (float)(a.hcw * a.w[r] * (double)a.Z[k * a.ldx + j]);
}

// Weighted parent sums over chunk c of kMaeChunk parents, one thread per
// column: wpart[c][0][j] = sum w_r z_{r:N, j}, wpart[c][1][j] = sum w_r d_{r:N, j}
// (fp64, parents in rank order).
__global__ __launch_bounds__(256) void k_mae_wsum(MaeArgs a)
{
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x, c = blockIdx.y;
    if (j >= a.D) return;
    const int64_t r0 = c * kMaeChunk, r1 = r0 + kMaeChunk < a.mu ? r0 + kMaeChunk : a.mu;
    double zw = 0.0, dw = 0.0;
    // unrolled so that several parents' loads are in flight (same order)
#pragma unroll 8
    for (int64_t r = r0; r < r1; ++r) {
        const int64_t k = a.sel[r];
        const double wr = a.w[r];
        zw += wr * (double)a.Z[k * a.ldx + j];
        dw += wr * (double)a.Dm[k * a.ldx + j];
    }
    a.wpart[(2 * c) * a.D + j] = zw;
    a.wpart[(2 * c + 1) * a.D + j] = dw;
}

// One thread per column j: <z>_w and <d>_w from the chunk sums (in chunk
// order), y_j <- y_j + sigma <d>_w, s_j <- (1 - c_s) s_j + c_z <z>_w, the last
// factor term (At[mu][j] = (M s')_j, Bt[mu][j] = c_1/2 s'_j; the terms past mu
// and the columns past D are zero from creation), and the block's sum of
// s'_j^2 (fp64, fixed order).  Term r < mu of the factors is
//     At[r][j] = d_{r:N, j},  Bt[r][j] = c_w/2 w_r z_{r:N, j}  (k_mae_gather).
__global__ __launch_bounds__(kMaeBlock) void k_mae_recombine(MaeArgs a, int64_t nchunks)
{
    __shared__ double red[kMaeBlock];
    const int64_t j = (int64_t)blockIdx.x * kMaeBlock + threadIdx.x;
    double sq = 0.0;
    if (j < a.D) {
        double zw = 0.0, dw = 0.0;
#pragma unroll 8
        for (int64_t c = 0; c < nchunks; ++c) {
            zw += a.wpart[(2 * c) * a.D + j];
            dw += a.wpart[(2 * c + 1) * a.D + j];
        }
        const double sig = (double)*a.sigma, keep = 1.0 - a.cs;
        const float sn = (float)(keep * (double)a.s[j] + a.cz * zw);
        a.At[a.mu * a.ldf + j] = (float)(keep * (double)a.Dm[a.N * a.ldx + j] + a.cz * dw);
        a.Bt[a.mu * a.ldf + j] = (float)(a.hc1 * (double)sn);
        a.y[j] = (float)((double)a.y[j] + sig * dw);
        a.s[j] = sn;
        sq = (double)sn * (double)sn;
    }
    red[threadIdx.x] = sq;
    __syncthreads();
    for (int w = kMaeBlock / 2; w > 0; w /= 2) {
        if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) a.part[blockIdx.x] = red[0];
}

// sigma <- sigma exp(c_s/d_s (|s'| / chi_D - 1)), |s'|^2 from the block sums
// in a fixed order.
__global__ __launch_bounds__(256) void k_mae_sigma(MaeArgs a, int64_t nparts)
{
    __shared__ double red[256];
    double acc = 0.0;
    for (int64_t q = threadIdx.x; q < nparts; q += 256) acc += a.part[q];
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int w = 128; w > 0; w /= 2) {
        if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) *a.sigma = (float)((double)*a.sigma * exp(a.damp * (sqrt(red[0]) / a.chi - 1.0)));
}

// M <- beta M + At^T Bt over 2 STEPS factor terms (the factors hold zeros
// past the mu + 1 real terms and past column D, up to their padded extents:
// kp = 2 STEPS terms, a pitch ldf that is a multiple of 128, so no operand
// load needs a guard).  A block of four waves owns a 128 x 64 tile of M, each
// wave a 32 x 64 slice of it accumulated in two 32x32x2 MFMA tiles.  The
// block first issues its operand loads (the 128 rows of At and 64 columns
// of Bt over all terms, float4 from the k-major factors), then each wave
// issues the 32 loads of its slice of M; the operands go to LDS as soon as
// they arrive (loads complete in order, so the slice is still on its way
// from HBM) and the products read them from LDS while the slice arrives.
// LDS holds each term pair interleaved ([pair][row][term of the pair]) so
// that lane l = col + 32 h reads float 2 col + h of a pair: 64 consecutive
// floats, no bank conflicts.  The barrier fences LDS only, keeping the
// slice's loads in flight.  Rows past D read as zero and are not stored.
// Waves per SIMD the staged operands leave room for: four blocks of up to
// 40 KB of LDS per CU, three past that.
template <int STEPS>
constexpr int kMaeRankWaves = STEPS * 48 * 32 <= 160 * 1024 / 4 ? 4 : 3;

template <int STEPS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(kMaeRankWaves<STEPS>))) void k_mae_rank(MaeArgs a, float *M,
                                                                                           float beta)
{
    constexpr int NA = STEPS * 32, NI = STEPS * 48, PER = (NI + 255) / 256;  // float4 pairs of terms to stage
    __shared__ float4 sA[STEPS * 64], sB[STEPS * 32];
    const int tid = threadIdx.x, lane = tid % 64, col = lane % 32, h = lane / 32, w = tid / 64;
    const int64_t tn = (a.D + 63) / 64, ldf = a.ldf, ld = a.ldx;
    const int64_t I0 = ((int64_t)blockIdx.x / tn) * 128, j0 = ((int64_t)blockIdx.x % tn) * 64;
    const int64_t i0 = I0 + 32 * w;
    float4 lo[PER], hi[PER];
#pragma unroll
    for (int p = 0; p < PER; ++p) {
        // the last round's spare threads load the last item again (no
        // branch around the loads, which would wait for them)
        const int it = tid + 256 * p < NI ? tid + 256 * p : NI - 1;
        const bool isA = it < NA;
        const int s = isA ? it / 32 : (it - NA) / 16, q = isA ? it % 32 : (it - NA) % 16;
        const float *f = (isA ? a.At + I0 : a.Bt + j0) + 2 * s * ldf + 4 * q;
        lo[p] = *reinterpret_cast<const float4 *>(f);
        hi[p] = *reinterpret_cast<const float4 *>(f + ldf);
    }
    // The wave's slice of M through a buffer descriptor based at its first
    // element and ending at the end of M: rows past D fall outside its range
    // and read as zero (they are not stored).  The row offset sits in the
    // lane offset because the range check ignores the scalar offset.  M is
    // read and written once per pass, with the non-temporal policy (aux 2),
    // which keeps the staged factors in the L2.
    const int64_t wi0 = I0 + 32 * __builtin_amdgcn_readfirstlane(w);  // = i0, known to be wave-uniform
    const int64_t left = wi0 < a.D ? ((a.D - wi0) * ld - j0) * 4 : 0;  // bytes from the slice to the end of M
    const __amdgpu_buffer_rsrc_t mr = __builtin_amdgcn_make_buffer_rsrc(
        M + (wi0 < a.D ? wi0 * ld + j0 : 0), 0, (int)(left < 0x7fffffffLL ? left : 0x7fffffffLL), 0x00020000);
    float old[2][16];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const int off = (((v / 4) * 8 + h * 4 + v % 4) * (int)ld + col) * 4;
        old[0][v] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(mr, off, 0, 2));  // the load returns bits
        old[1][v] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(mr, off + 128, 0, 2));
    }
#pragma unroll
    for (int p = 0; p < PER; ++p) {
        const int it = tid + 256 * p;
        if (p + 1 < PER || it < NI) {
            const bool isA = it < NA;
            const int s = isA ? it / 32 : (it - NA) / 16, q = isA ? it % 32 : (it - NA) % 16;
            float4 *d = isA ? sA + s * 64 + 2 * q : sB + s * 32 + 2 * q;
            d[0] = make_float4(lo[p].x, hi[p].x, lo[p].y, hi[p].y);
            d[1] = make_float4(lo[p].z, hi[p].z, lo[p].w, hi[p].w);
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
    if (i0 >= a.D) return;
    const float *la = reinterpret_cast<const float *>(sA) + (32 * w + col) * 2 + h;
    const float *lb = reinterpret_cast<const float *>(sB) + col * 2 + h;
    f32x16 acc[2];
#pragma unroll
    for (int n = 0; n < 2; ++n)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[n][v] = 0.0f;
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
        const float av = la[s * 256], b0 = lb[s * 128], b1 = lb[s * 128 + 64];
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, b0, acc[0], 0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, b1, acc[1], 0, 0, 0);
    }
    if (j0 + 64 <= a.D) {
        // every column is inside the matrix: store through the descriptor,
        // which drops the rows past D
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int off = (((v / 4) * 8 + h * 4 + v % 4) * (int)ld + col) * 4;
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(fmaf(1.0f, acc[0][v], beta * old[0][v])), mr, off, 0, 2);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(fmaf(1.0f, acc[1][v], beta * old[1][v])), mr, off + 128,
                                                  0, 2);
        }
        return;
    }
#pragma unroll
    for (int n = 0; n < 2; ++n)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int64_t i = i0 + (v / 4) * 8 + h * 4 + v % 4, j = j0 + 32 * n + col;
            if (i < a.D && j < a.D) M[i * ld + j] = fmaf(1.0f, acc[n][v], beta * old[n][v]);
        }
}

// The same update for any number of terms (a.kp, a multiple of 32): each
// wave owns a 32 x 64 tile of M and loads its MFMA operands directly from the
// k-major factors (lane l: row or column l % 32 of term 2 step + l / 32, one
// 128-byte line per half wave), 16 steps at a time, double-buffered: the
// next block's loads are in flight while the current block's products run.
// The tile of M is loaded first.  It holds two blocks of operands at one
// wave per SIMD, which measured faster than 2 or 3 waves with 8-step blocks.
__global__ __launch_bounds__(256) void k_mae_rank_any(MaeArgs a, float *M, float beta)
{
    constexpr int CH = 16;
    const int lane = threadIdx.x % 64, col = lane % 32, h = lane / 32;
    const int64_t tn = (a.D + 63) / 64;
    const int64_t wave = (int64_t)blockIdx.x * 4 + threadIdx.x / 64;
    const int64_t i0 = (wave / tn) * 32, j0 = (wave % tn) * 64;
    if (i0 >= a.D) return;
    float old[2][16];
#pragma unroll
    for (int n = 0; n < 2; ++n)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int64_t i = i0 + (v / 4) * 8 + h * 4 + v % 4, j = j0 + 32 * n + col;
            old[n][v] = (i < a.D && j < a.D) ? M[i * a.ldx + j] : 0.0f;
        }
    f32x16 acc[2];
#pragma unroll
    for (int n = 0; n < 2; ++n)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[n][v] = 0.0f;
    const float *pa = a.At + h * a.ldf + i0 + col;
    const float *pb = a.Bt + h * a.ldf + j0 + col;
    float av[2][CH], b0[2][CH], b1[2][CH];
    auto load = [&](int buf, int64_t c0) {
#pragma unroll
        for (int t = 0; t < CH; ++t) {
            const int64_t off = 2 * (c0 + t) * a.ldf;
            av[buf][t] = pa[off];
            b0[buf][t] = pb[off];
            b1[buf][t] = pb[off + 32];
        }
    };
    auto products = [&](int buf) {
#pragma unroll
        for (int t = 0; t < CH; ++t) {
            acc[0] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[buf][t], b0[buf][t], acc[0], 0, 0, 0);
            acc[1] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[buf][t], b1[buf][t], acc[1], 0, 0, 0);
        }
    };
    const int64_t steps = a.kp / 2;
    load(0, 0);
    for (int64_t c0 = 0; c0 < steps; c0 += 2 * CH) {
        if (c0 + CH < steps) load(1, c0 + CH);
        products(0);
        if (c0 + CH < steps) {
            if (c0 + 2 * CH < steps) load(0, c0 + 2 * CH);
            products(1);
        }
    }
#pragma unroll
    for (int n = 0; n < 2; ++n)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int64_t i = i0 + (v / 4) * 8 + h * 4 + v % 4, j = j0 + 32 * n + col;
            if (i < a.D && j < a.D) M[i * a.ldx + j] = fmaf(1.0f, acc[n][v], beta * old[n][v]);
        }
}

__global__ __launch_bounds__(256) void k_mae_identity(float *M, int64_t D, int64_t ldx)
{
    const int64_t total = D * ldx;
    for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < total; q += (int64_t)gridDim.x * 256)
        M[q] = (q / ldx == q % ldx) ? 1.0f : 0.0f;
}

unsigned blocks_for(int64_t n, int64_t per, int64_t cap)
{
    const int64_t b = (n + per - 1) / per;
    return (unsigned)(b < 1 ? 1 : b > cap ? cap : b);
}

}  // namespace

hipError_t launch_mae_sample(const MaeArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_mae_sample, dim3(blocks_for((a.N + 1) * (a.ldx / 4), 256, 16384)), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_mae_select(const MaeArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_mae_select, dim3(blocks_for(a.N, 256, 1 << 20)), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_mae_recombine(const MaeArgs &a, hipStream_t s)
{
    const int64_t nparts = (a.D + kMaeBlock - 1) / kMaeBlock, cols = (a.D + 255) / 256;
    const int64_t nchunks = (a.mu + kMaeChunk - 1) / kMaeChunk;
    hipLaunchKernelGGL(k_mae_gather, dim3((unsigned)cols, (unsigned)a.mu), dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_mae_wsum, dim3((unsigned)cols, (unsigned)nchunks), dim3(256), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_mae_recombine, dim3((unsigned)nparts), dim3(kMaeBlock), 0, s, a, nchunks);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_mae_sigma, dim3(1), dim3(256), 0, s, a, nparts);
    return hipGetLastError();
}

hipError_t launch_mae_rank(const MaeArgs &a, float *M, float beta, hipStream_t s)
{
    const int64_t waves = ((a.D + 31) / 32) * ((a.D + 63) / 64);
    const dim3 grid_any((unsigned)((waves + 3) / 4)), block(256);
    const dim3 grid((unsigned)(((a.D + 127) / 128) * ((a.D + 63) / 64)));
    const int64_t steps = (a.mu + 2) / 2;  // ceil((mu + 1) / 2)
    if (a.ldf % 128 != 0 || (steps <= kMaeRankUnrolled && a.kp != 2 * steps)) return hipErrorInvalidValue;
    switch (steps > kMaeRankUnrolled ? 0 : steps) {
#define EVOX_RANK_CASE(S) \
    case S: hipLaunchKernelGGL((k_mae_rank<S>), grid, block, 0, s, a, M, beta); break;
        EVOX_RANK_CASE(1) EVOX_RANK_CASE(2) EVOX_RANK_CASE(3) EVOX_RANK_CASE(4) EVOX_RANK_CASE(5)
        EVOX_RANK_CASE(6) EVOX_RANK_CASE(7) EVOX_RANK_CASE(8) EVOX_RANK_CASE(9) EVOX_RANK_CASE(10)
        EVOX_RANK_CASE(11) EVOX_RANK_CASE(12) EVOX_RANK_CASE(13) EVOX_RANK_CASE(14) EVOX_RANK_CASE(15)
        EVOX_RANK_CASE(16) EVOX_RANK_CASE(17) EVOX_RANK_CASE(18) EVOX_RANK_CASE(19) EVOX_RANK_CASE(20)
        EVOX_RANK_CASE(21) EVOX_RANK_CASE(22) EVOX_RANK_CASE(23) EVOX_RANK_CASE(24) EVOX_RANK_CASE(25)
        EVOX_RANK_CASE(26) EVOX_RANK_CASE(27) EVOX_RANK_CASE(28) EVOX_RANK_CASE(29) EVOX_RANK_CASE(30)
        EVOX_RANK_CASE(31) EVOX_RANK_CASE(32)
#undef EVOX_RANK_CASE
        default: hipLaunchKernelGGL(k_mae_rank_any, grid_any, block, 0, s, a, M, beta); break;
    }
    return hipGetLastError();
}

hipError_t launch_mae_identity(float *M, int64_t D, int64_t ldx, hipStream_t s)
{
    hipLaunchKernelGGL(k_mae_identity, dim3(blocks_for(D * ldx, 256, 16384)), dim3(256), 0, s, M, D, ldx);
    return hipGetLastError();
}

}  // namespace evox
