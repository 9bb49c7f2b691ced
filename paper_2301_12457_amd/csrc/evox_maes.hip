// The matrix-adaptation ES generation (CMA-ES of Table II in the form of
// Beyer and Sendhoff, 2017) apart from its two matrix products and the
// fitness pass: deviates, parent selection, recombination of the center and
// the path together with the factors of the rank-mu update, and the step
// size.  With s' the new path and d_i = M z_i the steps of the parents,
//     M [I + c_1/2 (s' s'^T - I) + c_w/2 (sum_i w_i z_i z_i^T - I)]
//   = (1 - (c_1 + c_w)/2) M + (M s') (c_1/2 s')^T + sum_i d_i (c_w/2 w_i z_i)^T,
// and M s' = (1 - c_s) M s + sqrt(mu_eff c_s (2 - c_s)) sum_i w_i d_i, so the
// update is one product of two D x (mu + 1) factors whose columns this file
// writes, and M s comes from the sampling product (the path rides along as
// an extra deviate row).
#include "evox_launch.hpp"

namespace evox {

namespace {

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

// One thread per column j: the weighted parent sums <z>_w and <d>_w in fp64,
// y_j <- y_j + sigma <d>_w, s_j <- (1 - c_s) s_j + c_z <z>_w, the factor rows
//     At[j] = (d_{1:N, j}, ..., d_{mu:N, j}, (M s')_j, 0 ...)
//     Bt[j] = (c_w/2 w_1 z_{1:N, j}, ..., c_w/2 w_mu z_{mu:N, j}, c_1/2 s'_j, 0 ...)
// and the block's sum of s'_j^2 (fp64, fixed order).
__global__ __launch_bounds__(kMaeBlock) void k_mae_recombine(MaeArgs a)
{
    __shared__ double red[kMaeBlock];
    const int64_t j = (int64_t)blockIdx.x * kMaeBlock + threadIdx.x;
    double sq = 0.0;
    if (j < a.D) {
        double zw = 0.0, dw = 0.0;
        float *at = a.At + j * a.kp, *bt = a.Bt + j * a.kp;
        for (int64_t r = 0; r < a.mu; ++r) {
            const int64_t k = a.sel[r];
            const double wr = a.w[r];
            const float z = a.Z[k * a.ldx + j], d = a.Dm[k * a.ldx + j];
            zw += wr * (double)z;
            dw += wr * (double)d;
            at[r] = d;
            bt[r] = (float)(a.hcw * wr * (double)z);
        }
        const double sig = (double)*a.sigma, keep = 1.0 - a.cs;
        const float sn = (float)(keep * (double)a.s[j] + a.cz * zw);
        at[a.mu] = (float)(keep * (double)a.Dm[a.N * a.ldx + j] + a.cz * dw);
        bt[a.mu] = (float)(a.hc1 * (double)sn);
        for (int64_t r = a.mu + 1; r < a.kp; ++r) at[r] = bt[r] = 0.0f;
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
    const int64_t nparts = (a.D + kMaeBlock - 1) / kMaeBlock;
    hipLaunchKernelGGL(k_mae_recombine, dim3((unsigned)nparts), dim3(kMaeBlock), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_mae_sigma, dim3(1), dim3(256), 0, s, a, nparts);
    return hipGetLastError();
}

hipError_t launch_mae_identity(float *M, int64_t D, int64_t ldx, hipStream_t s)
{
    hipLaunchKernelGGL(k_mae_identity, dim3(blocks_for(D * ldx, 256, 16384)), dim3(256), 0, s, M, D, ldx);
    return hipGetLastError();
}

}  // namespace evox
