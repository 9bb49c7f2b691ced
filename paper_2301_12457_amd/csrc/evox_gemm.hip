// Dense fp32 matrix product on the matrix cores (the contractions of the
// matrix-adaptation ES): C = alpha op(A) op(B) + beta C, row-major operands
// with leading dimensions, op(X) = X or X^T.
//
// Block tile 128 x 128, 256 threads as 2 x 2 waves of 64 x 64, each wave a
// 2 x 2 grid of v_mfma_f32_32x32x2f32 accumulators (16 floats per lane).
// The K loop stages a 128 x 16 tile of op(A) and a 16 x 128 tile of op(B) in
// LDS, k-major, so that every MFMA operand is a read of 32 consecutive floats
// by each half of the wave.  Operand lane layout of the 32x32x2 instruction:
// lane l holds A[l % 32][l / 32] and B[l / 32][l % 32]; result element v of
// lane l is C[(v / 4) 8 + (l / 32) 4 + v % 4][l % 32].  Loads outside the
// matrices read zero; stores outside are skipped.  The order of the
// additions is fixed, so results are reproducible.
#include "evox_launch.hpp"

namespace evox {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kBM = 128, kBN = 128, kBK = 16, kPad = 4;

// Element (r, c) of a row-major matrix with leading dimension ld, zero
// outside rows x cols.
__device__ __forceinline__ float at_or_zero(const float *X, int64_t ld, int64_t r, int64_t c, int64_t rows,
                                            int64_t cols)
{
    return (r < rows && c < cols) ? X[r * ld + c] : 0.0f;
}

// Four consecutive elements (r, c .. c+3) of a row-major matrix, zero outside;
// one 16-byte load when all four are inside (ld and c multiples of 4).
__device__ __forceinline__ float4 quad_or_zero(const float *X, int64_t ld, int64_t r, int64_t c, int64_t rows,
                                               int64_t cols)
{
    if (r < rows && c + 3 < cols) return *reinterpret_cast<const float4 *>(X + r * ld + c);
    return make_float4(at_or_zero(X, ld, r, c, rows, cols), at_or_zero(X, ld, r, c + 1, rows, cols),
                       at_or_zero(X, ld, r, c + 2, rows, cols), at_or_zero(X, ld, r, c + 3, rows, cols));
}

template <bool TA, bool TB>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs g)
{
    __shared__ float As[kBK][kBM + kPad];
    __shared__ float Bs[kBK][kBN + kPad];
    const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64;
    const int wm = wave / 2, wn = wave % 2;
    const int64_t i0 = (int64_t)blockIdx.y * kBM, j0 = (int64_t)blockIdx.x * kBN;
    f32x16 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.0f;

    for (int64_t k0 = 0; k0 < g.K; k0 += kBK) {
        // op(A) tile [i0, i0 + 128) x [k0, k0 + 16) into As[k][i]
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int q = tid + 256 * r;
            if constexpr (!TA) {  // A is M x K: a row's 16 k are contiguous
                const int row = q / 4, c4 = q % 4;
                const float4 v = quad_or_zero(g.A, g.lda, i0 + row, k0 + 4 * c4, g.M, g.K);
                As[4 * c4 + 0][row] = v.x;
                As[4 * c4 + 1][row] = v.y;
                As[4 * c4 + 2][row] = v.z;
                As[4 * c4 + 3][row] = v.w;
            } else {  // A is K x M: a k-row's 128 i are contiguous
                const int kr = q / 32, c4 = q % 32;
                const float4 v = quad_or_zero(g.A, g.lda, k0 + kr, i0 + 4 * c4, g.K, g.M);
                *reinterpret_cast<float4 *>(&As[kr][4 * c4]) = v;
            }
        }
        // op(B) tile [k0, k0 + 16) x [j0, j0 + 128) into Bs[k][j]
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int q = tid + 256 * r;
            if constexpr (!TB) {  // B is K x N
                const int kr = q / 32, c4 = q % 32;
                const float4 v = quad_or_zero(g.B, g.ldb, k0 + kr, j0 + 4 * c4, g.K, g.N);
                *reinterpret_cast<float4 *>(&Bs[kr][4 * c4]) = v;
            } else {  // B is N x K
                const int col = q / 4, c4 = q % 4;
                const float4 v = quad_or_zero(g.B, g.ldb, j0 + col, k0 + 4 * c4, g.N, g.K);
                Bs[4 * c4 + 0][col] = v.x;
                Bs[4 * c4 + 1][col] = v.y;
                Bs[4 * c4 + 2][col] = v.z;
                Bs[4 * c4 + 3][col] = v.w;
            }
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < kBK; kk += 2) {
            const int kr = kk + lane / 32;
            float a[2], b[2];
#pragma unroll
            for (int m = 0; m < 2; ++m) a[m] = As[kr][wm * 64 + m * 32 + lane % 32];
#pragma unroll
            for (int n = 0; n < 2; ++n) b[n] = Bs[kr][wn * 64 + n * 32 + lane % 32];
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int n = 0; n < 2; ++n) acc[m][n] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[m], b[n], acc[m][n], 0, 0, 0);
        }
        __syncthreads();
    }
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int n = 0; n < 2; ++n)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t i = i0 + wm * 64 + m * 32 + (v / 4) * 8 + (lane / 32) * 4 + v % 4;
                const int64_t j = j0 + wn * 64 + n * 32 + lane % 32;
                if (i < g.M && j < g.N) {
                    float *c = g.C + i * g.ldc + j;
                    *c = g.beta != 0.0f ? fmaf(g.alpha, acc[m][n][v], g.beta * *c) : g.alpha * acc[m][n][v];
                }
            }
}

}  // namespace

hipError_t launch_gemm(bool ta, bool tb, const GemmArgs &g, hipStream_t s)
{
    if (g.M <= 0 || g.N <= 0) return hipSuccess;
    const dim3 grid((unsigned)((g.N + kBN - 1) / kBN), (unsigned)((g.M + kBM - 1) / kBM));
    if (!ta && !tb) hipLaunchKernelGGL((k_gemm<false, false>), grid, dim3(256), 0, s, g);
    if (!ta && tb) hipLaunchKernelGGL((k_gemm<false, true>), grid, dim3(256), 0, s, g);
    if (ta && !tb) hipLaunchKernelGGL((k_gemm<true, false>), grid, dim3(256), 0, s, g);
    if (ta && tb) hipLaunchKernelGGL((k_gemm<true, true>), grid, dim3(256), 0, s, g);
    return hipGetLastError();
}

}  // namespace evox
