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
typedef float f32x4 __attribute__((ext_vector_type(4)));

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

// ---------------------------------------------------------------------------
// C = alpha A B^T + beta C with A [M x K] and B [N x K] both K-contiguous, the
// layout of the two contractions of the matrix-adaptation ES (samples times
// M^T, and the rank-mu update).  Block tile BM x BN (BM, BN in {64, 128}),
// 2 x 2 waves of (BM/2) x (BN/2), each a grid of 32x32x2 MFMA accumulators;
// K in tiles of 32, each staged in LDS row-major ([row][k], rows padded to 36
// floats so that every row starts 16-byte aligned) after being prefetched
// into registers while the previous tile is multiplied.  Within a tile, lane
// half h = l / 32 takes k = 16 h + step (steps 0..15), so each lane reads its
// operands as float4 runs along k; the order in which the products are summed
// is fixed.
// Split-K (gridDim.z = splits): block z sums k in [z kc, (z + 1) kc) and, with
// a workspace, stores its raw partial tile there; k_splitk_reduce then adds
// the partials in order z = 0, 1, ... and applies alpha and beta.  Without a
// workspace (one split) the block applies alpha and beta itself.
// ---------------------------------------------------------------------------
constexpr int kNtBK = 32, kNtLD = kNtBK + 4;
// register stages of the operand prefetch for the thin tiles (M <= 128,
// 64 output columns per block); the 128 x 128 tiles keep one stage
constexpr int kNtThinDepth = 2;

template <int BM, int BN, int DEPTH>
__global__ __launch_bounds__(256) void k_gemm_nt(GemmArgs g, float *work, int64_t kc)
{
    constexpr int TM = BM / 64, TN = BN / 64;            // 32x32 tiles per wave
    constexpr int QA = BM * kNtBK / 4 / 256, QB = BN * kNtBK / 4 / 256;  // float4 per thread
    __shared__ float As[BM * kNtLD];
    __shared__ float Bs[BN * kNtLD];
    const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64, col = lane % 32, h = lane / 32;
    const int wm = wave / 2, wn = wave % 2;
    const int64_t i0 = (int64_t)blockIdx.y * BM, j0 = (int64_t)blockIdx.x * BN;
    const int64_t kb = (int64_t)blockIdx.z * kc, ke = kb + kc < g.K ? kb + kc : g.K;
    // DEPTH register stages of the next K tiles' operands (compile-time
    // stage indices, so they stay in registers)
    float4 ra[DEPTH][QA], rb[DEPTH][QB];
    auto load = [&](int d, int64_t k0) {
#pragma unroll
        for (int q = 0; q < QA; ++q) {
            const int idx = tid + 256 * q, row = idx / 8, c4 = idx % 8;
            ra[d][q] = quad_or_zero(g.A, g.lda, i0 + row, k0 + 4 * c4, g.M, ke);
        }
#pragma unroll
        for (int q = 0; q < QB; ++q) {
            const int idx = tid + 256 * q, row = idx / 8, c4 = idx % 8;
            rb[d][q] = quad_or_zero(g.B, g.ldb, j0 + row, k0 + 4 * c4, g.N, ke);
        }
    };
    auto store = [&](int d) {
#pragma unroll
        for (int q = 0; q < QA; ++q) {
            const int idx = tid + 256 * q, row = idx / 8, c4 = idx % 8;
            *reinterpret_cast<float4 *>(&As[row * kNtLD + 4 * c4]) = ra[d][q];
        }
#pragma unroll
        for (int q = 0; q < QB; ++q) {
            const int idx = tid + 256 * q, row = idx / 8, c4 = idx % 8;
            *reinterpret_cast<float4 *>(&Bs[row * kNtLD + 4 * c4]) = rb[d][q];
        }
    };
    f32x16 acc[TM][TN];
#pragma unroll
    for (int m = 0; m < TM; ++m)
#pragma unroll
        for (int n = 0; n < TN; ++n)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[m][n][v] = 0.0f;

    auto compute = [&]() {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            float4 a4[TM], b4[TN];
#pragma unroll
            for (int m = 0; m < TM; ++m)
                a4[m] = *reinterpret_cast<const float4 *>(&As[(wm * TM * 32 + m * 32 + col) * kNtLD + h * 16 + 4 * c]);
#pragma unroll
            for (int n = 0; n < TN; ++n)
                b4[n] = *reinterpret_cast<const float4 *>(&Bs[(wn * TN * 32 + n * 32 + col) * kNtLD + h * 16 + 4 * c]);
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int m = 0; m < TM; ++m)
#pragma unroll
                    for (int n = 0; n < TN; ++n)
                        acc[m][n] = __builtin_amdgcn_mfma_f32_32x32x2f32(comp(a4[m], e), comp(b4[n], e),
                                                                         acc[m][n], 0, 0, 0);
        }
    };
    if (kb < ke) {
        // tile kb in LDS, tiles kb + d kNtBK (d < DEPTH) in register stage d
        load(0, kb);
        store(0);
        __syncthreads();
#pragma unroll
        for (int d = 1; d < DEPTH; ++d)
            if (kb + d * kNtBK < ke) load(d, kb + d * kNtBK);
        for (int64_t k0 = kb; k0 < ke; k0 += DEPTH * kNtBK) {
#pragma unroll
            for (int d = 0; d < DEPTH; ++d) {
                const int64_t kt = k0 + d * kNtBK;  // the tile in LDS (uniform)
                if (kt >= ke) break;
                // stage d held tile kt (now in LDS): refill it DEPTH tiles ahead
                if (kt + DEPTH * kNtBK < ke) load(d, kt + DEPTH * kNtBK);
                compute();
                __syncthreads();
                if (kt + kNtBK < ke) {
                    store((d + 1) % DEPTH);
                    __syncthreads();
                }
            }
        }
    }
#pragma unroll
    for (int m = 0; m < TM; ++m)
#pragma unroll
        for (int n = 0; n < TN; ++n)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t i = i0 + wm * TM * 32 + m * 32 + (v / 4) * 8 + h * 4 + v % 4;
                const int64_t j = j0 + wn * TN * 32 + n * 32 + col;
                if (i < g.M && j < g.N) {
                    if (work) {
                        work[((int64_t)blockIdx.z * g.M + i) * g.N + j] = acc[m][n][v];
                    } else {
                        float *c = g.C + i * g.ldc + j;
                        *c = g.beta != 0.0f ? fmaf(g.alpha, acc[m][n][v], g.beta * *c) : g.alpha * acc[m][n][v];
                    }
                }
            }
}

// A B^T for at most 16 RB rows of A (the thin sampling products): 16 x 16
// MFMA tiles (v_mfma_f32_16x16x4f32), so 101 rows pad to 112 instead of
// 128.  Block: all 16 RB rows x 64 columns, K tile kNtBK; wave w owns the
// 16-column block w and the RB row blocks.  Within a K tile, lane group
// q = lane / 16 takes the 8 consecutive k 8q .. 8q + 7, one per MFMA step
// (any split of k over the four k slots of the instruction is a valid
// product, since A and B use the same one), so each lane reads its
// operands as two float4 per row block.  Operand prefetch as in k_gemm_nt.
template <int RB, int DEPTH>
__global__ __launch_bounds__(256) void k_gemm_nt16(GemmArgs g, float *work, int64_t kc)
{
    constexpr int BM = 16 * RB, BN = 64;
    constexpr int FA = BM * kNtBK / 4, FB = BN * kNtBK / 4;  // float4 per tile
    constexpr int QA = (FA + 255) / 256, QB = FB / 256;      // float4 per thread
    __shared__ float As[BM * kNtLD];
    __shared__ float Bs[BN * kNtLD];
    const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64, r16 = lane % 16, q = lane / 16;
    const int64_t i0 = (int64_t)blockIdx.y * BM, j0 = (int64_t)blockIdx.x * BN;
    const int64_t kb = (int64_t)blockIdx.z * kc, ke = kb + kc < g.K ? kb + kc : g.K;
    float4 ra[DEPTH][QA], rb[DEPTH][QB];
    auto load = [&](int d, int64_t k0) {
#pragma unroll
        for (int u = 0; u < QA; ++u) {
            const int idx = tid + 256 * u, row = idx / 8, c4 = idx % 8;
            if (idx < FA) ra[d][u] = quad_or_zero(g.A, g.lda, i0 + row, k0 + 4 * c4, g.M, ke);
        }
#pragma unroll
        for (int u = 0; u < QB; ++u) {
            const int idx = tid + 256 * u, row = idx / 8, c4 = idx % 8;
            rb[d][u] = quad_or_zero(g.B, g.ldb, j0 + row, k0 + 4 * c4, g.N, ke);
        }
    };
    auto store = [&](int d) {
#pragma unroll
        for (int u = 0; u < QA; ++u) {
            const int idx = tid + 256 * u, row = idx / 8, c4 = idx % 8;
            if (idx < FA) *reinterpret_cast<float4 *>(&As[row * kNtLD + 4 * c4]) = ra[d][u];
        }
#pragma unroll
        for (int u = 0; u < QB; ++u) {
            const int idx = tid + 256 * u, row = idx / 8, c4 = idx % 8;
            *reinterpret_cast<float4 *>(&Bs[row * kNtLD + 4 * c4]) = rb[d][u];
        }
    };
    f32x4 acc[RB];
#pragma unroll
    for (int m = 0; m < RB; ++m)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[m][v] = 0.0f;
    auto compute = [&]() {
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {  // k 8q + 4hf .. 8q + 4hf + 3
            const float4 b4 = *reinterpret_cast<const float4 *>(&Bs[(wave * 16 + r16) * kNtLD + 8 * q + 4 * hf]);
#pragma unroll
            for (int m = 0; m < RB; ++m) {
                const float4 a4 = *reinterpret_cast<const float4 *>(&As[(m * 16 + r16) * kNtLD + 8 * q + 4 * hf]);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    acc[m] = __builtin_amdgcn_mfma_f32_16x16x4f32(comp(a4, e), comp(b4, e), acc[m], 0, 0, 0);
            }
        }
    };
    if (kb < ke) {
        load(0, kb);
        store(0);
        __syncthreads();
#pragma unroll
        for (int d = 1; d < DEPTH; ++d)
            if (kb + d * kNtBK < ke) load(d, kb + d * kNtBK);
        for (int64_t k0 = kb; k0 < ke; k0 += DEPTH * kNtBK) {
#pragma unroll
            for (int d = 0; d < DEPTH; ++d) {
                const int64_t kt = k0 + d * kNtBK;
                if (kt >= ke) break;
                if (kt + DEPTH * kNtBK < ke) load(d, kt + DEPTH * kNtBK);
                compute();
                __syncthreads();
                if (kt + kNtBK < ke) {
                    store((d + 1) % DEPTH);
                    __syncthreads();
                }
            }
        }
    }
    // result v of row block m: row 16 m + 4 q + v, column 16 wave + r16
#pragma unroll
    for (int m = 0; m < RB; ++m)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int64_t i = i0 + m * 16 + 4 * q + v, j = j0 + wave * 16 + r16;
            if (i < g.M && j < g.N) {
                if (work) {
                    work[((int64_t)blockIdx.z * g.M + i) * g.N + j] = acc[m][v];
                } else {
                    float *c = g.C + i * g.ldc + j;
                    *c = g.beta != 0.0f ? fmaf(g.alpha, acc[m][v], g.beta * *c) : g.alpha * acc[m][v];
                }
            }
        }
}

__global__ __launch_bounds__(256) void k_splitk_reduce(GemmArgs g, const float *work, int splits)
{
    const int64_t n = g.M * g.N;
    for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < n; q += (int64_t)gridDim.x * 256) {
        float acc = work[q];
        for (int z = 1; z < splits; ++z) acc += work[(int64_t)z * n + q];
        const int64_t i = q / g.N, j = q % g.N;
        float *c = g.C + i * g.ldc + j;
        *c = g.beta != 0.0f ? fmaf(g.alpha, acc, g.beta * *c) : g.alpha * acc;
    }
}

}  // namespace

int occupancy_gemm_nt_thin(int64_t M)
{
    int n = 0;
    const hipError_t e = M > 64 && M <= 112
                             ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_gemm_nt16<7, kNtThinDepth>, 256, 0)
                             : hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_gemm_nt<128, 64, kNtThinDepth>, 256, 0);
    return e == hipSuccess ? n : 0;
}

int64_t gemm_nt_chunk(int64_t K, int splits)
{
    const int64_t per = (K + splits - 1) / splits;
    return (per + kNtBK - 1) / kNtBK * kNtBK;
}

hipError_t launch_gemm_nt(const GemmArgs &g, int splits, float *work, hipStream_t s)
{
    if (g.M <= 0 || g.N <= 0) return hipSuccess;
    if (splits < 1 || (splits > 1 && !work)) return hipErrorInvalidValue;
    const int64_t kc = splits > 1 ? gemm_nt_chunk(g.K, splits) : (g.K > 0 ? g.K : 1);
    // 65..112 rows: 16 x 16 tiles (7 row blocks) instead of 128 padded rows
    const bool rows112 = g.M > 64 && g.M <= 112;
    const int bm = g.M <= 64 ? 64 : rows112 ? 112 : 128, bn = g.M <= 128 ? 64 : 128;
    const dim3 grid((unsigned)((g.N + bn - 1) / bn), (unsigned)((g.M + bm - 1) / bm), (unsigned)splits);
    float *w = splits > 1 ? work : nullptr;
    if (rows112) hipLaunchKernelGGL((k_gemm_nt16<7, kNtThinDepth>), grid, dim3(256), 0, s, g, w, kc);
    else if (bm == 64) hipLaunchKernelGGL((k_gemm_nt<64, 64, kNtThinDepth>), grid, dim3(256), 0, s, g, w, kc);
    else if (bn == 64) hipLaunchKernelGGL((k_gemm_nt<128, 64, kNtThinDepth>), grid, dim3(256), 0, s, g, w, kc);
    else hipLaunchKernelGGL((k_gemm_nt<128, 128, 1>), grid, dim3(256), 0, s, g, w, kc);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || splits == 1) return e;
    const int64_t n = g.M * g.N, blocks = (n + 255) / 256;
    hipLaunchKernelGGL(k_splitk_reduce, dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(256), 0, s, g,
                       (const float *)work, splits);
    return hipGetLastError();
}

hipError_t launch_gemm(bool ta, bool tb, const GemmArgs &g, hipStream_t s)
{
    if (g.M <= 0 || g.N <= 0) return hipSuccess;
    if (!ta && tb) return launch_gemm_nt(g, 1, nullptr, s);
    const dim3 grid((unsigned)((g.N + kBN - 1) / kBN), (unsigned)((g.M + kBM - 1) / kBM));
    if (!ta && !tb) hipLaunchKernelGGL((k_gemm<false, false>), grid, dim3(256), 0, s, g);
    if (!ta && tb) hipLaunchKernelGGL((k_gemm<false, true>), grid, dim3(256), 0, s, g);
    if (ta && !tb) hipLaunchKernelGGL((k_gemm<true, false>), grid, dim3(256), 0, s, g);
    if (ta && tb) hipLaunchKernelGGL((k_gemm<true, true>), grid, dim3(256), 0, s, g);
    return hipGetLastError();
}

}  // namespace evox
