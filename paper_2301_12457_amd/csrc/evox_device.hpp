// Device-side building blocks of the gfx950 generation kernels: Philox,
// benchmark-function row reductions, row layout, and the argmin order.
//
// Data layout: a population matrix is row-major fp32 with a row pitch ldx
// (multiple of 4 floats, 16-byte aligned rows).  One row is handled by a
// group of G consecutive lanes (G a power of two, 4..1024); lane g of the
// group holds the float4 chunks c = g + G * it, it = 0..MAXIT-1, i.e. the
// elements 4c..4c+3.  Every wave load instruction therefore reads G * 16
// contiguous bytes of a row (128-bit loads, fully coalesced), and a row's
// fitness is a per-lane partial over its chunks followed by a butterfly over
// the G lanes (DPP/ds_swizzle shuffles) and, for G > 64, an LDS step across
// the waves of the row.  The reduction order depends only on D, so every
// kernel that evaluates a row produces bit-identical fitness.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace evox {

enum { FN_SPHERE = 0, FN_ACKLEY, FN_RASTRIGIN, FN_GRIEWANK, FN_ROSENBROCK, FN_SCHWEFEL, FN_COUNT };

// Random-stream ids (fourth Philox counter word).
enum { STREAM_INIT_X = 0, STREAM_INIT_V = 1, STREAM_PSO = 2, STREAM_CSO = 3, STREAM_PERM = 4,
       STREAM_INIT_NORMAL = 5, STREAM_DE = 6, STREAM_ES = 7, STREAM_PGPE = 8,
       STREAM_MAES = 9, STREAM_NSGA_SEL = 10, STREAM_NSGA_VAR = 11, STREAM_NSGA_MUT = 12 };

constexpr int kBlock = 256;              // threads per block when a row takes <= 256 lanes
constexpr int kGridCap = 2048;           // blocks of the grid-stride kernels (8 per CU on 256 CUs)
constexpr int64_t kMaxGrid = 1 << 20;    // blocks of the row kernels at most (grid-stride beyond)
constexpr int kSlots = 2048;             // selection slots (atomicMin targets)
constexpr int kMaxG = 1024;

__host__ __device__ constexpr int block_for(int G) { return G > kBlock ? G : kBlock; }

// Row layout: G lanes per row, MAXIT float4 chunk registers per lane, nit of
// them used; G is the fewest lanes (a power of two) that hold the row in at
// most `family` chunks per lane (8 at G = 1024).  Three families, chosen by
// measurement on gfx950:
//   LAYOUT_EVAL   4 chunks per lane: evox_eval (one wave per row at D = 1000,
//                 no LDS step in the row reduction);
//   LAYOUT_PSO    2 chunks per lane: the PSO generation kernels (fewer
//                 registers per lane, more waves in flight);
//   LAYOUT_CSO    1 chunk per lane up to D = 4096: the CSO kernels, whose
//                 random row gathers want a row in one load instruction.
// The layout depends only on (D, family), so every kernel of a state reduces
// a row in the same order and produces bit-identical fitness.
enum { LAYOUT_CSO = 1, LAYOUT_PSO = 2, LAYOUT_EVAL = 4 };

struct Layout {
    int G, maxit, nit;
};

inline bool row_layout(int64_t D, int family, Layout *L)
{
    if (D < 1) return false;
    const int64_t c4 = (D + 3) / 4;
    int G = 4;
    while (G < kMaxG && (c4 + G - 1) / G > family) G *= 2;
    const int64_t nit = (c4 + G - 1) / G;
    // the kernels' compile-time chunk count: the family's, and at 1024 lanes
    // the smallest of (family, 4, 8) that holds the row (fewer registers for
    // rows that need only a few chunks per lane)
    const int maxit = G < kMaxG || nit <= family ? family : nit <= 4 ? 4 : 8;
    if (nit > maxit) return false;
    *L = Layout{G, maxit, (int)nit};
    return true;
}

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two
// 32x32->64 multiplies and key xors, Weyl-incremented key.  Everything stays
// in registers; the key is wave-uniform (SGPRs).  Each round's two
// three-input exclusive ors are single v_bitop3_b32 instructions (truth
// table 0x96, odd parity of the three input bits) when kXor3: 40 instead of
// 60 vector instructions per call.  kXor3 = false keeps the two-input form
// for kernels where the denser schedule costs occupancy (same words).
// ---------------------------------------------------------------------------
struct U4 {
    uint32_t x, y, z, w;
};

template <bool kXor3 = true>
__device__ __forceinline__ U4 philox(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                     uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t m0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
        const uint64_t m1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
        uint32_t n0, n2;
        if constexpr (kXor3) {
            n0 = __builtin_amdgcn_bitop3_b32((uint32_t)(m1 >> 32), c1, k0, 0x96);
            n2 = __builtin_amdgcn_bitop3_b32((uint32_t)(m0 >> 32), c3, k1, 0x96);
        } else {
            n0 = (uint32_t)(m1 >> 32) ^ c1 ^ k0;
            n2 = (uint32_t)(m0 >> 32) ^ c3 ^ k1;
        }
        c1 = (uint32_t)m1;
        c3 = (uint32_t)m0;
        c0 = n0;
        c2 = n2;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return U4{c0, c1, c2, c3};
}

// Top 24 bits times 2^-24: exact, in [0, 1).
__device__ __forceinline__ float u01(uint32_t w) { return (float)(w >> 8) * 0x1p-24f; }

// Streaming (nontemporal) 128-bit row accesses: population rows are touched
// once per generation, so they are loaded and stored with the nontemporal
// hint, which on gfx950 keeps them from displacing reused data in the caches
// and lets HBM run mixed read/write streams closer to peak.
typedef float v4f_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float4 ld_stream(const float *p)
{
    const v4f_t t = __builtin_nontemporal_load(reinterpret_cast<const v4f_t *>(p));
    return make_float4(t.x, t.y, t.z, t.w);
}

__device__ __forceinline__ void st_stream(float *p, float4 v)
{
    const v4f_t t = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(t, reinterpret_cast<v4f_t *>(p));
}

// Row access with the streaming hint only when `nt` (wave-uniform): a state
// that fits in the 256 MB last-level cache is better served by normal
// accesses, a larger one by streaming ones.
__device__ __forceinline__ float4 ld_row(const float *p, bool nt)
{
    return nt ? ld_stream(p) : *reinterpret_cast<const float4 *>(p);
}

__device__ __forceinline__ void st_row(float *p, float4 v, bool nt)
{
    if (nt)
        st_stream(p, v);
    else
        *reinterpret_cast<float4 *>(p) = v;
}

// Streamed bytes of one pass above which the streaming hint is used.
constexpr int64_t kStreamBytes = (int64_t)512 << 20;

__device__ __forceinline__ float comp(const float4 &v, int e)
{
    return e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w;
}
__device__ __forceinline__ float wcomp(const U4 &v, int e)
{
    return u01(e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w);
}

// ---------------------------------------------------------------------------
// Trigonometry.  cos(2 pi r) / sin(2 pi r) by exact reduction of r to
// [-1/2, 1/2] (r - rint(r) is exact in fp32) and the hardware v_cos_f32 /
// v_sin_f32, whose input is in revolutions.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float cos_rev(float r)
{
    return __builtin_amdgcn_cosf(r - __builtin_rintf(r));
}
__device__ __forceinline__ float sin_rev(float r)
{
    return __builtin_amdgcn_sinf(r - __builtin_rintf(r));
}

// Four standard normal deviates of float4 chunk c of row `row` at generation
// t of a stream: the Box-Muller transform of the word pairs (0, 1) and (2, 3)
// of one Philox call, u1 = ((a >> 8) + 1) 2^-24 in (0, 1], u2 = (b >> 8)
// 2^-24; the even element gets r cos(2 pi u2), the odd one r sin(2 pi u2),
// r = sqrt(-2 ln u1).  Stream 5 at generation 0 is the normal initial
// population, stream 7 the ES perturbations.
__device__ __forceinline__ float4 normal4(uint32_t c, uint32_t row, uint32_t t, uint32_t stream, uint32_t k0,
                                          uint32_t k1)
{
    const U4 w = philox(c, row, t, stream, k0, k1);
    // -2 ln u1 = -(2 ln 2) log2 u1 with the hardware log2 and square root
    // (u1 >= 2^-24 is never denormal; both within one ulp)
    constexpr float kTwoLn2 = 0x1.62e430p+0f;  // 2 ln 2 rounded to fp32
    const float r0 = __builtin_amdgcn_sqrtf(-kTwoLn2 * __builtin_amdgcn_logf((float)((w.x >> 8) + 1u) * 0x1p-24f));
    const float r1 = __builtin_amdgcn_sqrtf(-kTwoLn2 * __builtin_amdgcn_logf((float)((w.z >> 8) + 1u) * 0x1p-24f));
    const float a0 = u01(w.y), a1 = u01(w.w);
    return make_float4(r0 * cos_rev(a0), r0 * sin_rev(a0), r1 * cos_rev(a1), r1 * sin_rev(a1));
}

// ---------------------------------------------------------------------------
// Benchmark functions as row reductions.  Acc holds up to two partials; the
// per-element step sees x_j, its right neighbour x_{j+1} (Rosenbrock) and the
// 0-based index j; combine() merges two lanes' partials; finish() gives F.
// ---------------------------------------------------------------------------
struct Acc {
    float a, b;
};

template <int FN>
struct Fn;

template <>
struct Fn<FN_SPHERE> {  // sum x^2
    static constexpr bool kNeighbour = false;
    __device__ static Acc init() { return {0.f, 0.f}; }
    __device__ static void elem(Acc &s, float x, float, int64_t) { s.a = fmaf(x, x, s.a); }
    __device__ static Acc combine(Acc p, Acc q) { return {p.a + q.a, 0.f}; }
    __device__ static float finish(Acc s, int64_t) { return s.a; }
};

template <>
struct Fn<FN_ACKLEY> {  // a = sum x^2, b = sum cos(2 pi x)
    static constexpr bool kNeighbour = false;
    __device__ static Acc init() { return {0.f, 0.f}; }
    __device__ static void elem(Acc &s, float x, float, int64_t)
    {
        s.a = fmaf(x, x, s.a);
        s.b += cos_rev(x);
    }
    __device__ static Acc combine(Acc p, Acc q) { return {p.a + q.a, p.b + q.b}; }
    __device__ static float finish(Acc s, int64_t D)
    {
        const float n = (float)D;
        const float e1 = expf(-0.2f * sqrtf(s.a / n));
        const float e2 = expf(s.b / n);
        return (20.0f - 20.0f * e1) + (2.71828182845904523536f - e2);
    }
};

// sin(pi r) for |r| <= 1/2 as r P(r^2), P of degree 4 fitted to
// sin(pi r) / r on [0, 1/2] by iteratively reweighted least squares (fp32
// coefficients; within 3 ulp of sin(pi r) relative, at every r, evaluated
// with these fmas).
__device__ __forceinline__ float sinpi_reduced(float r)
{
    const float u = r * r;
    float p = fmaf(u, 0x1.3db0e6p-4f, -0x1.324cdcp-1f);
    p = fmaf(u, p, 0x1.4668b0p+1f);
    p = fmaf(u, p, -0x1.4abbc2p+2f);
    p = fmaf(u, p, 0x1.921fb6p+1f);
    return r * p;
}

template <>
struct Fn<FN_RASTRIGIN> {  // a = sum (x^2 + 20 sin^2(pi x)) = 10 D + sum (x^2 - 10 cos(2 pi x))
    static constexpr bool kNeighbour = false;
    __device__ static Acc init() { return {0.f, 0.f}; }
    __device__ static void elem(Acc &s, float x, float, int64_t)
    {
        // non-negative terms (1 - cos 2u = 2 sin^2 u): the sum is accurate
        // relative to F itself, also near the optimum; x - rint(x) is exact
        const float sn = sinpi_reduced(x - __builtin_rintf(x));
        s.a += fmaf(20.0f * sn, sn, x * x);
    }
    __device__ static Acc combine(Acc p, Acc q) { return {p.a + q.a, 0.f}; }
    __device__ static float finish(Acc s, int64_t) { return s.a; }
};

template <>
struct Fn<FN_GRIEWANK> {  // a = sum x^2, b = prod cos(x / sqrt(j + 1))
    static constexpr bool kNeighbour = false;
    __device__ static Acc init() { return {0.f, 1.f}; }
    __device__ static void elem(Acc &s, float x, float, int64_t j)
    {
        s.a = fmaf(x, x, s.a);
        s.b *= cosf(x * rsqrtf((float)(j + 1)));
    }
    __device__ static Acc combine(Acc p, Acc q) { return {p.a + q.a, p.b * q.b}; }
    __device__ static float finish(Acc s, int64_t) { return (1.0f - s.b) + s.a * (1.0f / 4000.0f); }
};

template <>
struct Fn<FN_ROSENBROCK> {  // sum_{j < D-1} 100 (x_{j+1} - x_j^2)^2 + (1 - x_j)^2
    static constexpr bool kNeighbour = true;
    __device__ static Acc init() { return {0.f, 0.f}; }
    __device__ static void elem(Acc &s, float x, float xn, int64_t)
    {
        const float d = fmaf(-x, x, xn);  // one rounding of x_{j+1} - x_j^2
        const float o = 1.0f - x;
        s.a += fmaf(100.0f * d, d, o * o);
    }
    __device__ static Acc combine(Acc p, Acc q) { return {p.a + q.a, 0.f}; }
    __device__ static float finish(Acc s, int64_t) { return s.a; }
};

template <>
struct Fn<FN_SCHWEFEL> {  // a = sum x sin(sqrt|x|)
    static constexpr bool kNeighbour = false;
    __device__ static Acc init() { return {0.f, 0.f}; }
    __device__ static void elem(Acc &s, float x, float, int64_t)
    {
        const float r = sqrtf(fabsf(x)) * 0.159154943091895335769f;  // revolutions
        s.a = fmaf(x, sin_rev(r), s.a);
    }
    __device__ static Acc combine(Acc p, Acc q) { return {p.a + q.a, 0.f}; }
    __device__ static float finish(Acc s, int64_t D) { return 418.9829f * (float)D - s.a; }
};

// ---------------------------------------------------------------------------
// Row fitness from the registers of a G-lane group.  xr[it] holds chunk
// g + G*it (zeros outside the row).  All lanes of the group return F.
// nbr: LDS scratch of block_for(G) * MAXIT floats, used for the Rosenbrock
// neighbour when a row spans several waves; red: LDS of block_for(G)/64 * 2
// floats for the cross-wave step.  Must be reached by every thread of the
// block (it contains barriers when G > 64).
// ---------------------------------------------------------------------------
template <int G>
__device__ __forceinline__ float shfl_xor_g(float v, int m)
{
    return __shfl_xor(v, m, G < 64 ? G : 64);
}

// Combines the partials of a G-lane row group: butterfly inside the wave,
// then (G > 64) across the group's waves through red (LDS of
// block_for(G)/64 * 2 floats).  Every lane returns the combined partial.
// Must be reached by every thread of the block (barriers when G > 64).
template <int FN, int G>
__device__ __forceinline__ Acc group_reduce(Acc s, float *red)
{
    using F = Fn<FN>;
#pragma unroll
    for (int m = (G < 64 ? G : 64) / 2; m >= 1; m >>= 1) {
        Acc o{shfl_xor_g<G>(s.a, m), shfl_xor_g<G>(s.b, m)};
        s = F::combine(s, o);
    }
    if constexpr (G > 64) {
        const int tid = threadIdx.x;
        constexpr int W = G / 64;  // waves per row
        const int wave = tid / 64;
        if ((tid & 63) == 0) {
            red[2 * wave] = s.a;
            red[2 * wave + 1] = s.b;
        }
        __syncthreads();
        const int w0 = (wave / W) * W;
        Acc t{red[2 * w0], red[2 * w0 + 1]};
#pragma unroll
        for (int q = 1; q < W; ++q) t = F::combine(t, Acc{red[2 * (w0 + q)], red[2 * (w0 + q) + 1]});
        __syncthreads();
        s = t;
    }
    return s;
}

template <int FN, int G, int MAXIT>
__device__ __forceinline__ float row_fitness(const float4 (&xr)[MAXIT], int g, int64_t D,
                                             float *nbr, float *red)
{
    using F = Fn<FN>;
    const int tid = threadIdx.x;
    // right neighbour of the last element of each chunk
    float nb[MAXIT];
    if constexpr (F::kNeighbour) {
        if constexpr (G <= 64) {
#pragma unroll
            for (int it = 0; it < MAXIT; ++it) {
                const float same = __shfl(xr[it].x, (g + 1) & (G - 1), G);
                const float next = it + 1 < MAXIT ? __shfl(xr[it + 1 < MAXIT ? it + 1 : it].x, 0, G)
                                                  : 0.0f;
                nb[it] = g == G - 1 ? next : same;
            }
        } else {
            const int base = (tid / G) * G * MAXIT;
#pragma unroll
            for (int it = 0; it < MAXIT; ++it) nbr[base + it * G + g] = xr[it].x;
            __syncthreads();
#pragma unroll
            for (int it = 0; it < MAXIT; ++it) {
                const int k = it * G + g + 1;
                nb[it] = k < G * MAXIT ? nbr[base + k] : 0.0f;
            }
            __syncthreads();
        }
    } else {
#pragma unroll
        for (int it = 0; it < MAXIT; ++it) nb[it] = 0.0f;
    }

    Acc s = F::init();
#pragma unroll
    for (int it = 0; it < MAXIT; ++it) {
        const int64_t j0 = 4 * ((int64_t)g + (int64_t)G * it);
        const float4 v = xr[it];
        const float n4[4] = {v.y, v.z, v.w, nb[it]};
        const int64_t lim = F::kNeighbour ? D - 1 : D;  // last element has no pair
        if (j0 + 3 < lim) {
#pragma unroll
            for (int e = 0; e < 4; ++e) F::elem(s, comp(v, e), n4[e], j0 + e);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (j0 + e < lim) F::elem(s, comp(v, e), n4[e], j0 + e);
        }
    }
    return F::finish(group_reduce<FN, G>(s, red), D);
}

// ---------------------------------------------------------------------------
// Selection order: smaller value, then lower index; -0 == +0; NaN after all
// numbers.  A total order, so any reduction tree gives the same winner.  It
// is encoded as one 64-bit key, (order-preserving value bits << 32) | index,
// so the order is an unsigned integer min and a block's candidate is folded
// into a slot with one atomicMin.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t sel_key(float v, int64_t i)
{
    uint32_t o;
    if (v != v) {
        o = 0xFFFFFFFFu;
    } else {
        uint32_t b = __float_as_uint(v);
        if ((b << 1) == 0) b = 0;  // -0 -> +0
        o = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
    }
    return ((uint64_t)o << 32) | (uint32_t)i;
}

__device__ __forceinline__ float key_value(uint64_t k)
{
    const uint32_t o = (uint32_t)(k >> 32);
    if (o == 0xFFFFFFFFu) return __builtin_nanf("");
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}

__device__ __forceinline__ int64_t key_index(uint64_t k) { return (int64_t)(uint32_t)k; }

constexpr uint64_t kNoKey = ~(uint64_t)0;

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m)
{
    const int lo = __shfl_xor((int)(uint32_t)v, m, 64);
    const int hi = __shfl_xor((int)(uint32_t)(v >> 32), m, 64);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

// Block-wide min of per-thread keys and sum of counts; thread 0 gets them.
// sk / sc: LDS of blockDim/64 entries each.  Reached by every thread.
__device__ __forceinline__ void block_min_key(uint64_t &k, uint32_t &cnt, uint64_t *sk, uint32_t *sc)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        const uint64_t o = shfl_xor_u64(k, m);
        k = o < k ? o : k;
        cnt += (uint32_t)__shfl_xor((int)cnt, m, 64);
    }
    const int wave = threadIdx.x / 64, nw = blockDim.x / 64;
    if ((threadIdx.x & 63) == 0) {
        sk[wave] = k;
        sc[wave] = cnt;
    }
    __syncthreads();
    if (threadIdx.x == 0)
        for (int q = 1; q < nw; ++q) {
            k = sk[q] < k ? sk[q] : k;
            cnt += sc[q];
        }
}

// Selection slots in device scratch: every block of a row kernel folds its
// candidate into key[blockIdx mod kSlots] (and its improved-row count into
// cnt); k_select reduces the slots and resets them.
struct SelSlots {
    uint64_t key[kSlots];
    uint32_t cnt[kSlots];
};

__device__ __forceinline__ void slot_commit(SelSlots *sl, uint64_t k, uint32_t cnt)
{
    const int s = blockIdx.x & (kSlots - 1);
    if (k != kNoKey) atomicMin((unsigned long long *)&sl->key[s], (unsigned long long)k);
    if (cnt) atomicAdd(&sl->cnt[s], cnt);
}

// Result of a selection, kept in device scratch.
struct DevBest {
    float f;
    int32_t pad;
    int64_t i;
    uint64_t improved;  // PSO: rows whose personal best improved, summed
};

}  // namespace evox
