// Function-independent kernels of the gfx950 path: initialisation, selection
// (second pass), fills, the CSO pairing sort and swarm mean, the Philox
// diagnostic, and the dispatch from a function id to its instantiation.
//
// Pairing (CSO).  The permutation is the order of the individuals by
// (key, index), key_i = Philox stream-4 word of individual i at generation t.
// Keys are uniform 32-bit numbers, so a superbucket sort does it in three
// light passes over 4096-individual chunks (kPermChunk):
//   k_perm_count  per-superbucket counts (top `bits` key bits; LDS
//                 histogram, one global atomic per nonempty bucket)
//   k_perm_place  scan of the counts, per-block range reservation, and
//                 placement of (key, index) into the superbucket ranges, as
//                 one 8-byte entry so a block's run of a bucket is contiguous
//   k_perm_sort   one block per superbucket (~1000 entries): counting sort on
//                 the next 8 key bits in LDS, then ranks inside sub-buckets,
//                 written as the permutation
// The permutation depends only on (seed, t), so a batch of generations is
// sorted at once (grid dimension y), which fills the GPU far better than one
// generation of these latency-bound passes.
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
            if (a.x_normal) {
                const float4 z = normal4((uint32_t)c, (uint32_t)row, 0u, STREAM_INIT_NORMAL, a.k0, a.k1);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (4 * c + e < a.D) xo[e] = fmaf(a.sigma, comp(z, e), a.mu);
            } else {
                const U4 rx = philox((uint32_t)c, (uint32_t)row, 0u, STREAM_INIT_X, a.k0, a.k1);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (4 * c + e < a.D) xo[e] = fmaf(wcomp(rx, e), xr, a.lb);
            }
            if (a.v && !a.v_zero) {
                const U4 rv = philox((uint32_t)c, (uint32_t)row, 0u, STREAM_INIT_V, a.k0, a.k1);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (4 * c + e < a.D) vo[e] = fmaf(wcomp(rv, e), vr, a.v_lo);
            }
        }
        const float4 X = make_float4(xo[0], xo[1], xo[2], xo[3]);
        reinterpret_cast<float4 *>(a.x)[q] = X;
        if (a.v) reinterpret_cast<float4 *>(a.v)[q] = make_float4(vo[0], vo[1], vo[2], vo[3]);
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
// Second pass of the selection: one block reduces the kSlots keys (and the
// improved-row counts), resets them for the next launch, stores the result,
// and copies the selected row (ldx floats) to row_out.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void k_select(SelSlots *sl, const float *rows, int64_t ldx,
                                                 float *row_out, DevBest *best, float *bf_out,
                                                 int64_t *bi_out)
{
    __shared__ uint64_t sk[16];
    __shared__ uint32_t sc[16];
    __shared__ int64_t sel;
    uint64_t k = kNoKey;
    uint32_t cnt = 0;
    for (int q = threadIdx.x; q < kSlots; q += blockDim.x) {
        const uint64_t kq = sl->key[q];
        k = kq < k ? kq : k;
        cnt += sl->cnt[q];
        sl->key[q] = kNoKey;
        sl->cnt[q] = 0;
    }
    block_min_key(k, cnt, sk, sc);
    if (threadIdx.x == 0) {
        const float v = key_value(k);
        const int64_t i = k == kNoKey ? 0 : key_index(k);
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

hipError_t launch_select(SelSlots *slots, const float *rows, int64_t ldx, float *row_out,
                         DevBest *best, float *best_f_out, int64_t *best_i_out, hipStream_t s)
{
    hipLaunchKernelGGL(k_select, dim3(1), dim3(1024), 0, s, slots, rows, ldx, row_out, best,
                       best_f_out, best_i_out);
    return hipGetLastError();
}

__global__ __launch_bounds__(1024) void k_slots_init(SelSlots *sl)
{
    for (int q = threadIdx.x; q < kSlots; q += blockDim.x) {
        sl->key[q] = kNoKey;
        sl->cnt[q] = 0;
    }
}

hipError_t launch_slots_init(SelSlots *slots, hipStream_t s)
{
    hipLaunchKernelGGL(k_slots_init, dim3(1), dim3(1024), 0, s, slots);
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

__global__ __launch_bounds__(256) void k_fill_u32(uint32_t *dst, int64_t n, uint32_t value)
{
    for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < n; j += (int64_t)gridDim.x * 256)
        dst[j] = value;
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

hipError_t launch_fill_u32(uint32_t *dst, int64_t n, uint32_t value, hipStream_t s)
{
    hipLaunchKernelGGL(k_fill_u32, dim3(flat_grid(n)), dim3(256), 0, s, dst, n, value);
    return hipGetLastError();
}

hipError_t launch_zero_u32(uint32_t *dst, int64_t n, hipStream_t s) { return launch_fill_u32(dst, n, 0u, s); }

// First pass of the selection over a stored fitness array.
__global__ __launch_bounds__(256) void k_argmin_slots(const float *f, int64_t n, SelSlots *sl)
{
    __shared__ uint64_t sk[4];
    __shared__ uint32_t sc[4];
    uint64_t k = kNoKey;
    uint32_t none = 0;
    for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < n; j += (int64_t)gridDim.x * 256) {
        const uint64_t kj = sel_key(f[j], j);
        k = kj < k ? kj : k;
    }
    block_min_key(k, none, sk, sc);
    if (threadIdx.x == 0) slot_commit(sl, k, 0);
}

hipError_t launch_argmin_slots(const float *f, int64_t N, SelSlots *slots, hipStream_t s)
{
    hipLaunchKernelGGL(k_argmin_slots, dim3(flat_grid(N)), dim3(256), 0, s, f, N, slots);
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

// Streaming copy (the bandwidth reference): one float4 per thread with
// nontemporal loads and stores (the fastest plain copy measured on the
// MI355X, ahead of 2-8 float4 per thread), the last n % 4 floats one by one.
__global__ __launch_bounds__(256) void k_stream_copy(const float *src, float *dst, int64_t n)
{
    const int64_t n4 = n / 4;
    for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < n4; q += (int64_t)gridDim.x * 256)
        st_stream(dst + 4 * q, ld_stream(src + 4 * q));
    if (blockIdx.x == 0 && threadIdx.x < (n & 3)) dst[4 * n4 + threadIdx.x] = src[4 * n4 + threadIdx.x];
}

hipError_t launch_stream_copy(const float *src, float *dst, int64_t n, hipStream_t s)
{
    int64_t grid = (n / 4 + 255) / 256;
    if (grid > kMaxGrid) grid = kMaxGrid;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(k_stream_copy, dim3((unsigned)grid), dim3(256), 0, s, src, dst, n);
    return hipGetLastError();
}

// Diagnostic: the 20 B per element stream of a PSO generation alone, one
// float4 per thread (grid-stride only beyond kMaxGrid blocks).
__global__ __launch_bounds__(256) void k_pso_stream(float *x, float *v, const float *p, int64_t n4)
{
    for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < n4; q += (int64_t)gridDim.x * 256) {
        const float4 xv = ld_stream(x + 4 * q), vv = ld_stream(v + 4 * q), pv = ld_stream(p + 4 * q);
        const float4 vn = make_float4(vv.x + (pv.x - xv.x), vv.y + (pv.y - xv.y), vv.z + (pv.z - xv.z),
                                      vv.w + (pv.w - xv.w));
        st_stream(v + 4 * q, vn);
        st_stream(x + 4 * q, make_float4(xv.x + vn.x, xv.y + vn.y, xv.z + vn.z, xv.w + vn.w));
    }
}

hipError_t launch_pso_stream(float *x, float *v, const float *p, int64_t n, hipStream_t s)
{
    const int64_t n4 = n / 4;
    int64_t grid = (n4 + 255) / 256;
    if (grid > kMaxGrid) grid = kMaxGrid;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(k_pso_stream, dim3((unsigned)grid), dim3(256), 0, s, x, v, p, n4);
    return hipGetLastError();
}

__device__ __forceinline__ uint32_t bucket_of(uint32_t key, int bits)
{
    return bits ? key >> (32 - bits) : 0u;
}

// A batch of permutations covers generations t0 .. t0 + gridDim.y - 1; block
// row blockIdx.y works on generation t0 + blockIdx.y and its slice of each
// array (counts nb, offsets nb + 1, keys / indices / permutation N).
struct PermSlice {
    uint32_t t;
    uint32_t *hist, *offs, *cursor;
    uint2 *tkv;
    uint32_t *perm;
    uint32_t *mate;  // null: no mate array
};

__device__ __forceinline__ PermSlice perm_slice(const PermArgs &a)
{
    const int64_t b = blockIdx.y, nb = (int64_t)1 << a.bits;
    return PermSlice{a.t0 + (uint32_t)b, a.hist + b * nb, a.offs + b * (nb + 1), a.cursor + b * nb,
                     a.tkv + b * a.N, a.perm + b * a.N, a.mate ? a.mate + b * a.N : nullptr};
}

// Mate entry of the individual at permutation position pos whose partner,
// at position pos ^ 1, is `other`: pairs are positions (2k, 2k + 1), the
// first of a pair wins ties.
__device__ __forceinline__ uint32_t mate_entry(uint32_t pos, uint32_t other)
{
    return other | ((pos & 1u) ? 0u : kMateFirst);
}

// Keys of the individuals 4 * (blockIdx.x * kPermChunk / 4 + r * 256 + tid)
// + e, r < kPermChunk / 1024, e < 4, handled by one thread of a perm block
// (kPermChunk per block): words of Philox stream 4, or the caller's keys.
template <typename F>
__device__ __forceinline__ void for_block_keys(const PermArgs &a, uint32_t t, F &&f)
{
    const int64_t q0 = (int64_t)blockIdx.x * (kPermChunk / 4);
#pragma unroll
    for (int r = 0; r < kPermChunk / 1024; ++r) {
        const int64_t q = q0 + r * 256 + threadIdx.x;
        if (4 * q < a.N) {
            uint32_t k4[4];
            if (a.keys) {
#pragma unroll
                for (int e = 0; e < 4; ++e) k4[e] = 4 * q + e < a.N ? a.keys[4 * q + e] : 0u;
            } else {
                const U4 w = philox((uint32_t)q, 0u, t, STREAM_PERM, a.k0, a.k1);
                k4[0] = w.x;
                k4[1] = w.y;
                k4[2] = w.z;
                k4[3] = w.w;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (4 * q + e < a.N) f(k4[e], 4 * q + e);
        }
    }
}

// Pass 1: per-superbucket counts (LDS histogram per block, then one global
// atomic per nonempty bucket).
__global__ __launch_bounds__(256) void k_perm_count(PermArgs a)
{
    __shared__ uint32_t h[kPermMaxBuckets];
    const PermSlice sl = perm_slice(a);
    const int nb = 1 << a.bits;
    for (int b = threadIdx.x; b < nb; b += 256) h[b] = 0;
    __syncthreads();
    for_block_keys(a, sl.t, [&](uint32_t key, int64_t) { atomicAdd(&h[bucket_of(key, a.bits)], 1u); });
    __syncthreads();
    for (int b = threadIdx.x; b < nb; b += 256)
        if (h[b]) atomicAdd(&sl.hist[b], h[b]);
}

// Exclusive scan of n <= kPermMaxBuckets counts into off (LDS), 256 threads.
__device__ __forceinline__ void lds_exclusive_scan(const uint32_t *cnt, int n, uint32_t *off)
{
    __shared__ uint32_t tsum[256];
    const int per = (n + 255) / 256, lo = threadIdx.x * per;
    const int hi = lo + per < n ? lo + per : n;
    uint32_t s = 0;
    for (int b = lo; b < hi; ++b) s += cnt[b];
    tsum[threadIdx.x] = s;
    __syncthreads();
    for (int d = 1; d < 256; d <<= 1) {
        const uint32_t v = threadIdx.x >= d ? tsum[threadIdx.x - d] : 0u;
        __syncthreads();
        tsum[threadIdx.x] += v;
        __syncthreads();
    }
    uint32_t run = threadIdx.x ? tsum[threadIdx.x - 1] : 0u;
    for (int b = lo; b < hi; ++b) {
        off[b] = run;
        run += cnt[b];
    }
    __syncthreads();
}

// Pass 2: every block scans the counts (block 0 also publishes the offsets),
// reserves a range per bucket for its own keys, and places (key, index).
__global__ __launch_bounds__(256) void k_perm_place(PermArgs a)
{
    __shared__ uint32_t cnt[kPermMaxBuckets];
    __shared__ uint32_t off[kPermMaxBuckets];
    const PermSlice sl = perm_slice(a);
    const int nb = 1 << a.bits;
    for (int b = threadIdx.x; b < nb; b += 256) cnt[b] = sl.hist[b];
    __syncthreads();
    lds_exclusive_scan(cnt, nb, off);
    if (blockIdx.x == 0) {
        for (int b = threadIdx.x; b < nb; b += 256) sl.offs[b] = off[b];
        if (threadIdx.x == 0) sl.offs[nb] = (uint32_t)a.N;
    }
    for (int b = threadIdx.x; b < nb; b += 256) cnt[b] = 0;
    __syncthreads();
    for_block_keys(a, sl.t, [&](uint32_t key, int64_t) { atomicAdd(&cnt[bucket_of(key, a.bits)], 1u); });
    __syncthreads();
    for (int b = threadIdx.x; b < nb; b += 256)
        if (cnt[b]) off[b] += atomicAdd(&sl.cursor[b], cnt[b]);
    __syncthreads();
    for_block_keys(a, sl.t, [&](uint32_t key, int64_t i) {
        const uint32_t pos = atomicAdd(&off[bucket_of(key, a.bits)], 1u);
        sl.tkv[pos] = make_uint2(key, (uint32_t)i);
    });
}

// Pass 3: one block per superbucket orders its entries by (key, index): a
// counting sort on the next 8 key bits (256 sub-buckets of ~4 entries) in
// LDS, then each entry's rank inside its sub-bucket by comparison; the
// ordered indices are written as the permutation.  The bucket's count and
// cursor are then cleared for the next batch.  A bucket larger than the LDS
// capacity (not expected for uniform keys) is ranked in global memory.
__global__ __launch_bounds__(256) void k_perm_sort(PermArgs a)
{
    __shared__ uint32_t K[kPermSortCap], I[kPermSortCap], S[kPermSortCap];
    __shared__ uint32_t cnt[256], start[256], cur[256];
    const PermSlice sl = perm_slice(a);
    const int b = blockIdx.x;
    const uint32_t lo = sl.offs[b], n = sl.hist[b];
    const int shift = 24 - a.bits;  // the 8 key bits below the superbucket bits
    if (n <= (uint32_t)kPermSortCap) {
        cnt[threadIdx.x] = 0;
        __syncthreads();
        for (uint32_t q = threadIdx.x; q < n; q += 256)
            atomicAdd(&cnt[(sl.tkv[lo + q].x >> shift) & 255u], 1u);
        __syncthreads();
        if (threadIdx.x < 64) {  // exclusive scan of 256 counts by one wave, 4 per lane
            const int l = threadIdx.x;
            const uint32_t c0 = cnt[4 * l], c1 = cnt[4 * l + 1], c2 = cnt[4 * l + 2], c3 = cnt[4 * l + 3];
            uint32_t tot = c0 + c1 + c2 + c3, inc = tot;
            for (int d = 1; d < 64; d <<= 1) {
                const uint32_t o = __shfl_up(inc, d, 64);
                if (l >= d) inc += o;
            }
            const uint32_t ex = inc - tot;
            start[4 * l] = ex;
            start[4 * l + 1] = ex + c0;
            start[4 * l + 2] = ex + c0 + c1;
            start[4 * l + 3] = ex + c0 + c1 + c2;
        }
        __syncthreads();
        cur[threadIdx.x] = start[threadIdx.x];
        __syncthreads();
        for (uint32_t q = threadIdx.x; q < n; q += 256) {
            const uint2 e = sl.tkv[lo + q];
            const uint32_t pos = atomicAdd(&cur[(e.x >> shift) & 255u], 1u);
            K[pos] = e.x;
            I[pos] = e.y;
        }
        __syncthreads();
        for (uint32_t q = threadIdx.x; q < n; q += 256) {
            const uint32_t key = K[q], idx = I[q], sb = (key >> shift) & 255u;
            const uint32_t s0 = start[sb], s1 = s0 + cnt[sb];
            uint32_t rank = 0;
            // bitwise, not short-circuit: no branch per entry
            for (uint32_t r = s0; r < s1; ++r) rank += (uint32_t)((K[r] < key) | ((K[r] == key) & (I[r] < idx)));
            S[s0 + rank] = idx;
        }
        __syncthreads();
        for (uint32_t q = threadIdx.x; q < n; q += 256) sl.perm[lo + q] = S[q];
        if (sl.mate) {
            // pairs inside this superbucket's range; a pair that straddles two
            // ranges is written by k_perm_edges
            for (uint32_t q = threadIdx.x; q < n; q += 256) {
                const uint32_t pos = lo + q, other = pos ^ 1u;
                if ((int64_t)other >= a.N)
                    sl.mate[S[q]] = kUnpaired;
                else if (other >= lo && other < lo + n)
                    sl.mate[S[q]] = mate_entry(pos, S[other - lo]);
            }
        }
    } else {
        for (uint32_t p = threadIdx.x; p < n; p += 256) {
            const uint32_t key = sl.tkv[lo + p].x, idx = sl.tkv[lo + p].y;
            uint32_t rank = 0;
            for (uint32_t q = 0; q < n; ++q) {
                const uint32_t kq = sl.tkv[lo + q].x, iq = sl.tkv[lo + q].y;
                rank += (uint32_t)((kq < key) | ((kq == key) & (iq < idx)));
            }
            sl.perm[lo + rank] = idx;
        }
        if (sl.mate) {
            __syncthreads();  // the block's permutation entries are written
            for (uint32_t q = threadIdx.x; q < n; q += 256) {
                const uint32_t pos = lo + q, other = pos ^ 1u;
                if ((int64_t)other >= a.N)
                    sl.mate[sl.perm[pos]] = kUnpaired;
                else if (other >= lo && other < lo + n)
                    sl.mate[sl.perm[pos]] = mate_entry(pos, sl.perm[other]);
            }
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        sl.hist[b] = 0;
        sl.cursor[b] = 0;
    }
}

// Pass 4 (mate arrays only): the pairs that straddle two superbucket ranges,
// one thread per range start.  A range that starts at an odd position lo
// splits the pair (lo - 1, lo); empty ranges share their start with the next
// range and write the same two entries again.
__global__ __launch_bounds__(256) void k_perm_edges(PermArgs a)
{
    const PermSlice sl = perm_slice(a);
    const int b = blockIdx.x * 256 + threadIdx.x, nb = 1 << a.bits;
    if (b < 1 || b >= nb) return;
    const uint32_t lo = sl.offs[b];
    if ((int64_t)lo >= a.N || (lo & 1u) == 0) return;
    const uint32_t first = sl.perm[lo - 1], second = sl.perm[lo];
    sl.mate[first] = second | kMateFirst;
    sl.mate[second] = first;
}

hipError_t launch_perm(const PermArgs &a, hipStream_t s)
{
    const unsigned chunks = (unsigned)((a.N + kPermChunk - 1) / kPermChunk);
    const unsigned nb = 1u << a.bits;
    hipLaunchKernelGGL(k_perm_count, dim3(chunks, a.batch), dim3(256), 0, s, a);
    hipLaunchKernelGGL(k_perm_place, dim3(chunks, a.batch), dim3(256), 0, s, a);
    hipLaunchKernelGGL(k_perm_sort, dim3(nb, a.batch), dim3(256), 0, s, a);
    if (a.mate) hipLaunchKernelGGL(k_perm_edges, dim3((nb + 255) / 256, a.batch), dim3(256), 0, s, a);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Diagnostic: the data movement of one swarm-mean CSO generation alone, in
// the generation kernel's traversal (ranges of kCsoSweep individuals, the
// losers listed in index order, one row group per listed loser): gather the
// winner's row, read the loser's x and v, write v + (x_w - x) and the moved
// x.  No random numbers, no fitness, no column sums: the floor the
// generation kernel's row traffic sets on this hardware.
// ---------------------------------------------------------------------------
template <int G>
__global__ __launch_bounds__(block_for(G)) void k_pair_move(float *x, float *v, int64_t N, int64_t D, int64_t ldx,
                                                            const int32_t *winner_of)
{
    constexpr int B = block_for(G), RPB = B / G, NW = B / 64, R = kCsoSweep;
    static_assert(R <= B, "one individual per thread in the listing phase");
    __shared__ int32_t lst_l[R], lst_w[R];
    __shared__ int32_t wcnt[NW];
    const int tid = threadIdx.x, g = tid % G, slot = tid / G, lane = tid & 63, wave = tid >> 6;
    const int64_t C4 = (D + 3) >> 2;
    for (int64_t base = (int64_t)blockIdx.x * R; base < N; base += (int64_t)gridDim.x * R) {
        int32_t w = -1;
        if (tid < R && base + tid < N) w = winner_of[base + tid];
        const bool listed = w >= 0 && w < N;  // an index out of range is ignored
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
            lst_l[at] = (int32_t)(base + tid);
            lst_w[at] = w;
        }
        __syncthreads();
        for (int q = slot; q < total; q += RPB) {
            const int64_t l = lst_l[q], wr = lst_w[q];
            for (int64_t c = g; c < C4; c += G) {
                const int64_t off_l = l * ldx + 4 * c;
                const float4 xw = *reinterpret_cast<const float4 *>(x + wr * ldx + 4 * c);
                const float4 xl = ld_stream(x + off_l);
                const float4 vl = ld_stream(v + off_l);
                const float4 vn = make_float4(vl.x + (xw.x - xl.x), vl.y + (xw.y - xl.y), vl.z + (xw.z - xl.z),
                                              vl.w + (xw.w - xl.w));
                st_stream(v + off_l, vn);
                st_stream(x + off_l, make_float4(xl.x + vn.x, xl.y + vn.y, xl.z + vn.z, xl.w + vn.w));
            }
        }
        __syncthreads();  // the next range overwrites the list
    }
}

template <int G>
static hipError_t launch_pair_move_g(float *x, float *v, int64_t N, int64_t D, int64_t ldx, const int32_t *winner_of,
                                     hipStream_t s)
{
    int occ = 0, dev = 0, cus = 0;
    (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, k_pair_move<G>, block_for(G), 0);
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                                 hipSuccess)
        cus = 256;
    int64_t grid = (N + kCsoSweep - 1) / kCsoSweep;
    const int64_t resident = (int64_t)cus * (occ > 0 ? occ : 1);
    if (grid > resident) grid = resident;
    hipLaunchKernelGGL((k_pair_move<G>), dim3((unsigned)grid), dim3(block_for(G)), 0, s, x, v, N, D, ldx, winner_of);
    return hipGetLastError();
}

hipError_t launch_pair_move(int G, float *x, float *v, int64_t N, int64_t D, int64_t ldx, const int32_t *winner_of,
                            hipStream_t s)
{
    switch (G) {
        case 4: return launch_pair_move_g<4>(x, v, N, D, ldx, winner_of, s);
        case 8: return launch_pair_move_g<8>(x, v, N, D, ldx, winner_of, s);
        case 16: return launch_pair_move_g<16>(x, v, N, D, ldx, winner_of, s);
        case 32: return launch_pair_move_g<32>(x, v, N, D, ldx, winner_of, s);
        case 64: return launch_pair_move_g<64>(x, v, N, D, ldx, winner_of, s);
        case 128: return launch_pair_move_g<128>(x, v, N, D, ldx, winner_of, s);
        case 256: return launch_pair_move_g<256>(x, v, N, D, ldx, winner_of, s);
        case 512: return launch_pair_move_g<512>(x, v, N, D, ldx, winner_of, s);
        case 1024: return launch_pair_move_g<1024>(x, v, N, D, ldx, winner_of, s);
        default: return hipErrorInvalidValue;
    }
}

// Block (0, 0) also finishes the selection (slots -> best) when asked.
// xbar = (sum of the per-block partial rows) / N, rounded once, in two
// stages.  Block (tile, rg) of 64 columns x 4 lanes: lane l sums partial rows
// rg + S (l + 4 u), u = 0, 1, ... (S = m.stages) in that order, the four
// lanes are added in lane order into s1[rg].  The last block of a tile to
// finish sums s1[0..S) the same way (lane l: stages l + 4 u) and writes the
// mean.  Padding columns get 0.  Loads go out in batches of 8.
__device__ __forceinline__ double strided_sum(const double *base, int64_t first, int64_t step,
                                              int64_t end, int64_t pitch)
{
    double s = 0.0;
    for (int64_t q0 = first; q0 < end; q0 += 8 * step) {
        double v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int64_t q = q0 + u * step;
            v[u] = q < end ? __hip_atomic_load(base + q * pitch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                           : 0.0;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) s += v[u];
    }
    return s;
}

__global__ __launch_bounds__(256) void k_cso_mean(MeanArgs m)
{
    __shared__ double part[4][64];
    __shared__ int last;
    if (m.slots && blockIdx.x == 0 && blockIdx.y == 0) {
        // second pass of the selection over the generation kernel's slots
        __shared__ uint64_t sk[4];
        __shared__ uint32_t sc[4];
        // all of a thread's slot loads issued before any of the resets, so
        // the pass costs one memory latency instead of one per slot row
        constexpr int R = kSlots / 256;
        static_assert(kSlots % 256 == 0, "whole slot rows per thread");
        uint64_t kq[R];
#pragma unroll
        for (int u = 0; u < R; ++u) kq[u] = m.slots->key[threadIdx.x + 256 * u];
        uint64_t k = kNoKey;
        uint32_t none = 0;
#pragma unroll
        for (int u = 0; u < R; ++u) {
            k = kq[u] < k ? kq[u] : k;
            m.slots->key[threadIdx.x + 256 * u] = kNoKey;
            m.slots->cnt[threadIdx.x + 256 * u] = 0;
        }
        block_min_key(k, none, sk, sc);
        if (threadIdx.x == 0) {
            m.best->f = key_value(k);
            m.best->i = k == kNoKey ? 0 : key_index(k);
        }
    }
    const int col = threadIdx.x & 63, lane = threadIdx.x >> 6;
    const int64_t tile = blockIdx.x, rg = blockIdx.y;
    const int64_t j = tile * 64 + col;
    double s = 0.0;
    if (j < m.D) s = strided_sum(m.xsum + j, rg + (int64_t)m.stages * lane, 4 * (int64_t)m.stages, m.nparts, m.ldx);
    part[lane][col] = s;
    __syncthreads();
    if (lane == 0) {  // wave 0 writes this block's stage sums and releases them
        if (j < m.D) m.s1[rg * m.ldx + j] = ((part[0][col] + part[1][col]) + part[2][col]) + part[3][col];
        __threadfence();
    }
    __syncthreads();
    if (threadIdx.x == 0) last = atomicAdd(&m.ticket[tile], 1u) == (uint32_t)(m.stages - 1);
    __syncthreads();
    if (last) {
        __threadfence();
        double t = 0.0;
        if (j < m.D) t = strided_sum(m.s1 + j, lane, 4, m.stages, m.ldx);
        part[lane][col] = t;
        __syncthreads();
        if (lane == 0 && j < m.ldx) {
            const double u = ((part[0][col] + part[1][col]) + part[2][col]) + part[3][col];
            m.xbar[j] = j < m.D ? (float)(u / (double)m.N) : 0.0f;
        }
        if (threadIdx.x == 0) m.ticket[tile] = 0;
    }
}

hipError_t launch_cso_mean(const MeanArgs &m, hipStream_t s)
{
    const unsigned tiles = (unsigned)((m.ldx + 63) / 64);
    if (m.stages < 1 || m.stages > kMeanStages) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_cso_mean, dim3(tiles, (unsigned)m.stages), dim3(256), 0, s, m);
    return hipGetLastError();
}

#define EVOX_LAUNCH_COLSUM(GG, MM, UNUSED) \
    hipLaunchKernelGGL((k_colsum<GG, MM>), dim3(grid), dim3(block_for(GG)), 0, s, x, N, D, ldx, xsum)

hipError_t launch_colsum(Layout L, const float *x, int64_t N, int64_t D, int64_t ldx, double *xsum,
                         int grid, hipStream_t s)
{
    switch (L.G * 16 + L.maxit) {
        EVOX_FAMILY_CASES(EVOX_LAUNCH_COLSUM, LAYOUT_CSO, 0)
        EVOX_BIG_CASES(EVOX_LAUNCH_COLSUM, LAYOUT_CSO, 0)
        default: return hipErrorInvalidValue;
    }
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

hipError_t launch_pso(int fn, Layout L, int mode, const PsoArgs &a, int grid, hipStream_t s)
{
    if (mode == PSO_MOVE) fn = FN_SPHERE;  // the move does not evaluate
#define EVOX_CALL_PSO(F) launch_pso_t<F>(L, mode, a, grid, s)
    EVOX_FN_SWITCH(EVOX_CALL_PSO)
}

hipError_t launch_pso_small(int fn, Layout L, const PsoArgs &a, int64_t n_gens, float *gbest_out, DevBest *best,
                            hipStream_t s)
{
#define EVOX_CALL_PSO_SMALL(F) launch_pso_small_t<F>(L, a, n_gens, gbest_out, best, s)
    EVOX_FN_SWITCH(EVOX_CALL_PSO_SMALL)
}

hipError_t launch_eval(int fn, Layout L, bool vec, const EvalArgs &a, int grid, hipStream_t s)
{
#define EVOX_CALL_EVAL(F) launch_eval_t<F>(L, vec, a, grid, s)
    EVOX_FN_SWITCH(EVOX_CALL_EVAL)
}

hipError_t launch_cso(int fn, Layout L, const CsoArgs &a, int grid, hipStream_t s)
{
#define EVOX_CALL_CSO(F) launch_cso_t<F>(L, a, grid, s)
    EVOX_FN_SWITCH(EVOX_CALL_CSO)
}

hipError_t launch_de(int fn, Layout L, const DeArgs &a, int grid, hipStream_t s)
{
#define EVOX_CALL_DE(F) launch_de_t<F>(L, a, grid, s)
    EVOX_FN_SWITCH(EVOX_CALL_DE)
}

hipError_t launch_es_eval(int fn, Layout L, const EsArgs &a, int grid, hipStream_t s)
{
#define EVOX_CALL_ES(F) launch_es_eval_t<F>(L, a, grid, s)
    EVOX_FN_SWITCH(EVOX_CALL_ES)
}

hipError_t launch_mae_eval(int fn, Layout L, const MaeEvalArgs &a, int grid, hipStream_t s)
{
#define EVOX_CALL_MAE(F) launch_mae_eval_t<F>(L, a, grid, s)
    EVOX_FN_SWITCH(EVOX_CALL_MAE)
}

// ---------------------------------------------------------------------------
// OpenES centered ranks: rank_i = #{j : key_j < key_i} with key = (orderable
// fitness, index), the argmin order, so the ranks are a permutation and NaN
// ranks last.  Block (tile of 256 kEsRankPer samples i, kEsRankPer per
// thread, range of kEsRankSpan samples j) stages its j-keys in LDS, counts
// (each key read from LDS serves kEsRankPer comparisons), and adds each
// count to rank_i with one integer atomic per i (exact, so the result does
// not depend on the order of the additions).  rank is zeroed by k_es_eval
// of the same generation.
// ---------------------------------------------------------------------------
constexpr int kEsRankSpan = 128, kEsRankPer = 4;

__global__ __launch_bounds__(256) void k_es_rank(const float *fit, int64_t N, uint32_t *rank)
{
    __shared__ uint64_t kj[kEsRankSpan];
    const int64_t i0 = (int64_t)blockIdx.x * (256 * kEsRankPer) + threadIdx.x;
    const int64_t j0 = (int64_t)blockIdx.y * kEsRankSpan;
    const int64_t nj = N - j0 < kEsRankSpan ? N - j0 : kEsRankSpan;
    for (int q = threadIdx.x; q < nj; q += 256) kj[q] = sel_key(fit[j0 + q], j0 + q);
    __syncthreads();
    uint64_t ki[kEsRankPer];
    uint32_t below[kEsRankPer];
#pragma unroll
    for (int u = 0; u < kEsRankPer; ++u) {
        const int64_t i = i0 + 256 * u;
        ki[u] = i < N ? sel_key(fit[i], i) : 0;  // key 0 counts nothing below it
        below[u] = 0;
    }
    for (int q = 0; q < nj; ++q) {
        const uint64_t k = kj[q];
#pragma unroll
        for (int u = 0; u < kEsRankPer; ++u) below[u] += k < ki[u] ? 1u : 0u;
    }
#pragma unroll
    for (int u = 0; u < kEsRankPer; ++u) {
        const int64_t i = i0 + 256 * u;
        if (i < N && below[u]) atomicAdd(&rank[i], below[u]);
    }
}

hipError_t launch_es_rank(const float *fit, int64_t N, uint32_t *rank, hipStream_t s)
{
    const unsigned tiles = (unsigned)((N + 256 * kEsRankPer - 1) / (256 * kEsRankPer)),
                   spans = (unsigned)((N + kEsRankSpan - 1) / kEsRankSpan);
    hipLaunchKernelGGL(k_es_rank, dim3(tiles, spans), dim3(256), 0, s, fit, N, rank);
    return hipGetLastError();
}

// Gradient, pass 1: thread (pair chunk b, column chunk c) sums, over its
// kEsPairChunk pairs and in fp64, the deviates z_k regenerated from Philox
// exactly as the samples drew them, weighted by the pair's centered ranks
// u = rank / (N - 1) - 1/2:
//   OpenES  w_k z_k,               w_k = (u_{2k} - u_{2k+1}) / (N sigma)
//   PGPE    m_k z_k and s_k (z_k^2 - 1),
//           m_k = (u_{2k} - u_{2k+1}) / (2H), s_k = (u_{2k} + u_{2k+1}) / (2H)
// (the per-dimension sigma_j factor of PGPE is applied in pass 2).
template <bool PGPE>
__global__ __launch_bounds__(256) void k_es_grad(EsGradArgs a)
{
    // the chunk's pair weights, computed once per block (three fp64
    // divisions per pair) and read from LDS by every column
    __shared__ double wts[PGPE ? 2 : 1][kEsPairChunk];
    static_assert(kEsPairChunk <= 256, "one thread per pair of the chunk");
    const int64_t C4 = (a.D + 3) / 4;
    const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x, b = blockIdx.y;
    const int64_t k0 = b * kEsPairChunk, k1 = k0 + kEsPairChunk < a.H ? k0 + kEsPairChunk : a.H;
    if (threadIdx.x < k1 - k0) {
        const int64_t k = k0 + threadIdx.x;
        const double nm1 = (double)(2 * a.H - 1);
        const double u0 = (double)a.rank[2 * k] / nm1 - 0.5, u1 = (double)a.rank[2 * k + 1] / nm1 - 0.5;
        if constexpr (PGPE) {
            wts[0][threadIdx.x] = 0.5 * (u0 - u1) / (double)a.H;
            wts[1][threadIdx.x] = 0.5 * (u0 + u1) / (double)a.H;
        } else {
            wts[0][threadIdx.x] = (u0 - u1) / ((double)(2 * a.H) * (double)a.sigma);
        }
    }
    __syncthreads();
    if (c >= C4) return;
    double s[4] = {0.0, 0.0, 0.0, 0.0}, q[4] = {0.0, 0.0, 0.0, 0.0};
    for (int64_t k = k0; k < k1; ++k) {
        const float4 z = normal4((uint32_t)c, (uint32_t)k, a.t, a.stream, a.k0, a.k1);
        const double zz[4] = {(double)z.x, (double)z.y, (double)z.z, (double)z.w};
        if constexpr (PGPE) {
            const double m = wts[0][k - k0], sw = wts[1][k - k0];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                s[e] = fma(m, zz[e], s[e]);
                q[e] = fma(sw, zz[e] * zz[e] - 1.0, q[e]);
            }
        } else {
            const double w = wts[0][k - k0];
#pragma unroll
            for (int e = 0; e < 4; ++e) s[e] = fma(w, zz[e], s[e]);
        }
    }
    const int64_t chunks = (a.H + kEsPairChunk - 1) / kEsPairChunk;
    double *dst = a.part + b * 4 * C4 + 4 * c;
#pragma unroll
    for (int e = 0; e < 4; ++e) dst[e] = s[e];
    if constexpr (PGPE) {
        double *dq = dst + chunks * 4 * C4;
#pragma unroll
        for (int e = 0; e < 4; ++e) dq[e] = q[e];
    }
}

// Pass 2: per column, the chunks' partial sums -- kEsUpdSlices slice sums in
// chunk order, combined in a fixed order in LDS -- then the steps, each gradient
// rounded to fp32 once:
//   theta_j <- fma(-lr, g_j, theta_j)       (PGPE: g_j = sigma_j * sum)
//   PGPE: d_j = -sig_lr * (sigma_j * sum'), clamped to +-max_change sigma_j,
//         sigma_j <- sigma_j + d_j.
// Block: 64 columns x kEsUpdSlices slices.
constexpr int kEsUpdSlices = 16;  // chunk-row slices summed in parallel per column

template <bool PGPE>
__global__ __launch_bounds__(64 * kEsUpdSlices) void k_es_update(EsGradArgs a, int64_t chunks)
{
    __shared__ double qs[2][kEsUpdSlices][64];
    const int64_t C4 = (a.D + 3) / 4;
    const int col = threadIdx.x & 63, qt = threadIdx.x >> 6;
    const int64_t j = (int64_t)blockIdx.x * 64 + col;
    const int64_t per = (chunks + kEsUpdSlices - 1) / kEsUpdSlices, b0 = qt * per,
                  b1 = b0 + per < chunks ? b0 + per : chunks;
    double g = 0.0, h = 0.0;
    if (j < a.D)
        for (int64_t b = b0; b < b1; ++b) {
            g += a.part[b * 4 * C4 + j];
            if constexpr (PGPE) h += a.part[(chunks + b) * 4 * C4 + j];
        }
    qs[0][qt][col] = g;
    qs[1][qt][col] = h;
    __syncthreads();
    if (qt == 0 && j < a.D) {
        double gj = qs[0][0][col], hj = qs[1][0][col];
#pragma unroll
        for (int r = 1; r < kEsUpdSlices; ++r) {
            gj += qs[0][r][col];
            hj += qs[1][r][col];
        }
        if constexpr (PGPE) {
            const float sj = a.sig[j];
            a.theta[j] = fmaf(-a.lr, (float)((double)sj * gj), a.theta[j]);
            const float cap = a.max_change * sj;
            const float d = fminf(fmaxf(-a.sig_lr * (float)((double)sj * hj), -cap), cap);
            a.sig[j] = sj + d;
        } else {
            (void)hj;
            a.theta[j] = fmaf(-a.lr, (float)gj, a.theta[j]);
        }
    }
}

hipError_t launch_es_grad(const EsGradArgs &a, hipStream_t s)
{
    const int64_t C4 = (a.D + 3) / 4, chunks = (a.H + kEsPairChunk - 1) / kEsPairChunk;
    const dim3 grid((unsigned)((C4 + 255) / 256), (unsigned)chunks), upd((unsigned)((a.D + 63) / 64));
    if (a.sig) {
        hipLaunchKernelGGL(k_es_grad<true>, grid, dim3(256), 0, s, a);
        hipLaunchKernelGGL(k_es_update<true>, upd, dim3(64 * kEsUpdSlices), 0, s, a, chunks);
    } else {
        hipLaunchKernelGGL(k_es_grad<false>, grid, dim3(256), 0, s, a);
        hipLaunchKernelGGL(k_es_update<false>, upd, dim3(64 * kEsUpdSlices), 0, s, a, chunks);
    }
    return hipGetLastError();
}

int occupancy_cso(int fn, Layout L, bool local)
{
    switch (fn) {
    case FN_SPHERE: return occupancy_cso_t<FN_SPHERE>(L, local);
    case FN_ACKLEY: return occupancy_cso_t<FN_ACKLEY>(L, local);
    case FN_RASTRIGIN: return occupancy_cso_t<FN_RASTRIGIN>(L, local);
    case FN_GRIEWANK: return occupancy_cso_t<FN_GRIEWANK>(L, local);
    case FN_ROSENBROCK: return occupancy_cso_t<FN_ROSENBROCK>(L, local);
    case FN_SCHWEFEL: return occupancy_cso_t<FN_SCHWEFEL>(L, local);
    default: return 0;
    }
}

}  // namespace evox
