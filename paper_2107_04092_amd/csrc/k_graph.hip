// gfx950 kernels of the graph builder (Fig. 1 data structures): an int64
// scan for row pointers, random Bernoulli and fixed-fan-out rows, grouping of
// an edge list by source, per-row LDS sort by (target, weight), and slice
// pivots with plastic prefixes.
#include "snn_device.h"

namespace snn {
namespace {

// ---------------------------------------------------------------------------
// inclusive scan of int64 in place: chunks of 4*kBlock, chunk totals, offsets

constexpr int kScanChunk = 4 * kBlock;

__device__ long long block_incl_scan_i64(long long v, long long *sh)
{
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const long long u = __shfl_up(v, off, kWave);
        if (lane >= off) v += u;
    }
    __syncthreads();
    if (lane == kWave - 1) sh[wave] = v;
    __syncthreads();
    for (int q = 0; q < wave; ++q) v += sh[q];
    return v;
}

__global__ __launch_bounds__(kBlock) void k_scan_local(int64_t *d, int64_t count, int64_t *bsum)
{
    __shared__ long long sh[kBlock / kWave];
    const int64_t base = (int64_t)blockIdx.x * kScanChunk + threadIdx.x * 4;
    long long x[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) x[q] = base + q < count ? d[base + q] : 0;
    x[1] += x[0];
    x[2] += x[1];
    x[3] += x[2];
    const long long incl = block_incl_scan_i64(x[3], sh);
    const long long excl = incl - x[3];
#pragma unroll
    for (int q = 0; q < 4; ++q)
        if (base + q < count) d[base + q] = x[q] + excl;
    if (threadIdx.x == kBlock - 1) bsum[blockIdx.x] = incl;
}

__global__ __launch_bounds__(kBlock) void k_scan_bsum(int64_t *bsum, int64_t nb)
{
    __shared__ long long sh[kBlock / kWave];
    __shared__ long long carry;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int64_t b0 = 0; b0 < nb; b0 += kBlock) {
        const int64_t i = b0 + threadIdx.x;
        const long long v = i < nb ? bsum[i] : 0;
        const long long incl = block_incl_scan_i64(v, sh);
        const long long c = carry;
        if (i < nb) bsum[i] = c + incl - v;  // exclusive offsets
        __syncthreads();
        if (threadIdx.x == kBlock - 1) carry = c + incl;
        __syncthreads();
    }
}

__global__ __launch_bounds__(kBlock) void k_scan_add(int64_t *d, int64_t count, const int64_t *bsum)
{
    const long long off = bsum[blockIdx.x];
    const int64_t base = (int64_t)blockIdx.x * kScanChunk;
    for (int q = threadIdx.x; q < kScanChunk; q += kBlock)
        if (base + q < count) d[base + q] += off;
}

// ---------------------------------------------------------------------------
// graph builder (Fig. 1 data structures)

// Bernoulli rows: count the pairs (k, j), j != k, whose stream-0 draw is
// below the threshold; row_ptr[k+1] = count (scanned afterwards).
__global__ __launch_bounds__(kBlock) void k_count_bernoulli(GraphArgs a)
{
    __shared__ long long sh[kBlock / kWave];
    const int k = blockIdx.x;
    long long c = 0;
    for (int j = threadIdx.x; j < a.n; j += kBlock)
        c += (j != k) && rng32(a.seed, 0, (uint64_t)k, (uint64_t)j) < a.thr;
    c = block_sum_i64(c, sh);
    if (threadIdx.x == 0) {
        a.row_ptr[k + 1] = c;
        if (k == 0) a.row_ptr[0] = 0;
    }
}

// Bernoulli rows: write the present targets in ascending order (ballot-rank
// within each wave, wave offsets through LDS) with the source's weight.
__global__ __launch_bounds__(kBlock) void k_fill_bernoulli(GraphArgs a)
{
    __shared__ int s_wc[kBlock / kWave];
    const int k = blockIdx.x, tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    const int64_t base = a.row_ptr[k];
    const float wk = k < a.n_exc ? a.w_exc : a.w_inh;
    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    int64_t off = 0;
    for (int j0 = 0; j0 < a.n; j0 += kBlock) {
        const int j = j0 + tid;
        const bool f = j < a.n && j != k && rng32(a.seed, 0, (uint64_t)k, (uint64_t)j) < a.thr;
        const uint64_t m = ballot64(f);
        if (lane == 0) s_wc[wave] = __popcll(m);
        __syncthreads();
        int pre = 0, tot = 0;
#pragma unroll
        for (int q = 0; q < kBlock / kWave; ++q) {
            pre += q < wave ? s_wc[q] : 0;
            tot += s_wc[q];
        }
        if (f) {
            const int64_t pos = base + off + pre + __popcll(m & below);
            a.col[pos] = j;
            a.w[pos] = wk;
        }
        off += tot;
        __syncthreads();
    }
}

__global__ __launch_bounds__(kBlock) void k_rowptr_fanout(GraphArgs a)
{
    const int64_t k = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (k <= a.n) a.row_ptr[k] = k * a.fanout;
}

// Fixed fan-out: edge (k, b) targets (u32 * n) >> 32 of stream 1 at (k, b).
__global__ __launch_bounds__(kBlock) void k_fill_fanout(GraphArgs a)
{
    const int64_t total = (int64_t)a.n * a.fanout;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < total; e += stride) {
        const int64_t k = e / a.fanout, b = e - k * a.fanout;
        const uint32_t u = rng32(a.seed, 1, (uint64_t)k, (uint64_t)b);
        a.col[e] = (int32_t)(((uint64_t)u * (uint64_t)a.n) >> 32);
        a.w[e] = k < a.n_exc ? a.w_exc : a.w_inh;
    }
}

// Edge list: validate indices and count per source into row_ptr[src+1].
__global__ __launch_bounds__(kBlock) void k_edges_count(GraphArgs a, const int32_t *src,
                                                        const int32_t *dst, int64_t e)
{
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < e; i += stride) {
        const int32_t s = src[i], d = dst[i];
        if (s < 0 || s >= a.n || d < 0 || d >= a.n) {
            atomicOr(a.err, kErrIndex);
            continue;
        }
        atomicAdd((unsigned long long *)(a.row_ptr + s + 1), 1ull);
    }
}

__global__ __launch_bounds__(kBlock) void k_edges_scatter(GraphArgs a, const int32_t *src,
                                                          const int32_t *dst, const float *w,
                                                          int64_t e, int64_t *cursor)
{
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < e; i += stride) {
        const int32_t s = src[i], d = dst[i];
        if (s < 0 || s >= a.n || d < 0 || d >= a.n) continue;
        const int64_t pos = (int64_t)atomicAdd((unsigned long long *)(cursor + s), 1ull);
        a.col[pos] = d;
        a.w[pos] = w[i];
    }
}

__global__ __launch_bounds__(kBlock) void k_row_maxlen(GraphArgs a)
{
    const int k = blockIdx.x * kBlock + threadIdx.x;
    int len = 0;
    if (k < a.n) {
        const int64_t l = a.row_ptr[k + 1] - a.row_ptr[k];
        len = (int)(l > 0x7fffffff ? 0x7fffffff : l);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) len = max(len, __shfl_xor(len, off, kWave));
    if (threadIdx.x % kWave == 0 && len > 0) atomicMax(a.maxlen, len);  // one per wave
}

// Order-preserving map of fp32 bits to uint32 (negative floats reversed).
__device__ __forceinline__ uint32_t f2ord(float f)
{
    const uint32_t b = __float_as_uint(f);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float ord2f(uint32_t o)
{
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}

// Sorts each row by (target, weight) with a bitonic network in LDS.
constexpr int kSortBlock = 1024;
__global__ __launch_bounds__(kSortBlock) void k_row_sort(GraphArgs a)
{
    extern __shared__ unsigned long long keys[];
    const int k = blockIdx.x, tid = threadIdx.x;
    const int64_t rs = a.row_ptr[k];
    const int len = (int)(a.row_ptr[k + 1] - rs);
    if (len <= 1) return;
    if (len > kMaxSortRow) {
        if (tid == 0) atomicOr(a.err, kErrRowTooLong);
        return;
    }
    int p2 = 2;
    while (p2 < len) p2 <<= 1;
    for (int x = tid; x < p2; x += kSortBlock)
        keys[x] = x < len ? (((unsigned long long)(uint32_t)a.col[rs + x] << 32) |
                             f2ord(a.w[rs + x]))
                          : ~0ull;
    __syncthreads();
    for (int size = 2; size <= p2; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int x = tid; x < (p2 >> 1); x += kSortBlock) {
                const int lo = 2 * stride * (x / stride) + (x % stride);
                const int hi = lo + stride;
                const bool up = (lo & size) == 0;
                const unsigned long long u = keys[lo], v = keys[hi];
                if ((u > v) == up) {
                    keys[lo] = v;
                    keys[hi] = u;
                }
            }
            __syncthreads();
        }
    }
    for (int x = tid; x < len; x += kSortBlock) {
        const unsigned long long key = keys[x];
        a.col[rs + x] = (int32_t)(key >> 32);
        a.w[rs + x] = ord2f((uint32_t)key);
    }
}

// First index in the row [p, p+len) (sorted by target) whose target is >= v.
__device__ __forceinline__ int lower_bound_col(const int32_t *p, int len, int64_t v)
{
    int lo = 0, hi = len;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if ((int64_t)p[mid] < v) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// Pivots (Fig. 1): piv[k][s] = lower_bound(row k, s*W), s = 0..S, so that
// row entries piv[k][s] .. piv[k][s+1]-1 target slice s. One wave per row,
// lanes over slices. Also the plastic prefix end of each row.
__global__ __launch_bounds__(kBlock) void k_pivots(GraphArgs a)
{
    const int lane = threadIdx.x % kWave;
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    for (int64_t k = ((int64_t)blockIdx.x * kBlock + threadIdx.x) / kWave; k < a.n;
         k += waves) {  // wave-uniform
        const int64_t rs = a.row_ptr[k];
        const int len = (int)(a.row_ptr[k + 1] - rs);
        const int32_t *row = a.col + rs;
        int32_t *out = a.piv + k * (int64_t)(a.n_slices + 1);
        for (int s = lane; s <= a.n_slices; s += kWave)
            out[s] = s == a.n_slices ? len : lower_bound_col(row, len, (int64_t)s * a.width);
        if (lane == 0) {
            int pe = 0;
            if (a.plastic == 2) pe = len;
            else if (a.plastic == 1 && k < a.n_exc) pe = lower_bound_col(row, len, a.n_exc);
            a.pend[k] = pe;
        }
    }
}

// Compressed targets: each entry's slice-local index, target - sW for the
// slice s = target / W that holds it (16 bits for W <= 65536).
__global__ __launch_bounds__(kBlock) void k_encode_targets(GraphArgs a, int64_t n_edges)
{
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < n_edges; e += stride)
        a.col16[e] = (uint16_t)(a.col[e] % a.width);
}

}  // namespace

hipError_t launch_scan_i64(hipStream_t s, int64_t *data, int64_t count, int64_t *bsum)
{
    if (count <= 0) return hipSuccess;
    const int64_t nb = (count + kScanChunk - 1) / kScanChunk;
    hipLaunchKernelGGL(k_scan_local, dim3((unsigned)nb), dim3(kBlock), 0, s, data, count, bsum);
    hipLaunchKernelGGL(k_scan_bsum, dim3(1), dim3(kBlock), 0, s, bsum, nb);
    hipLaunchKernelGGL(k_scan_add, dim3((unsigned)nb), dim3(kBlock), 0, s, data, count, bsum);
    return hipGetLastError();
}

hipError_t launch_graph_count_bernoulli(hipStream_t s, const GraphArgs &a)
{
    hipLaunchKernelGGL(k_count_bernoulli, dim3(a.n), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_graph_fill_bernoulli(hipStream_t s, const GraphArgs &a)
{
    hipLaunchKernelGGL(k_fill_bernoulli, dim3(a.n), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_graph_fill_fanout(hipStream_t s, const GraphArgs &a)
{
    hipLaunchKernelGGL(k_rowptr_fanout, dim3(blocks_for((int64_t)a.n + 1)), dim3(kBlock), 0, s,
                       a);
    if (a.col != nullptr) {
        hipLaunchKernelGGL(k_fill_fanout, dim3(blocks_for((int64_t)a.n * a.fanout, kBlock,
                                                          1 << 16)),
                           dim3(kBlock), 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_edges_count(hipStream_t s, const GraphArgs &a, const int32_t *src,
                              const int32_t *dst, int64_t e)
{
    if (e <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_edges_count, dim3(blocks_for(e, kBlock, 1 << 16)), dim3(kBlock), 0, s,
                       a, src, dst, e);
    return hipGetLastError();
}

hipError_t launch_edges_scatter(hipStream_t s, const GraphArgs &a, const int32_t *src,
                                const int32_t *dst, const float *w, int64_t e,
                                int64_t *cursor)
{
    if (e <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_edges_scatter, dim3(blocks_for(e, kBlock, 1 << 16)), dim3(kBlock), 0,
                       s, a, src, dst, w, e, cursor);
    return hipGetLastError();
}

hipError_t launch_row_maxlen(hipStream_t s, const GraphArgs &a)
{
    hipLaunchKernelGGL(k_row_maxlen, dim3(blocks_for(a.n)), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_row_sort(hipStream_t s, const GraphArgs &a, int pow2len)
{
    static std::mutex mu;
    static int granted = 64 * 1024;
    const size_t lds = (size_t)pow2len * sizeof(unsigned long long);
    const hipError_t e = allow_dynamic_lds((const void *)k_row_sort, (int)lds, mu, granted);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_row_sort, dim3(a.n), dim3(kSortBlock), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_pivots(hipStream_t s, const GraphArgs &a)
{
    hipLaunchKernelGGL(k_pivots, dim3(blocks_for((int64_t)a.n * kWave)), dim3(kBlock), 0, s,
                       a);
    return hipGetLastError();
}

hipError_t launch_encode_targets(hipStream_t s, const GraphArgs &a, int64_t n_edges)
{
    if (n_edges <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_encode_targets, dim3(blocks_for(n_edges, kBlock, 1 << 16)), dim3(kBlock),
                       0, s, a, n_edges);
    return hipGetLastError();
}

}  // namespace snn
