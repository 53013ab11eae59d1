// gfx950 (CDNA4) kernels of the synapse pass: neuron update, spike-list
// compaction, lazy + event-driven STDP, slice (LDS) and global-atomic
// delivery, and the sliced-CSR graph builder.
//
// Built with -ffp-contract=off: the neuron update must reproduce a fixed
// fp32 operation order, so no multiply-add is ever fused.
#include "snn_internal.h"

#include <mutex>

namespace snn {
namespace {

// ---------------------------------------------------------------------------
// helpers

// SplitMix64 output function (Steele, Lea & Flood 2014) of seed XOR key, with
// key = stream << 58 | a << 24 | b: a counter-based draw per (stream, a, b).
__device__ __forceinline__ uint32_t rng32(uint64_t seed, uint32_t stream, uint64_t a,
                                          uint64_t b)
{
    uint64_t z = (seed ^ (((uint64_t)stream << 58) | (a << 24) | b)) + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    return (uint32_t)(z >> 32);
}

__device__ __forceinline__ uint64_t ballot64(bool p) { return __builtin_amdgcn_ballot_w64(p); }

// fp32 -> fixed point (x * 2^32 is exact in fp32; only |x| < 2^-9 loses bits)
__device__ __forceinline__ long long to_fix(float x) { return __float2ll_rn(x * kFixScale); }
// fixed point -> fp32, one correctly rounded conversion (the scaling is exact)
__device__ __forceinline__ float from_fix(long long s) { return __ll2float_rn(s) * kFixUnit; }

__device__ __forceinline__ int wave_sum_i32(int v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

__device__ __forceinline__ long long wave_sum_i64(long long v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

// Sum over a kBlock-thread workgroup; every thread gets the total.
__device__ __forceinline__ long long block_sum_i64(long long v, long long *sh)
{
    v = wave_sum_i64(v);
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    __syncthreads();
    if (lane == 0) sh[wave] = v;
    __syncthreads();
    long long t = 0;
#pragma unroll
    for (int q = 0; q < kBlock / kWave; ++q) t += sh[q];
    return t;
}

// Sum / inclusive scan over a NT-thread workgroup (sh: NT/64 entries).
template <int NT>
__device__ __forceinline__ long long block_sum_i64_n(long long v, long long *sh)
{
    v = wave_sum_i64(v);
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    __syncthreads();
    if (lane == 0) sh[wave] = v;
    __syncthreads();
    long long t = 0;
#pragma unroll
    for (int q = 0; q < NT / kWave; ++q) t += sh[q];
    return t;
}

template <int NT>
__device__ __forceinline__ long long block_incl_scan_i64_n(long long v, long long *sh)
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

// ---------------------------------------------------------------------------
// state initialisation and fills (kernels instead of memsets so that a
// captured step never contains a memset node)

__global__ __launch_bounds__(kBlock) void k_init_state(float *v, int32_t *ref, float *ie,
                                                       float *ii, uint64_t *hist, float *ypost,
                                                       int32_t *t_last, float *xpre, int32_t n)
{
    const int i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= n) return;
    v[i] = 0.f;
    ref[i] = 0;
    ie[i] = 0.f;
    ii[i] = 0.f;
    hist[i] = 0ull;
    ypost[i] = 0.f;
    t_last[i] = -1;
    xpre[i] = 0.f;
}

template <typename T>
__global__ __launch_bounds__(kBlock) void k_fill(T *p, int64_t count, T value)
{
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < count; i += stride)
        p[i] = value;
}

// ---------------------------------------------------------------------------
// (1) neuron update. One thread per neuron, one wave64 per mask word.

__global__ __launch_bounds__(kBlock) void k_neuron(NeuronArgs a)
{
    const int tid = threadIdx.x;
    const int i = blockIdx.x * kBlock + tid;
    int s = 0, trig = 0;
    if (i < a.n) {
        if (a.model == 2) {
            s = rng32(a.seed, 4, (uint64_t)a.t, (uint64_t)i) < a.fire_thr;
        } else {
            float ae, ai = 0.f;
            if (a.input_forced) {
                ae = a.ain[i];
                if (a.model == 1) ai = a.ain[a.n + i];
            } else {
                long long se = a.apart[i];
                for (int c = 1; c < a.n_parts; ++c) se += a.apart[c * a.part_stride + i];
                ae = from_fix(se);
                if (a.model == 1) {
                    long long si = a.apart[a.n + i];
                    for (int c = 1; c < a.n_parts; ++c) si += a.apart[c * a.part_stride + a.n + i];
                    ai = from_fix(si);
                }
            }
            float v = a.v[i];
            int r = a.ref[i];
            if (a.model == 1) {
                const float ie = __fadd_rn(__fmul_rn(a.ie[i], a.d_e), ae);
                const float ii = __fadd_rn(__fmul_rn(a.ii[i], a.d_i), ai);
                a.ie[i] = ie;
                a.ii[i] = ii;
                if (r > 0) {
                    r -= 1;
                    v = a.v_reset;
                } else {
                    float x = __fsub_rn(a.v_inf, v);
                    x = __fadd_rn(x, ie);
                    x = __fadd_rn(x, ii);
                    v = __fadd_rn(v, __fmul_rn(x, a.k_m));
                    if (v >= a.v_th) {
                        s = 1;
                        v = a.v_reset;
                        r = a.ref_steps;
                    }
                }
            } else {
                if (r > 0) {
                    r -= 1;
                    v = a.v_reset;
                } else {
                    float x = 0.f;
                    if (a.poisson_len > 0) {
                        const uint32_t u = rng32(a.seed, 3, (uint64_t)a.t, (uint64_t)i);
                        int k = 0;
                        for (int q = 0; q < a.poisson_len; ++q) k += (a.poisson[q] <= u);
                        x = __fmul_rn(a.j_ext, (float)k);
                    }
                    const float d = __fsub_rn(a.v_inf, v);
                    const float b = __fmul_rn(d, a.k_m);
                    const float c = __fadd_rn(v, b);
                    v = __fadd_rn(c, ae);
                    v = __fadd_rn(v, x);
                    if (v >= a.v_th) {
                        s = 1;
                        v = a.v_reset;
                        r = a.ref_steps;
                    }
                }
            }
            a.v[i] = v;
            a.ref[i] = r;
        }
        uint64_t h = a.hist[i];
        if (a.n_plastic_rows > 0) {
            // post trace seen by a pre spike at step t: posts strictly before t
            const float y = __fmul_rn(__fadd_rn(a.ypost[i], (float)(h & 1ull)), a.d_minus);
            a.ypost[i] = y;
        }
        h = (h << 1) | (uint64_t)s;
        a.hist[i] = h;
        if (i < a.n_plastic_rows) {
            const int tx = (int)((h >> a.dm1) & 1ull);
            trig = tx | (a.t - (int64_t)a.t_last[i] >= 64);
        }
    }
    const uint64_t m = ballot64(s), rm = ballot64(trig);
    const int wave = tid / kWave, lane = tid % kWave;
    const int64_t word = (int64_t)blockIdx.x * (kBlock / kWave) + wave;
    __shared__ int s_cnt[2][kBlock / kWave];
    if (lane == 0) {
        if (word * kWave < a.n) {
            a.mask[word] = m;
            a.rmask[word] = rm;
        }
        s_cnt[0][wave] = __popcll(m);
        s_cnt[1][wave] = __popcll(rm);
    }
    __syncthreads();
    if (tid == 0) {
        int c0 = 0, c1 = 0;
#pragma unroll
        for (int q = 0; q < kBlock / kWave; ++q) {
            c0 += s_cnt[0][q];
            c1 += s_cnt[1][q];
        }
        a.blk_spk[blockIdx.x] = c0;
        a.blk_row[blockIdx.x] = c1;
    }
}

// Ascending spike list and plastic-row list from the masks: each workgroup
// adds the counts of the workgroups before it, then ranks its bits.
__global__ __launch_bounds__(kBlock) void k_compact(CompactArgs a)
{
    __shared__ long long sh[kBlock / kWave];
    __shared__ int s_pc[2][kBlock / kWave];
    const int tid = threadIdx.x, b = blockIdx.x;
    long long p0 = 0, p1 = 0;
    for (int q = tid; q < b; q += kBlock) {
        p0 += a.blk_spk[q];
        p1 += a.blk_row[q];
    }
    // pack both prefix sums into one reduction (each < 2^31)
    const long long packed = block_sum_i64((p0 << 32) | p1, sh);
    p0 = packed >> 32;
    p1 = packed & 0xffffffffll;
    const int wave = tid / kWave, lane = tid % kWave;
    const int64_t word = (int64_t)b * (kBlock / kWave) + wave;
    const uint64_t m = word < a.nw ? a.mask[word] : 0ull;
    const uint64_t rm = word < a.nw ? a.rmask[word] : 0ull;
    if (lane == 0) {
        s_pc[0][wave] = __popcll(m);
        s_pc[1][wave] = __popcll(rm);
    }
    __syncthreads();
    int o0 = (int)p0, o1 = (int)p1, t0 = 0, t1 = 0;
#pragma unroll
    for (int q = 0; q < kBlock / kWave; ++q) {
        if (q < wave) {
            o0 += s_pc[0][q];
            o1 += s_pc[1][q];
        }
        t0 += s_pc[0][q];
        t1 += s_pc[1][q];
    }
    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    const int i = (int)(word * kWave) + lane;
    if ((m >> lane) & 1ull) a.spk_list[o0 + __popcll(m & below)] = i;
    if ((rm >> lane) & 1ull) a.row_list[o1 + __popcll(rm & below)] = i;
    if (b == (int)gridDim.x - 1 && tid == 0) {
        *a.spk_cnt = (int)p0 + t0;
        *a.row_cnt = (int)p1 + t1;
        a.gstats[kGSpikes] += (int)p0 + t0;
    }
}

// ---------------------------------------------------------------------------
// (2) lazy + event-driven STDP (Sec. III-A, Fig. 2(b,c)).
//
// Row k was last brought up to date at step t_last; its age is t - t_last
// (1..64). A wave takes one row at a time; each lane one synapse k->j per
// 64-wide column of the row. The post spikes of j in the window are the set
// bits age-1..0 of hist[j] (bit i = spike at step t-i); they are visited
// oldest first via count-leading-zeros, each potentiating with the pre trace
// decayed to its step. A row transmitting at t then depresses with the post
// trace y_j(t), and a post at t itself potentiates with the pre trace that
// includes the pre spike at t.
//
// Memory-level parallelism: a lane issues the loads of its U synapses of a
// 64*U chunk (targets, weights), then all their history (and post-trace)
// gathers, before any arithmetic, so one wave keeps up to 2U (3U) loads in
// flight and a 1000-synapse row costs about one load and one gather latency.

template <int U>
__global__ __launch_bounds__(kBlock) void k_stdp(StdpArgs a)
{
    __shared__ float s_dpow[65];
    __shared__ long long sh[kBlock / kWave];
    const int tid = threadIdx.x;
    for (int q = tid; q < 65; q += kBlock) s_dpow[q] = a.dpow[q];
    __syncthreads();
    const int32_t *__restrict__ col = a.col;
    float *__restrict__ wgt = a.w;
    const uint64_t *__restrict__ hist = a.hist;
    const float *__restrict__ ypost = a.ypost;
    const int lane = tid % kWave;
    const int gw = (blockIdx.x * kBlock + tid) / kWave;
    const int nwv = gridDim.x * (kBlock / kWave);
    const bool flush = a.rows == nullptr;
    const int nrows = flush ? a.n_rows_all : *a.row_cnt;
    long long st_rows = 0, st_forced = 0, st_syn = 0, st_written = 0;
    for (int r = gw; r < nrows; r += nwv) {
        const int k = flush ? r : a.rows[r];
        int age = (int)(a.t - (int64_t)a.t_last[k]);
        if (age <= 0) continue;  // flush: row already current (wave-uniform)
        if (age > 64) {
            // the plasticity part was skipped for this row: posts older than
            // the history word are lost; flag it and stay inside the table
            if (lane == 0) atomicOr(a.err, kErrWindow);
            age = 64;
        }
        const int pre = flush ? 0 : (int)((hist[k] >> a.dm1) & 1ull);
        const float xp0 = a.xpre[k];
        const int64_t rs = a.row_ptr[k];
        const int len = a.pend[k];
        const uint64_t win = age >= 64 ? ~0ull : ((1ull << age) - 1ull);
        const float xp_now = __fadd_rn(__fmul_rn(xp0, s_dpow[age]), (float)pre);
        for (int base = 0; base < len; base += kWave * U) {
            int j[U];
            float w[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int q = base + u * kWave + lane;
                j[u] = q < len ? col[rs + q] : -1;
                w[u] = q < len ? wgt[rs + q] : 0.f;
            }
            uint64_t h[U];
#pragma unroll
            for (int u = 0; u < U; ++u) h[u] = j[u] >= 0 ? (hist[j[u]] & win) : 0ull;
            float y[U];
            if (pre) {
#pragma unroll
                for (int u = 0; u < U; ++u) y[u] = j[u] >= 0 ? ypost[j[u]] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (j[u] < 0) continue;
                float ww = w[u];
                bool changed = false;
                uint64_t older = h[u] & ~1ull;
                while (older) {
                    const int bit = 63 - __clzll((long long)older);
                    older ^= 1ull << bit;
                    const float xp = __fmul_rn(xp0, s_dpow[age - bit]);
                    ww = ww + a.c_pot * powf(ww, a.mu) * xp;
                    changed = true;
                }
                if (pre) {
                    ww = ww - a.c_dep * ww * y[u];
                    ww = fmaxf(ww, 0.f);
                    changed = true;
                }
                if (h[u] & 1ull) {
                    ww = ww + a.c_pot * powf(ww, a.mu) * xp_now;
                    changed = true;
                }
                if (changed) {
                    wgt[rs + base + u * kWave + lane] = ww;
                    ++st_written;
                }
            }
        }
        if (lane == 0) {
            a.t_last[k] = (int32_t)a.t;
            a.xpre[k] = xp_now;
            ++st_rows;
            st_forced += (!flush && !pre);
            st_syn += len;
        }
    }
    st_rows = block_sum_i64(st_rows, sh);
    st_forced = block_sum_i64(st_forced, sh);
    st_syn = block_sum_i64(st_syn, sh);
    st_written = block_sum_i64(st_written, sh);
    if (tid == 0) {
        int64_t *slot = a.stats + (int64_t)blockIdx.x * kStFields;
        slot[kStRows] += st_rows;
        slot[kStForced] += st_forced;
        slot[kStSyn] += st_syn;
        slot[kStWritten] += st_written;
    }
}

// ---------------------------------------------------------------------------
// (3) delivery.
//
// Slice delivery (Sec. III-B, Fig. 3(b)): work item q = (slice s, chunk c)
// owns targets [sW, (s+1)W) for the c-th 1/C of the transmitted spikes. The
// slice accumulator lives in LDS as exact 64-bit fixed point. For a batch of
// spikes the workgroup first gathers each spike's in-slice segment
// (row start + piv[k][s], length piv[k][s+1] - piv[k][s]) into LDS and
// prefix-sums the lengths; then every thread takes flattened elements of the
// concatenated segments, so lanes stay busy whatever the segment lengths and
// consecutive lanes read consecutive entries of a segment. Each element adds
// its weight into acc[target - sW] with an LDS 64-bit integer atomic. With
// C = 1 the workgroup owns the slice and stores the fp32 input directly;
// with C > 1 it stores fixed-point partial sum c. Workgroup b runs on XCD
// b mod 8, so work items are dealt out so that each XCD gets a contiguous
// range of slices (neighbouring segments of one row share cache lines).

constexpr int kDlvBlock = 1024;
constexpr int kDlvBatch = 1024;  // spikes whose segments are staged at once
constexpr int kDlvUnroll = 4;

__global__ __launch_bounds__(kDlvBlock) void k_deliver_lds(DeliverArgs a)
{
    extern __shared__ long long acc[];
    __shared__ long long s_start[kDlvBatch];
    __shared__ int s_off[kDlvBatch + 1];
    __shared__ int s_half[kDlvBatch];
    __shared__ long long sh[kDlvBlock / kWave];
    const int tid = threadIdx.x;
    const int nb = gridDim.x;  // multiple of 8
    const int q = (blockIdx.x & 7) * (nb >> 3) + (blockIdx.x >> 3);
    if (q >= a.n_work) return;  // whole workgroup, before any barrier
    const int s = q / a.chunks, c = q - s * a.chunks;
    const int base = s * a.width;
    const int span = a.nacc * a.width;
    for (int x = tid; x < span; x += kDlvBlock) acc[x] = 0;
    const int cnt = *a.cnt;
    const int lo = (int)((int64_t)cnt * c / a.chunks);
    const int hi = (int)((int64_t)cnt * (c + 1) / a.chunks);
    const int piv_stride = a.n_slices + 1;
    const int32_t *__restrict__ col = a.col;
    const float *__restrict__ wgt = a.w;
    long long ev = 0;
    for (int b0 = lo; b0 < hi; b0 += kDlvBatch) {
        const int nbt = min(kDlvBatch, hi - b0);
        // stage segment starts and lengths (one spike per thread)
        int len = 0;
        if (tid < nbt) {
            const int k = a.list[b0 + tid];
            const int32_t *pv = a.piv + (int64_t)k * piv_stride + s;
            const int p0 = pv[0], p1 = pv[1];
            s_start[tid] = a.row_ptr[k] + p0;
            s_half[tid] = (a.nacc == 2 && k >= a.n_exc) ? a.width : 0;
            len = p1 - p0;
        }
        // exclusive prefix of the lengths over the workgroup
        const long long incl = block_incl_scan_i64_n<kDlvBlock>(len, sh);
        if (tid < nbt) s_off[tid] = (int)(incl - len);
        if (tid == kDlvBlock - 1) s_off[nbt] = (int)incl;  // = total (threads >= nbt add 0)
        __syncthreads();
        const int total = s_off[nbt];
        ev += tid == 0 ? total : 0;
        for (int e0 = 0; e0 < total; e0 += kDlvBlock * kDlvUnroll) {
            int tgt[kDlvUnroll];
            float wv[kDlvUnroll];
#pragma unroll
            for (int u = 0; u < kDlvUnroll; ++u) {
                const int e = e0 + u * kDlvBlock + tid;
                tgt[u] = -1;
                wv[u] = 0.f;
                if (e < total) {
                    // segment holding element e: last i with s_off[i] <= e
                    int l = 0, r = nbt;
                    while (r - l > 1) {
                        const int m = (l + r) >> 1;
                        if (s_off[m] <= e) l = m;
                        else r = m;
                    }
                    const long long idx = s_start[l] + (e - s_off[l]);
                    tgt[u] = col[idx] - base + s_half[l];
                    wv[u] = wgt[idx];
                }
            }
#pragma unroll
            for (int u = 0; u < kDlvUnroll; ++u)
                if (tgt[u] >= 0)
                    atomicAdd((unsigned long long *)(acc + tgt[u]),
                              (unsigned long long)to_fix(wv[u]));
        }
        __syncthreads();  // staging arrays are rewritten by the next batch
    }
    __syncthreads();
    if (a.chunks == 1) {
        for (int x = tid; x < a.width; x += kDlvBlock) {
            const int j = base + x;
            if (j < a.n) {
                a.ain[j] = from_fix(acc[x]);
                if (a.nacc == 2) a.ain[a.n + j] = from_fix(acc[a.width + x]);
            }
        }
    } else {
        long long *out = a.apart + (int64_t)c * a.part_stride;
        for (int x = tid; x < a.width; x += kDlvBlock) {
            const int j = base + x;
            if (j < a.n) {
                out[j] = acc[x];
                if (a.nacc == 2) out[a.n + j] = acc[a.width + x];
            }
        }
    }
    ev = block_sum_i64_n<kDlvBlock>(ev, sh);
    if (tid == 0) a.stats[blockIdx.x] += ev;
}

// Row-wise delivery with global atomics (Fig. 3(a)): a wave per transmitted
// spike, lanes over its row, hardware 64-bit integer atomics on the same
// fixed-point accumulator in HBM/L2. A lane loads U entries before issuing
// their atomics, so a 1000-synapse row needs about one load latency.
constexpr int kGlobalUnroll = 16;

__global__ __launch_bounds__(kBlock) void k_deliver_global(DeliverArgs a)
{
    __shared__ long long sh[kBlock / kWave];
    const int tid = threadIdx.x, lane = tid % kWave;
    const int gw = (blockIdx.x * kBlock + tid) / kWave;
    const int nwv = gridDim.x * (kBlock / kWave);
    const int cnt = *a.cnt;
    const int32_t *__restrict__ col = a.col;
    const float *__restrict__ wgt = a.w;
    long long ev = 0;
    for (int x = gw; x < cnt; x += nwv) {
        const int k = a.list[x];
        const int64_t rs = a.row_ptr[k], re = a.row_ptr[k + 1];
        long long *dst = (a.nacc == 2 && k >= a.n_exc) ? a.apart + a.n : a.apart;
        for (int64_t e0 = rs; e0 < re; e0 += kWave * kGlobalUnroll) {
            int tgt[kGlobalUnroll];
            float wv[kGlobalUnroll];
#pragma unroll
            for (int u = 0; u < kGlobalUnroll; ++u) {
                const int64_t e = e0 + u * kWave + lane;
                tgt[u] = e < re ? col[e] : -1;
                wv[u] = e < re ? wgt[e] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < kGlobalUnroll; ++u)
                if (tgt[u] >= 0)
                    atomicAdd((unsigned long long *)(dst + tgt[u]),
                              (unsigned long long)to_fix(wv[u]));
        }
        if (lane == 0) ev += re - rs;
    }
    ev = block_sum_i64(ev, sh);
    if (tid == 0) a.stats[blockIdx.x] += ev;
}

// The fp32 input the next neuron update would compute from the partial sums.
__global__ __launch_bounds__(kBlock) void k_materialize_input(const long long *apart,
                                                              int64_t stride, int32_t parts,
                                                              float *ain, int64_t count)
{
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= count) return;
    long long v = apart[i];
    for (int c = 1; c < parts; ++c) v += apart[c * stride + i];
    ain[i] = from_fix(v);
}

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
    if (k >= a.n) return;
    const int64_t len = a.row_ptr[k + 1] - a.row_ptr[k];
    atomicMax(a.maxlen, (int32_t)(len > 0x7fffffff ? 0x7fffffff : len));
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

// First index in the sorted range [p, p+len) whose value is >= v.
__device__ __forceinline__ int lower_bound_i32(const int32_t *p, int len, int64_t v)
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
    const int64_t k = ((int64_t)blockIdx.x * kBlock + threadIdx.x) / kWave;
    const int lane = threadIdx.x % kWave;
    if (k >= a.n) return;  // wave-uniform
    const int64_t rs = a.row_ptr[k];
    const int len = (int)(a.row_ptr[k + 1] - rs);
    const int32_t *row = a.col + rs;
    int32_t *out = a.piv + k * (int64_t)(a.n_slices + 1);
    for (int s = lane; s <= a.n_slices; s += kWave)
        out[s] = s == a.n_slices ? len : lower_bound_i32(row, len, (int64_t)s * a.width);
    if (lane == 0) {
        int pe = 0;
        if (a.plastic == 2) pe = len;
        else if (a.plastic == 1 && k < a.n_exc) pe = lower_bound_i32(row, len, a.n_exc);
        a.pend[k] = pe;
    }
}

inline int blocks_for(int64_t count, int per = kBlock, int64_t cap = 1 << 20)
{
    int64_t b = (count + per - 1) / per;
    if (b < 1) b = 1;
    if (b > cap) b = cap;
    return (int)b;
}

}  // namespace

// ---------------------------------------------------------------------------
// launchers

hipError_t launch_init_state(hipStream_t s, float *v, int32_t *ref, float *ie, float *ii,
                             uint64_t *hist, float *ypost, int32_t *t_last, float *xpre,
                             int32_t n)
{
    hipLaunchKernelGGL(k_init_state, dim3(blocks_for(n)), dim3(kBlock), 0, s, v, ref, ie, ii,
                       hist, ypost, t_last, xpre, n);
    return hipGetLastError();
}

hipError_t launch_fill_f32(hipStream_t s, float *p, int64_t count, float value)
{
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill<float>, dim3(blocks_for(count, kBlock, 4096)), dim3(kBlock), 0,
                       s, p, count, value);
    return hipGetLastError();
}

hipError_t launch_fill_i64(hipStream_t s, int64_t *p, int64_t count, int64_t value)
{
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill<int64_t>, dim3(blocks_for(count, kBlock, 4096)), dim3(kBlock),
                       0, s, p, count, value);
    return hipGetLastError();
}

hipError_t launch_fill_i32(hipStream_t s, int32_t *p, int64_t count, int32_t value)
{
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill<int32_t>, dim3(blocks_for(count, kBlock, 4096)), dim3(kBlock),
                       0, s, p, count, value);
    return hipGetLastError();
}

hipError_t launch_fill_ll(hipStream_t s, long long *p, int64_t count, long long value)
{
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill<long long>, dim3(blocks_for(count, kBlock, 4096)), dim3(kBlock),
                       0, s, p, count, value);
    return hipGetLastError();
}

hipError_t launch_copy_bytes(hipStream_t s, void *dst, const void *src, int64_t bytes)
{
    if (bytes <= 0) return hipSuccess;
    return hipMemcpyAsync(dst, src, (size_t)bytes, hipMemcpyDeviceToDevice, s);
}

hipError_t launch_neuron(hipStream_t s, const NeuronArgs &a)
{
    hipLaunchKernelGGL(k_neuron, dim3(blocks_for(a.n)), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_compact(hipStream_t s, const CompactArgs &a)
{
    hipLaunchKernelGGL(k_compact, dim3(blocks_for(a.n)), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_stdp(hipStream_t s, const StdpArgs &a, int blocks)
{
    hipLaunchKernelGGL(k_stdp<kStdpUnroll>, dim3(blocks), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

// Raises a kernel's dynamic-LDS limit to `bytes` (once per size increase).
hipError_t allow_dynamic_lds(const void *kernel, int bytes, std::mutex &mu, int &granted)
{
    std::lock_guard<std::mutex> lock(mu);
    if (bytes <= granted) return hipSuccess;
    const hipError_t e =
        hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) {
        (void)hipGetLastError();  // do not leave the error for the next launch
        return e;
    }
    granted = bytes;
    return hipSuccess;
}

hipError_t launch_deliver_lds(hipStream_t s, const DeliverArgs &a, int blocks, size_t lds)
{
    static std::mutex mu;
    static int granted = 64 * 1024;
    const hipError_t e = allow_dynamic_lds((const void *)k_deliver_lds, (int)lds, mu, granted);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_deliver_lds, dim3(blocks), dim3(kDlvBlock), lds, s, a);
    return hipGetLastError();
}

int deliver_lds_static_bytes()
{
    hipFuncAttributes attr{};
    if (hipFuncGetAttributes(&attr, (const void *)k_deliver_lds) != hipSuccess) {
        (void)hipGetLastError();
        return -1;
    }
    return (int)attr.sharedSizeBytes;
}

hipError_t launch_deliver_global(hipStream_t s, const DeliverArgs &a, int blocks)
{
    hipLaunchKernelGGL(k_deliver_global, dim3(blocks), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_materialize_input(hipStream_t s, const long long *apart, int64_t part_stride,
                                    int32_t n_parts, float *ain, int64_t count)
{
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_materialize_input, dim3(blocks_for(count)), dim3(kBlock), 0, s, apart,
                       part_stride, n_parts, ain, count);
    return hipGetLastError();
}

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

}  // namespace snn
